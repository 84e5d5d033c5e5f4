"""GPU parity of the prefill path (B > 8 tokens): decode to codes, then the
W8A16 MFMA GEMM with the scale applied per output (Sec. 2.1 linear layer on
the dequantised weights; the paper's decompress-then-FP8-GEMM pipeline).

Bar: max|y - y_ref| / max|y_ref| <= 1e-2 per token row against the oracle's
fp64 GEMM on the decoded BF16 weights (as for the GEMV), plus exact outputs
for one-hot tokens (y = s_i v(q_ij), a single product), on ragged shapes
(tokens, rows and columns not multiples of the 128 x 128 x 64 tile), both
base formats, and sampled rows and tokens of the full-size 8192 x 28672
layer.  Batches of up to 8 tokens go to the fused decode-GEMV instead, with
its results."""
import sys

import numpy as np
import pytest

import oracle
import synth
from synth.configs import config_matrices, small_spec

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def eq():
    import paper_2601_22787_amd as m
    m.lib()
    assert torch.cuda.is_available()
    return m


def _dev():
    return torch.device("cuda:0")


def encode(eq, w, bits, C, lanes, fmt):
    alpha, _ = eq.eqe_alpha_search(w, bits, base_format=fmt)
    return eq.eqe_encode(w, alpha, chunk_syms=C, lanes=lanes, base_format=fmt)


def tokens(spec, B):
    return np.stack([synth.vector(spec.seed, 100 + t, spec.cols) for t in range(B)])


def gpu_gemm(eq, L, x_bits, bias_bits=None):
    B = x_bits.shape[0]
    x = torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(_dev())
    bias = None if bias_bits is None else torch.from_numpy(bias_bits.view(np.int16)).to(_dev())
    y = torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
    eq.eq_decode_gemm(L, x, B, bias, y, L.gemm_workspace(B))
    return y.cpu().numpy()


def rel_err(y, y_ref):
    return np.abs(y - y_ref).max(axis=1) / np.maximum(np.abs(y_ref).max(axis=1), 1e-30)


SHAPES = [
    # M, N, C, lanes, bits, B
    (64, 256, 4096, 64, 2.0, 16),
    (100, 320, 1024, 64, 3.0, 37),     # ragged rows, columns (320 = 5 x 64) and tokens
    (256, 1024, 4096, 128, 2.0, 129),  # one 256 x 256 tile, 4 slices; 129 tokens
    (37, 4096, 16384, 256, 4.0, 300),
    (300, 208, 2048, 64, 2.5, 9),      # N = 208: a partial 64-column stage
]


@pytest.mark.parametrize("fmt", [1, 2])
@pytest.mark.parametrize("M,N,C,lanes,bits,B", SHAPES)
def test_gemm_shapes(eq, M, N, C, lanes, bits, B, fmt):
    say("gemm", M, N, B, "format", fmt)
    spec = small_spec(M, N, bits=bits, chunk=C, lanes=lanes, seed=4000 + M + N)
    w = synth.weights(spec)
    blob = encode(eq, w, bits, C, lanes, fmt)
    L = eq.Layer(blob, _dev())
    rc, q = oracle.container_decode(blob)
    assert rc == oracle.OK
    w_ref = oracle.dequant(q, oracle.container_scales(blob), fmt)
    x = tokens(spec, B)
    bias = synth.bias(spec)
    for b in (None, bias):
        y = gpu_gemm(eq, L, x, b)
        err = rel_err(y, oracle.gemv(w_ref, x, b))
        assert np.isfinite(y).all() and (err <= TOL).all(), err.max()
    assert eq.eq_get_status(L) == eq.EQ_OK


@pytest.mark.parametrize("fmt", [1, 2])
def test_gemm_one_hot_exact(eq, fmt):
    """One-hot tokens select single weights: y_ti = s_i v(q_ij) exactly (one
    product, no rounding), over every code of the base format."""
    if fmt == 1:
        codes = [c for c in range(256) if (c & 0x7F) != 0x7F and c != 0x80]
    else:
        codes = [c for c in range(256) if c != 0x80]
    vals = np.array([oracle.code_value(fmt, c) for c in codes])
    M, N = 40, 512
    w = np.zeros((M, N), dtype=np.uint16)
    for i in range(M):
        row = np.resize(np.roll(vals, 29 * i), N) * (2.0 ** ((i % 7) - 3))
        w[i] = [synth.to_bf16(float(v)) for v in row]
    blob = eq.eqe_encode(w, 1.0, chunk_syms=4096, lanes=64, base_format=fmt)
    L = eq.Layer(blob, _dev())
    rc, q = oracle.container_decode(blob)
    assert rc == oracle.OK and len(np.unique(q)) == len(codes)
    scale = synth.bf16_to_f32(oracle.container_scales(blob)).astype(np.float64)
    cols = np.arange(0, N, 3)
    x = np.zeros((cols.size, N), dtype=np.uint16)
    x[np.arange(cols.size), cols] = 0x3F80
    exact = {j: scale * np.array([oracle.code_value(fmt, int(c)) for c in q[:, j]])
             for j in cols}
    # 171 tokens: 128 x 128 blocks; 50 and 20: the 64- and 32-token blocks
    for n in (cols.size, 50, 20):
        y = gpu_gemm(eq, L, x[:n])
        for t, j in enumerate(cols[:n]):
            assert np.array_equal(y[t].astype(np.float64), exact[j]), (n, j)


def test_gemm_codes_entry_and_checks(eq):
    spec = small_spec(96, 512, bits=2.0, chunk=4096, lanes=64, seed=4100)
    w = synth.weights(spec)
    blob = encode(eq, w, 2.0, 4096, 64, 1)
    L = eq.Layer(blob, _dev())
    x_bits = tokens(spec, 20)
    x = torch.from_numpy(x_bits.view(np.int16)).to(_dev())
    codes = torch.empty(spec.params, dtype=torch.uint8, device=_dev())
    eq.eq_decode_codes(L, codes)
    y1 = torch.empty(20, spec.rows, dtype=torch.float32, device=_dev())
    nws = eq.eq_gemm_codes_workspace_bytes(L, 20)
    ws = torch.empty(nws, dtype=torch.uint8, device=_dev()) if nws else None
    eq.eq_gemm_codes(L, codes, x, 20, None, y1, ws)
    y2 = torch.from_numpy(gpu_gemm(eq, L, x_bits)).to(_dev())
    assert torch.equal(y1, y2)
    # the GEMV computes the same products (different summation order)
    y3 = torch.empty(8, spec.rows, dtype=torch.float32, device=_dev())
    eq.eq_decode_gemv(L, x[:8].contiguous(), 8, None, y3, L.workspace(8))
    assert (rel_err(y3.cpu().numpy(), y1[:8].cpu().numpy()) < 1e-5).all()
    with pytest.raises(eq.EqError):  # misaligned activations
        eq.eq_gemm_codes(L, codes, x.view(-1)[1:].view(torch.int16), 1, None, y1, ws)
    with pytest.raises(eq.EqError):  # workspace too small
        eq.eq_decode_gemm(L, x, 20, None, y1, L.gemm_workspace(20)[:100])
    spec2 = small_spec(8, 200, bits=2.0, chunk=1600, lanes=64, seed=4101)
    L2 = eq.Layer(encode(eq, synth.weights(spec2), 2.0, 1600, 64, 1), _dev())
    with pytest.raises(eq.EqError):  # N not a multiple of 16
        eq.eq_decode_gemm(L2, torch.zeros(200, dtype=torch.int16, device=_dev()), 1, None,
                          torch.empty(8, dtype=torch.float32, device=_dev()),
                          torch.empty(256, dtype=torch.uint8, device=_dev()))


@pytest.mark.parametrize("N,B", [(4096, 20), (4112, 9), (4096, 48), (2048, 128)])
def test_gemm_split_k(eq, N, B):
    """Few output tiles and long rows: the input columns are cut into slices
    (32-token blocks: 16 slices of 4 stages, 13 uneven slices of 5 of 65
    stages; 64-token blocks: 16 of 4; 128 x 128 blocks: 8 of 4), the partial
    sums reduced in slice order.  Within the bar, deterministic, and the
    workspace is required."""
    say("split-K", N, B)
    spec = small_spec(100, N, bits=2.0, chunk=8192, lanes=64, seed=4300 + N + B)
    w = synth.weights(spec)
    blob = encode(eq, w, 2.0, 8192, 64, 1)
    L = eq.Layer(blob, _dev())
    assert eq.eq_gemm_codes_workspace_bytes(L, B) > 0
    rc, q = oracle.container_decode(blob)
    w_ref = oracle.dequant(q, oracle.container_scales(blob))
    x = tokens(spec, B)
    bias = synth.bias(spec)
    y = gpu_gemm(eq, L, x, bias)
    err = rel_err(y, oracle.gemv(w_ref, x, bias))
    assert np.isfinite(y).all() and (err <= TOL).all(), err.max()
    assert np.array_equal(y, gpu_gemm(eq, L, x, bias))
    codes = torch.empty(spec.params, dtype=torch.uint8, device=_dev())
    eq.eq_decode_codes(L, codes)
    xt = torch.from_numpy(x.view(np.int16)).to(_dev())
    yt = torch.empty(B, spec.rows, dtype=torch.float32, device=_dev())
    with pytest.raises(eq.EqError):  # the slices need the workspace
        eq.eq_gemm_codes(L, codes, xt, B, None, yt, None)


def test_gemm_large_tiles_split_k(eq):
    """256 x 256 tiles with split-K: 300 rows x 250 tokens (two row tiles, one
    token tile) over 1040 columns, 17 stages with a 16-column last one, cut
    into slices of 5, 5, 5 and 2 stages; within the bar, deterministic."""
    spec = small_spec(300, 1040, bits=2.0, chunk=8192, lanes=64, seed=4400)
    w = synth.weights(spec)
    blob = encode(eq, w, 2.0, 8192, 64, 1)
    L = eq.Layer(blob, _dev())
    assert eq.eq_gemm_codes_workspace_bytes(L, 250) > 0
    rc, q = oracle.container_decode(blob)
    w_ref = oracle.dequant(q, oracle.container_scales(blob))
    x = tokens(spec, 250)
    bias = synth.bias(spec)
    y = gpu_gemm(eq, L, x, bias)
    err = rel_err(y, oracle.gemv(w_ref, x, bias))
    assert np.isfinite(y).all() and (err <= TOL).all(), err.max()
    assert np.array_equal(y, gpu_gemm(eq, L, x, bias))


def _sampled(eq, spec, w, blob, L, B, fmt, seed):
    """Sampled rows x sampled tokens (always the first and last) of the
    prefill output against the oracle's fp64 GEMM of the same rows, whose
    codes come from the oracle's quantiser on the generated weights."""
    x = tokens(spec, B)
    y = gpu_gemm(eq, L, x)
    assert eq.eq_get_status(L) == eq.EQ_OK and np.isfinite(y).all()
    r = np.random.default_rng(seed)
    rows = sorted(set(r.choice(spec.rows, 8, replace=False).tolist()) | {0, spec.rows - 1})
    toks = sorted(set(r.choice(B, 6, replace=False).tolist()) | {0, B - 1})
    scale = oracle.container_scales(blob)
    w_rows = oracle.dequant(oracle.quantize(w[rows], scale[rows], fmt), scale[rows], fmt)
    err = rel_err(y[np.ix_(toks, rows)], oracle.gemv(w_rows, x[toks]))
    assert (err <= TOL).all(), err


@pytest.mark.parametrize("fmt", [1, 2])
def test_gemm_config4_full_size_sampled(eq, fmt):
    """The 8192x28672 layer at 256 tokens (32 tiles of 256 x 256, 8 slices of
    56 stages) and the 28672x8192 layer at 768 tokens (336 blocks of 256 x
    256)."""
    for spec, B in zip(config_matrices(4), (256, 768)):
        say("gemm config 4", spec.name, B, fmt)
        w = synth.weights(spec)
        alpha, _ = eq.eqe_alpha_search(w, spec.target_bits, sample_rows=512, base_format=fmt)
        blob = eq.eqe_encode(w, alpha, chunk_syms=spec.chunk_syms, lanes=spec.lanes,
                             base_format=fmt)
        L = eq.Layer(blob, _dev())
        _sampled(eq, spec, w, blob, L, B, fmt, 12 + B)
        del L


def test_gemm_large_tiles_ragged(eq):
    """256 x 256 tiles on a shape ragged in every dimension: 4000 rows, 272
    columns (four 64-column stages and a 16-column one), 4100 tokens."""
    spec = small_spec(4000, 272, bits=3.0, chunk=16384, lanes=64, seed=4200)
    w = synth.weights(spec)
    blob = encode(eq, w, 3.0, 16384, 64, 1)
    L = eq.Layer(blob, _dev())
    _sampled(eq, spec, w, blob, L, 4100, 1, 99)


def test_block_codes_buffer_feeds_gemm(eq):
    """Sec. 2.2 block-wise pipeline: the codes of three layers into one block
    buffer by one launch of eq_decode_codes_multi, then eq_gemm_codes from
    that buffer:
    codes bit-exact against the oracle, outputs equal to eq_decode_gemm's and
    within the bar against the oracle's fp64 GEMM."""
    shapes = [(200, 512, 4096, 64, 4200), (96, 512, 2048, 64, 4201), (64, 1024, 8192, 64, 4202)]
    layers = []
    for M, N, C, lanes, seed in shapes:
        spec = small_spec(M, N, bits=2.5, chunk=C, lanes=lanes, seed=seed)
        w = synth.weights(spec)
        blob = encode(eq, w, 2.5, C, lanes, 1)
        layers.append((spec, blob, eq.Layer(blob, _dev())))
    sizes = [s.params for s, _, _ in layers]
    block = torch.full((sum(sizes) + 64,), 0xA5, dtype=torch.uint8, device=_dev())
    starts = np.cumsum([0] + sizes)
    views = [block[starts[i]:starts[i + 1]] for i in range(len(layers))]
    eq.eq_decode_codes_multi([L for _, _, L in layers], views)
    assert (block[sum(sizes):] == 0xA5).all()
    B = 24
    for (spec, blob, L), cv in zip(layers, views):
        rc, q_ref = oracle.container_decode(blob)
        assert rc == oracle.OK
        assert np.array_equal(cv.cpu().numpy().reshape(spec.rows, spec.cols), q_ref)
        x_bits = tokens(spec, B)
        x = torch.from_numpy(x_bits.view(np.int16)).to(_dev())
        y = torch.full((B, spec.rows), float("nan"), dtype=torch.float32, device=_dev())
        nws = eq.eq_gemm_codes_workspace_bytes(L, B)
        ws = torch.empty(nws, dtype=torch.uint8, device=_dev()) if nws else None
        eq.eq_gemm_codes(L, cv, x, B, None, y, ws)
        yn = y.cpu().numpy()
        assert np.array_equal(yn, gpu_gemm(eq, L, x_bits))
        w_ref = oracle.dequant(q_ref, oracle.container_scales(blob))
        assert (rel_err(yn, oracle.gemv(w_ref, x_bits)) <= TOL).all()
        assert eq.eq_get_status(L) == eq.EQ_OK


@pytest.mark.parametrize("version", [1, 2, "2-ordered"])
@pytest.mark.parametrize("fmt", [1, 2])
def test_small_batches_take_the_fused_gemv(eq, version, fmt):
    """Up to 8 tokens eq_decode_gemm runs the fused decode-GEMV: its outputs
    equal eq_decode_gemv's bit for bit (same workspace size rule), meet the
    GEMV bar against the oracle, and 9 tokens go through the GEMM (after a
    decode to codes in matrix order, also for a layer with a row order)."""
    M, N = 96, 1024
    seed = 4321 + (3 if version == "2-ordered" else version) + fmt
    spec = small_spec(M, N, bits=2.5, chunk=4096, lanes=64, seed=seed)
    w = synth.weights(spec)
    alpha, _ = eq.eqe_alpha_search(w, 2.5, base_format=fmt)
    if version == 1:
        blob = eq.eqe_encode(w, alpha, chunk_syms=4096, lanes=64, base_format=fmt)
    else:
        blob = eq.eqe_encode2(w, alpha, tile_rows=64, tile_cols=64, base_format=fmt,
                              row_order=version == "2-ordered")
    L = eq.Layer(blob, _dev())
    rc, q = (oracle.container_decode(blob) if version == 1 else oracle.container2_decode(blob))
    assert rc == oracle.OK
    w_ref = oracle.dequant(q, oracle.container_scales(blob), fmt)
    bias = synth.bias(spec)
    bias_t = torch.from_numpy(bias.view(np.int16)).to(_dev())
    for B in (1, 5, 8, 9):
        x_bits = tokens(spec, B)
        x = torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(_dev())
        assert eq.eq_gemm_workspace_bytes(L, B) >= (eq.eq_gemv_workspace_bytes(L, B)
                                                    if B <= 8 else 0)
        y = gpu_gemm(eq, L, x_bits, bias)
        err = rel_err(y, oracle.gemv(w_ref, x_bits, bias))
        assert np.isfinite(y).all() and (err <= TOL).all(), (B, err)
        if B <= 8:
            y2 = torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
            eq.eq_decode_gemv(L, x, B, bias_t, y2, L.workspace(B))
            assert np.array_equal(y, y2.cpu().numpy()), B
    assert eq.eq_get_status(L) == eq.EQ_OK
