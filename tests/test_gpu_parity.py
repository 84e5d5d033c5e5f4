"""GPU parity: libeq's gfx950 kernels against the CPU oracle.

Codes and dequantised BF16 weights must be bit-exact; the fused GEMV must be
within max|y - y_ref| / max|y_ref| <= 1e-2 per batch row against the oracle's
fp64 GEMV on the decoded BF16 weights (the bar stated for this path; the
kernel's own error is fp32 accumulation plus the BF16 rounding of W_hat that
it skips, about 1e-3 of the row norm at worst).
"""
import sys

import numpy as np
import pytest

import oracle
import synth
from gemv_ref import TOL_EXACT, exact_gemv, normwise
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
    m.lib()  # fails loudly if the library is not built
    assert torch.cuda.is_available()
    return m


def _dev():
    return torch.device("cuda:0")


def gpu_codes(eq, L):
    out = torch.empty(L.rows * L.cols, dtype=torch.uint8, device=_dev())
    eq.eq_decode_codes(L, out)
    return out.cpu().numpy().reshape(L.rows, L.cols)


def gpu_bf16(eq, L):
    out = torch.empty(L.rows * L.cols, dtype=torch.int16, device=_dev())
    eq.eq_decode_bf16(L, out)
    return out.cpu().numpy().view(np.uint16).reshape(L.rows, L.cols)


def gpu_gemv(eq, L, x_bits, bias_bits=None, stream=None):
    B = x_bits.shape[0]
    x = torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(_dev())
    bias = None if bias_bits is None else torch.from_numpy(bias_bits.view(np.int16)).to(_dev())
    y = torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
    eq.eq_decode_gemv(L, x, B, bias, y, L.workspace(B), stream)
    return y.cpu().numpy()


def rel_err(y, y_ref):
    return np.abs(y - y_ref).max(axis=1) / np.maximum(np.abs(y_ref).max(axis=1), 1e-30)


def check_full(eq, blob, spec_like, batches=(1,), with_bias=True):
    """Whole-matrix comparison (sizes the oracle finishes in seconds)."""
    L = eq.Layer(blob, _dev())
    rc, q_ref = oracle.container_decode(blob)
    assert rc == oracle.OK
    q = gpu_codes(eq, L)
    assert np.array_equal(q, q_ref), "codes differ"
    w_ref = oracle.dequant(q_ref, oracle.container_scales(blob))
    w = gpu_bf16(eq, L)
    assert np.array_equal(w, w_ref), "bf16 differs"
    for B in batches:
        x = synth.activations(spec_like, B)
        bias = synth.bias(spec_like) if with_bias else None
        y = gpu_gemv(eq, L, x, bias)
        y_ref = oracle.gemv(w_ref, x, bias)
        err = rel_err(y, y_ref)
        assert np.isfinite(y).all() and (err <= TOL).all(), (B, err)
        y_ex = exact_gemv(q_ref, oracle.container_scales(blob), x, bias_bits=bias)
        assert (normwise(y, y_ex) <= TOL_EXACT).all(), (B, normwise(y, y_ex))
    assert eq.eq_get_status(L) == eq.EQ_OK
    return L


EDGE = [
    # M, N, C, lanes, bits, outliers
    (1, 64, 64, 64, 2.0, False),       # a single full step
    (1, 1, 64, 64, 2.0, False),        # one symbol, one partial step
    (3, 77, 128, 64, 3.0, False),      # ragged N, partial last chunk
    (5, 100, 256, 256, 2.0, False),    # N < W: steps span several rows
    (40, 640, 1024, 64, 2.0, False),   # rows split between chunks
    (6, 8192, 4096, 64, 2.5, False),   # rows longer than chunks
    (64, 512, 4096, 128, 4.0, True),   # W = 128, outliers
    (37, 1280, 65536, 256, 2.0, False),  # W = 256, single partial chunk
    (16, 4160, 8192, 256, 3.0, False), # ragged at W = 256; B = 8 reads x from global memory
    (24, 1024, 2048, 128, 6.0, False), # near-flat distribution (many symbols)
    # B = 8 of these does not fit LDS: tiled GEMV (17 start-column classes,
    # partial last chunk; W = 128)
    (24, 4352, 8192, 256, 2.0, False),
    (32, 4224, 4096, 128, 3.0, True),
    # 4001 chunks in 17 classes: 16 wavefronts per block on 256 compute units,
    # where two 48 KiB tiles no longer fit LDS beside the tables and windows
    # (tiles of 11 steps); 16-step chunks, partial last tile and chunk
    (3765, 4352, 4096, 256, 2.0, False),
]


@pytest.mark.parametrize("M,N,C,lanes,bits,outliers", EDGE)
def test_edge_shapes(eq, M, N, C, lanes, bits, outliers):
    say("edge", M, N, C, lanes, bits)
    spec = small_spec(M, N, bits=bits, chunk=C, lanes=lanes, seed=1000 + M * 7 + N,
                      outliers=outliers)
    w = synth.weights(spec)
    alpha, _ = eq.eqe_alpha_search(w, bits)
    blob = eq.eqe_encode(w, alpha, chunk_syms=C, lanes=lanes)
    check_full(eq, blob, spec, batches=(1, 3, 8))


def test_single_symbol_layer(eq):
    say("single symbol")
    spec = small_spec(8, 128, chunk=256, lanes=64)
    w = np.zeros((8, 128), dtype=np.uint16)
    blob = eq.eqe_encode(w, 1.0, chunk_syms=256, lanes=64)
    assert oracle.container_info(blob).n_syms == 1
    check_full(eq, blob, spec, batches=(1, 2))


def test_oracle_built_container(eq, c1_container):
    """A container written by the oracle's own encoder decodes identically."""
    say("oracle-built c1")
    spec, w, alpha, blob = c1_container
    check_full(eq, blob, spec, batches=(1, 8))


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_config_full(eq, cfg):
    for spec in config_matrices(cfg):
        say("config", cfg, spec.name, spec.rows, spec.cols)
        w = synth.weights(spec)
        alpha, _ = eq.eqe_alpha_search(w, spec.target_bits, sample_rows=1024)
        blob = eq.eqe_encode(w, alpha, chunk_syms=spec.chunk_syms, lanes=spec.lanes,
                             seed=spec.seed, target_bits=spec.target_bits)
        info = oracle.container_info(blob)
        assert abs(info.entropy_bits - spec.target_bits) <= 0.05
        check_full(eq, blob, spec, batches=(1, 8) if cfg < 3 else (1,))


@pytest.mark.parametrize("lanes", [64, 256])
def test_every_e4m3_code(eq, lanes):
    """A layer whose codes are all 253 finite E4M3FN codes (rows hold s * v(q)
    for every q, so AbsMax with alpha = 1 reproduces each code exactly):
    decode, dequantisation and the GEMV's code-to-value conversion are
    checked on every code."""
    say("every code", lanes)
    codes = [c for c in range(256) if (c & 0x7F) != 0x7F and c != 0x80]
    vals = np.array([oracle.e4m3_value(c) for c in codes])
    M, N = 6, 512
    w = np.zeros((M, N), dtype=np.uint16)
    for i in range(M):
        row = np.resize(np.roll(vals, 37 * i), N) * (2.0 ** (i - 2))
        w[i] = [synth.to_bf16(float(v)) for v in row]
    blob = eq.eqe_encode(w, 1.0, chunk_syms=1024, lanes=lanes)
    rc, q_ref = oracle.container_decode(blob)
    assert rc == oracle.OK and len(np.unique(q_ref)) == len(codes)
    spec = small_spec(M, N, chunk=1024, lanes=lanes, seed=3)
    L = check_full(eq, blob, spec, batches=(1, 2))
    # one-hot activations: y_i = s_i * v(q_ij) exactly, for every column
    scale = synth.bf16_to_f32(oracle.container_scales(blob)).astype(np.float64)
    for j0 in range(0, N, 8):
        x = np.zeros((8, N), dtype=np.uint16)
        for b in range(8):
            x[b, j0 + b] = 0x3F80
        y = gpu_gemv(eq, L, x)
        for b in range(8):
            exact = scale * np.array([oracle.e4m3_value(int(c)) for c in q_ref[:, j0 + b]])
            assert np.array_equal(y[b].astype(np.float64), exact), (j0 + b)


def test_one_hot_and_zero_inputs(eq):
    say("one-hot")
    spec = small_spec(48, 1024, bits=3.0, chunk=4096, lanes=64, seed=5)
    w = synth.weights(spec)
    blob = eq.eqe_encode(w, eq.eqe_alpha_search(w, 3.0)[0], chunk_syms=4096, lanes=64)
    L = eq.Layer(blob, _dev())
    _, q_ref = oracle.container_decode(blob)
    scale = oracle.container_scales(blob)
    w_ref = oracle.dequant(q_ref, scale)
    cols = [0, 1, 63, 64, 511, 1023]
    x = np.zeros((len(cols), 1024), dtype=np.uint16)
    for b, j in enumerate(cols):
        x[b, j] = 0x3F80  # 1.0
    y = gpu_gemv(eq, L, x)
    for b, j in enumerate(cols):
        exact = synth.bf16_to_f32(scale).astype(np.float64) * \
            np.array([oracle.e4m3_value(int(c)) for c in q_ref[:, j]])
        assert np.array_equal(y[b].astype(np.float64), exact)   # s_i * v(q_ij), exact in fp32
        back = torch.from_numpy(y[b]).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(back, w_ref[:, j])
    bias = synth.bias(spec)
    y0 = gpu_gemv(eq, L, np.zeros((2, 1024), dtype=np.uint16), bias)
    assert np.array_equal(y0, np.stack([synth.bf16_to_f32(bias)] * 2))


def test_bias_view_at_odd_element(eq):
    """A bias that is a view one element into a tensor (2-byte aligned, not
    4): rows that a chunk holds whole (config-1 shape: four rows per
    4096-symbol chunk) and rows split between chunks read the same bias
    entry as the oracle."""
    for M, N, C in ((256, 1024, 4096), (40, 640, 1024)):
        say("bias view", M, N, C)
        spec = small_spec(M, N, bits=2.0, chunk=C, lanes=64, seed=4400 + M)
        w = synth.weights(spec)
        blob = eq.eqe_encode(w, eq.eqe_alpha_search(w, 2.0)[0], chunk_syms=C, lanes=64)
        L = eq.Layer(blob, _dev())
        _, q_ref = oracle.container_decode(blob)
        w_ref = oracle.dequant(q_ref, oracle.container_scales(blob))
        bias_bits = synth.bias(spec)
        backing = torch.zeros(M + 2, dtype=torch.int16, device=_dev())
        backing[1:M + 1] = torch.from_numpy(bias_bits.view(np.int16)).to(_dev())
        bias = backing[1:M + 1]
        assert bias.data_ptr() % 4 == 2
        for B in (1, 8):
            x = synth.activations(spec, B)
            xt = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(_dev())
            y = torch.full((B, M), float("nan"), dtype=torch.float32, device=_dev())
            eq.eq_decode_gemv(L, xt, B, bias, y, L.workspace(B))
            y = y.cpu().numpy()
            assert (rel_err(y, oracle.gemv(w_ref, x, bias_bits)) <= TOL).all()
            # x = 0: y is the bias, exactly
            y0 = torch.full((B, M), float("nan"), dtype=torch.float32, device=_dev())
            eq.eq_decode_gemv(L, torch.zeros_like(xt), B, bias, y0, L.workspace(B))
            assert np.array_equal(y0.cpu().numpy(), np.stack([synth.bf16_to_f32(bias_bits)] * B))


def test_deterministic_and_streams(eq):
    say("determinism")
    spec = small_spec(256, 2048, bits=2.0, chunk=16384, lanes=64, seed=8)
    w = synth.weights(spec)
    blob = eq.eqe_encode(w, eq.eqe_alpha_search(w, 2.0)[0], chunk_syms=16384, lanes=64)
    L = eq.Layer(blob, _dev())
    x = synth.activations(spec, 2)
    y0 = gpu_gemv(eq, L, x)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        y1 = gpu_gemv(eq, L, x, stream=s)
    torch.cuda.synchronize()
    y2 = gpu_gemv(eq, L, x)
    assert np.array_equal(y0, y1) and np.array_equal(y0, y2)


def test_corrupted_stream_flagged(eq):
    """A flipped stream bit: the GPU must reach the oracle's verdict, and
    when the oracle still decodes cleanly the codes must agree."""
    say("corruption")
    spec = small_spec(32, 1024, bits=2.0, chunk=4096, lanes=64, seed=9)
    w = synth.weights(spec)
    blob = eq.eqe_encode(w, eq.eqe_alpha_search(w, 2.0)[0], chunk_syms=4096, lanes=64)
    info = oracle.container_info(blob)
    r = np.random.default_rng(3)
    flagged = 0
    for trial in range(6):
        bad = blob.copy()
        word = int(r.integers(info.total_words))
        bad[info.off_words + 2 * word + int(r.integers(2))] ^= np.uint8(1 << int(r.integers(8)))
        L = eq.Layer(bad, _dev())
        q = gpu_codes(eq, L)
        rc_gpu = eq.eq_get_status(L)
        rc_ref, q_ref = oracle.container_decode(bad)
        if rc_ref == oracle.ECORRUPT:
            assert rc_gpu == eq.EQ_ECORRUPT
            flagged += 1
        else:
            assert rc_gpu == eq.EQ_OK and np.array_equal(q, q_ref)
        eq.eq_layer_prepare(L)  # clears the status word
        assert eq.eq_get_status(L) == eq.EQ_OK
    assert flagged >= 1


@pytest.mark.parametrize("lanes,N", [(128, 1024), (256, 2048)])
def test_bf16_output_alignment(eq, lanes, N):
    """Full steps of W = 128 and 256 write a step's values through the
    wavefront's LDS staging area, G adjacent columns per lane and store, when
    the output is aligned to G values; otherwise one value per state and
    store.  Both give the oracle's BF16 and codes bit for bit, through the
    single-layer and the block-wise launch, at output offsets of 0 to 3
    elements."""
    say("bf16 alignment", lanes, N)
    spec = small_spec(48, N, bits=2.0, chunk=8192, lanes=lanes, seed=5100 + lanes)
    w = synth.weights(spec)
    alpha, _ = eq.eqe_alpha_search(w, 2.0)
    blob = eq.eqe_encode(w, alpha, chunk_syms=8192, lanes=lanes)
    L = eq.Layer(blob, _dev())
    rc, q_ref = oracle.container_decode(blob)
    assert rc == oracle.OK
    w_ref = oracle.dequant(q_ref, oracle.container_scales(blob))
    n = spec.rows * spec.cols
    for off in range(4):
        full = torch.full((n + 8,), -1, dtype=torch.int16, device=_dev())
        eq.eq_decode_bf16(L, full[off:off + n])
        got = full.cpu().numpy().view(np.uint16)
        assert np.array_equal(got[off:off + n].reshape(spec.rows, N), w_ref), off
        assert (got[:off] == 0xFFFF).all() and (got[off + n:] == 0xFFFF).all(), off
        full.fill_(-1)
        eq.eq_decode_bf16_multi([L, L], [full[off:off + n], full[off:off + n]])
        got = full.cpu().numpy().view(np.uint16)
        assert np.array_equal(got[off:off + n].reshape(spec.rows, N), w_ref), off
        codes = torch.full((n + 8,), 0xA5, dtype=torch.uint8, device=_dev())
        eq.eq_decode_codes(L, codes[off:off + n])
        got = codes.cpu().numpy()
        assert np.array_equal(got[off:off + n].reshape(spec.rows, N), q_ref), off
        assert (got[:off] == 0xA5).all() and (got[off + n:] == 0xA5).all(), off
    assert eq.eq_get_status(L) == eq.EQ_OK
