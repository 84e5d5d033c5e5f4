"""GPU parity of container version 2 (tile-ordered chunks, phrase alphabet)
against the oracle.

Codes and BF16 weights bit-exact against the oracle's decode and
dequantiser; the fused GEMV within max|y - y_ref| / max|y_ref| <= 1e-2 per
batch row against the oracle's fp64 GEMV on the decoded BF16 weights; one-hot
inputs exact.  Shapes cover partial tiles in both directions, fewer rows than
a tile, N not a multiple of 4 (segments ending in pairs and single codes),
every tile height, narrow and wide tiles, both base formats and a
single-phrase layer.
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
    m.lib()
    assert torch.cuda.is_available()
    return m


def _dev():
    return torch.device("cuda:0")


def gpu_codes(eq, L, off=0):
    n = L.rows * L.cols
    out = torch.full((n + off + 8,), 0xA5, dtype=torch.uint8, device=_dev())
    eq.eq_decode_codes(L, out[off:off + n])
    got = out.cpu().numpy()
    assert (got[:off] == 0xA5).all() and (got[off + n:] == 0xA5).all()
    return got[off:off + n].reshape(L.rows, L.cols)


def gpu_bf16(eq, L, off=0):
    n = L.rows * L.cols
    out = torch.full((n + off + 8,), -1, dtype=torch.int16, device=_dev())
    eq.eq_decode_bf16(L, out[off:off + n])
    got = out.cpu().numpy().view(np.uint16)
    assert (got[:off] == 0xFFFF).all() and (got[off + n:] == 0xFFFF).all()
    return got[off:off + n].reshape(L.rows, L.cols)


def gpu_gemv(eq, L, x_bits, bias_bits=None):
    B = x_bits.shape[0]
    x = torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(_dev())
    bias = None if bias_bits is None else torch.from_numpy(bias_bits.view(np.int16)).to(_dev())
    y = torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
    eq.eq_decode_gemv(L, x, B, bias, y, L.workspace(B))
    return y.cpu().numpy()


def rel_err(y, y_ref):
    return np.abs(y - y_ref).max(axis=1) / np.maximum(np.abs(y_ref).max(axis=1), 1e-30)


def check_full(eq, blob, spec, batches=(1, 2, 3, 5, 8), with_bias=True, offsets=(0,)):
    L = eq.Layer(blob, _dev())
    assert L.raw.version == 2
    rc, q_ref = oracle.container2_decode_par(blob)
    assert rc == oracle.OK
    w_ref = oracle.dequant_par(q_ref, oracle.container_scales(blob),
                               oracle.container2_info(blob).base_format)
    for off in offsets:
        assert np.array_equal(gpu_codes(eq, L, off), q_ref), ("codes", off)
        assert np.array_equal(gpu_bf16(eq, L, off), w_ref), ("bf16", off)
    for B in batches:
        x = synth.activations(spec, B)
        bias = synth.bias(spec) if with_bias else None
        y = gpu_gemv(eq, L, x, bias)
        err = rel_err(y, oracle.gemv_par(w_ref, x, bias))
        assert np.isfinite(y).all() and (err <= TOL).all(), (B, err)
        y_ex = exact_gemv(q_ref, oracle.container_scales(blob), x,
                          oracle.container2_info(blob).base_format, bias)
        assert (normwise(y, y_ex) <= TOL_EXACT).all(), (B, normwise(y, y_ex))
    assert eq.eq_get_status(L) == eq.EQ_OK
    return L, q_ref, w_ref


def build(eq, spec, TR, TC, bits, fmt=1, row_order=False):
    w = synth.weights(spec)
    alpha, _ = eq.eqe_alpha_search(w, bits, base_format=fmt)
    return w, eq.eqe_encode2(w, alpha, tile_rows=TR, tile_cols=TC, base_format=fmt,
                             row_order=row_order)


EDGE = [
    # M, N, TR, TC, bits, outliers
    (1, 4, 64, 4, 2.0, False),           # one phrase slot
    (1, 1, 64, 4, 2.0, False),           # one code
    (3, 77, 64, 64, 3.0, False),         # N odd: pairs and singles at segment ends
    (5, 100, 256, 32, 2.0, False),       # rows far below a tile
    (40, 640, 64, 256, 2.0, False),      # partial last column tile
    (300, 1000, 64, 256, 2.5, False),    # partial tiles both ways
    (130, 4096, 128, 512, 4.0, True),    # 4 bits, outliers, wide tiles
    (37, 1283, 128, 64, 3.0, False),
    (520, 2048, 256, 256, 2.0, False),   # the config-4 tile, partial last tile row
    (24, 1024, 64, 1024, 6.0, False),    # near-flat distribution, long segments
    (777, 260, 256, 4, 2.0, True),       # the narrowest tiles
]


@pytest.mark.parametrize("M,N,TR,TC,bits,outliers", EDGE)
def test_v2_edge_shapes(eq, M, N, TR, TC, bits, outliers):
    say("v2 edge", M, N, TR, TC, bits)
    spec = small_spec(M, N, bits=bits, seed=2000 + 7 * M + N, outliers=outliers)
    _, blob = build(eq, spec, TR, TC, bits)
    check_full(eq, blob, spec)


def test_v2_output_offsets(eq):
    """Phrases are stored with 8-byte (BF16) and 4-byte (codes) stores at any
    element offset: outputs that start 1-3 elements into a buffer are
    bit-exact and nothing outside them is written."""
    spec = small_spec(70, 1000, bits=2.0, seed=2100)
    _, blob = build(eq, spec, 64, 256, 2.0)
    check_full(eq, blob, spec, batches=(1,), offsets=(0, 1, 2, 3))


def test_v2_single_phrase_and_oracle_built(eq):
    spec = small_spec(70, 512, seed=2200)
    w = np.zeros((70, 512), dtype=np.uint16)
    blob = eq.eqe_encode2(w, 1.0, tile_rows=64, tile_cols=256)
    assert oracle.container2_info(blob).n_syms == 1
    check_full(eq, blob, spec, batches=(1, 2))
    # a container written by the oracle's own encoder
    spec = small_spec(200, 768, bits=2.0, seed=2201)
    w = synth.weights(spec)
    alpha, _ = oracle.alpha_search(w, 2.0)
    check_full(eq, oracle.container2_build(w, alpha, 128, 128), spec, batches=(1, 8))


@pytest.mark.parametrize("TR", [64, 256])
def test_v2_every_code_and_one_hot(eq, TR):
    """All 253 finite E4M3FN codes in one layer (each row holds s * v(q) for
    every q, so AbsMax with alpha = 1 reproduces each code), and one-hot
    inputs: y_i = s_i * v(q_ij) exactly, for every column."""
    codes = [c for c in range(256) if (c & 0x7F) != 0x7F and c != 0x80]
    vals = np.array([oracle.e4m3_value(c) for c in codes])
    M, N = 6, 512
    w = np.zeros((M, N), dtype=np.uint16)
    for i in range(M):
        row = np.resize(np.roll(vals, 37 * i), N) * (2.0 ** (i - 2))
        w[i] = [synth.to_bf16(float(v)) for v in row]
    blob = eq.eqe_encode2(w, 1.0, tile_rows=TR, tile_cols=128)
    spec = small_spec(M, N, seed=2300)
    L, q_ref, _ = check_full(eq, blob, spec, batches=(1, 2))
    assert len(np.unique(q_ref)) == len(codes)
    scale = synth.bf16_to_f32(oracle.container_scales(blob)).astype(np.float64)
    for j0 in range(0, N, 8):
        x = np.zeros((8, N), dtype=np.uint16)
        for b in range(8):
            x[b, j0 + b] = 0x3F80
        y = gpu_gemv(eq, L, x)
        for b in range(8):
            exact = scale * np.array([oracle.e4m3_value(int(c)) for c in q_ref[:, j0 + b]])
            assert np.array_equal(y[b].astype(np.float64), exact), (j0 + b)


def test_v2_int8(eq):
    for (M, N, TR, TC) in ((96, 1000, 64, 256), (300, 2048, 256, 256)):
        say("v2 int8", M, N)
        spec = small_spec(M, N, bits=2.0, seed=2400 + M)
        _, blob = build(eq, spec, TR, TC, 2.0, fmt=eq.FMT_INT8)
        assert oracle.container2_info(blob).base_format == eq.FMT_INT8
        check_full(eq, blob, spec, batches=(1, 8))


def test_v2_zero_input_and_bias_view(eq):
    spec = small_spec(300, 1024, bits=2.0, seed=2500)
    _, blob = build(eq, spec, 64, 256, 2.0)
    L = eq.Layer(blob, _dev())
    bias_bits = synth.bias(spec)
    backing = torch.zeros(302, dtype=torch.int16, device=_dev())
    backing[1:301] = torch.from_numpy(bias_bits.view(np.int16)).to(_dev())
    for B in (1, 8):
        y = torch.full((B, 300), float("nan"), dtype=torch.float32, device=_dev())
        eq.eq_decode_gemv(L, torch.zeros((B, 1024), dtype=torch.int16, device=_dev()), B,
                          backing[1:301], y, L.workspace(B))
        assert np.array_equal(y.cpu().numpy(), np.stack([synth.bf16_to_f32(bias_bits)] * B))


def test_v2_deterministic(eq):
    spec = small_spec(256, 4096, bits=2.0, seed=2600)
    _, blob = build(eq, spec, 64, 256, 2.0)
    L = eq.Layer(blob, _dev())
    x = synth.activations(spec, 3)
    y0 = gpu_gemv(eq, L, x)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        y1 = torch.full((3, 256), float("nan"), dtype=torch.float32, device=_dev())
        xt = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(_dev())
        eq.eq_decode_gemv(L, xt, 3, None, y1, L.workspace(3), s)
    torch.cuda.synchronize()
    assert np.array_equal(y0, y1.cpu().numpy()) and np.array_equal(y0, gpu_gemv(eq, L, x))


def test_v2_corrupted_stream_flagged(eq):
    spec = small_spec(64, 1024, bits=2.0, seed=2700)
    _, blob = build(eq, spec, 64, 256, 2.0)
    info = oracle.container2_info(blob)
    r = np.random.default_rng(5)
    flagged = 0
    for trial in range(6):
        bad = blob.copy()
        word = int(r.integers(info.total_words))
        bad[info.off_words + 2 * word + int(r.integers(2))] ^= np.uint8(1 << int(r.integers(8)))
        L = eq.Layer(bad, _dev())
        out = torch.empty(L.rows * L.cols, dtype=torch.uint8, device=_dev())
        eq.eq_decode_codes(L, out)
        q = out.cpu().numpy().reshape(L.rows, L.cols)
        rc_gpu = eq.eq_get_status(L)
        rc_ref, q_ref = oracle.container2_decode(bad)
        if rc_ref == oracle.ECORRUPT:
            assert rc_gpu == eq.EQ_ECORRUPT
            flagged += 1
        else:
            assert rc_gpu == eq.EQ_OK and np.array_equal(q, q_ref)
        eq.eq_layer_prepare(L)
        assert eq.eq_get_status(L) == eq.EQ_OK
    assert flagged >= 1


def bench_tiles(spec):
    """The benchmark's version-2 tiles below 65536-symbol chunks: C / 128
    columns, 128 rows when the matrix has at least 2048 such tiles, else 64."""
    tc = spec.chunk_syms // 128
    return (128 if -(-spec.rows // 128) * -(-spec.cols // tc) >= 2048 else 64), tc


@pytest.mark.parametrize("cfg", [1, 2, 3])
@pytest.mark.parametrize("shape,row_order", [("C/64", False), ("bench", False),
                                             ("bench", True)])
def test_v2_configs_1_to_3(eq, cfg, shape, row_order):
    """Whole matrices of configs 1-3 at 64-row tiles of C symbols and at the
    benchmark's tiles (64 or 128 rows of C / 128 columns), in matrix order
    and with the row order (which moves config 3's outlier-free rows
    together)."""
    for spec in config_matrices(cfg):
        TR, TC = (64, spec.chunk_syms // 64) if shape == "C/64" else bench_tiles(spec)
        say("v2 config", cfg, spec.name, spec.rows, spec.cols, TR, TC, row_order)
        w = synth.weights(spec)
        alpha, _ = eq.eqe_alpha_search(w, spec.target_bits, sample_rows=1024)
        blob = eq.eqe_encode2(w, alpha, tile_rows=TR, tile_cols=TC, seed=spec.seed,
                              target_bits=spec.target_bits, row_order=row_order)
        check_full(eq, blob, spec, batches=(1, 8))


@pytest.mark.parametrize("B", [1, 3, 8])
def test_v2_gemv_multi_joint(eq, B):
    """Layers sharing an input (as q|k|v) in one version-2 launch: outputs
    identical to the single-layer launches (same per-tile work, same merge
    order) and within the bar against the oracle; layers of different tile
    heights fall back to one launch each."""
    shapes = [(300, 1024, 64, 256, 2900), (64, 1024, 64, 256, 2901), (97, 1024, 64, 128, 2902)]
    layers = []
    for M, N, TR, TC, seed in shapes:
        spec = small_spec(M, N, bits=2.0, seed=seed)
        _, blob = build(eq, spec, TR, TC, 2.0)
        layers.append((spec, blob, eq.Layer(blob, _dev())))
    spec0 = layers[0][0]
    x_bits = synth.activations(spec0, B)
    x = torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(_dev())
    Ls = [L for _, _, L in layers]
    for group in (Ls, Ls + [eq.Layer(build(eq, small_spec(40, 1024, seed=2903), 128, 256,
                                             2.0)[1], _dev())]):
        ys = [torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
              for L in group]
        eq.eq_decode_gemv_multi(group, x, B, None, ys, eq.multi_workspace(group, B))
        for L, y in zip(group, ys):
            assert np.array_equal(y.cpu().numpy(), gpu_gemv(eq, L, x_bits))
    for (spec, blob, L), y in zip(layers, ys):
        rc, q = oracle.container2_decode(blob)
        assert rc == oracle.OK
        w_ref = oracle.dequant(q, oracle.container_scales(blob))
        err = rel_err(y.cpu().numpy(), oracle.gemv(w_ref, x_bits))
        assert (err <= TOL).all(), err
        assert eq.eq_get_status(L) == eq.EQ_OK


@pytest.mark.parametrize("single_phrase", [False, True])
def test_v2_block_wise_codes_and_bf16(eq, single_phrase):
    """Block-wise decode of version-2 layers (Sec. 2.2): one launch over
    ragged layers of different widths, tile widths and base formats (with a
    single-phrase layer: the split table for all), each layer's codes and
    BF16 bit-exact against the oracle and nothing written outside its
    output; with a layer of another tile height the launch runs each block's
    tiles at its layer's height, with the same results."""
    shapes = [(130, 512, 64, 2.0, 1), (40, 640, 256, 3.0, 2), (5, 100, 32, 2.0, 1),
              (300, 1000, 256, 2.5, 1)]
    blobs, specs = [], []
    for i, (M, N, TC, bits, fmt) in enumerate(shapes):
        spec = small_spec(M, N, bits=bits, seed=2600 + i)
        w = synth.weights(spec)
        if single_phrase and i == 2:
            w = np.zeros_like(w)
        alpha, _ = eq.eqe_alpha_search(w, bits, base_format=fmt) if w.any() else (1.0, 0)
        blobs.append(eq.eqe_encode2(w, alpha, tile_rows=64, tile_cols=TC, base_format=fmt))
        specs.append(spec)
    Ls = [eq.Layer(b, _dev()) for b in blobs]
    sizes = [L.rows * L.cols for L in Ls]
    for heights in ("one", "mixed"):
        layers, bl = list(Ls), list(blobs)
        if heights == "mixed":
            spec = small_spec(200, 768, bits=2.0, seed=2650)
            w = synth.weights(spec)
            alpha, _ = eq.eqe_alpha_search(w, 2.0)
            bl.append(eq.eqe_encode2(w, alpha, tile_rows=128, tile_cols=128))
            layers.append(eq.Layer(bl[-1], _dev()))
        n = [L.rows * L.cols for L in layers]
        codes = torch.full((sum(n) + 64,), 0xA5, dtype=torch.uint8, device=_dev())
        starts = np.cumsum([0] + n)
        cviews = [codes[starts[i]:starts[i + 1]] for i in range(len(layers))]
        eq.eq_decode_codes_multi(layers, cviews)
        bufs = [torch.full((k + 8,), -1, dtype=torch.int16, device=_dev()) for k in n]
        eq.eq_decode_bf16_multi(layers, [b[:k] for b, k in zip(bufs, n)])
        assert (codes[sum(n):] == 0xA5).all()
        for L, blob, cv, b, k in zip(layers, bl, cviews, bufs, n):
            rc, q_ref = oracle.container2_decode(blob)
            assert rc == oracle.OK
            fmt = oracle.container2_info(blob).base_format
            w_ref = oracle.dequant(q_ref, oracle.container_scales(blob), fmt)
            assert np.array_equal(cv.cpu().numpy().reshape(q_ref.shape), q_ref), heights
            got = b.cpu().numpy().view(np.uint16)
            assert np.array_equal(got[:k].reshape(w_ref.shape), w_ref), heights
            assert (got[k:] == 0xFFFF).all()
            assert eq.eq_get_status(L) == eq.EQ_OK


# ---- row order: tiles cut over the rows sorted by phrase count ----

def _mixed_rows(spec):
    """Weights whose rows are of two kinds, with and without outliers (the
    rows the order groups), so that the stored order is far from the
    identity."""
    w = synth.weights(spec).copy()
    plain = synth.weights(small_spec(spec.rows, spec.cols, seed=spec.seed + 1, outliers=False))
    w[1::5] = plain[1::5]
    return w


@pytest.mark.parametrize("M,N,TR,TC,bits,outliers", EDGE)
def test_v2_row_order_edge_shapes(eq, M, N, TR, TC, bits, outliers):
    """Every entry point on ordered layers: codes and BF16 bit-exact in
    matrix order, the GEMV (merged partials, and tiles of whole rows) within
    the bar, at the edge shapes of the matrix-order case."""
    say("v2 row order edge", M, N, TR, TC, bits)
    spec = small_spec(M, N, bits=bits, seed=2000 + 7 * M + N, outliers=outliers)
    _, blob = build(eq, spec, TR, TC, bits, row_order=True)
    assert oracle.container2_info(blob).flags == 1
    check_full(eq, blob, spec)


@pytest.mark.parametrize("TR,TC", [(64, 256), (128, 128), (256, 256), (64, 1024)])
def test_v2_row_order_mixed_rows_and_offsets(eq, TR, TC):
    """Rows of two kinds in one layer: the order moves most rows; outputs
    starting 0-3 elements into a buffer are bit-exact (stores at any byte
    address) and nothing outside them is written."""
    M, N = 700, 1024
    spec = small_spec(M, N, bits=2.0, seed=2800 + TR + TC, outliers=True)
    w = _mixed_rows(spec)
    alpha, _ = eq.eqe_alpha_search(w, 2.0)
    blob = eq.eqe_encode2(w, alpha, tile_rows=TR, tile_cols=TC, row_order=True)
    order = oracle.container2_row_order(blob)
    say("v2 row order mixed", TR, TC, "rows moved", int((order != np.arange(M)).sum()))
    assert (order != np.arange(M)).sum() > M // 2
    check_full(eq, blob, spec, batches=(1, 2, 8), offsets=(0, 1, 2, 3))


def test_v2_row_order_multi(eq):
    """Joint launches over ordered and matrix-order layers together: the
    GEMV of layers sharing an input equals the single-layer launches, and
    block-wise codes and BF16 (one launch over tile heights 64 and 128) are
    bit-exact against the oracle."""
    shapes = [(300, 1024, 64, 256, True), (64, 1024, 64, 128, False),
              (97, 1024, 64, 256, True), (200, 1024, 128, 256, True)]
    layers = []
    for i, (M, N, TR, TC, ordered) in enumerate(shapes):
        spec = small_spec(M, N, bits=2.0, seed=2950 + i, outliers=True)
        w = _mixed_rows(spec)
        alpha, _ = eq.eqe_alpha_search(w, 2.0)
        blob = eq.eqe_encode2(w, alpha, tile_rows=TR, tile_cols=TC, row_order=ordered)
        layers.append((spec, blob, eq.Layer(blob, _dev())))
    Ls = [L for _, _, L in layers]
    for B in (1, 8):
        x_bits = synth.activations(layers[0][0], B)
        x = torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(_dev())
        ys = [torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
              for L in Ls]
        eq.eq_decode_gemv_multi(Ls, x, B, None, ys, eq.multi_workspace(Ls, B))
        for L, y in zip(Ls, ys):
            assert np.array_equal(y.cpu().numpy(), gpu_gemv(eq, L, x_bits)), B
    n = [L.rows * L.cols for L in Ls]
    codes = [torch.full((k + 8,), 0xA5, dtype=torch.uint8, device=_dev()) for k in n]
    bufs = [torch.full((k + 8,), -1, dtype=torch.int16, device=_dev()) for k in n]
    eq.eq_decode_codes_multi(Ls, [c[:k] for c, k in zip(codes, n)])
    eq.eq_decode_bf16_multi(Ls, [b[:k] for b, k in zip(bufs, n)])
    for (spec, blob, L), c, b, k in zip(layers, codes, bufs, n):
        rc, q_ref = oracle.container2_decode(blob)
        assert rc == oracle.OK
        w_ref = oracle.dequant(q_ref, oracle.container_scales(blob))
        got_c = c.cpu().numpy()
        got_b = b.cpu().numpy().view(np.uint16)
        assert np.array_equal(got_c[:k].reshape(q_ref.shape), q_ref)
        assert np.array_equal(got_b[:k].reshape(w_ref.shape), w_ref)
        assert (got_c[k:] == 0xA5).all() and (got_b[k:] == 0xFFFF).all()
        assert eq.eq_get_status(L) == eq.EQ_OK


@pytest.mark.parametrize("TC", [256, 1024])
def test_v2_row_order_damaged_on_device(eq, TC):
    """An order entry out of range in the device copy only (the host checked
    its own): every entry point marks the layer corrupt, keeps that row in
    place and writes nothing outside its outputs."""
    M, N = 70, 1024
    spec = small_spec(M, N, bits=2.0, seed=2990)
    _, blob = build(eq, spec, 64, TC, 2.0, row_order=True)
    info = oracle.container2_info(blob)
    L = eq.Layer(blob, _dev())
    o = info.off_order + 4 * 3
    L.dev_blob[o:o + 4] = torch.from_numpy(np.frombuffer(np.uint32(M + 5).tobytes(),
                                                         dtype=np.uint8).copy()).to(_dev())
    torch.cuda.synchronize()
    for what in ("codes", "bf16", "gemv1", "gemv8"):
        eq.eq_layer_prepare(L)
        assert eq.eq_get_status(L) == eq.EQ_OK
        if what == "codes":
            gpu_codes(eq, L, 1)
        elif what == "bf16":
            gpu_bf16(eq, L, 1)
        else:
            gpu_gemv(eq, L, synth.activations(spec, 1 if what == "gemv1" else 8))
        assert eq.eq_get_status(L) == eq.EQ_ECORRUPT, what


def test_v2_row_order_int8_and_single_phrase(eq):
    """Ordered layers through the other table and value paths: the Int8 base
    format (its own BF16 conversion at write-out), and a single-phrase layer
    (the split table; every row costs the same, so the order is the
    identity, stored and used all the same)."""
    spec = small_spec(300, 1000, bits=2.0, seed=2995, outliers=True)
    w = _mixed_rows(spec)
    alpha, _ = eq.eqe_alpha_search(w, 2.0, base_format=oracle.INT8)
    blob = eq.eqe_encode2(w, alpha, tile_rows=128, tile_cols=256, base_format=oracle.INT8,
                          row_order=True)
    assert oracle.container2_info(blob).base_format == oracle.INT8
    check_full(eq, blob, spec, batches=(1, 8), offsets=(0, 1))
    z = np.zeros((70, 512), dtype=np.uint16)
    blob = eq.eqe_encode2(z, 1.0, tile_rows=64, tile_cols=256, row_order=True)
    info = oracle.container2_info(blob)
    assert info.flags == 1 and info.n_syms == 1
    assert np.array_equal(oracle.container2_row_order(blob), np.arange(70))
    check_full(eq, blob, small_spec(70, 512, seed=2996), batches=(1, 3), offsets=(0, 3))
