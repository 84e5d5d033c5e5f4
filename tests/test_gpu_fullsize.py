"""Whole-matrix GPU parity at the full sizes of the Llama-70B workloads.

Config 4 (the 8192x28672 / 28672x8192 MLP pair) and the three distinct layers
of the config-5 stack (one per entropy class, all seven matrices) are
compared element by element against the oracle, with no sampling:
  - codes (Alg. 2, entropy decoding and view) and BF16 weights (plus the dequantiser of
    Sec. 2.1) bit-exact, through the single-layer entry points and through
    the block-wise launches (Sec. 2.2 block-wise decompression: to BF16 as
    the benchmark times it, and to one code buffer for the whole block);
  - the codes also equal the oracle quantiser applied to the generated
    weights;
  - every output of the fused GEMV (Alg. 2, QMatMul) within the normwise bar
    max|y - y_ref| / max|y_ref| <= 1e-2 per batch row against the oracle's
    fp64 GEMV on the decoded BF16 weights; the elementwise error over the
    entries with |y_ref| >= 1e-3 max|y_ref| is printed beside it.  That
    comparison is dominated by the rounding of W_hat to BF16 (about 1e-3),
    which the fused GEMV never does: it forms s_i * sum_j v(q_ij) x_j from
    the exact code values.  So every output is also held to 1e-4 (normwise)
    of that exact product in fp64, where only the fp32 accumulation differs
    (about 1e-6 expected; one missing term of a row would be about 1e-3).
The same checks run on version-2 containers of the same matrices (tiles of
256 x 256 for the 65536-symbol chunks), the containers of the benchmark's
target row and of its version-2 leg.
The oracle decodes chunk by chunk on several host threads (chunks are
independent), which gives its single-threaded result exactly.
"""
import sys

import numpy as np
import pytest

import oracle
import synth
from gemv_ref import TOL_EXACT, exact_gemv
from synth.configs import config_matrices

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


def errors(y, y_ref):
    """(normwise, elementwise) error per batch row: max|dy| / max|y_ref|, and
    max |dy| / |y_ref| over entries with |y_ref| >= 1e-3 max|y_ref|."""
    d = np.abs(y.astype(np.float64) - y_ref)
    m = np.abs(y_ref).max(axis=1, keepdims=True)
    norm = d.max(axis=1) / np.maximum(m[:, 0], 1e-300)
    big = np.abs(y_ref) >= 1e-3 * m
    elem = np.where(big, d / np.maximum(np.abs(y_ref), 1e-300), 0.0).max(axis=1)
    return norm, elem


def build(eq, spec):
    w = synth.weights(spec)
    alpha, _ = eq.eqe_alpha_search(w, spec.target_bits, sample_rows=512)
    blob = eq.eqe_encode(w, alpha, chunk_syms=spec.chunk_syms, lanes=spec.lanes, seed=spec.seed,
                         target_bits=spec.target_bits)
    assert abs(oracle.container_info(blob).entropy_bits - spec.target_bits) <= 0.05
    return w, blob


def v2_tiles(spec):
    """Tile shape of the version-2 containers the benchmark times: 256
    columns for 65536-symbol chunks, C / 128 below; the taller of (256, 128),
    or (128, 64) below 65536 symbols, when the matrix has at least 2048 such
    tiles, else the shorter."""
    tall, tc = (256, 256) if spec.chunk_syms >= 65536 else (128, spec.chunk_syms // 128)
    tiles = -(-spec.rows // tall) * -(-spec.cols // tc)
    return (tall if tiles >= 2048 else tall // 2), tc


def build2(eq, spec, row_order=False):
    w = synth.weights(spec)
    alpha, _ = eq.eqe_alpha_search(w, spec.target_bits, sample_rows=512)
    tr, tc = v2_tiles(spec)
    blob = eq.eqe_encode2(w, alpha, tile_rows=tr, tile_cols=tc, seed=spec.seed,
                          target_bits=spec.target_bits, row_order=row_order)
    assert oracle.container_version(blob) == 2
    return w, blob


def reference(w, blob):
    """Oracle codes and BF16 weights of a whole container (either version)."""
    if oracle.container_version(blob) == 2:
        rc, q_ref = oracle.container2_decode_par(blob)
    else:
        rc, q_ref = oracle.container_decode_par(blob)
    assert rc == oracle.OK
    scale = oracle.container_scales(blob)
    assert np.array_equal(oracle.quantize_par(w, scale), q_ref)
    return q_ref, oracle.dequant_par(q_ref, scale)


def gpu_codes(eq, L):
    out = torch.empty(L.rows * L.cols, dtype=torch.uint8, device=_dev())
    eq.eq_decode_codes(L, out)
    return out.cpu().numpy().reshape(L.rows, L.cols)


def to_np_bf16(t, L):
    return t.cpu().numpy().view(np.uint16).reshape(L.rows, L.cols)


def check_gemv(eq, name, L, w_ref, x_bits, y, q_ref, scale):
    y_ref = oracle.gemv_par(w_ref, x_bits)
    norm, elem = errors(y, y_ref)
    exact, _ = errors(y, exact_gemv(q_ref, scale, x_bits))
    say(f"  {name} B={x_bits.shape[0]} GEMV error normwise {norm.max():.2e} "
        f"elementwise {elem.max():.2e}; against the exact product {exact.max():.2e}")
    assert np.isfinite(y).all() and (norm <= TOL).all(), (name, norm)
    assert (exact <= TOL_EXACT).all(), (name, exact)


def gemv_single(eq, L, x_bits):
    B = x_bits.shape[0]
    x = torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(_dev())
    y = torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
    eq.eq_decode_gemv(L, x, B, None, y, L.workspace(B))
    return y.cpu().numpy()


def test_config4_whole_matrices(eq):
    """Both config-4 matrices, every chunk and every GEMV row: codes; BF16
    through the block-wise launch of the pair (7168 chunks in one grid, as the
    benchmark launches it) and through the single-layer entry point; GEMV at
    B = 1 and B = 8 through the launches the benchmark times."""
    layers = []
    for spec in config_matrices(4):
        say("config 4 build", spec.name, spec.rows, spec.cols)
        w, blob = build(eq, spec)
        layers.append((spec, w, blob, eq.Layer(blob, _dev())))
    Ls = [L for _, _, _, L in layers]
    outs = [torch.full((L.rows * L.cols,), -1, dtype=torch.int16, device=_dev()) for L in Ls]
    eq.eq_decode_bf16_multi(Ls, outs)
    # the pair's codes into one block buffer (one launch), as the prefill reads them
    sizes = [L.rows * L.cols for L in Ls]
    block = torch.full((sum(sizes) + 64,), 0xA5, dtype=torch.uint8, device=_dev())
    views = [block[:sizes[0]], block[sizes[0]:sizes[0] + sizes[1]]]
    eq.eq_decode_codes_multi(Ls, views)
    assert (block[sum(sizes):] == 0xA5).all()
    for (spec, w, blob, L), out, cv in zip(layers, outs, views):
        say("config 4 parity", spec.name)
        q_ref, w_ref = reference(w, blob)
        assert np.array_equal(gpu_codes(eq, L), q_ref), spec.name
        assert np.array_equal(cv.cpu().numpy().reshape(L.rows, L.cols), q_ref), spec.name
        assert np.array_equal(to_np_bf16(out, L), w_ref), spec.name
        one = torch.empty(L.rows * L.cols, dtype=torch.int16, device=_dev())
        eq.eq_decode_bf16(L, one)
        assert torch.equal(one, out)
        del one
        for B in (1, 8):
            x_bits = synth.activations(spec, B)
            check_gemv(eq, spec.name, L, w_ref, x_bits, gemv_single(eq, L, x_bits), q_ref,
                       oracle.container_scales(blob))
        assert eq.eq_get_status(L) == eq.EQ_OK
        del w_ref, q_ref


# Inputs of a config-5 block: attention input (q, k, v), o input, MLP input
# (gate, up), down input.
GROUPS = ((("q", "k", "v"), 8192), (("o",), 8192), (("gate", "up"), 8192), (("down",), 28672))


@pytest.mark.parametrize("layer", [0, 1, 2])
def test_config5_layer_whole(eq, layer):
    """One config-5 layer of each entropy class (layer l at (2, 3, 4)[l mod 3]
    bits), all seven matrices whole: codes and BF16 through the single-layer
    entry points and through one block-wise BF16 launch of the whole layer;
    the GEMV at B = 1 through the block-wise launches the benchmark times
    (q|k|v, o, gate|up, down sharing their inputs) and per matrix."""
    specs = {s.name.split(".")[-1]: s for s in config_matrices(5, layers=[layer])}
    built = {}
    for n, spec in specs.items():
        say("config 5 build", layer, n, spec.rows, spec.cols, spec.target_bits)
        w, blob = build(eq, spec)
        built[n] = (w, blob, eq.Layer(blob, _dev()))
    names = list(specs)
    Ls = [built[n][2] for n in names]
    outs = [torch.full((L.rows * L.cols,), -1, dtype=torch.int16, device=_dev()) for L in Ls]
    eq.eq_decode_bf16_multi(Ls, outs)
    # the whole layer's codes into one block buffer by one launch
    sizes = [L.rows * L.cols for L in Ls]
    block = torch.full((sum(sizes) + 64,), 0xA5, dtype=torch.uint8, device=_dev())
    starts = np.cumsum([0] + sizes)
    code_views = [block[starts[i]:starts[i + 1]] for i in range(len(Ls))]
    eq.eq_decode_codes_multi(Ls, code_views)
    assert (block[sum(sizes):] == 0xA5).all()
    ys = {}
    for i, (g, ncols) in enumerate(GROUPS):
        x_bits = synth.vector(0x5EED, 16 + i, ncols).reshape(1, ncols)
        x = torch.from_numpy(x_bits.view(np.int16)).to(_dev()).view(1, ncols)
        gl = [built[n][2] for n in g]
        gy = [torch.full((1, L.rows), float("nan"), dtype=torch.float32, device=_dev())
              for L in gl]
        eq.eq_decode_gemv_multi(gl, x, 1, None, gy, eq.multi_workspace(gl, 1))
        for n, y in zip(g, gy):
            ys[n] = (x_bits, y.cpu().numpy())
    for n, out, cv in zip(names, outs, code_views):
        w, blob, L = built[n]
        say("config 5 parity", layer, n)
        q_ref, w_ref = reference(w, blob)
        assert np.array_equal(gpu_codes(eq, L), q_ref), n
        assert np.array_equal(cv.cpu().numpy().reshape(L.rows, L.cols), q_ref), n
        assert np.array_equal(to_np_bf16(out, L), w_ref), n
        one = torch.empty(L.rows * L.cols, dtype=torch.int16, device=_dev())
        eq.eq_decode_bf16(L, one)
        assert torch.equal(one, out), n
        del one
        x_bits, y_blk = ys[n]
        assert np.array_equal(y_blk, gemv_single(eq, L, x_bits)), n
        check_gemv(eq, n, L, w_ref, x_bits, y_blk, q_ref, oracle.container_scales(blob))
        assert eq.eq_get_status(L) == eq.EQ_OK
        del w_ref, q_ref


@pytest.mark.parametrize("row_order", [False, True])
def test_config4_whole_matrices_v2(eq, row_order):
    """Version-2 containers of both config-4 matrices (256 x 256 tiles, the
    target row's container; with and without the row order), every tile and
    every row: codes and BF16 through the single-layer entry points; the GEMV
    at B = 1 (the target row), 3 (the pair table of 4 rows) and 8 (the pair
    table in two halves)."""
    for spec in config_matrices(4):
        say("config 4 version 2 build", spec.name, spec.rows, spec.cols, row_order)
        w, blob = build2(eq, spec, row_order)
        L = eq.Layer(blob, _dev())
        say("config 4 version 2 parity", spec.name)
        q_ref, w_ref = reference(w, blob)
        assert np.array_equal(gpu_codes(eq, L), q_ref), spec.name
        out = torch.full((L.rows * L.cols,), -1, dtype=torch.int16, device=_dev())
        eq.eq_decode_bf16(L, out)
        assert np.array_equal(to_np_bf16(out, L), w_ref), spec.name
        del out
        for B in (1, 3, 8):
            x_bits = synth.activations(spec, B)
            check_gemv(eq, spec.name, L, w_ref, x_bits, gemv_single(eq, L, x_bits), q_ref,
                       oracle.container_scales(blob))
        assert eq.eq_get_status(L) == eq.EQ_OK
        del w_ref, q_ref, L


@pytest.mark.parametrize("layer,row_order", [(0, False), (1, False), (2, False), (0, True)])
def test_config5_layer_whole_v2(eq, layer, row_order):
    """Version-2 containers of one config-5 layer of each entropy class (and
    one with the row order), all seven matrices whole: codes and BF16 through
    the single-layer entry points and the block-wise calls; the GEMV at B = 1
    through the joint launches the benchmark times (q|k|v and gate|up in one
    launch each, o and down alone), equal to the per-matrix launches and
    against the oracle."""
    specs = {s.name.split(".")[-1]: s for s in config_matrices(5, layers=[layer])}
    built = {}
    for n, spec in specs.items():
        say("config 5 version 2 build", layer, n, spec.rows, spec.cols, spec.target_bits,
            row_order)
        w, blob = build2(eq, spec, row_order)
        built[n] = (w, blob, eq.Layer(blob, _dev()))
    names = list(specs)
    Ls = [built[n][2] for n in names]
    outs = [torch.full((L.rows * L.cols,), -1, dtype=torch.int16, device=_dev()) for L in Ls]
    eq.eq_decode_bf16_multi(Ls, outs)
    sizes = [L.rows * L.cols for L in Ls]
    block = torch.full((sum(sizes) + 64,), 0xA5, dtype=torch.uint8, device=_dev())
    starts = np.cumsum([0] + sizes)
    code_views = [block[starts[i]:starts[i + 1]] for i in range(len(Ls))]
    eq.eq_decode_codes_multi(Ls, code_views)
    assert (block[sum(sizes):] == 0xA5).all()
    ys = {}
    for i, (g, ncols) in enumerate(GROUPS):
        x_bits = synth.vector(0x5EED, 16 + i, ncols).reshape(1, ncols)
        x = torch.from_numpy(x_bits.view(np.int16)).to(_dev()).view(1, ncols)
        gl = [built[n][2] for n in g]
        gy = [torch.full((1, L.rows), float("nan"), dtype=torch.float32, device=_dev())
              for L in gl]
        eq.eq_decode_gemv_multi(gl, x, 1, None, gy, eq.multi_workspace(gl, 1))
        for n, y in zip(g, gy):
            ys[n] = (x_bits, y.cpu().numpy())
    for n, out, cv in zip(names, outs, code_views):
        w, blob, L = built[n]
        say("config 5 version 2 parity", layer, n)
        q_ref, w_ref = reference(w, blob)
        assert np.array_equal(gpu_codes(eq, L), q_ref), n
        assert np.array_equal(cv.cpu().numpy().reshape(L.rows, L.cols), q_ref), n
        assert np.array_equal(to_np_bf16(out, L), w_ref), n
        x_bits, y_blk = ys[n]
        assert np.array_equal(y_blk, gemv_single(eq, L, x_bits)), n
        check_gemv(eq, n, L, w_ref, x_bits, y_blk, q_ref, oracle.container_scales(blob))
        assert eq.eq_get_status(L) == eq.EQ_OK
        del w_ref, q_ref
