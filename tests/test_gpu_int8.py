"""GPU parity of the Int8 base format (the paper's alternative to Float8,
Sec. 3.5; symmetric quantiser of Sec. 2.1 with Qmax = 127).

Same bars as for E4M3: codes and dequantised BF16 weights bit-exact against
the oracle (decoded with the Int8 value of each code), the fused GEMV within
max|y - y_ref| / max|y_ref| <= 1e-2 per batch row against the oracle's fp64
GEMV on the decoded weights.  The shapes cover every kernel path: general
shapes (rows not whole steps), whole-row steps at 64, 128 and 256 lanes,
activations staged whole or in tiles (batch 8 on wide rows), block-wise
launches, and the full-size 8192x28672 / 28672x8192 pair.
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
INT8 = oracle.INT8


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


def encode8(eq, w, bits, C, lanes, sample_rows=0):
    alpha, _ = eq.eqe_alpha_search(w, bits, sample_rows=sample_rows, base_format=eq.FMT_INT8)
    return eq.eqe_encode(w, alpha, chunk_syms=C, lanes=lanes, base_format=eq.FMT_INT8)


def gpu_codes(eq, L):
    out = torch.empty(L.rows * L.cols, dtype=torch.uint8, device=_dev())
    eq.eq_decode_codes(L, out)
    return out.cpu().numpy().reshape(L.rows, L.cols)


def gpu_bf16(eq, L):
    out = torch.empty(L.rows * L.cols, dtype=torch.int16, device=_dev())
    eq.eq_decode_bf16(L, out)
    return out.cpu().numpy().view(np.uint16).reshape(L.rows, L.cols)


def gpu_gemv(eq, L, x_bits, bias_bits=None):
    B = x_bits.shape[0]
    x = torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(_dev())
    bias = None if bias_bits is None else torch.from_numpy(bias_bits.view(np.int16)).to(_dev())
    y = torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
    eq.eq_decode_gemv(L, x, B, bias, y, L.workspace(B))
    return y.cpu().numpy()


def rel_err(y, y_ref):
    return np.abs(y - y_ref).max(axis=1) / np.maximum(np.abs(y_ref).max(axis=1), 1e-30)


def oracle_bf16(blob):
    rc, q = oracle.container_decode(blob)
    assert rc == oracle.OK
    return q, oracle.dequant(q, oracle.container_scales(blob), INT8)


def check_full(eq, blob, spec_like, batches):
    L = eq.Layer(blob, _dev())
    assert L.base_format == eq.FMT_INT8
    q_ref, w_ref = oracle_bf16(blob)
    assert np.array_equal(gpu_codes(eq, L), q_ref), "codes differ"
    assert np.array_equal(gpu_bf16(eq, L), w_ref), "bf16 differs"
    for B in batches:
        x = synth.activations(spec_like, B)
        bias = synth.bias(spec_like)
        y = gpu_gemv(eq, L, x, bias)
        err = rel_err(y, oracle.gemv(w_ref, x, bias))
        assert np.isfinite(y).all() and (err <= TOL).all(), (B, err)
        y_ex = exact_gemv(q_ref, oracle.container_scales(blob), x, INT8, bias)
        assert (normwise(y, y_ex) <= TOL_EXACT).all(), (B, normwise(y, y_ex))
    assert eq.eq_get_status(L) == eq.EQ_OK
    return L


EDGE = [
    # M, N, C, lanes, bits, outliers
    (3, 77, 128, 64, 3.0, False),       # ragged N, partial last chunk (general shapes)
    (5, 100, 256, 256, 2.0, False),     # N < W: steps span several rows
    (40, 640, 1024, 64, 2.0, False),    # rows split between chunks, 64 lanes
    (64, 512, 4096, 128, 4.0, True),    # 128 lanes: paired in-register conversion
    (37, 1280, 65536, 256, 2.0, False),  # 256 lanes, single partial chunk
    (16, 4160, 8192, 256, 3.0, False),  # ragged at 256 lanes; B = 8 from global memory
    (24, 4352, 8192, 256, 2.0, False),  # B = 8 too large for LDS: tiled activations
    (32, 4224, 4096, 128, 3.0, True),   # tiled at 128 lanes
]


@pytest.mark.parametrize("M,N,C,lanes,bits,outliers", EDGE)
def test_int8_edge_shapes(eq, M, N, C, lanes, bits, outliers):
    say("int8 edge", M, N, C, lanes, bits)
    spec = small_spec(M, N, bits=bits, chunk=C, lanes=lanes, seed=2000 + M * 7 + N,
                      outliers=outliers)
    w = synth.weights(spec)
    check_full(eq, encode8(eq, w, bits, C, lanes), spec, batches=(1, 3, 8))


@pytest.mark.parametrize("lanes", [64, 256])
def test_every_int8_code(eq, lanes):
    """All 255 codes of [-127, 127]: row i holds v * 2^(i-2) for every v, so
    AbsMax (alpha = 1) gives s_i = 2^(i-2) and q = v exactly.  Decode,
    dequantisation and the GEMV's conversion of every code are checked; a
    one-hot input gives y_i = s_i * v(q_ij) exactly."""
    say("int8 every code", lanes)
    vals = np.arange(-127, 128, dtype=np.float64)
    M, N = 6, 512
    w = np.zeros((M, N), dtype=np.uint16)
    for i in range(M):
        row = np.resize(np.roll(vals, 41 * i), N) * (2.0 ** (i - 2))
        w[i] = [synth.to_bf16(float(v)) for v in row]
    blob = eq.eqe_encode(w, 1.0, chunk_syms=1024, lanes=lanes, base_format=eq.FMT_INT8)
    q_ref, _ = oracle_bf16(blob)
    assert len(np.unique(q_ref)) == 255 and not (q_ref == 0x80).any()
    assert np.array_equal(q_ref.view(np.int8).astype(np.float64) *
                          (2.0 ** (np.arange(M) - 2))[:, None], synth.bf16_to_f32(w))
    spec = small_spec(M, N, chunk=1024, lanes=lanes, seed=4)
    L = check_full(eq, blob, spec, batches=(1, 2))
    scale = synth.bf16_to_f32(oracle.container_scales(blob)).astype(np.float64)
    for j0 in range(0, N, 64):
        x = np.zeros((8, N), dtype=np.uint16)
        for b in range(8):
            x[b, j0 + 8 * b + 3] = 0x3F80
        y = gpu_gemv(eq, L, x)
        for b in range(8):
            exact = scale * q_ref[:, j0 + 8 * b + 3].view(np.int8).astype(np.float64)
            assert np.array_equal(y[b].astype(np.float64), exact), (j0, b)


def test_int8_block_wise_and_mixed_formats(eq):
    """Block-wise launches of Int8 layers equal the single-layer paths and the
    oracle; a call mixing E4M3 and Int8 layers runs each layer on its own and
    gives the same results."""
    shapes = [(512, 2048, 8192, 256, 2.0), (128, 2048, 8192, 256, 3.0),
              (96, 2048, 4096, 256, 4.0)]
    layers = []
    for i, (M, N, C, lanes, bits) in enumerate(shapes):
        spec = small_spec(M, N, bits=bits, chunk=C, lanes=lanes, seed=3000 + i)
        w = synth.weights(spec)
        blob = encode8(eq, w, bits, C, lanes)
        layers.append((eq.Layer(blob, _dev()), blob, spec))
    w4 = synth.weights(small_spec(64, 2048, seed=3100))
    blob4 = eq.eqe_encode(w4, eq.eqe_alpha_search(w4, 2.0)[0], chunk_syms=8192, lanes=256)
    e4m3 = (eq.Layer(blob4, _dev()), blob4, None)
    for group, name in ((layers, "int8 joint"), (layers[:1] + [e4m3] + layers[1:], "mixed")):
        say("int8 block-wise", name)
        Ls = [L for L, _, _ in group]
        outs = [torch.full((L.rows * L.cols,), -1, dtype=torch.int16, device=_dev()) for L in Ls]
        eq.eq_decode_bf16_multi(Ls, outs)
        for (L, blob, _), out in zip(group, outs):
            got = out.cpu().numpy().view(np.uint16).reshape(L.rows, L.cols)
            assert np.array_equal(got, gpu_bf16(eq, L))
            if L.base_format == eq.FMT_INT8:
                assert np.array_equal(got, oracle_bf16(blob)[1])
        for B in (1, 8):
            x_bits = synth.activations(group[0][2], B)
            x = torch.from_numpy(x_bits.view(np.int16)).to(_dev())
            ys = [torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
                  for L in Ls]
            eq.eq_decode_gemv_multi(Ls, x, B, None, ys, eq.multi_workspace(Ls, B))
            for (L, blob, _), y in zip(group, ys):
                y1 = torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
                eq.eq_decode_gemv(L, x, B, None, y1, L.workspace(B))
                assert torch.equal(y, y1), (name, B)
                if L.base_format == eq.FMT_INT8:
                    err = rel_err(y.cpu().numpy(), oracle.gemv(oracle_bf16(blob)[1], x_bits))
                    assert (err <= TOL).all(), err
        for L in Ls:
            assert eq.eq_get_status(L) == eq.EQ_OK


def test_int8_config4_whole(eq):
    """The 8192x28672 and 28672x8192 layers coded as Int8 at ~2 bits, in the
    launch configuration of the benchmark, whole: codes against the oracle's
    decode and quantiser, BF16 against its dequantiser, every GEMV output at
    B = 1 and 8 against its fp64 GEMV."""
    for spec in config_matrices(4):
        say("int8 config 4", spec.name)
        w = synth.weights(spec)
        blob = encode8(eq, w, spec.target_bits, spec.chunk_syms, spec.lanes, sample_rows=512)
        info = oracle.container_info(blob)
        assert info.base_format == INT8 and abs(info.entropy_bits - spec.target_bits) <= 0.05
        L = eq.Layer(blob, _dev())
        scale = oracle.container_scales(blob)
        rc, q_ref = oracle.container_decode_par(blob)
        assert rc == oracle.OK
        assert np.array_equal(oracle.quantize_par(w, scale, INT8), q_ref)
        w_ref = oracle.dequant_par(q_ref, scale, INT8)
        assert np.array_equal(gpu_codes(eq, L), q_ref)
        assert np.array_equal(gpu_bf16(eq, L), w_ref)
        assert eq.eq_get_status(L) == eq.EQ_OK
        for B in (1, 8):
            x = synth.activations(spec, B)
            y = gpu_gemv(eq, L, x)
            err = rel_err(y, oracle.gemv_par(w_ref, x))
            assert np.isfinite(y).all() and (err <= TOL).all(), (spec.name, B, err)
        del L, w_ref, q_ref
