"""HIP graph capture of the library's entry points.  A call only launches
kernels on the given stream (no allocation, memset or synchronisation), so a
serving loop can capture a layer's decode, GEMVs and prefill GEMM once and
replay them.  Every replay, with other work on the stream between replays,
must give the eager results bit for bit: every kernel adds its partial sums
in a fixed order (codes, BF16, whole-row GEMV, the general-shape GEMV over
decoded codes, GEMM with split-K).  The outputs are overwritten before each
replay, so stale values cannot pass."""
import sys

import numpy as np
import pytest

import synth
from synth.configs import small_spec

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


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


def layer(eq, M, N, C, lanes, seed):
    spec = small_spec(M, N, bits=2.0, chunk=C, lanes=lanes, seed=seed)
    w = synth.weights(spec)
    alpha, _ = eq.eqe_alpha_search(w, 2.0)
    return eq.Layer(eq.eqe_encode(w, alpha, chunk_syms=C, lanes=lanes), _dev()), spec


def xs(spec, B):
    return torch.from_numpy(synth.activations(spec, B).view(np.int16)).to(_dev())


def test_graph_replays_match_eager(eq):
    Lu, su = layer(eq, 64, 2048, 8192, 256, 6000)    # whole-row steps
    Lv, _ = layer(eq, 48, 2048, 8192, 256, 6001)
    Lg, sg = layer(eq, 37, 1000, 4096, 64, 6002)     # rows across steps (GEMV on decoded codes)
    x1, x8, xg, xb = xs(su, 1), xs(su, 8), xs(sg, 3), xs(su, 40)
    bias = torch.from_numpy(synth.bias(su).view(np.int16)).to(_dev())
    n = su.rows * su.cols
    bufs = {
        "codes": torch.empty(n, dtype=torch.uint8, device=_dev()),
        "bf16": torch.empty(n, dtype=torch.int16, device=_dev()),
        "m0": torch.empty(n, dtype=torch.int16, device=_dev()),
        "m1": torch.empty(Lv.rows * Lv.cols, dtype=torch.int16, device=_dev()),
        "c0": torch.empty(n, dtype=torch.uint8, device=_dev()),
        "c1": torch.empty(Lv.rows * Lv.cols, dtype=torch.uint8, device=_dev()),
        "y1": torch.empty(1, Lu.rows, dtype=torch.float32, device=_dev()),
        "y8": torch.empty(8, Lu.rows, dtype=torch.float32, device=_dev()),
        "yg": torch.empty(3, Lg.rows, dtype=torch.float32, device=_dev()),
        "yb": torch.empty(40, Lu.rows, dtype=torch.float32, device=_dev()),
    }
    ws1, ws8, wsg, wsb = Lu.workspace(1), Lu.workspace(8), Lg.workspace(3), Lu.gemm_workspace(40)
    assert eq.eq_gemm_codes_workspace_bytes(Lu, 40) > 0  # split-K path

    def calls():
        eq.eq_decode_codes(Lu, bufs["codes"])
        eq.eq_decode_bf16(Lu, bufs["bf16"])
        eq.eq_decode_bf16_multi([Lu, Lv], [bufs["m0"], bufs["m1"]])
        eq.eq_decode_codes_multi([Lu, Lv], [bufs["c0"], bufs["c1"]])
        eq.eq_decode_gemv(Lu, x1, 1, None, bufs["y1"], ws1)
        eq.eq_decode_gemv(Lu, x8, 8, bias, bufs["y8"], ws8)
        eq.eq_decode_gemv(Lg, xg, 3, None, bufs["yg"], wsg)
        eq.eq_decode_gemm(Lu, xb, 40, None, bufs["yb"], wsb)

    calls()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in bufs.items()}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        calls()
    for rep in range(3):
        say("replay", rep)
        for v in bufs.values():
            v.fill_(-1 if v.dtype != torch.float32 else float("nan"))
        # other work on the stream between replays
        other = torch.empty(1, Lu.rows, dtype=torch.float32, device=_dev())
        eq.eq_decode_gemv(Lu, x1, 1, None, other, Lu.workspace(1))
        (torch.randn(256, 256, device=_dev()) @ torch.randn(256, 256, device=_dev())).sum()
        g.replay()
        torch.cuda.synchronize()
        for k in bufs:
            assert torch.equal(bufs[k], ref[k]), (rep, k)
        assert torch.equal(other, ref["y1"])
    for L in (Lu, Lv, Lg):
        assert eq.eq_get_status(L) == eq.EQ_OK


def layer2(eq, M, N, TR, TC, seed, row_order=False):
    spec = small_spec(M, N, bits=2.0, seed=seed, outliers=row_order)
    w = synth.weights(spec)
    alpha, _ = eq.eqe_alpha_search(w, 2.0)
    blob = eq.eqe_encode2(w, alpha, tile_rows=TR, tile_cols=TC, row_order=row_order)
    return eq.Layer(blob, _dev()), spec


@pytest.mark.parametrize("row_order", [False, True])
def test_graph_replays_match_eager_v2(eq, row_order):
    """The same for container version 2 (in matrix order, and with the row
    order): codes and BF16 (rings in LDS), the GEMV at batch 1 and 8 with its
    column-tile merge, the joint GEMV of two layers sharing an input,
    block-wise codes, and the no-alloc GEMV (its static scratch address is
    taken on the eager call before capture)."""
    La, sa = layer2(eq, 300, 1024, 256, 256, 6100, row_order)
    Lb, _ = layer2(eq, 70, 1024, 256, 256, 6101)
    x1, x8 = xs(sa, 1), xs(sa, 8)
    bias = torch.from_numpy(synth.bias(sa).view(np.int16)).to(_dev())
    n = sa.rows * sa.cols
    bufs = {
        "codes": torch.empty(n, dtype=torch.uint8, device=_dev()),
        "bf16": torch.empty(n, dtype=torch.int16, device=_dev()),
        "c0": torch.empty(n, dtype=torch.uint8, device=_dev()),
        "c1": torch.empty(Lb.rows * Lb.cols, dtype=torch.uint8, device=_dev()),
        "y1": torch.empty(1, La.rows, dtype=torch.float32, device=_dev()),
        "y8": torch.empty(8, La.rows, dtype=torch.float32, device=_dev()),
        "ja": torch.empty(8, La.rows, dtype=torch.float32, device=_dev()),
        "jb": torch.empty(8, Lb.rows, dtype=torch.float32, device=_dev()),
        "na": torch.empty(8, La.rows, dtype=torch.float32, device=_dev()),
    }
    ws1, ws8, wsm = La.workspace(1), La.workspace(8), eq.multi_workspace([La, Lb], 8)

    def calls():
        eq.eq_decode_codes(La, bufs["codes"])
        eq.eq_decode_bf16(La, bufs["bf16"])
        eq.eq_decode_codes_multi([La, Lb], [bufs["c0"], bufs["c1"]])
        eq.eq_decode_gemv(La, x1, 1, None, bufs["y1"], ws1)
        eq.eq_decode_gemv(La, x8, 8, bias, bufs["y8"], ws8)
        eq.eq_decode_gemv_multi([La, Lb], x8, 8, None, [bufs["ja"], bufs["jb"]], wsm)
        eq.eq_decode_gemv_noalloc(La, x8, 8, bias, bufs["na"])

    calls()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in bufs.items()}
    assert torch.equal(ref["na"], ref["y8"]) and torch.equal(ref["c0"], ref["codes"])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        calls()
    for rep in range(3):
        say("replay v2", rep)
        for v in bufs.values():
            v.fill_(-1 if v.dtype != torch.float32 else float("nan"))
        other = torch.empty(1, La.rows, dtype=torch.float32, device=_dev())
        eq.eq_decode_gemv(La, x1, 1, None, other, La.workspace(1))
        (torch.randn(256, 256, device=_dev()) @ torch.randn(256, 256, device=_dev())).sum()
        g.replay()
        torch.cuda.synchronize()
        for k in bufs:
            assert torch.equal(bufs[k], ref[k]), (rep, k)
        assert torch.equal(other, ref["y1"])
    for L in (La, Lb):
        assert eq.eq_get_status(L) == eq.EQ_OK
