"""eq_decode_gemv_noalloc (workspace in the library's static per-device
scratch) against eq_decode_gemv with a caller workspace: identical y, bit for
bit, on two calls in a row where the second input is smaller (the scratch
then holds the first call's contents), for each way the GEMV uses its
workspace -- version-2 partial sums over column tiles, version-1 row
partials with activation pairs, version-1 codes for rows that are not whole
steps -- and the outputs within the oracle's tolerance; a call that needs
more than the scratch fails with EQ_ESCRATCH before any device work.
"""
import sys

import numpy as np
import pytest

import oracle
import synth
from synth.configs import small_spec

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


def _v2(eq, M, N, TR, TC, seed, row_order=False):
    spec = small_spec(M, N, bits=2.0, seed=seed, outliers=row_order)
    w = synth.weights(spec)
    alpha, _ = eq.eqe_alpha_search(w, 2.0)
    return spec, eq.eqe_encode2(w, alpha, tile_rows=TR, tile_cols=TC, row_order=row_order)


def _v1(eq, M, N, C, lanes, seed):
    spec = small_spec(M, N, bits=2.5, seed=seed)
    w = synth.weights(spec)
    alpha, _ = eq.eqe_alpha_search(w, 2.5)
    return spec, eq.eqe_encode(w, alpha, chunk_syms=C, lanes=lanes)


def _inputs(spec, B, bias):
    x = synth.activations(spec, B)
    b = synth.bias(spec) if bias else None
    xt = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(_dev())
    bt = None if b is None else torch.from_numpy(b.view(np.int16)).to(_dev())
    return x, b, xt, bt


def _run_pair(eq, cases):
    """cases: [(spec, blob, B, bias)], run back to back through the no-alloc
    entry point, then each again through eq_decode_gemv."""
    layers, got = [], []
    for spec, blob, B, bias in cases:
        L = eq.Layer(blob, _dev())
        x, b, xt, bt = _inputs(spec, B, bias)
        assert eq.eq_gemv_workspace_bytes(L, B) <= eq.NOALLOC_SCRATCH_BYTES
        y = torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
        say("noalloc", spec.rows, spec.cols, "B", B, "version", L.raw.version,
            "ws", eq.eq_gemv_workspace_bytes(L, B))
        eq.eq_decode_gemv_noalloc(L, xt, B, bt, y)
        layers.append((L, x, b, xt, bt, B))
        got.append(y)
    torch.cuda.synchronize()
    for (L, x, b, xt, bt, B), y in zip(layers, got):
        ref = torch.full((B, L.rows), float("nan"), dtype=torch.float32, device=_dev())
        eq.eq_decode_gemv(L, xt, B, bt, ref, L.workspace(B))
        yn, rn = y.cpu().numpy(), ref.cpu().numpy()
        assert np.array_equal(yn.view(np.uint32), rn.view(np.uint32))
        blob = L.blob
        if oracle.container_version(blob) == 2:
            rc, q = oracle.container2_decode_par(blob)
            fmt = oracle.container2_info(blob).base_format
        else:
            rc, q = oracle.container_decode_par(blob)
            fmt = oracle.container_info(blob).base_format
        assert rc == oracle.OK
        w_ref = oracle.dequant_par(q, oracle.container_scales(blob), fmt)
        y_ref = oracle.gemv_par(w_ref, x, b)
        err = np.abs(yn - y_ref).max(axis=1) / np.maximum(np.abs(y_ref).max(axis=1), 1e-30)
        assert np.isfinite(yn).all() and (err <= TOL).all(), err
        assert eq.eq_get_status(L) == eq.EQ_OK


def test_noalloc_v2_partials(eq):
    big = _v2(eq, 1024, 4096, 256, 256, 3100)
    small = _v2(eq, 300, 1000, 64, 256, 3101)
    _run_pair(eq, [(*big, 8, True), (*small, 3, False)])


def test_noalloc_v2_row_order(eq):
    """Ordered layers (row sums merged into matrix rows, and tiles of whole
    rows written in place) through the static scratch, then a smaller one."""
    big = _v2(eq, 1024, 4096, 256, 256, 3102, row_order=True)
    whole_rows = _v2(eq, 300, 1000, 64, 1024, 3103, row_order=True)
    _run_pair(eq, [(*big, 1, True), (*whole_rows, 8, False)])


def test_noalloc_v1_row_partials(eq):
    big = _v1(eq, 512, 2048, 4096 + 1024, 256, 3200)   # rows split between chunks
    small = _v1(eq, 96, 1024, 1536, 128, 3201)
    _run_pair(eq, [(*big, 8, True), (*small, 1, True)])


def test_noalloc_v1_codes_workspace(eq):
    big = _v1(eq, 200, 1000, 2048, 64, 3300)            # 1000 not a multiple of 64
    small = _v1(eq, 37, 300, 1024, 64, 3301)
    _run_pair(eq, [(*big, 2, True), (*small, 5, False)])


def test_noalloc_rejects_oversize(eq):
    # 129 column tiles x 8192 rows x batch 8 x 4 bytes of partials > 32 MiB
    w = np.zeros((8192, 516), dtype=np.uint16)
    L = eq.Layer(eq.eqe_encode2(w, 1.0, tile_rows=64, tile_cols=4), _dev())
    assert eq.eq_gemv_workspace_bytes(L, 8) > eq.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((8, 516), dtype=torch.int16, device=_dev())
    y = torch.full((8, 8192), float("nan"), dtype=torch.float32, device=_dev())
    with pytest.raises(eq.EqError) as e:
        eq.eq_decode_gemv_noalloc(L, x, 8, None, y)
    assert e.value.code == eq.EQ_ESCRATCH
    torch.cuda.synchronize()
    assert torch.isnan(y).all()
    # a batch that fits runs
    eq.eq_decode_gemv_noalloc(L, x[:1], 1, None, y[:1])
    torch.cuda.synchronize()
    assert (y[:1] == 0).all()
