"""Scale optimisation of the encoder (Sec. 2.2, eq. optimization; Alg. 1, scale optimisation).

Oracle pins: hand-worked objective and straight-through gradient values for
single weights (E4M3 and Int8, inside and outside the clamp, both signs);
invariance under scaling W and S by a power of two; a matrix of exactly
representable weights (zero distortion, R = mean |v|); the closed-form
gradient of the regulariser; L-BFGS reaching the exact minimiser of a
coupled quadratic.  Paper-level facts on a config-1 matrix: entropy falls
and sparsity rises with lambda (Fig. entropy_vs_reg_param,
Fig. entropy_vs_sparsity), the optimised scales beat AbsMax scaled by one
factor at matched entropy (the point of eq. optimization), and the optimiser
lowers F from its AbsMax start.  Product against oracle: objective and
gradient, optimised objective, lambda search and scaled containers.
"""
import numpy as np
import pytest

import oracle
import paper_2601_22787_amd as eq
import synth
from synth.configs import config_matrices, small_spec

E4M3, INT8 = oracle.E4M3, oracle.INT8


def one(w: float) -> np.ndarray:
    return np.array([[synth.to_bf16(w)]], dtype=np.uint16)


@pytest.mark.parametrize("fmt,w,s,F0,R,gd,gr", [
    # w = 1, s = 0.3: u = 3.33.., E4M3 rounds to 3.25, Int8 to 3; dv/ds = -1/0.09
    (E4M3, 1.0, 0.3, 0.025, 3.25, 3.3333333333333335 - 3.25, -1 / 0.09),
    (INT8, 1.0, 0.3, 0.1, 3.0, 3.3333333333333335 - 3.0, -1 / 0.09),
    # the same with w = -1: the sign flips the code and dv/ds, not F or the gradient
    (E4M3, -1.0, 0.3, 0.025, 3.25, 3.3333333333333335 - 3.25, -1 / 0.09),
    # clamp active (u = 1000 > 448): v = 448, dv/ds = 0, dW_hat/ds = v
    (E4M3, 1.0, 0.001, 0.552, 448.0, -448.0, 0.0),
    (INT8, 1.0, 0.001, 0.873, 127.0, -127.0, 0.0),
])
def test_single_weight_worked_values(fmt, w, s, F0, R, gd, gr):
    for lam in (0.0, 0.5, 7.0):
        f, g, d = oracle.rd_objective(one(w), np.array([s]), lam, fmt)
        assert d == pytest.approx(F0, rel=1e-9)
        assert f == pytest.approx(F0 + lam * R, rel=1e-9)
        assert g[0] == pytest.approx(gd + lam * gr, rel=1e-7, abs=1e-9)


@pytest.fixture(scope="module")
def small():
    return synth.weights(small_spec(24, 96, seed=71))


@pytest.mark.parametrize("fmt", [E4M3, INT8])
def test_scaling_invariance(small, fmt):
    """F(2^k W, 2^k S) = F(W, S) and the gradient scales by 2^-k (d is
    relative, R sees the same codes)."""
    r = np.random.default_rng(3)
    amax = np.abs(synth.bf16_to_f32(small)).max(axis=1).astype(np.float64)
    s = amax / oracle.qmax(fmt) * r.uniform(0.5, 300.0, small.shape[0])
    f0, g0, d0 = oracle.rd_objective(small, s, 2.0, fmt)
    for k in (-3, 5):
        wk = (small.astype(np.int32) + (k << 7)).astype(np.uint16)  # exponent shift: exact
        assert np.array_equal(synth.bf16_to_f32(wk), synth.bf16_to_f32(small) * 2.0 ** k)
        f, g, d = oracle.rd_objective(wk, s * 2.0 ** k, 2.0, fmt)
        assert f == pytest.approx(f0, rel=1e-12) and d == pytest.approx(d0, rel=1e-12)
        assert np.allclose(g, g0 * 2.0 ** -k, rtol=1e-12, atol=0)


@pytest.mark.parametrize("fmt", [E4M3, INT8])
def test_exactly_representable_matrix(fmt):
    """W_ij = s_i v_ij with v in the base format and s_i a power of two:
    zero distortion and R = mean |v| (the value's l1 norm per entry)."""
    r = np.random.default_rng(9)
    if fmt == E4M3:
        codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)
    else:
        codes = np.arange(-127, 128).astype(np.int8).view(np.uint8)
    vals = np.array([oracle.code_value(fmt, int(c)) for c in codes])
    M, N = 6, 80
    v = r.choice(vals, (M, N))
    s = 2.0 ** r.integers(-8, 4, M).astype(np.float64)
    w = np.array([[synth.to_bf16(float(x)) for x in row] for row in v * s[:, None]],
                 dtype=np.uint16)
    assert np.array_equal(synth.bf16_to_f32(w).astype(np.float64), v * s[:, None])
    for lam in (0.0, 3.0):
        f, g, d = oracle.rd_objective(w, s, lam, fmt)
        assert d == 0.0
        assert f == pytest.approx(lam * np.abs(v).mean(), rel=1e-12)


def test_regulariser_gradient_closed_form():
    """With no zero code and no clamping, the straight-through derivative of
    lambda mean|W_q| is -lambda sum_j |W_ij| / (M N s_i^2)."""
    r = np.random.default_rng(4)
    M, N = 12, 64
    vals = r.choice([-1.0, 1.0], (M, N)) * r.uniform(1.0, 8.0, (M, N))
    w = np.array([[synth.to_bf16(float(x)) for x in row] for row in vals], dtype=np.uint16)
    wf = synth.bf16_to_f32(w).astype(np.float64)
    s = np.abs(wf).min(axis=1) / 1.5 * r.uniform(0.9, 1.0, M)  # every |u| >= 1.5, <= 448
    assert (np.abs(wf).max(axis=1) / s <= 448).all()
    for fmt in (E4M3, INT8):
        _, g0, _ = oracle.rd_objective(w, s, 0.0, fmt)
        _, g1, _ = oracle.rd_objective(w, s, 1.0, fmt)
        assert np.allclose(g1 - g0, -np.abs(wf).sum(axis=1) / (M * N * s ** 2), rtol=1e-10)


def test_lbfgs_reaches_quadratic_minimiser():
    """f = 1/2 sum a_i (x_i - c_i)^2 + 1/2 b (sum (x_i - c_i))^2 is strictly
    convex with minimiser c and minimum 0 (closed form)."""
    r = np.random.default_rng(2)
    n = 40
    a = r.uniform(1.0, 4.0, n)
    c = r.normal(0, 3, n)
    x, f = oracle.lbfgs_quadratic(a, 0.3, c, np.zeros(n), iters=200, history=10, lr=1.0)
    assert np.allclose(x, c, atol=1e-6) and f < 1e-10


@pytest.fixture(scope="module")
def c1_rows():
    return synth.weights(config_matrices(1)[0])[:48, :512]


def _alpha_curve(w, fmt):
    """(entropy, distortion) of AbsMax scaled by alpha over a range of alpha."""
    out = []
    for a in 2.0 ** np.arange(0, 18, 0.25):
        s = oracle.row_scales(w, float(a), fmt)
        q = oracle.quantize(w, s, fmt)
        _, _, d = oracle.rd_objective(w, synth.bf16_to_f32(s).astype(np.float64), 0.0, fmt)
        out.append((oracle.entropy_codes(q), d))
    return sorted(out)


@pytest.mark.parametrize("fmt", [E4M3, INT8])
def test_paper_rate_distortion_behaviour(c1_rows, fmt):
    w = c1_rows
    amax = np.abs(synth.bf16_to_f32(w)).max(axis=1).astype(np.float64)
    s0 = amax / oracle.qmax(fmt)
    lams = (1.0, 10.0, 100.0, 1000.0) if fmt == E4M3 else (0.03, 0.3, 3.0, 30.0)
    hs, sp, ds = [], [], []
    for lam in lams:
        s, f = oracle.rd_scales(w, lam, iters=200, fmt=fmt)
        assert f < oracle.rd_objective(w, s0, lam, fmt)[0]   # the optimiser makes progress
        q = oracle.quantize(w, _bf16(s), fmt)
        hs.append(oracle.entropy_codes(q))
        sp.append((q == 0).mean())
        ds.append(oracle.rd_objective(w, s, 0.0, fmt)[2])
    assert all(h1 > h2 for h1, h2 in zip(hs, hs[1:])), hs      # entropy falls with lambda
    assert all(a <= b for a, b in zip(sp, sp[1:])), sp         # sparsity rises
    curve = _alpha_curve(w, fmt)
    for h, d in zip(hs, ds):
        # distortion of alpha-scaled AbsMax at the same entropy (interpolated)
        d_alpha = np.interp(h, [c[0] for c in curve], [c[1] for c in curve])
        if 1.0 < h < 5.0:
            assert d < d_alpha, (h, d, d_alpha)


def _bf16(s: np.ndarray) -> np.ndarray:
    return np.array([oracle.bf16_round(float(v)) for v in s], dtype=np.uint16)


@pytest.mark.parametrize("fmt", [E4M3, INT8])
def test_product_objective_matches_oracle(small, fmt):
    r = np.random.default_rng(17)
    amax = np.abs(synth.bf16_to_f32(small)).max(axis=1).astype(np.float64)
    for scale in (1.0, 20.0, 3000.0, 0.2):
        s = amax / oracle.qmax(fmt) * scale * r.uniform(0.7, 1.4, small.shape[0])
        for lam in (0.0, 2.5):
            f0, g0, d0 = oracle.rd_objective(small, s, lam, fmt)
            f1, g1, d1 = eq.eqe_rd_objective(small, s, lam, base_format=fmt, threads=3)
            assert f1 == pytest.approx(f0, rel=1e-12) and d1 == pytest.approx(d0, rel=1e-12)
            assert np.allclose(g1, g0, rtol=1e-10, atol=1e-14 * np.abs(g0).max())


@pytest.mark.parametrize("fmt,lam", [(E4M3, 3.0), (E4M3, 300.0), (INT8, 1.0)])
def test_product_optimiser_matches_oracle(c1_rows, fmt, lam):
    w = c1_rows[:16]
    s_ref, f_ref = oracle.rd_scales(w, lam, iters=200, fmt=fmt)
    s64, s16, f = eq.eqe_rd_scales(w, lam, iters=200, base_format=fmt, threads=2)
    assert f == pytest.approx(f_ref, rel=2e-3)
    assert np.array_equal(s16, _bf16(s64))
    q_ref = oracle.quantize(w, _bf16(s_ref), fmt)
    q = oracle.quantize(w, s16, fmt)
    assert abs(oracle.entropy_codes(q) - oracle.entropy_codes(q_ref)) < 0.03


@pytest.mark.parametrize("fmt", [E4M3, INT8])
def test_lambda_search_and_scaled_container(c1_rows, fmt):
    w = c1_rows
    lam, h = eq.eqe_rd_lambda_search(w, 2.0, 0, iters=150, base_format=fmt)
    assert abs(h - 2.0) <= 0.05
    _, s16, _ = eq.eqe_rd_scales(w, lam, iters=150, base_format=fmt)
    q = oracle.quantize(w, s16, fmt)
    assert oracle.entropy_codes(q) == pytest.approx(h, abs=1e-9)
    blob = eq.eqe_encode(w, 0.0, chunk_syms=4096, lanes=64, base_format=fmt, scale_bf16=s16)
    ref = oracle.container_build_scaled(w, s16, 12, 4096, 64, fmt=fmt)
    assert np.array_equal(blob, ref)
    rc, q_dec = oracle.container_decode(blob)
    assert rc == oracle.OK and np.array_equal(q_dec, q)
    with pytest.raises(eq.EqError):  # a zero scale cannot be dequantised exactly
        bad = s16.copy()
        bad[3] = 0
        eq.eqe_encode(w, 0.0, chunk_syms=4096, lanes=64, base_format=fmt, scale_bf16=bad)
