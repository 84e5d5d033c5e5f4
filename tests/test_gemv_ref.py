"""The exact GEMV reference of the GPU tests (gemv_ref.exact_gemv) against a
scalar loop over the definition y_b[i] = s_i * sum_j v(q_ij) x_b[j] + bias_i,
on tiny seeded inputs, for both base formats, with and without bias."""
import numpy as np
import pytest

import oracle
from gemv_ref import exact_gemv, normwise


def scalar_gemv(q, scale, x, fmt, bias):
    M, N = q.shape
    y = np.zeros((x.shape[0], M))
    for b in range(x.shape[0]):
        for i in range(M):
            acc = 0.0
            for j in range(N):
                acc += oracle.code_value(fmt, int(q[i, j])) * oracle.bf16_value(int(x[b, j]))
            y[b, i] = oracle.bf16_value(int(scale[i])) * acc
            if bias is not None:
                y[b, i] += oracle.bf16_value(int(bias[i]))
    return y


def bf16_bits(rng, shape):
    return (rng.standard_normal(shape).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


@pytest.mark.parametrize("fmt", [oracle.E4M3, oracle.INT8])
@pytest.mark.parametrize("with_bias", [False, True])
def test_exact_gemv_matches_scalar_loop(fmt, with_bias):
    rng = np.random.default_rng(7 + fmt)
    M, N, B = 19, 53, 3
    w = bf16_bits(rng, (M, N))
    scale = oracle.row_scales(w, 1.0, fmt)
    q = oracle.quantize(w, scale, fmt)
    x = bf16_bits(rng, (B, N))
    bias = bf16_bits(rng, (M,)) if with_bias else None
    y = exact_gemv(q, scale, x, fmt, bias)
    ref = scalar_gemv(q, scale, x, fmt, bias)
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_exact_gemv_differs_from_bf16_weights_by_their_rounding():
    """The oracle's GEMV on BF16 W_hat differs from the exact product by the
    rounding of each weight (at most 2^-9 of it): the normwise gap is
    nonzero and below 2^-9 * max_i sum_j |w_ij x_j| / max|y|."""
    rng = np.random.default_rng(3)
    M, N = 64, 512
    w = bf16_bits(rng, (M, N))
    scale = oracle.row_scales(w, 1.0)
    q = oracle.quantize(w, scale)
    x = bf16_bits(rng, (2, N))
    y_ex = exact_gemv(q, scale, x)
    y_w = oracle.gemv(oracle.dequant(q, scale), x)
    gap = normwise(y_w, y_ex)
    table = np.array([oracle.code_value(oracle.E4M3, c) for c in range(256)])
    s = (scale.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    xf = (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    bound = 2.0 ** -9 * (np.abs(table[q] * s[:, None]) @ np.abs(xf).T).T.max(axis=1)
    assert (gap > 0).all() and (gap * np.abs(y_ex).max(axis=1) <= bound).all()
