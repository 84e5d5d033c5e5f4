"""Exact reference product for the fused-GEMV tests (a helper module of the
tests, not a test file).

The fused GEMV forms y_b[i] = s_i * sum_j v(q_ij) x_b[j] + bias_i from the
exact code values (Sec. 2.1: the quantised weights times their row scales,
applied once per output).  The oracle's GEMV multiplies the dequantised BF16
weights W_hat instead, whose rounding (up to 2^-9 of each weight) dominates a
comparison with it: about 1e-3 of max|y|, normwise.  exact_gemv is the
product without that rounding, in fp64 from the oracle's code values and
BF16 conversions, so that against it only the kernel's fp32 accumulation
differs (about 1e-6; one term missing from a row shows as about 1e-3).
"""
import numpy as np

import oracle

TOL_EXACT = 1e-4


def _bf16(bits):
    b = np.asarray(bits).astype(np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def exact_gemv(q, scale, x_bits, fmt=oracle.E4M3, bias_bits=None):
    """y[b][i] = s_i * sum_j v(q_ij) x_b[j] (+ bias_i) in fp64, for codes
    q [M][N], BF16 row scales [M], BF16 inputs [B][N] and an optional BF16
    bias [M]; row block by row block."""
    table = np.array([oracle.code_value(fmt, c) for c in range(256)], dtype=np.float64)
    x = _bf16(np.atleast_2d(x_bits))
    s = _bf16(scale)
    q = np.asarray(q).reshape(s.size, -1)
    y = np.empty((x.shape[0], q.shape[0]), dtype=np.float64)
    for r0 in range(0, q.shape[0], 2048):
        r1 = min(r0 + 2048, q.shape[0])
        y[:, r0:r1] = (table[q[r0:r1]] @ x.T).T * s[r0:r1]
    if bias_bits is not None:
        y += _bf16(bias_bits)
    return y


def normwise(y, y_ref):
    """max|y - y_ref| / max|y_ref| per batch row."""
    y = np.asarray(y, dtype=np.float64)
    return np.abs(y - y_ref).max(axis=1) / np.maximum(np.abs(y_ref).max(axis=1), 1e-300)
