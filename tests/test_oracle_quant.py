"""Oracle quantiser / dequantiser / scale choice (Sec. 2.1; Alg. 1: AbsMax
initialisation, scale choice, quantisation).

Pins: torch's float32 -> float8_e4m3fn cast (round to nearest even) for Q,
torch's float32 -> bfloat16 cast of the exact product for the dequantiser,
AbsMax mapping the row maximum to +-Qmax, nearest-BF16 property of the scales,
and the qualitative facts of Tab. unique_val.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth.configs import small_spec


def _f32(bits):
    return synth.bf16_to_f32(bits)


@pytest.fixture(scope="module")
def small_w():
    return synth.weights(small_spec(192, 320, seed=11))


def test_quantize_matches_torch_cast(small_w):
    for alpha in (1.0, 37.5, 41547.44):
        s = oracle.row_scales(small_w, alpha)
        q = oracle.quantize(small_w, s)
        v = torch.from_numpy(_f32(small_w)) / torch.from_numpy(_f32(s))[:, None]
        ref = v.clamp(-448, 448).to(torch.float8_e4m3fn).view(torch.uint8).numpy().copy()
        ref[ref == 0x80] = 0
        assert (q == ref).all(), alpha


def test_absmax_maps_row_max_to_qmax(small_w):
    s = oracle.row_scales(small_w, 1.0)
    q = oracle.quantize(small_w, s)
    a = np.abs(_f32(small_w))
    jmax = a.argmax(axis=1)
    top = q[np.arange(q.shape[0]), jmax]
    assert np.isin(top, [0x7E, 0xFE]).all()


def test_scales_are_nearest_bf16(small_w):
    alpha = 3.7
    s = oracle.row_scales(small_w, alpha)
    amax = np.abs(_f32(small_w).astype(np.float64)).max(axis=1)
    target = np.float64(np.float32(alpha)) * amax / 448.0
    sv = _f32(s).astype(np.float64)
    up = _f32((s + 1).astype(np.uint16)).astype(np.float64)
    dn = _f32((s - 1).astype(np.uint16)).astype(np.float64)
    err = np.abs(sv - target)
    assert (err <= np.abs(up - target)).all() and (err <= np.abs(dn - target)).all()


def test_zero_row_gets_unit_scale():
    w = np.zeros((3, 64), dtype=np.uint16)
    w[1, 5] = synth.to_bf16(2.0)
    s = oracle.row_scales(w, 1.0)
    assert s[0] == 0x3F80 and s[2] == 0x3F80
    q = oracle.quantize(w, s)
    assert (q[0] == 0).all() and (q[2] == 0).all() and q[1, 5] == 0x7E


def test_symmetry_and_no_negative_zero(small_w):
    s = oracle.row_scales(small_w, 500.0)
    q = oracle.quantize(small_w, s)
    qn = oracle.quantize((small_w ^ 0x8000).astype(np.uint16), s)
    nz = q != 0
    assert (qn[nz] == (q[nz] ^ 0x80)).all()
    assert (qn[~nz] == 0).all()
    assert not (q == 0x80).any()


def test_dequant_matches_torch_exact_product(small_w):
    s = oracle.row_scales(small_w, 41.0)
    q = oracle.quantize(small_w, s)
    w_hat = oracle.dequant(q, s)
    qt = torch.from_numpy(q).view(torch.float8_e4m3fn).to(torch.float32)
    prod = torch.from_numpy(_f32(s))[:, None] * qt     # exact in fp32
    ref = prod.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (w_hat == ref).all()


@pytest.fixture(scope="module")
def c1_quarter():
    from synth.configs import config_matrices
    return synth.weights(config_matrices(1)[0])[:256]


@pytest.mark.parametrize("bits", [2.0, 3.0, 4.0])
def test_alpha_search_hits_target(c1_quarter, bits):
    alpha, h = oracle.alpha_search(c1_quarter, bits)
    assert abs(h - bits) <= 0.05
    q = oracle.quantize(c1_quarter, oracle.row_scales(c1_quarter, alpha))
    assert oracle.entropy_codes(q) == pytest.approx(h, abs=1e-12)


def test_unique_values_behave_as_tab_unique_val(c1_quarter):
    """Tab. unique_val: more distinct values than a fixed 2^bits grid, and the
    count grows with the bit budget (exact counts need LLaMA-2 weights)."""
    uniq = {}
    for bits in (2.0, 3.0, 4.0):
        alpha, _ = oracle.alpha_search(c1_quarter, bits)
        q = oracle.quantize(c1_quarter, oracle.row_scales(c1_quarter, alpha))
        uniq[bits] = len(np.unique(q))
        assert uniq[bits] > 2 ** bits
    assert uniq[2.0] < uniq[3.0] < uniq[4.0]
