"""Oracle Int8 base format (Sec. 2.1 symmetric quantiser; Sec. 3.5 ablation).

Pins: numpy's two's complement view for the code values, numpy's clip + rint
(round half to even) for the quantiser on random values and on every exact
half-integer, AbsMax mapping each row maximum to +-127, the nearest-BF16
property of the scales with Qmax = 127, torch's bf16 cast of the exact
product for the dequantiser, the alpha search reaching its target, and a
container round trip whose header names the format.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from synth.configs import small_spec

INT8 = oracle.INT8


def _f32(bits):
    return synth.bf16_to_f32(bits)


@pytest.fixture(scope="module")
def small_w():
    return synth.weights(small_spec(160, 384, seed=23))


def test_int8_values_are_twos_complement():
    ref = np.arange(256, dtype=np.uint8).view(np.int8).astype(np.float64)
    got = np.array([oracle.int8_value(c) for c in range(256)])
    assert (got == ref).all()
    assert all(oracle.code_value(INT8, c) == ref[c] for c in range(256))
    assert oracle.qmax(INT8) == 127.0 and oracle.qmax(oracle.E4M3) == 448.0


def _numpy_int8(v: np.ndarray) -> np.ndarray:
    return np.rint(np.clip(v.astype(np.float64), -127.0, 127.0)).astype(np.int8).view(np.uint8)


def test_int8_round_matches_numpy_random():
    r = np.random.default_rng(5)
    v = np.concatenate([r.normal(0, 3, 20000), r.normal(0, 200, 5000)]).astype(np.float32)
    got = np.array([oracle.int8_round(float(x)) for x in v], dtype=np.uint8)
    assert (got == _numpy_int8(v)).all()


def test_int8_round_halves_and_clamp():
    halves = (np.arange(-130, 130) + 0.5).astype(np.float32)
    cases = np.concatenate([halves, np.nextafter(halves, np.float32(-1e9)),
                            np.nextafter(halves, np.float32(1e9)),
                            np.float32([127.0, -127.0, 127.49, -127.6, 1e30, -1e30, -0.0, 0.0,
                                        -0.5, 0.5, -0.49])])
    got = np.array([oracle.int8_round(float(x)) for x in cases], dtype=np.uint8)
    assert (got == _numpy_int8(cases)).all()
    # ties go to the even integer; the range is symmetric, so 0x80 never occurs
    assert oracle.int8_round(2.5) == 2 and oracle.int8_round(3.5) == 4
    assert oracle.int8_round(-2.5) == 0xFE and oracle.int8_round(-1e9) == 0x81
    assert oracle.int8_round(-0.25) == 0


def test_int8_quantize_matches_numpy(small_w):
    for alpha in (1.0, 9.0, 60.0):
        s = oracle.row_scales(small_w, alpha, INT8)
        q = oracle.quantize(small_w, s, INT8)
        v = _f32(small_w) / _f32(s)[:, None]  # one fp32 division, as in Sec. 2.1
        assert (q == _numpy_int8(v)).all(), alpha
        assert not (q == 0x80).any()


def test_int8_absmax_maps_row_max_to_qmax(small_w):
    s = oracle.row_scales(small_w, 1.0, INT8)
    q = oracle.quantize(small_w, s, INT8)
    jmax = np.abs(_f32(small_w)).argmax(axis=1)
    top = q[np.arange(q.shape[0]), jmax].view(np.int8)
    assert (np.abs(top.astype(np.int32)) == 127).all()


def test_int8_scales_are_nearest_bf16(small_w):
    alpha = 5.3
    s = oracle.row_scales(small_w, alpha, INT8)
    amax = np.abs(_f32(small_w).astype(np.float64)).max(axis=1)
    target = np.float64(np.float32(alpha)) * amax / 127.0
    sv = _f32(s).astype(np.float64)
    up = _f32((s + 1).astype(np.uint16)).astype(np.float64)
    dn = _f32((s - 1).astype(np.uint16)).astype(np.float64)
    err = np.abs(sv - target)
    assert (err <= np.abs(up - target)).all() and (err <= np.abs(dn - target)).all()


def test_int8_dequant_matches_torch_exact_product(small_w):
    s = oracle.row_scales(small_w, 7.0, INT8)
    q = oracle.quantize(small_w, s, INT8)
    w_hat = oracle.dequant(q, s, INT8)
    qt = torch.from_numpy(q.view(np.int8).astype(np.float32))
    prod = torch.from_numpy(_f32(s))[:, None] * qt  # exact: 8-bit x 7-bit significands
    ref = prod.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (w_hat == ref).all()
    # the E4M3 reading of the same codes is a different weight matrix
    assert not (oracle.dequant(q, s) == w_hat).all()


@pytest.mark.parametrize("bits", [2.0, 3.0, 4.0])
def test_int8_alpha_search_hits_target(bits):
    from synth.configs import config_matrices
    w = synth.weights(config_matrices(1)[0])[:128]
    alpha, h = oracle.alpha_search(w, bits, INT8)
    assert abs(h - bits) <= 0.05
    q = oracle.quantize(w, oracle.row_scales(w, alpha, INT8), INT8)
    assert oracle.entropy_codes(q) == pytest.approx(h, abs=1e-12)


def test_int8_container_round_trip(small_w):
    alpha, _ = oracle.alpha_search(small_w, 2.5, INT8)
    blob = oracle.container_build(small_w, alpha, 12, 2048, 64, fmt=INT8)
    info = oracle.container_info(blob)
    assert info.base_format == INT8
    rc, q = oracle.container_decode(blob)
    assert rc == oracle.OK
    s = oracle.row_scales(small_w, alpha, INT8)
    assert (oracle.container_scales(blob) == s).all()
    assert (q == oracle.quantize(small_w, s, INT8)).all()
    # an unknown base format is rejected
    bad = blob.copy()
    bad[12] = 3
    with pytest.raises(ValueError):
        oracle.container_info(bad)
