"""Oracle number formats pinned against library routines and special values.

E4M3FN (App. A.1 Float8 base format) and BF16 (scales, weights) are checked
against torch's CPU casts, which implement the OCP / bfloat16 definitions with
round-to-nearest-even, and against the format's known extremes.
"""
import math

import numpy as np
import pytest
import torch

import oracle


def test_e4m3_all_codes_match_torch():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = np.array([oracle.e4m3_value(c) for c in range(256)])
    nan_ref, nan_got = np.isnan(ref), np.isnan(got)
    assert (nan_ref == nan_got).all()
    assert nan_got.sum() == 2  # 0x7F and 0xFF
    assert (ref[~nan_ref] == got[~nan_got]).all()


def test_e4m3_extremes():
    assert oracle.e4m3_value(0x7E) == 448.0        # Qmax
    assert oracle.e4m3_value(0x01) == 2.0 ** -9    # smallest subnormal
    assert oracle.e4m3_value(0x08) == 2.0 ** -6    # smallest normal
    assert oracle.e4m3_value(0x38) == 1.0
    assert math.isnan(oracle.e4m3_value(0x7F))
    assert oracle.e4m3_value(0x80) == 0.0 and math.copysign(1, oracle.e4m3_value(0x80)) < 0


def _torch_e4m3(v: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(v.astype(np.float32)).clamp(-448.0, 448.0)
    c = t.to(torch.float8_e4m3fn).view(torch.uint8).numpy().copy()
    c[c == 0x80] = 0x00  # signed zero resolved to +0 (App. A.1)
    return c


def test_e4m3_round_matches_torch_random():
    r = np.random.default_rng(1)
    mag = np.exp2(r.uniform(-12, 9.2, 20000)).astype(np.float32)
    v = (mag * r.choice([-1.0, 1.0], mag.size)).astype(np.float32)
    got = np.array([oracle.e4m3_round(float(x)) for x in v], dtype=np.uint8)
    assert (got == _torch_e4m3(v)).all()


def test_e4m3_round_ties_and_neighbours():
    vals = np.array([oracle.e4m3_value(c) for c in range(0x7F)])
    mids = (vals[:-1] + vals[1:]) / 2  # exact ties between neighbours
    cases = []
    for m in mids:
        m32 = np.float32(m)
        assert float(m32) == m
        cases += [m32, np.nextafter(m32, np.float32(0)), np.nextafter(m32, np.float32(1e9))]
    cases += [np.float32(v) for v in vals]
    v = np.array(cases, dtype=np.float32)
    v = np.concatenate([v, -v])
    got = np.array([oracle.e4m3_round(float(x)) for x in v], dtype=np.uint8)
    assert (got == _torch_e4m3(v)).all()
    # a tie between codes 0x38 (1.0) and 0x39 (1.125) goes to the even code
    assert oracle.e4m3_round(1.0625) == 0x38
    assert oracle.e4m3_round(1.1875) == 0x3A


def test_e4m3_round_clamps_and_zero():
    assert oracle.e4m3_round(1e6) == 0x7E
    assert oracle.e4m3_round(-1e6) == 0xFE
    assert oracle.e4m3_round(460.0) == 0x7E
    assert oracle.e4m3_round(-0.0) == 0x00
    assert oracle.e4m3_round(-1e-9) == 0x00   # rounds to zero: stored as +0
    assert oracle.e4m3_round(2.0 ** -10) == 0x00  # tie between 0 and 2^-9 -> even (0)
    assert oracle.e4m3_round(2.0 ** -10 * 1.0001) == 0x01


def test_bf16_round_matches_torch_on_f32():
    r = np.random.default_rng(2)
    bits = r.integers(0, 2 ** 32, 50000, dtype=np.uint64).astype(np.uint32)
    f = bits.view(np.float32)
    f = f[np.isfinite(f) & (np.abs(f) < 3.0e38)]
    # add exact ties (low 16 bits 0x8000) and subnormals
    ties = ((bits[:2000] & 0x7F7F0000) | 0x8000).view(np.float32)
    sub = (bits[:2000] & 0x007FFFFF).view(np.float32)
    f = np.concatenate([f, ties, sub, -sub]).astype(np.float32)
    ref = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([oracle.bf16_round(float(x)) for x in f], dtype=np.uint16)
    assert (got == ref).all()


def test_bf16_round_once_from_fp64():
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even significand -> 1.0
    assert oracle.bf16_round(1.0 + 2 ** -8) == 0x3F80
    # 1 + 3*2^-8 is a tie between 1+2^-7 and 1+2^-6 -> 1+2^-6 (even)
    assert oracle.bf16_round(1.0 + 3 * 2 ** -8) == 0x3F82
    # just above the tie: must round up.  Rounding through fp32 first would
    # drop the 2^-40 and land on the tie (-> 1.0): the oracle rounds once.
    assert oracle.bf16_round(1.0 + 2 ** -8 + 2 ** -40) == 0x3F81
    assert oracle.bf16_round(-2.5) == 0xC020
    assert oracle.bf16_value(0x3F80) == 1.0 and oracle.bf16_value(0xC020) == -2.5


@pytest.mark.parametrize("code", [0x01, 0x07, 0x08, 0x38, 0x7E])
def test_bf16_holds_every_e4m3_value(code):
    v = oracle.e4m3_value(code)
    assert oracle.bf16_value(oracle.bf16_round(v)) == v
