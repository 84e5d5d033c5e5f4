"""The seeded input generator: determinism and the distributions it promises."""
import numpy as np
import pytest
import torch

import synth
from synth.configs import config_matrices, small_spec


def test_deterministic_across_thread_counts():
    spec = small_spec(97, 301, seed=5)
    a = synth.weights(spec, threads=1)
    b = synth.weights(spec, threads=7)
    assert (a == b).all()


def test_uniform_range_and_moments():
    u = np.array([synth.uniform(1, 0, k) for k in range(20000)])
    assert (u > 0).all() and (u < 1).all()
    assert abs(u.mean() - 0.5) < 0.01 and abs(u.var() - 1 / 12) < 0.003


def test_bf16_rounding_matches_torch():
    r = np.random.default_rng(0)
    v = r.standard_normal(5000) * np.exp(r.uniform(-8, 8, 5000))
    v32 = v.astype(np.float32)
    ref = torch.from_numpy(v32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([synth.to_bf16(float(x)) for x in v32], dtype=np.uint16)
    assert (got == ref).all()


def test_student_t_moments():
    spec = small_spec(512, 1024, nu=5, sigma=0.0, seed=2)
    w = synth.bf16_to_f32(synth.weights(spec)).astype(np.float64)
    # t(5): mean 0, variance nu/(nu-2) = 5/3
    assert abs(w.mean()) < 0.01
    assert w.var() == pytest.approx(5 / 3, rel=0.04)


def test_row_scales_lognormal():
    spec = small_spec(2000, 256, nu=5, sigma=0.5, seed=3)
    w = synth.bf16_to_f32(synth.weights(spec)).astype(np.float64)
    log_rms = np.log(np.sqrt((w ** 2).mean(axis=1)))
    assert log_rms.std() == pytest.approx(0.5, rel=0.1)


def test_outlier_rate_and_magnitude():
    spec = small_spec(400, 2500, sigma=0.0, seed=4, outliers=True)
    w = synth.bf16_to_f32(synth.weights(spec))
    out = np.abs(w) == 20.0
    assert out.mean() == pytest.approx(1e-3, rel=0.15)
    assert (w[out] > 0).mean() == pytest.approx(0.5, abs=0.1)


def test_config_shapes():
    assert [(m.rows, m.cols) for m in config_matrices(4)] == [(8192, 28672), (28672, 8192)]
    c5 = config_matrices(5)
    assert len(c5) == 560
    assert sum(m.params for m in c5) == 80 * 855638016
    assert {m.target_bits for m in c5} == {2.0, 3.0, 4.0}
    assert len({m.seed for m in c5}) == 560
