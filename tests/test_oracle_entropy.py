"""Oracle entropy functions pinned to the paper's printed values and closed forms.

eq. emp_entropy defines the empirical entropy; App. B.1 gives the sparse-mixture
closed form and prints Tab. sparsity_entropy.
"""
import math
import os

import numpy as np
import pytest
import scipy.stats

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "sparsity_entropy.txt")


def _table():
    rows = {}
    with open(GOLDEN) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            name, *vals = line.split()
            rows[name] = [float(v) for v in vals]
    return rows


def test_tab_sparsity_entropy_uniform_row_from_histograms():
    """Row 1: a histogram with zero mass s and 255 equally likely non-zero
    codes; the empirical entropy must reproduce the printed values."""
    t = _table()
    for s, printed in zip(t["s"], t["uniform"]):
        n = 255 * 10000
        counts = np.zeros(256, dtype=np.uint64)
        zeros = int(round(s * n))
        counts[0] = zeros
        counts[1:] = (n - zeros) // 255
        assert counts.sum() == n
        h = oracle.entropy_counts(counts)
        assert round(h, 2) == printed, (s, h, printed)


def test_tab_sparsity_entropy_closed_form_both_rows():
    t = _table()
    for s, u, o in zip(t["s"], t["uniform"], t["original"]):
        assert round(oracle.sparsity_entropy(s, math.log2(255)), 2) == u
        assert round(oracle.sparsity_entropy(s, 6.5), 2) == o


def test_sparsity_entropy_limits():
    assert oracle.sparsity_entropy(0.0, 5.0) == 5.0
    assert oracle.sparsity_entropy(1.0, 5.0) == 0.0
    assert abs(oracle.sparsity_entropy(0.5, 0.0) - 1.0) < 1e-15


@pytest.mark.parametrize("k", [0, 1, 3, 8])
def test_uniform_histogram_has_k_bits(k):
    counts = np.zeros(256, dtype=np.uint64)
    counts[: 2 ** k] = 7
    assert oracle.entropy_counts(counts) == pytest.approx(k, abs=1e-12)


def test_codes_entropy_matches_scipy():
    r = np.random.default_rng(3)
    q = r.choice(256, size=100000, p=np.r_[np.full(16, 0.05), np.full(240, 0.2 / 240)])
    q = q.astype(np.uint8)
    ref = scipy.stats.entropy(np.bincount(q, minlength=256), base=2)
    assert oracle.entropy_codes(q) == pytest.approx(ref, rel=1e-12)
