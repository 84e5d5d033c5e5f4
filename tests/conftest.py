import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle
    return oracle


@pytest.fixture(scope="session")
def c1_weights():
    import synth
    from synth.configs import config_matrices
    spec = config_matrices(1)[0]
    return spec, synth.weights(spec)


@pytest.fixture(scope="session")
def c1_container(c1_weights):
    """Config-1 container built by the oracle (alpha from the oracle's search)."""
    import oracle
    spec, w = c1_weights
    alpha, h = oracle.alpha_search(w, spec.target_bits)
    blob = oracle.container_build(w, alpha, 12, spec.chunk_syms, spec.lanes, spec.seed,
                                  spec.target_bits)
    return spec, w, alpha, blob


def rng(seed=0):
    return np.random.default_rng(seed)
