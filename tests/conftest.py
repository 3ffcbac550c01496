import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running case (large synthetic layer)")


@pytest.fixture(scope="session")
def oracle():
    import oracle as _oracle
    return _oracle


@pytest.fixture(scope="session")
def qe():
    """The HIP library binding; GPU tests fail (not skip) if it cannot run."""
    import torch
    assert torch.cuda.is_available(), "GPU test run without a visible GPU"
    import paper_2309_01885_amd as P
    P.load()
    return P


@pytest.fixture(scope="session")
def c2_x():
    """The attention-projection workload's activations (4096 x 262144
    heavy-tailed tokens); the MLP up-projection and the outlier-aware
    workload draw the very same X."""
    import synth
    spec = synth.CONFIGS["c2"]
    print(f"[c2] drawing X {spec.p}x{spec.n}", flush=True)
    return synth.activations(spec)


@pytest.fixture(scope="session")
def c2_sigma64(c2_x, oracle):
    """The oracle's undamped fp64 Gram of all 262144 tokens of c2_x."""
    print("[c2] oracle Gram of all tokens (fp64)", flush=True)
    return oracle.gram_blas(c2_x)
