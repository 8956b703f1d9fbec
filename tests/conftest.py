import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU or GPU run (full-size model shapes)")


@pytest.fixture(scope="session")
def model8b():
    """The 8B-shaped decoder (seed 42) loaded once per session on the GPU."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    from workloads import SHAPE_8B, make_weights
    print("generating 8B weights", flush=True)
    w = make_weights(SHAPE_8B, seed=42)
    model = hvd.Model(SHAPE_8B, w)
    del w
    return model


def load_golden(name):
    import json
    path = os.path.join(ROOT, "tests", "golden", name)
    if not os.path.exists(path):
        pytest.skip(f"{name} not generated (tests/golden/make_golden.py)")
    with open(path) as f:
        return json.load(f)
