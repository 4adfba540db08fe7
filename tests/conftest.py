import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU reference case")


@pytest.fixture(scope="session")
def model_7b():
    """The 7B decoder drawn on the device once per session, with the fp64 reference's view of
    exactly those weights (layers decoded on first use)."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_10259_amd import workload as W
    from paper_2508_10259_amd.runtime import DeviceModel
    from ref_bridge import oracle_params
    spec = W.MODELS["7b"]
    w = W.make_device_weights(spec, seed=0)
    return spec, DeviceModel(w), oracle_params(w)
