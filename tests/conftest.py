import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def gpu_available() -> bool:
    try:
        import torch
        return bool(torch.cuda.is_available())
    except Exception:
        return False


@pytest.fixture(scope="session")
def tiny_cfg():
    import synth
    return synth.get("tiny")


@pytest.fixture(scope="session")
def tiny_weights(tiny_cfg):
    import synth
    w = synth.make_weights(tiny_cfg, seed=0)
    synth.add_w8a16(w)
    return w
