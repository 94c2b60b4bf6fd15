import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
GOLDEN = os.path.join(ROOT, "tests", "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def read_golden(name):
    """parse a `key: value` fixture; repeated keys collect into a list"""
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            k, v = line.split(":", 1)
            out.setdefault(k.strip(), []).append(v.split())
    return {k: (v[0] if len(v) == 1 else v) for k, v in out.items()}


@pytest.fixture(scope="session")
def orc():
    import oracle
    oracle.lib()
    return oracle


def pytest_runtest_setup(item):
    if item.get_closest_marker("gpu") is not None:
        import torch
        if not torch.cuda.is_available():
            pytest.fail("a gpu-marked test needs an MI355X; run `-m 'not gpu'` on machines without one")


@pytest.fixture(scope="session")
def tc():
    """the GPU binding; the HIP library must be built and loadable"""
    from paper_2401_07788_amd import tc as _tc
    _tc.lib()
    return _tc
