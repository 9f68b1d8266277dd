import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))
for _p in (ROOT, HERE):
    if _p not in sys.path:
        sys.path.insert(0, _p)

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


@pytest.fixture(scope="session")
def paper():
    """Values printed in the paper, each with its citation."""
    with open(os.path.join(GOLDEN, "paper_values.json")) as f:
        data = json.load(f)
    return {k: v["value"] for k, v in data.items() if not k.startswith("_")}


@pytest.fixture(scope="session")
def gpu_lib():
    """The HIP library, loaded once; GPU tests fail loudly if it is missing."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a visible GPU")
    from paper_2608_06812_amd import ozfp4
    ozfp4.load()
    return ozfp4
