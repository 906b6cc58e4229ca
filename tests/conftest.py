import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


@pytest.fixture(autouse=True)
def _sentinel_outputs(request):
    """GPU tests run with every output and workspace the binding allocates
    pre-filled (NaN floats, 0xAB bytes), so an unwritten output cannot pass."""
    if request.node.get_closest_marker("gpu") is None:
        yield
        return
    from paper_2301_13659_amd import spk
    spk.set_output_sentinel(True)
    try:
        yield
    finally:
        spk.set_output_sentinel(False)
