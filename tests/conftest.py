import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


GOLDEN = os.path.join(ROOT, "tests", "golden")


def read_golden(name):
    """Rows of whitespace-separated numbers from tests/golden/<name>;
    lines starting with '#' are comments (each file states its derivation)."""
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            rows.append(line.split())
    return rows


@pytest.fixture(autouse=True)
def _device_error_flags_clear(request):
    """After every GPU test: no library handle that is still open may hold a
    raised device error flag (a timed-out wait of the persistent decode, an
    activation beyond the fp16 range, an out-of-range token id).  Tests that
    raise a flag on purpose read (and so clear) it themselves."""
    yield
    if request.node.get_closest_marker("gpu") is None:
        return
    b = sys.modules.get("paper_2607_15865_amd.binding")
    if b is None:
        return
    raised = []
    for obj in list(b._live):
        if getattr(obj, "handle", None):
            f = obj.error()
            if f:
                raised.append((type(obj).__name__, f))
    assert not raised, f"device error flags raised: {raised}"
