import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU-side oracle runs")


_PARITY_RECORD: dict = {}


@pytest.fixture(scope="session")
def parity_record():
    """Measured parity margins of the GPU tests (row-normwise logit errors, label
    agreement, every excused mismatch with its top-2 gap), keyed by case.  Written as
    JSON at the end of the session to the path in RAFIKI_PARITY_OUT, if set."""
    yield _PARITY_RECORD
    out = os.environ.get("RAFIKI_PARITY_OUT")
    if out and _PARITY_RECORD:
        import json
        os.makedirs(os.path.dirname(os.path.abspath(out)), exist_ok=True)
        with open(out, "w") as f:
            json.dump(_PARITY_RECORD, f, indent=1, sort_keys=True)
