import os
import sys

import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if REPO not in sys.path:
    sys.path.insert(0, REPO)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def oracle():
    """The CPU oracle module (its C half is built on first use if it is missing)."""
    from oracle import focus_oracle
    focus_oracle._lib()
    return focus_oracle


@pytest.fixture(scope="session")
def golden_cases():
    import json
    with open(os.path.join(REPO, "tests", "golden", "fake_quant_examples.json")) as f:
        return json.load(f)["cases"]
