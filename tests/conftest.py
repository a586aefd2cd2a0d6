"""Shared fixtures.  GPU tests are marked `gpu`; everything else runs on CPU."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU sweep")


@pytest.fixture(scope="session")
def orc():
    from oracle import oracle
    oracle.build()
    return oracle


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Tolerance tally of the GPU parity comparisons: elements compared, elements
    that passed only through the one-BF16-ulp clause (|x| >= 2), and the
    largest difference among outputs below 2 in magnitude (held to 1e-2)."""
    try:
        from tests import helpers
    except Exception:
        return
    t = helpers.TALLY
    if t["elements"]:
        terminalreporter.write_line(
            f"bf16 parity tally: {t['elements']} elements compared, {t['ulp_clause_only']} passed only "
            f"through the one-ulp clause (|x| >= 2), max |d| below 2: {t['max_abs_below_2']:.3e}")
