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
    config.addinivalue_line("markers", "gpu: needs a gfx950 GPU (runs through the C-ABI library)")
    config.addinivalue_line("markers", "slow: long CPU test")


@pytest.fixture(scope="session")
def opool():
    """Process pool running the CPU oracle for the GPU parity tests (created on first use)."""
    from parity_util import OraclePool
    p = OraclePool()
    yield p
    p.close()


@pytest.fixture(scope="session")
def root_dir():
    return ROOT


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Parity tallies of the GPU-versus-oracle cases that ran: per stage, comparisons that matched exactly /
    that differed only at a decision whose own oracle margin was below 1e-5 (flagged)."""
    from tally import REGISTRY
    if not REGISTRY:
        return
    tr = terminalreporter
    tr.section("parity tallies (exact/flagged per stage; any other difference fails its test)")
    for t in REGISTRY:
        tr.write_line(t.line())
    tr.write_line("total: exact %d, flagged %d, over %d request-steps"
                  % (sum(t.total_exact for t in REGISTRY), sum(t.flagged for t in REGISTRY),
                     sum(t.request_steps for t in REGISTRY)))
