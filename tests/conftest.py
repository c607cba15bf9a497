import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (HIP device); run with -m gpu")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle
    oracle.build(force=False)
    return oracle


def pytest_terminal_summary(terminalreporter):
    """Near-ties of fp32 top-k lists (R27) seen by the parity checks."""
    import sys
    mod = sys.modules.get("tests.topk_check")
    if mod and mod.NEAR_TIES["queries"]:
        nt = mod.NEAR_TIES
        terminalreporter.write_line(
            f"top-k parity: {nt['queries']} query lists checked, {nt['near_ties']} fp32 near-ties")
