import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session", autouse=True)
def _oracle_built():
    import oracle
    oracle.build(force=False)
    yield


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Near-tie counts of every GPU-vs-oracle comparison of the run (groups
    compared, stop mismatches excused as near-ties, comparisons made)."""
    try:
        import parity
    except Exception:  # pragma: no cover
        return
    if not parity.SUMMARY:
        return
    tot_g = sum(v[0] for v in parity.SUMMARY.values())
    tot_t = sum(v[1] for v in parity.SUMMARY.values())
    terminalreporter.write_line(f"parity: {tot_g} groups compared, {tot_t} near-ties excused")
    for name in sorted(parity.SUMMARY):
        g, t, n = parity.SUMMARY[name]
        terminalreporter.write_line(f"  {name}: groups={g} near_ties={t} calls={n}")
