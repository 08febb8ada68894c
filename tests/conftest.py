import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle

    oracle.build()
    return oracle.LIB_PATH


@pytest.fixture(scope="session")
def synth_lib():
    import synth

    synth.build()
    return synth


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """The parity counts of every GPU run (re-syncs after near ties, first
    divergence steps, largest output errors), also under -q."""
    harness = sys.modules.get("harness")
    if harness is None or not harness.REPORTS:
        return
    tr = terminalreporter
    tr.write_sep("=", "parity counts (%d runs)" % len(harness.REPORTS))
    flagged = resynced = 0
    for test, tag, rep in harness.REPORTS:
        tr.write_line("%s  %s" % (test, rep.line(tag)))
        flagged += rep.flagged_steps
        resynced += rep.flagged_divergences
    tr.write_line("total: near-tie unit-steps %d, re-synced %d" % (flagged, resynced))
