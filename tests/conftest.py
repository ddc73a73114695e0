import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU; runs the HIP path")


class ParityCounts:
    """Rows per GPU parity case that sat near a decision boundary (several
    admissible outcomes), took an outcome other than the oracle's own, or
    went through the exact slow path; printed in the terminal summary."""

    def __init__(self):
        self.rows = []

    def add(self, label, rows, near, alt, fallback):
        self.rows.append((label, int(rows), int(near), int(alt), int(fallback)))


def pytest_sessionstart(session):
    session.config._parity_counts = ParityCounts()


def _counts_of(config):
    if not hasattr(config, "_parity_counts"):
        config._parity_counts = ParityCounts()
    return config._parity_counts


import pytest  # noqa: E402


@pytest.fixture(scope="session")
def parity_counts(request):
    return _counts_of(request.config)


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    c = _counts_of(config)
    if not c.rows:
        return
    tot = [sum(r[i] for r in c.rows) for i in range(1, 5)]
    terminalreporter.write_line(
        "parity counts: %d rows in %d cases; near-boundary rows %d; outcome other than the oracle's own %d; "
        "exact slow path (fallback) rows %d" % (tot[0], len(c.rows), tot[1], tot[2], tot[3]))
    for label, rows, near, alt, fb in c.rows:
        if near or alt or fb:
            terminalreporter.write_line("  %-28s rows=%-6d near=%-4d other=%-4d fallback=%d" % (label, rows, near, alt, fb))
