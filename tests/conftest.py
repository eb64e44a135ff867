import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library)")


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle
    oracle._load()
    return oracle


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Selection tie statistics of the GPU parity calls: tokens exempt from
    bit-exact selection by kind (cumulative-mass band, logit tie at the cut,
    LTE threshold band) and consecutive kept logits tied (order only)."""
    helpers = sys.modules.get("gpu_helpers")
    log = getattr(helpers, "TIE_LOG", None)
    if not log:
        return
    tr = terminalreporter
    tot = {}
    calls = tokens = 0
    for _, T, _, c in log:
        calls += 1
        tokens += T
        for k, v in c.items():
            tot[k] = tot.get(k, 0) + v
    tr.write_sep("-", "selection ties: %d parity calls, %d tokens" % (calls, tokens))
    tr.write_line("exempt %d (cumulative mass %d, logit tie at the cut %d, LTE band %d); "
                  "tied kept logits (order only) %d" % (
                      tot.get("exempt", 0), tot.get("mass", 0), tot.get("cut_order", 0),
                      tot.get("lte", 0), tot.get("prefix_order", 0)))
    for label, T, tau, c in log:
        if c["exempt"] or c["prefix_order"]:
            tr.write_line("  %-28s T=%-5d tau=%-6g exempt %d (mass %d, cut %d, lte %d), "
                          "order-only %d" % (label[:28], T, tau, c["exempt"], c["mass"],
                                             c["cut_order"], c["lte"], c["prefix_order"]))
