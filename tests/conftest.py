import os
import sys

import pytest

ROOT = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(ROOT)
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session", autouse=True)
def _oracle_built():
    import oracle

    if not os.path.exists(oracle.lib_path()):
        oracle.build(force=False)
    yield


@pytest.fixture(autouse=True)
def _parity_case(request):
    """Names the running test in the routing-parity records."""
    import parity

    parity.CURRENT_CASE = request.node.nodeid.split("::", 1)[-1]
    yield


def pytest_terminal_summary(terminalreporter):
    """Near-tie counts of every routing comparison of the session: tokens
    whose oracle gap z_(k) - z_(k+1) is below 1e-5 (the only exemption from
    bit-exact ids), how many of them the GPU resolved differently, and the
    largest gate and gap differences."""
    parity = sys.modules.get("parity")
    if parity is None or not parity.RECORDS:
        return
    tr = terminalreporter
    recs = parity.RECORDS
    tr.write_sep("-", "routing parity: near ties (oracle z_(k) - z_(k+1) < 1e-5)")
    tot = {k: sum(r[k] for r in recs) for k in ("tokens", "near_ties", "near_tie_swaps",
                                                  "inner_ties", "inner_reorders")}
    tr.write_line(f"{len(recs)} comparisons, {tot['tokens']} tokens: {tot['near_ties']} near ties "
                  f"({tot['near_tie_swaps']} resolved differently), {tot['inner_ties']} ties inside "
                  f"the top k ({tot['inner_reorders']} reordered); max |dw| "
                  f"{max(r['max_dw'] for r in recs):.3g}, max |dgap| "
                  f"{max(r['max_dgap'] for r in recs):.3g}")
    for r in recs:
        if r["near_ties"] or r["inner_ties"]:
            tr.write_line(f"  {r['case']} [{r['what']}]: {r['tokens']} tokens, near ties "
                          f"{r['near_ties']} (swapped {r['near_tie_swaps']}), inner ties "
                          f"{r['inner_ties']} (reordered {r['inner_reorders']})")
