import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)

# Where the near-tie record of a session's parity comparisons goes (the parity bar counts and
# reports near-ties); TS_PARITY_RECORD overrides it.
RECORD_PATH = os.environ.get("TS_PARITY_RECORD", os.path.join(ROOT, "gpurun_out", "parity_near_ties.json"))


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP path)")
    config.addinivalue_line("markers", "slow: long-running statistical test")


def _records():
    mod = sys.modules.get("helpers")
    return list(getattr(mod, "RECORDS", [])) if mod else []


def pytest_sessionfinish(session, exitstatus):
    recs = _records()
    if not recs:
        return
    total = {k: sum(r[k] for r in recs) for k in ("compared", "near_ties", "units", "units_compared")}
    try:
        os.makedirs(os.path.dirname(RECORD_PATH), exist_ok=True)
        with open(RECORD_PATH, "w") as f:
            json.dump({"tie_bar": 1e-5, "total": total, "comparisons": recs}, f, indent=1)
    except OSError:
        pass


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    recs = _records()
    if not recs:
        return
    tr = terminalreporter
    tr.section("parity near-ties (competing scores within 1e-5 relative)")
    for r in recs:
        tr.write_line(f"{r['test']} [{r['what']}]: {r['compared']} compared, {r['near_ties']} near-ties, "
                      f"{r['units_compared']}/{r['units']} nodes or levels compared, "
                      f"max rel err {r['max_rel_err']:.2e}")
