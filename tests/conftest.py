import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session")
def orc():
    import oracle
    return oracle.default()


def _parity_records():
    h = sys.modules.get("harness")
    return list(getattr(h, "RECORDS", []) or [])


def _parity_summary(records):
    """Totals per configuration of the parity checks' exclusion counts."""
    per = {}
    for r in records:
        t = per.setdefault(r["config"], dict(checks=0, rows=0, near_tie_rows=0, seqs=0,
                                              near_threshold_seqs=0, max_err={}))
        t["checks"] += 1
        for k in ("rows", "near_tie_rows", "seqs", "near_threshold_seqs"):
            t[k] += r[k]
        for k, v in r["max_err"].items():
            t["max_err"][k] = max(t["max_err"].get(k, 0.0), v)
    return per


def pytest_sessionfinish(session, exitstatus):
    """Write the parity checks' exclusion counts (near-threshold sequences,
    near-tie rows, largest errors) to a JSON record: the path in
    FORK_PARITY_RECORD, else test_records/parity_counts.json at the
    repository root."""
    records = _parity_records()
    if not records:
        return
    import json
    path = os.environ.get("FORK_PARITY_RECORD") or os.path.join(ROOT, "test_records",
                                                                 "parity_counts.json")
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w") as f:
        json.dump({"per_config": _parity_summary(records), "checks": records}, f, indent=1)


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    records = _parity_records()
    if not records:
        return
    tr = terminalreporter
    tr.section("parity exclusion counts (per configuration)")
    tr.write_line("%-16s %6s %9s %9s %9s %11s  %s" % ("config", "checks", "rows", "near-tie",
                                                       "seq-steps", "near-thresh", "max err"))
    for name, t in sorted(_parity_summary(records).items()):
        err = " ".join("%s=%.1e" % (k, v) for k, v in sorted(t["max_err"].items()))
        tr.write_line("%-16s %6d %9d %9d %9d %11d  %s" % (
            name, t["checks"], t["rows"], t["near_tie_rows"], t["seqs"],
            t["near_threshold_seqs"], err))
