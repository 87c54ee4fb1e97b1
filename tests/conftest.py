import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


# ---- parity report: every code and output comparison of the session
# (tests/helpers.py) as JSON, for runs that keep it: the path in
# NOVA_KV_PARITY_REPORT, else gpurun_out/parity_report.json when that folder
# exists at the repository root.

@pytest.fixture(autouse=True)
def _parity_test_id(request):
    import helpers
    helpers.CURRENT_TEST["id"] = request.node.nodeid
    yield


def pytest_sessionfinish(session, exitstatus):
    import json
    try:
        import helpers
    except ImportError:
        return
    if not helpers.REPORT:
        return
    path = os.environ.get("NOVA_KV_PARITY_REPORT")
    if not path:
        out = os.path.join(ROOT, "gpurun_out")
        if not os.path.isdir(out):
            return
        path = os.path.join(out, "parity_report.json")
    codes = [r for r in helpers.REPORT if r["kind"] == "codes"]
    outs = [r for r in helpers.REPORT if r["kind"] == "output"]
    summary = {
        "codes_compared": sum(r["codes"] for r in codes),
        "code_mismatches": sum(r["mismatches"] for r in codes),
        "near_ties": sum(r["near_ties"] for r in codes),
        "near_tie_mismatches": sum(r["near_tie_mismatches"] for r in codes),
        "output_rows_compared": sum(r["rows"] for r in outs),
        "worst_rel_err": max([r["worst_rel_err"] for r in outs] or [0.0]),
        "failed_comparisons": sum(1 for r in helpers.REPORT if not r["ok"]),
    }
    with open(path, "w") as f:
        json.dump({"summary": summary, "entries": helpers.REPORT}, f, indent=1)
