import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Near-tie accounting of the GPU parity tests: every comparison that
    allowed a near-tie records its counts, shown here even under -q and
    written as parity_record.json to the run's output folder
    (SELKV_RECORD_DIR, by default the one GPU runs hand back)."""
    try:
        from tests.parity_util import RECORDS
    except ImportError:
        return
    if not RECORDS:
        return
    tr = terminalreporter
    tr.write_sep("-", "near-tie accounting (selection swaps within 1e-6 relative of the threshold, "
                      "route ties within 1e-6 relative)")
    keys = sorted({k for r in RECORDS for k in r if k not in ("test", "case")})
    totals = {k: 0 for k in keys if k not in ("score_rel_err",)}
    worst_err = 0.0
    for r in RECORDS:
        fields = " ".join(f"{k}={r[k]:.2e}" if k == "score_rel_err" else f"{k}={r[k]}"
                          for k in keys if k in r)
        tr.write_line(f"{r['test']} [{r['case']}]: {fields}")
        for k in totals:
            totals[k] += int(r.get(k, 0))
        worst_err = max(worst_err, float(r.get("score_rel_err", 0.0)))
    tr.write_line("totals: " + " ".join(f"{k}={v}" for k, v in totals.items())
                  + f" max score_rel_err={worst_err:.2e} over {len(RECORDS)} comparisons")
    out = os.environ.get("SELKV_RECORD_DIR", os.path.join(ROOT, "gpurun_out"))
    try:
        os.makedirs(out, exist_ok=True)
        with open(os.path.join(out, "parity_record.json"), "w") as f:
            json.dump({"records": RECORDS, "totals": totals, "max_score_rel_err": worst_err}, f, indent=1)
    except OSError:
        pass
