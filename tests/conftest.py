import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """The oracle comparisons of the session: one line per compared request
    (exact = the tree equals the free-running oracle's bit for bit; min_gap =
    the narrowest selection boundary; max_dev = the largest |score deviation|),
    also written to gpurun_out/parity_report.json when that folder exists."""
    import json

    compare = sys.modules.get("compare")
    rows = getattr(compare, "REPORTS", None) if compare else None
    if not rows:
        return
    tr = terminalreporter
    tr.section("oracle comparisons")
    n_exact = sum(1 for r in rows if r["exact"])
    n_same = sum(1 for r in rows if r.get("identical"))
    tr.write_line(f"{len(rows)} requests compared with the oracle: {n_exact} required bit-exact "
                  f"and were, {n_same} identical to the oracle's tree, max |score deviation| "
                  f"{max(r['max_dev'] for r in rows):.3g}")
    for r in rows:
        tr.write_line(f"  {r['label']:<34} req {r['request']:>3}  exact={int(r['exact'])}  "
                      f"identical={int(r.get('identical', 0))}  "
                      f"min_gap={r['min_gap']:.3g}  max_dev={r['max_dev']:.3g}  "
                      f"count={r['count']}")
    out_dir = os.path.join(ROOT, "gpurun_out")
    if os.path.isdir(out_dir):
        with open(os.path.join(out_dir, "parity_report.json"), "w") as f:
            json.dump(rows, f, indent=1, default=float)
