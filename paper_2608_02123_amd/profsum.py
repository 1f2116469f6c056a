"""Summaries of rocprofv3 CSV output for the round kernel.

``python -m paper_2608_02123_amd.profsum stats DIR`` prints the per-kernel
table of a ``--kernel-trace --stats`` run as markdown.

``python -m paper_2608_02123_amd.profsum traffic FETCH_DIR WRITE_DIR OUT.json [WORKLOAD [KERNEL [STEPS]]]``
turns two ``--pmc FETCH_SIZE`` / ``--pmc WRITE_SIZE`` runs of
``bench.py --calibrate-copy`` into HBM bytes per round-kernel launch.  Each
counter is scaled by what it reads for the calibration pass (an elementwise
negation of a float32 tensor: 256 MiB read and 256 MiB written), so that the
figure is in bytes whatever unit and sampling the counter has on the device.
"""
from __future__ import annotations

import csv
import glob
import hashlib
import json
import os
import sys

COPY_KERNEL = "neg_kernel"
COPY_BYTES = 256 << 20
KERNEL_SRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "pctree_kernels.hip")


def _one(dirname: str, suffix: str) -> str:
    hits = sorted(glob.glob(os.path.join(dirname, "**", f"*{suffix}"), recursive=True))
    if not hits:
        raise SystemExit(f"no *{suffix} under {dirname}")
    return hits[0]


def stats_markdown(dirname: str) -> str:
    rows = list(csv.DictReader(open(_one(dirname, "kernel_stats.csv"))))
    out = ["| kernel | calls | avg us | min us | max us | % time |", "|---|---:|---:|---:|---:|---:|"]
    for r in rows:
        out.append(f"| `{r['Name'][:90]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                   f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                   f"{float(r['Percentage']):.2f} |")
    return "\n".join(out)


def counter_means(dirname: str, counter: str) -> dict[str, tuple[float, int]]:
    """Mean counter value per dispatch (KiB for the size counters), by kernel name."""
    acc: dict[str, list[float]] = {}
    for r in csv.DictReader(open(_one(dirname, "counter_collection.csv"))):
        if r["Counter_Name"] != counter:
            continue
        acc.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return {k: (sum(v) / len(v), len(v)) for k, v in acc.items()}


def _pick(means: dict[str, tuple[float, int]], needle: str) -> tuple[str, float, int]:
    hits = [(k, v) for k, v in means.items() if needle in k]
    if not hits:
        raise SystemExit(f"no dispatch of a kernel named like {needle!r}")
    k, (val, n) = max(hits, key=lambda kv: kv[1][1])
    return k, val, n


def traffic(fetch_dir: str, write_dir: str, kernel: str = "round_kernel",
            workload: str = "qwen4b_b16", steps: int = 20) -> dict:
    f = counter_means(fetch_dir, "FETCH_SIZE")
    w = counter_means(write_dir, "WRITE_SIZE")
    _, f_copy, _ = _pick(f, COPY_KERNEL)
    _, w_copy, _ = _pick(w, COPY_KERNEL)
    name, f_k, nf = _pick(f, kernel)
    _, w_k, nw = _pick(w, kernel)
    ff = COPY_BYTES / (f_copy * 1024.0)
    fw = COPY_BYTES / (w_copy * 1024.0)
    with open(KERNEL_SRC, "rb") as fh:
        sha = hashlib.sha256(fh.read()).hexdigest()[:16]
    bench = (f"python3 bench.py --workload {workload} --configs \"\" --steps {steps} "
             f"--warmup {2 if steps >= 20 else 1} --no-cpu-baseline --cold-steps 0 --calibrate-copy")
    return {
        "workload": workload,
        "commands": [
            f"rocprofv3 --pmc FETCH_SIZE -d {fetch_dir} -o fetch --output-format csv -- {bench}",
            f"rocprofv3 --pmc WRITE_SIZE -d {write_dir} -o write --output-format csv -- {bench}",
        ],
        "kernel": name,
        "kernel_source_sha256_16": sha,
        "fetch_kib_per_launch": f_k, "write_kib_per_launch": w_k,
        "dispatches": [nf, nw],
        "copy_fetch_kib": f_copy, "copy_write_kib": w_copy,
        "fetch_scale": ff, "write_scale": fw,
        "read_bytes_per_launch": f_k * 1024.0 * ff,
        "written_bytes_per_launch": w_k * 1024.0 * fw,
        "bytes_per_launch": f_k * 1024.0 * ff + w_k * 1024.0 * fw,
    }


def main(argv: list[str]) -> None:
    if len(argv) >= 2 and argv[0] == "stats":
        print(stats_markdown(argv[1]))
    elif len(argv) >= 4 and argv[0] == "traffic":
        t = traffic(argv[1], argv[2], workload=argv[4] if len(argv) > 4 else "qwen4b_b16",
                    kernel=argv[5] if len(argv) > 5 else "round_kernel",
                    steps=int(argv[6]) if len(argv) > 6 else 20)
        with open(argv[3], "w") as fh:
            json.dump(t, fh, indent=1)
        print(json.dumps(t, indent=1))
    else:
        raise SystemExit(__doc__)


if __name__ == "__main__":
    main(sys.argv[1:])
