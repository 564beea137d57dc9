"""Summarise a rocprofv3 kernel trace of bench.py as a short markdown table.

    python -m paper_2605_07243_amd.profile_summary TRACE.csv --last-steps N \
        --step-marker block1_reset_kernel [--title ...]

The window is the last N hot-path steps, delimited by the first kernel of
each step (``--step-marker``).  For every kernel family the table lists
dispatches per step, total and mean duration, so the mean duration of a
kernel can be compared with the HIP-event timing bench.py reports.
"""
from __future__ import annotations

import argparse
import collections
import csv
import re
import sys


def family(name: str) -> str:
    name = name.split("(")[0].replace("void ", "").strip()
    name = re.sub(r"^sb::", "", name)
    return name


def summarise(path: str, last_steps: int, marker: str):
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    starts = [i for i, r in enumerate(rows) if marker in r["Kernel_Name"]]
    if len(starts) < last_steps + 1:
        raise SystemExit(f"only {len(starts)} steps found")
    lo, hi = starts[-last_steps - 1], starts[-1]
    win = rows[lo:hi]
    agg = collections.defaultdict(lambda: [0, 0.0])
    for r in win:
        d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        a = agg[family(r["Kernel_Name"])]
        a[0] += 1
        a[1] += d
    busy = sum(v[1] for v in agg.values())
    return agg, busy, len(win)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("trace")
    ap.add_argument("--last-steps", type=int, default=5)
    ap.add_argument("--step-marker", default="block1_reset_kernel")
    ap.add_argument("--top", type=int, default=24)
    a = ap.parse_args(argv)
    agg, busy, n = summarise(a.trace, a.last_steps, a.step_marker)
    k = a.last_steps
    out = [f"Window: last {k} steps, {n} dispatches, kernel busy "
           f"{busy / k:.1f} us/step.", "",
           "| kernel | dispatches/step | us/step | mean us | share |",
           "|---|---:|---:|---:|---:|"]
    fams = sorted(agg.items(), key=lambda kv: -kv[1][1])
    gemm = [0, 0.0]
    for name, (cnt, tot) in fams:
        if name.startswith("gemm_"):
            gemm[0] += cnt
            gemm[1] += tot
    for name, (cnt, tot) in fams[:a.top]:
        out.append(f"| `{name}` | {cnt / k:.1f} | {tot / k:.1f} | "
                   f"{tot / cnt:.2f} | {100 * tot / busy:.1f}% |")
    out += ["", f"All projection GEMM dispatches (`gemm_*`): "
                f"{gemm[0] / k:.1f}/step, mean {gemm[1] / max(gemm[0], 1):.2f} "
                f"us, {gemm[1] / k:.1f} us/step."]
    print("\n".join(out))


if __name__ == "__main__":
    sys.exit(main())
