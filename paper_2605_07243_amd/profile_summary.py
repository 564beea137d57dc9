"""Summarise rocprofv3 output of bench.py as short markdown tables.

    python -m paper_2605_07243_amd.profile_summary TRACE.csv --last-steps N \
        --step-marker block1_reset_kernel
    python -m paper_2605_07243_amd.profile_summary --pmc COUNTERS.csv \
        --last-steps N --calib-bytes B [--json OUT.json]

The window is the last N complete hot-path steps, delimited by the first
kernel of each step (``--step-marker``), leaving out steps that contain a
kernel named by ``--skip-steps-with`` (by default the one-thread row-count
copy that only bench.py's profiled pass launches, so that the window holds
the timed steps).  With a kernel trace, every kernel family gets
its dispatches per step, total and mean duration, so the mean duration of a
kernel can be compared with the HIP-event timing bench.py reports.  With a
counter collection (``--pmc``), every family gets the mean value of each
counter per dispatch (and, given SQ_VALU_MFMA_BUSY_CYCLES and
GRBM_GUI_ACTIVE, the fraction of SIMD cycles its MFMAs kept busy); the
calibration copy (bench.py --calib-mib, an
elementwise kernel that reads and writes B bytes) gives the factor by which
the counter over- or under-states bytes moved.
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


def step_window(names, last_steps: int, marker: str, skip: str):
    """Indices into `names` (kernel names in launch order) of the last
    `last_steps` complete steps that launch no kernel containing `skip`."""
    starts = [i for i, n in enumerate(names) if marker in n]
    steps = [range(a, b) for a, b in zip(starts, starts[1:])]
    if skip:
        steps = [r for r in steps if not any(skip in names[i] for i in r)]
    if len(steps) < last_steps:
        raise SystemExit(f"only {len(steps)} complete steps found")
    return [i for r in steps[len(steps) - last_steps:] for i in r]


def summarise(path: str, last_steps: int, marker: str, skip: str = ""):
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    win = [rows[i] for i in step_window([r["Kernel_Name"] for r in rows],
                                        last_steps, marker, skip)]
    agg = collections.defaultdict(lambda: [0, 0.0])
    for r in win:
        d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        a = agg[family(r["Kernel_Name"])]
        a[0] += 1
        a[1] += d
    busy = sum(v[1] for v in agg.values())
    return agg, busy, len(win)


def summarise_pmc(path: str, last_steps: int, marker: str, calib: str,
                  skip: str = ""):
    """Per family and counter: (dispatches in window, mean value); plus the
    calibration kernel's mean per counter (over all its dispatches)."""
    per = collections.defaultdict(dict)     # dispatch -> counter -> value
    names = {}
    for r in csv.DictReader(open(path)):
        d = int(r["Dispatch_Id"])
        names[d] = r["Kernel_Name"]
        c = r["Counter_Name"]
        per[d][c] = per[d].get(c, 0.0) + float(r["Counter_Value"])
    order = sorted(per)
    win = [order[i] for i in step_window([names[d] for d in order],
                                         last_steps, marker, skip)]
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    for d in win:
        for c, v in per[d].items():
            agg[family(names[d])][c].append(v)
    cal = collections.defaultdict(list)
    for d in order:
        if calib in names[d]:
            for c, v in per[d].items():
                cal[c].append(v)
    return agg, {c: sum(v) / len(v) for c, v in cal.items()}


def main_pmc(a):
    import json
    agg, cal = summarise_pmc(a.pmc, a.last_steps, a.step_marker, a.calib,
                             a.skip_steps_with)
    k = a.last_steps
    counters = sorted({c for f in agg.values() for c in f})
    kib = a.calib_bytes / 1024.0
    factor = {c: cal[c] / kib for c in cal if kib > 0}
    out = [f"Window: last {k} steps.  Calibration copy ({a.calib}, "
           f"{a.calib_bytes} B read and written): " +
           ", ".join(f"{c} {cal[c]:.0f} KiB (factor {factor[c]:.3f})"
                     for c in sorted(cal)), "",
           "| kernel | dispatches/step | " +
           " | ".join(f"{c} KiB/dispatch" for c in counters) + " |",
           "|---|---:|" + "---:|" * len(counters)]
    fams = sorted(agg.items(), key=lambda kv: -sum(
        sum(v) for v in kv[1].values()))
    table = {}
    for name, cs in fams:
        n = max(len(v) for v in cs.values())
        means = {c: (sum(cs[c]) / len(cs[c]) if cs.get(c) else 0.0)
                 for c in counters}
        table[name] = {"dispatches_per_step": n / k, **means}
        out.append(f"| `{name}` | {n / k:.1f} | " +
                   " | ".join(f"{means[c]:.0f}" for c in counters) + " |")
    # MFMA utilisation: SQ_VALU_MFMA_BUSY_CYCLES is summed over every SIMD
    # (256 CUs x 4), GRBM_GUI_ACTIVE over the 8 XCDs (each counts the
    # dispatch's active cycles)
    if "SQ_VALU_MFMA_BUSY_CYCLES" in counters and "GRBM_GUI_ACTIVE" in counters:
        out += ["", "| kernel | MFMA busy (% of SIMD cycles) |", "|---|---:|"]
        for name, row in table.items():
            act = row["GRBM_GUI_ACTIVE"] / 8.0
            if act > 0 and row["SQ_VALU_MFMA_BUSY_CYCLES"] > 0:
                util = row["SQ_VALU_MFMA_BUSY_CYCLES"] / (act * 1024.0)
                row["mfma_busy_frac"] = util
                out.append(f"| `{name}` | {100 * util:.1f} |")
    print("\n".join(out))
    if a.json:
        with open(a.json, "w") as f:
            json.dump({"calibration_kib": cal, "factor": factor,
                       "per_dispatch_kib": table}, f, indent=1)


# the GEMM kernels, their launch planning and the helpers they inline
# (declarations in kernels.h do not change the kernels)
GEMM_SOURCES = ("csrc/gemm.hip", "csrc/common.h")


def gemm_sources_sha256() -> str:
    """Hash of the sources of the projection GEMM kernel: counter figures
    taken from another version of them no longer describe the kernel."""
    import hashlib
    import os
    h = hashlib.sha256()
    here = os.path.dirname(os.path.abspath(__file__))
    for f in GEMM_SOURCES:
        with open(os.path.join(here, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def combine(fetch_json: str, write_json: str, out: str):
    """HBM bytes per projection-GEMM dispatch (all gemm_* families, weighted
    by dispatch count) from a FETCH_SIZE and a WRITE_SIZE summary, each
    divided by its calibration factor."""
    import json
    res = {"kernel": "gemm_* (all projection GEMMs)",
           "sources_sha256": gemm_sources_sha256()}
    total = 0.0
    for key, path, counter in (("fetch", fetch_json, "FETCH_SIZE"),
                               ("write", write_json, "WRITE_SIZE")):
        d = json.load(open(path))
        n = kib = 0.0
        for fam, row in d["per_dispatch_kib"].items():
            if fam.startswith("gemm_"):
                n += row["dispatches_per_step"]
                kib += row["dispatches_per_step"] * row[counter]
        f = d["factor"][counter]
        res[key] = {"counter_kib_per_dispatch": kib / n,
                    "calibration_factor": f,
                    "bytes_per_dispatch": kib / n * 1024 / f,
                    "dispatches_per_step": n}
        total += kib / n * 1024 / f
    res["bytes_per_dispatch"] = total
    with open(out, "w") as fh:
        json.dump(res, fh, indent=1)
    print(json.dumps(res, indent=1))


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--combine", nargs=3, metavar=("FETCH_JSON", "WRITE_JSON",
                                                   "OUT_JSON"))
    ap.add_argument("trace", nargs="?")
    ap.add_argument("--pmc", help="counter_collection.csv of a --pmc run")
    ap.add_argument("--calib", default="neg_kernel",
                    help="name fragment of the calibration copy kernel")
    ap.add_argument("--calib-bytes", type=float, default=0.0)
    ap.add_argument("--json")
    ap.add_argument("--last-steps", type=int, default=5)
    ap.add_argument("--step-marker", default="block1_reset_kernel")
    ap.add_argument("--skip-steps-with", default="copy_int_kernel",
                    help="leave out steps that launch this kernel ('' keeps all)")
    ap.add_argument("--top", type=int, default=24)
    a = ap.parse_args(argv)
    if a.combine:
        return combine(*a.combine)
    if a.pmc:
        return main_pmc(a)
    agg, busy, n = summarise(a.trace, a.last_steps, a.step_marker,
                             a.skip_steps_with)
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
