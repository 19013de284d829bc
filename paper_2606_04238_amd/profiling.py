"""Summaries of rocprofv3 runs of the decode MLP kernels, and the HBM traffic
figure that bench.py reports from them.

``summarize`` turns the CSV output of three rocprofv3 runs of the same
command -- ``--kernel-trace --stats``, ``--pmc FETCH_SIZE`` and
``--pmc WRITE_SIZE`` -- into a short markdown summary.  The byte counters
are calibrated against a copy-like elementwise dispatch of known size that
bench.py launches with ``--calibrate-copy-mib N`` (it reads N MiB and writes
N MiB): the factor known bytes / counted bytes of that dispatch scales the
counters of the kernel under study.

The summary records a digest of the HIP sources; ``read_traffic`` returns
the traffic figure only while the sources still hash to that digest, so a
figure taken on an older kernel is never reported for a newer one.

Usage (on the CPU, after the three runs):
    python3 -m paper_2606_04238_amd.profiling KT_DIR PF_DIR PW_DIR KERNEL_SUBSTR \
        COPY_MIB OUT.md "COMMAND ..." ["COMMAND ..." ...]
"""
from __future__ import annotations

import csv
import glob
import hashlib
import os
import statistics
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))
_ROOT = os.path.dirname(_HERE)


def source_digest() -> str:
    """sha256 over the HIP sources and the C header, in a fixed order."""
    files = sorted(glob.glob(os.path.join(_HERE, "csrc", "*")))
    files.append(os.path.join(_ROOT, "include", "qmlp.h"))
    h = hashlib.sha256()
    for p in files:
        if os.path.isfile(p):
            h.update(os.path.basename(p).encode())
            with open(p, "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()[:16]


def _one(path_glob):
    hits = glob.glob(path_glob)
    if len(hits) != 1:
        raise FileNotFoundError("expected one file for %s, found %d" % (path_glob, len(hits)))
    return hits[0]


def _counter_means(pmc_dir):
    """{kernel name: [values per dispatch]} of the one counter in a --pmc run."""
    rows = list(csv.DictReader(open(_one(os.path.join(pmc_dir, "*counter_collection.csv")))))
    name = rows[0]["Counter_Name"] if rows else "?"
    out = {}
    for r in rows:
        out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return name, out


def _copy_dispatch(per_kernel, counter, copy_kib):
    """Counted KiB of the calibration dispatch: the elementwise dispatch whose
    counter lies closest to the known size (the fill that precedes it reads
    almost nothing, so the pick is unambiguous)."""
    best = None
    for k, vals in per_kernel.items():
        if "elementwise" not in k:
            continue
        for v in vals:
            if best is None or abs(v - copy_kib) < abs(best - copy_kib):
                best = v
    if best is None or best <= 0:
        raise ValueError("no calibration dispatch found for %s" % counter)
    return best


def summarize(kt_dir, pf_dir, pw_dir, kernel, copy_mib, out_md, commands):
    stats = list(csv.DictReader(open(_one(os.path.join(kt_dir, "*kernel_stats.csv")))))
    krow = [r for r in stats if kernel in r["Name"]]
    if len(krow) != 1:
        raise ValueError("kernel %r matches %d rows of the stats" % (kernel, len(krow)))
    krow = krow[0]
    copy_kib = copy_mib * 1024.0
    lines = ["# %s -- rocprofv3 summary" % kernel, ""]
    lines += ["Commands (run from the repository root on one MI355X; `R` is that root):", ""]
    lines += ["    " + c for c in commands]
    lines += ["", "## Kernel trace (--kernel-trace --stats), top dispatches", "",
              "| kernel | calls | avg us | min us | max us | share % |",
              "|---|---|---|---|---|---|"]
    for r in stats[:6]:
        lines.append("| `%s` | %s | %.3f | %.3f | %.3f | %s |" % (
            r["Name"][:90], r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
            float(r["MaxNs"]) / 1e3, r["Percentage"]))
    total = 0.0
    lines += ["", "## HBM byte counters (--pmc, one counter per run)", "",
              "| counter | kernel KiB/dispatch (mean) | dispatches | copy dispatch KiB | known KiB "
              "| factor | kernel bytes/dispatch |", "|---|---|---|---|---|---|---|"]
    for d in (pf_dir, pw_dir):
        counter, per = _counter_means(d)
        vals = [v for k, vs in per.items() if kernel in k for v in vs]
        if not vals:
            raise ValueError("kernel %r not in %s" % (kernel, d))
        counted = _copy_dispatch(per, counter, copy_kib)
        factor = copy_kib / counted
        kib = statistics.mean(vals)
        b = kib * 1024.0 * factor
        total += b
        lines.append("| %s | %.1f | %d | %.1f | %.0f | %.4f | %.0f |" % (
            counter, kib, len(vals), counted, copy_kib, factor, b))
    lines += ["", "traffic_bytes_per_launch: %.0f" % total,
              "kernel_avg_us: %.3f" % (float(krow["AverageNs"]) / 1e3),
              "kernel: %s" % kernel,
              "source_digest: %s" % source_digest(), ""]
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    return total


def read_traffic(profile_md, kernel):
    """HBM bytes per launch recorded in a summary, or None when the summary is
    missing, covers another kernel, or was taken on different sources."""
    if not os.path.isfile(profile_md):
        return None
    kv = {}
    for line in open(profile_md):
        if ":" in line and not line.startswith(("|", " ", "#")):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel") != kernel or kv.get("source_digest") != source_digest():
        return None
    try:
        return float(kv["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


if __name__ == "__main__":
    a = sys.argv[1:]
    if len(a) < 7:
        print(__doc__)
        sys.exit(2)
    t = summarize(a[0], a[1], a[2], a[3], int(a[4]), a[5], a[6:])
    print("traffic bytes per launch: %.0f" % t)
