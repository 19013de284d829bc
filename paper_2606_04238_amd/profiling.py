"""Summaries of rocprofv3 runs of the decode MLP kernels, and the HBM traffic
figure that bench.py reports from them.

``summarize`` turns the CSV output of three rocprofv3 runs of the same
command -- ``--kernel-trace --stats``, ``--pmc FETCH_SIZE`` and
``--pmc WRITE_SIZE`` -- into a short markdown summary.  The byte counters
are calibrated against reference dispatches of known size that bench.py
launches after its timing:

* ``--calibrate-stream-mib S``: the read-only streaming probe reads S MiB
  with the same non-temporal 128-bit loads as the weight stream, then S MiB
  with plain loads;
* ``--calibrate-copy-mib N``: a copy-like elementwise dispatch reads N MiB
  and writes N MiB.

FETCH_SIZE is scaled by known / counted bytes of the non-temporal probe
(the load kind of the weight stream) when it ran, else of the copy;
WRITE_SIZE by those of the copy.  Every factor found is listed.

The summary records a digest of the HIP sources; ``read_traffic`` returns
the traffic figure only while the sources still hash to that digest, so a
figure taken on an older kernel is never reported for a newer one.

Usage (on the CPU, after the runs):
    python3 -m paper_2606_04238_amd.profiling [--stream-mib=S] [--pmc-dir=DIR ...] \
        KT_DIR PF_DIR PW_DIR KERNEL_SUBSTR[|KERNEL_SUBSTR...] COPY_MIB OUT.md \
        "COMMAND ..." ["COMMAND ..." ...]
Each --pmc-dir adds a table of every counter of that --pmc run for the
kernels named.
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
    """{kernel name: [values per dispatch]} of the one counter in a --pmc run,
    and the run's rows."""
    rows = list(csv.DictReader(open(_one(os.path.join(pmc_dir, "*counter_collection.csv")))))
    name = rows[0]["Counter_Name"] if rows else "?"
    out = {}
    for r in rows:
        out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return name, out, rows


def step_dispatches(rows, parts, name_key):
    """Dispatch ids of the step's launches, one list per part: every run of
    consecutive dispatches (in dispatch order) whose kernel names contain
    parts[0], parts[1], ... in turn.  A command may launch the same kernel
    outside the step (one block per call, other precisions); those
    dispatches do not follow the step's order and are left out.  None when
    the rows carry no dispatch ids or no such run exists."""
    if not rows or "Dispatch_Id" not in rows[0]:
        return None
    seq = sorted({int(r["Dispatch_Id"]): r[name_key] for r in rows}.items())
    out = [[] for _ in parts]
    i = 0
    while i + len(parts) <= len(seq):
        if all(parts[j] in seq[i + j][1] for j in range(len(parts))):
            for j in range(len(parts)):
                out[j].append(seq[i + j][0])
            i += len(parts)
        else:
            i += 1
    return out if out[0] else None


def _part_values(rows, per, parts):
    """Per part: the counter values of the step's dispatches (by dispatch
    order when the rows allow it, else every dispatch of that name)."""
    ids = step_dispatches(rows, parts, "Kernel_Name")
    if ids is None:
        return [[v for k, vs in per.items() if part in k for v in vs] for part in parts]
    by_id = {}
    for r in rows:
        by_id.setdefault(int(r["Dispatch_Id"]), []).append(float(r["Counter_Value"]))
    return [[v for i in idl for v in by_id[i]] for idl in ids]


def _closest(per_kernel, substr, known_kib):
    """Counted KiB of the reference dispatch whose kernel name contains
    `substr` and whose counter lies closest to the known size (fills and
    other small dispatches of the same name read almost nothing, so the pick
    is unambiguous); None if no such dispatch ran."""
    best = None
    for k, vals in per_kernel.items():
        if substr not in k:
            continue
        for v in vals:
            if best is None or abs(v - known_kib) < abs(best - known_kib):
                best = v
    return best if best and best > 0 else None


NT_PROBE, PLAIN_PROBE, COPY = "stream_read_kernel<true>", "stream_read_kernel<false>", "elementwise"


def _factors(per_kernel, counter, copy_kib, stream_kib):
    """{reference: (counted KiB, known KiB, factor)} for every reference
    dispatch of this run that applies to the counter."""
    out = {}
    refs = [(COPY, copy_kib)]
    if counter.startswith("FETCH") and stream_kib:
        refs = [(NT_PROBE, stream_kib), (PLAIN_PROBE, stream_kib)] + refs
    for name, known in refs:
        if not known:
            continue
        c = _closest(per_kernel, name, known)
        if c is not None:
            out[name] = (c, known, known / c)
    return out


def summarize(kt_dir, pf_dir, pw_dir, kernel, copy_mib, out_md, commands, stream_mib=0,
              extra=None):
    """Write the summary; `extra` is a list of (title, markdown lines) that
    other counter passes contribute (they do not enter the traffic figure)."""
    stats = list(csv.DictReader(open(_one(os.path.join(kt_dir, "*kernel_stats.csv")))))
    # `kernel` may name several launches of one step, joined by "|": the
    # step's duration and bytes are the sums of their per-dispatch means
    parts = kernel.split("|")
    krows = []
    for part in parts:
        rows = [r for r in stats if part in r["Name"]]
        if len(rows) != 1:
            raise ValueError("kernel %r matches %d rows of the stats" % (part, len(rows)))
        krows.append(dict(rows[0]))
    # with the per-dispatch trace, the step's own dispatches give the figures
    traces = glob.glob(os.path.join(kt_dir, "*kernel_trace.csv"))
    if len(traces) == 1:
        trows = list(csv.DictReader(open(traces[0])))
        ids = step_dispatches(trows, parts, "Kernel_Name")
        if ids is not None:
            dur = {int(r["Dispatch_Id"]): int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
                   for r in trows}
            for kr, idl in zip(krows, ids):
                ns = [dur[i] for i in idl]
                kr.update(Calls=len(ns), AverageNs=statistics.mean(ns), MinNs=min(ns), MaxNs=max(ns))
    avg_us = sum(float(r["AverageNs"]) for r in krows) / 1e3
    copy_kib = copy_mib * 1024.0
    stream_kib = stream_mib * 1024.0
    lines = ["# %s -- rocprofv3 summary" % kernel, ""]
    lines += ["Commands (run from the repository root on one MI355X; `R` is that root):", ""]
    lines += ["    " + c for c in commands]
    def trace_rows(rs):
        return ["| `%s` | %s | %.3f | %.3f | %.3f | %s |" % (
            r["Name"][:90], r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
            float(r["MaxNs"]) / 1e3, r["Percentage"]) for r in rs]
    head = ["| kernel | calls | avg us | min us | max us | share % |", "|---|---|---|---|---|---|"]
    lines += ["", "## Kernel trace (--kernel-trace --stats), the launches of one step", "",
              "Dispatches taken in the step's launch order; the share is that of every "
              "dispatch of the kernel in the run.", ""]
    lines += head + trace_rows(krows)
    lines += ["", "Sum of their average durations: %.3f us." % avg_us]
    lines += ["", "## Kernel trace, the run's top dispatches (all kernels of the command)", ""]
    lines += head + trace_rows(stats[:6])
    total = 0.0
    cal = ["", "## Calibration dispatches (known bytes / counted bytes)", "",
           "| counter | reference dispatch | counted KiB | known KiB | factor |", "|---|---|---|---|---|"]
    lines += ["", "## HBM byte counters (--pmc, one counter per run)", "",
              "| counter | KiB per step (sum of the kernels' means) | dispatches | reference | factor "
              "| bytes per step |", "|---|---|---|---|---|---|"]
    for d in (pf_dir, pw_dir):
        counter, per, crows = _counter_means(d)
        kib = 0.0
        nd = 0
        for part, vals in zip(parts, _part_values(crows, per, parts)):
            if not vals:
                raise ValueError("kernel %r not in %s" % (part, d))
            kib += statistics.mean(vals)
            nd += len(vals)
        facs = _factors(per, counter, copy_kib, stream_kib)
        if not facs:
            raise ValueError("no calibration dispatch found for %s" % counter)
        for name, (c, known, fac) in facs.items():
            cal.append("| %s | `%s` | %.1f | %.0f | %.4f |" % (counter, name, c, known, fac))
        ref = NT_PROBE if NT_PROBE in facs else COPY
        factor = facs[ref][2]
        b = kib * 1024.0 * factor
        total += b
        lines.append("| %s | %.1f | %d | `%s` | %.4f | %.0f |" % (counter, kib, nd, ref, factor, b))
    lines += cal
    for title, body in (extra or []):
        lines += ["", "## " + title, ""] + list(body)
    lines += ["", "traffic_bytes_per_launch: %.0f" % total,
              "kernel_avg_us: %.3f" % avg_us,
              "kernel: %s" % kernel,
              "source_digest: %s" % source_digest(), ""]
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines))
    return total


def counter_table(pmc_dir, kernels):
    """Markdown rows of every counter of one --pmc run, mean per dispatch, for
    each kernel whose name contains one of `kernels` (the step's dispatches
    when the rows carry dispatch ids)."""
    rows = list(csv.DictReader(open(_one(os.path.join(pmc_dir, "*counter_collection.csv")))))
    ids = step_dispatches(rows, kernels, "Kernel_Name")
    keep = None if ids is None else {i: kn for kn, idl in zip(kernels, ids) for i in idl}
    acc = {}
    for r in rows:
        for kn in kernels:
            if kn in r["Kernel_Name"] and (keep is None or keep.get(int(r["Dispatch_Id"])) == kn):
                acc.setdefault((kn, r["Counter_Name"]), []).append(float(r["Counter_Value"]))
    out = ["| kernel | counter | mean per dispatch | dispatches |", "|---|---|---|---|"]
    for (kn, cn), vs in sorted(acc.items()):
        out.append("| `%s` | %s | %.6g | %d |" % (kn, cn, statistics.mean(vs), len(vs)))
    return out


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
    stream = 0
    extra_dirs = []
    rest = []
    for v in a:
        if v.startswith("--stream-mib="):
            stream = int(v.split("=", 1)[1])
        elif v.startswith("--pmc-dir="):
            extra_dirs.append(v.split("=", 1)[1])
        else:
            rest.append(v)
    if len(rest) < 7:
        print(__doc__)
        sys.exit(2)
    kern = rest[3]
    extra = [("Counters (--pmc %s)" % os.path.basename(d.rstrip("/")), counter_table(d, kern.split("|")))
             for d in extra_dirs]
    t = summarize(rest[0], rest[1], rest[2], kern, int(rest[4]), rest[5], rest[6:], stream_mib=stream,
                  extra=extra)
    print("traffic bytes per launch: %.0f" % t)
