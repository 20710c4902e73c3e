"""Summaries of rocprofv3 output for one scoring level (the files under profiles/).

    python -m paper_2608_21131_amd.rocprof_summary traffic FETCH.csv WRITE.csv
    python -m paper_2608_21131_amd.rocprof_summary trace KERNEL_TRACE.csv
    python -m paper_2608_21131_amd.rocprof_summary valu VALUBUSY.csv
    python -m paper_2608_21131_amd.rocprof_summary waves SQ1.csv [SQ2.csv ...]

`traffic` takes the counter_collection.csv of two `rocprofv3 --pmc FETCH_SIZE` /
`--pmc WRITE_SIZE` runs of `bench.py --copy-calib ...`.  The run's calibration
kernels (torch's fill, copy and sum of one plain 1 GiB buffer) fix the scale of
each counter: the fill writes 1 GiB, the copy reads and writes 1 GiB, the sum
reads 1 GiB.  The level is the span of dispatches after the second-to-last
multiply-accumulate launch up to and including the last one: one giant-step
phase, one baby-step phase and one multiply-accumulate, the same work as one
timed step.  `trace` lists the kernels of the same span with their durations,
`valu` their duration-weighted VALUBusy from a `--pmc VALUBusy` run.
`waves` sums SQ counters (one or more `--pmc SQ_...` runs, SQ_WAVE_CYCLES
among them) over the same span and gives each as a fraction of the kernel's
wave-cycles.
"""
import csv
import hashlib
import os
import re
import sys
from collections import OrderedDict

GIB = 1 << 30
MAC = "k_mac_diag"
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def sources_sha256():
    """sha256 over the library's kernel and host sources (any change voids a traffic summary)."""
    h = hashlib.sha256()
    for f in ("fa_kernels.hip", "fa_host.cpp", "fa_internal.h"):
        h.update(open(os.path.join(ROOT, "paper_2608_21131_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def _rows(path):
    rows = list(csv.DictReader(open(path)))
    key = "Dispatch_Id" if "Dispatch_Id" in rows[0] else "Start_Timestamp"
    rows.sort(key=lambda r: int(r[key]))
    return rows


def _name(k):
    m = re.search(r"(k_[a-z0-9_]+)", k)
    if m:
        return m.group(1)
    for tag in ("FillFunctor", "reduce_kernel", "copyBuffer", "fillBuffer"):
        if tag in k:
            return tag
    return k[:40]


def _span(rows):
    """Rows of the dispatches after the second-to-last multiply-accumulate launch up to the last one
    (a counter file holds one row per counter per dispatch)."""
    key = "Dispatch_Id" if "Dispatch_Id" in rows[0] else "Start_Timestamp"
    mac = sorted({int(r[key]) for r in rows if MAC in r["Kernel_Name"]})
    if len(mac) < 2:
        raise SystemExit("need at least two multiply-accumulate launches (a warm-up and a timed step)")
    return [r for r in rows if mac[-2] < int(r[key]) <= mac[-1]]


def _calib(rows, counter):
    """KiB the counter reports per GiB of known traffic, from the 1 GiB calibration kernels."""
    big = [r for r in rows if int(r.get("Grid_Size", 0) or 0) >= (1 << 17)]
    val = {}
    for r in big:
        n = _name(r["Kernel_Name"])
        if n in ("FillFunctor", "copyBuffer", "reduce_kernel") and n not in val:
            val[n] = float(r["Counter_Value"])
    gib_kib = GIB / 1024
    if counter == "FETCH_SIZE":
        reads = [val[k] for k in ("copyBuffer", "reduce_kernel") if k in val]
        return (sum(reads) / len(reads)) / gib_kib if reads else None, val
    writes = [val[k] for k in ("FillFunctor", "copyBuffer") if k in val]
    return (sum(writes) / len(writes)) / gib_kib if writes else None, val


def traffic(fetch_csv, write_csv):
    fr, wr = _rows(fetch_csv), _rows(write_csv)
    cf, vf = _calib(fr, "FETCH_SIZE")
    cw, vw = _calib(wr, "WRITE_SIZE")
    if not cf or not cw:
        raise SystemExit("calibration kernels not found (run bench.py with --copy-calib)")
    sf, sw = _span(fr), _span(wr)
    if [_name(r["Kernel_Name"]) for r in sf] != [_name(r["Kernel_Name"]) for r in sw]:
        raise SystemExit("the two runs dispatched different kernels")
    agg = OrderedDict()
    for f, w in zip(sf, sw):
        a = agg.setdefault(_name(f["Kernel_Name"]), [0, 0.0, 0.0, 0.0])
        a[0] += 1
        a[1] += float(f["Counter_Value"]) * 1024 / cf
        a[2] += float(w["Counter_Value"]) * 1024 / cw
        a[3] += (int(f["End_Timestamp"]) - int(f["Start_Timestamp"])) / 1e3
    out = ["Calibration (KiB reported per GiB of known traffic): FETCH_SIZE "
           f"{cf * GIB / 1024:.0f} (copy {vf.get('copyBuffer', 0):.0f}, sum {vf.get('reduce_kernel', 0):.0f} "
           f"KiB), WRITE_SIZE {cw * GIB / 1024:.0f} (fill {vw.get('FillFunctor', 0):.0f}, copy "
           f"{vw.get('copyBuffer', 0):.0f} KiB); read factor {1 / cf:.4f}, write factor {1 / cw:.4f}.", "",
           "| kernel | launches | read GB | written GB | total GB | us (counter run) | GB/s |",
           "|---|---:|---:|---:|---:|---:|---:|"]
    tr = tw = 0.0
    for k, (cnt, r, w, us) in sorted(agg.items(), key=lambda kv: -(kv[1][1] + kv[1][2])):
        out.append(f"| {k} | {cnt} | {r / 1e9:.3f} | {w / 1e9:.3f} | {(r + w) / 1e9:.3f} | {us:.1f} | "
                   f"{(r + w) / (us * 1e-6) / 1e9:.0f} |")
        tr += r
        tw += w
    out.append(f"| **level** | {sum(a[0] for a in agg.values())} | {tr / 1e9:.3f} | {tw / 1e9:.3f} | "
               f"{(tr + tw) / 1e9:.3f} | | |")
    out += ["", f"level_read_bytes: {int(tr)}", f"level_write_bytes: {int(tw)}",
            f"level_traffic_bytes: {int(tr + tw)}", f"sources_sha256: {sources_sha256()}"]
    return "\n".join(out)


def trace(trace_csv):
    rows = _span(_rows(trace_csv))
    t0 = int(rows[0]["Start_Timestamp"])
    agg = OrderedDict()
    for r in rows:
        a = agg.setdefault(_name(r["Kernel_Name"]), [0, 0.0])
        a[0] += 1
        a[1] += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    span = (int(rows[-1]["End_Timestamp"]) - t0) / 1e3
    out = [f"Span of one level (first dispatch to the multiply-accumulate's end): {span:.1f} us; kernels "
           "on two streams overlap, so their durations sum to more than the span.", "",
           "| kernel | launches | total us | avg us |", "|---|---:|---:|---:|"]
    for k, (cnt, us) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        out.append(f"| {k} | {cnt} | {us:.1f} | {us / cnt:.1f} |")
    return "\n".join(out)


def valu(valu_csv):
    rows = _span(_rows(valu_csv))
    agg = OrderedDict()
    for r in rows:
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        a = agg.setdefault(_name(r["Kernel_Name"]), [0, 0.0, 0.0])
        a[0] += 1
        a[1] += us
        a[2] += us * float(r["Counter_Value"])
    out = ["| kernel | launches | us (counter run) | VALUBusy |", "|---|---:|---:|---:|"]
    for k, (cnt, us, w) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        out.append(f"| {k} | {cnt} | {us:.1f} | {w / us:.1f}% |")
    return "\n".join(out)


def waves(*csvs):
    agg = OrderedDict()
    names = []
    for path in csvs:
        for r in _span(_rows(path)):
            c = r["Counter_Name"]
            if c not in names:
                names.append(c)
            agg.setdefault(_name(r["Kernel_Name"]), {}).setdefault(c, 0.0)
            agg[_name(r["Kernel_Name"])][c] += float(r["Counter_Value"])
    if "SQ_WAVE_CYCLES" not in names:
        raise SystemExit("SQ_WAVE_CYCLES is needed as the denominator")
    cols = [c for c in names if c != "SQ_WAVE_CYCLES"]
    out = ["| kernel | " + " | ".join(c.replace("SQ_", "") for c in cols) + " |",
           "|---|" + "---:|" * len(cols)]
    for k, v in sorted(agg.items(), key=lambda kv: -kv[1].get("SQ_WAVE_CYCLES", 0.0)):
        wc = v.get("SQ_WAVE_CYCLES", 0.0) or 1.0
        out.append(f"| {k} | " + " | ".join(f"{v.get(c, 0.0) / wc:.2f}" for c in cols) + " |")
    return "\n".join(out)


if __name__ == "__main__":
    if len(sys.argv) == 4 and sys.argv[1] == "traffic":
        print(traffic(sys.argv[2], sys.argv[3]))
    elif len(sys.argv) == 3 and sys.argv[1] == "trace":
        print(trace(sys.argv[2]))
    elif len(sys.argv) == 3 and sys.argv[1] == "valu":
        print(valu(sys.argv[2]))
    elif len(sys.argv) >= 3 and sys.argv[1] == "waves":
        print(waves(*sys.argv[2:]))
    else:
        raise SystemExit(__doc__)
