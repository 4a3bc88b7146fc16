"""Summarise rocprofv3 CSV output (kernel stats and per-dispatch counters).

    python -m paper_1801_09866_amd.profsum <rocprofv3 output dir> [--copy-bytes N]

Prints, per kernel: calls, average duration; and for counter runs the mean
of every collected counter per dispatch. With --copy-bytes, the counters of
the plain copy kernel (the largest-grid elementwise copy in the run) are
used to print a bytes-per-counter-unit scale factor.
"""
import argparse
import collections
import csv
import glob
import os


def short(name, width=60):
    name = name.split("(")[0]
    return name if len(name) <= width else name[:width - 3] + "..."


def kernel_stats(d):
    rows = []
    for p in glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True):
        with open(p) as f:
            for r in csv.DictReader(f):
                rows.append(r)
    return rows


def counters(d):
    acc = collections.defaultdict(lambda: collections.defaultdict(list))
    for p in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(p) as f:
            for r in csv.DictReader(f):
                acc[r["Kernel_Name"]][r["Counter_Name"]].append(float(r["Counter_Value"]))
    return acc


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("dir")
    ap.add_argument("--copy-bytes", type=float, default=None)
    a = ap.parse_args()
    ks = kernel_stats(a.dir)
    if ks:
        print("%-60s %8s %12s %12s %7s" % ("kernel", "calls", "avg_us", "total_ms", "pct"))
        for r in sorted(ks, key=lambda r: -float(r["TotalDurationNs"])):
            print("%-60s %8s %12.2f %12.3f %7.2f" % (short(r["Name"]), r["Calls"], float(r["AverageNs"]) / 1e3,
                                                  float(r["TotalDurationNs"]) / 1e6, float(r["Percentage"])))
    cs = counters(a.dir)
    if cs:
        names = sorted({c for k in cs.values() for c in k})
        print("%-60s %8s " % ("kernel", "dispatch") + " ".join("%16s" % n for n in names))
        for k, v in sorted(cs.items()):
            n = max(len(x) for x in v.values())
            print("%-60s %8d " % (short(k), n) + " ".join(
                "%16.1f" % (sum(v[c]) / len(v[c]) if v.get(c) else float("nan")) for c in names))
        if a.copy_bytes:
            cands = [k for k in cs if "copy" in k.lower() or "elementwise" in k.lower()]
            for k in cands:
                for c in names:
                    if cs[k].get(c):
                        mx = max(cs[k][c])
                        if mx > 0:
                            print("scale %s on %s: %.4f bytes per unit (max dispatch %.1f units for %.0f bytes)"
                                  % (c, short(k, 40), a.copy_bytes / mx, mx, a.copy_bytes))


if __name__ == "__main__":
    main()
