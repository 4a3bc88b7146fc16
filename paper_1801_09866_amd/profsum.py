"""Summarise rocprofv3 CSV output (kernel stats and per-dispatch counters).

    python -m paper_1801_09866_amd.profsum <rocprofv3 output dir> [--copy-bytes N]
    python -m paper_1801_09866_amd.profsum --traffic WORKLOAD --fetch DIR --write DIR \
        --fetch-scale B --write-scale B

The first form prints, per kernel: calls, average duration; and for counter
runs the mean of every collected counter per dispatch. With --copy-bytes, the
counters of the plain copy kernel in the run are used to print a
bytes-per-counter-unit scale factor. With --dispatches NAME, it also lists
the counters of every dispatch of the kernels whose name contains NAME, in
dispatch order.

The second form prints one line per library kernel,
    traffic WORKLOAD STAGE fetch_bytes=F write_bytes=W source_sha256=S
with the mean FETCH_SIZE and WRITE_SIZE per dispatch scaled to bytes, and a
hash of the sources the kernel is built from, so that a reader (bench.py) can
tell whether the kernel has changed since the counters were taken.

    python -m paper_1801_09866_amd.profsum --sweep-trace DIR --fetch DIR --write DIR \
        --mfma DIR --fetch-scale B --write-scale B [--group 6]

The third form summarises bench.py --sweep: per library kernel and sweep
size, mean duration, HBM bytes and MFMA utilisation per launch.

    python -m paper_1801_09866_amd.profsum --span WORKLOAD --warmup W --steps K \
        --trace DIR [--fetch DIR --write DIR --fetch-scale B --write-scale B] [--mfma DIR] [--leg 0[,1..]]

The fourth form selects the frames bench.py times: a frame is the run of
library kernels that starts with one k_hist_key launch, a leg is the run of
frames after one cache reset (the fill launches of rnnlm_cache_reset), and
the timed frames are frames W .. W+K-1 of leg 0 (the first leg; legs 1..3 are
bench.py's stamped replays of the same frames). It prints, per library kernel, the launches and
mean duration over those frames from the kernel trace, the mean HBM bytes and
MFMA counters from the counter runs, one line per frame for the GRU, and
traffic lines for WORKLOAD:framesW-E as in the second form.
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


def dispatches(d, name):
    """Counter values of each dispatch of the kernels matching `name`:
    [(dispatch id, kernel, {counter: value})] in dispatch order."""
    rows = collections.defaultdict(dict)
    kern = {}
    for p in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(p) as f:
            for r in csv.DictReader(f):
                if name in r["Kernel_Name"]:
                    i = int(r["Dispatch_Id"])
                    rows[i][r["Counter_Name"]] = rows[i].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
                    kern[i] = r["Kernel_Name"]
    return [(i, kern[i], rows[i]) for i in sorted(rows)]


# library kernel -> (benchmark stage, source files it is built from)
KERNELS = {
    "rn::k_hist_key": ("hist_key", ["keys.hip"]),
    "rn::k_frame_plan": ("frame_plan", ["plan.hip"]),
    "rn::k_gru": ("gru_gemm", ["gru.hip"]),
    "rn::k_score_finish": ("score_finish", ["score.hip"]),
    "rn::k_lognorm_gemm": ("lognorm_gemm", ["lognorm.hip"]),
    "rn::k_lognorm_combine": ("lognorm_combine", ["lognorm.hip"]),
}
SHARED = ["common.hpp", "kernels.hpp"]


def source_sha(files):
    import hashlib
    d = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
    h = hashlib.sha256()
    for f in files + SHARED:
        with open(os.path.join(d, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def stage_of(kernel_name):
    base = kernel_name.split("(")[0].replace("void ", "").split("<")[0].strip()
    return KERNELS.get(base)


def trace_dispatches(d):
    """Kernel-trace rows: [(dispatch id, kernel, duration in ns)] in dispatch order."""
    out = []
    for p in glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True):
        with open(p) as f:
            for r in csv.DictReader(f):
                out.append((int(r["Dispatch_Id"]), r["Kernel_Name"],
                            int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
    return sorted(out)


def family(kernel_name):
    return kernel_name.split("(")[0].replace("void ", "").split("<")[0].strip()


def sweep(a):
    """Saturation sweep: each library kernel family's dispatches in order,
    in groups of `group` launches of one size (the first of each group is a
    warm-up and left out): mean duration, HBM bytes (counter units times the
    scales) and MFMA utilisation per launch."""
    fam_of = lambda k: family(k) if stage_of(k) else None
    dur = collections.defaultdict(list)
    for _, k, ns in trace_dispatches(a.sweep_trace):
        if fam_of(k):
            dur[fam_of(k)].append(ns)
    cnt = collections.defaultdict(lambda: collections.defaultdict(list))
    for dd in (a.fetch, a.write, a.mfma):
        if not dd:
            continue
        rows = collections.defaultdict(dict)
        kern = {}
        for p in glob.glob(os.path.join(dd, "**", "*counter_collection.csv"), recursive=True):
            with open(p) as f:
                for r in csv.DictReader(f):
                    i = int(r["Dispatch_Id"])
                    rows[i][r["Counter_Name"]] = rows[i].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
                    kern[i] = r["Kernel_Name"]
        for i in sorted(rows):
            if fam_of(kern[i]):
                for c, v in rows[i].items():
                    cnt[fam_of(kern[i])][c].append(v)
    g = a.group
    print("%-22s %5s %10s %12s %12s %9s" % ("kernel", "size", "us", "fetch_MB", "write_MB", "MfmaUtil"))
    for fam in sorted(dur):
        # a launch of a kernel that runs once per layer is several dispatches:
        # merge them (times and bytes summed, MfmaUtil averaged)
        per = max(1, len(dur[fam]) // (a.sizes * g))

        def merged(v, avg=False):
            out = []
            for k in range(0, len(v) - per + 1, per):
                x = v[k:k + per]
                out.append(sum(x) / len(x) if avg else sum(x))
            return out
        d_ = merged(dur[fam])
        c_ = {c: merged(v, c == "MfmaUtil") for c, v in cnt[fam].items()}
        n = len(d_) // g
        for s in range(n):
            sl = slice(s * g + 1, (s + 1) * g)
            mean = lambda v: sum(v[sl]) / len(v[sl]) if len(v) >= (s + 1) * g else float("nan")
            us = mean(d_) / 1e3
            fb = mean(c_["FETCH_SIZE"]) * a.fetch_scale / 1e6 if c_.get("FETCH_SIZE") else float("nan")
            wb = mean(c_["WRITE_SIZE"]) * a.write_scale / 1e6 if c_.get("WRITE_SIZE") else float("nan")
            mu = mean(c_["MfmaUtil"]) if c_.get("MfmaUtil") else float("nan")
            print("%-22s %5d %10.2f %12.2f %12.2f %9.1f" % (fam, s, us, fb, wb, mu))


def traffic(a):
    fetch, write = counters(a.fetch), counters(a.write)
    for k in sorted(set(fetch) | set(write)):
        st = stage_of(k)
        if st is None:
            continue
        f = fetch.get(k, {}).get("FETCH_SIZE")
        w = write.get(k, {}).get("WRITE_SIZE")
        if not f or not w:
            continue
        fb = sum(f) / len(f) * a.fetch_scale
        wb = sum(w) / len(w) * a.write_scale
        print("traffic %s %s fetch_bytes=%d write_bytes=%d source_sha256=%s"
              % (a.traffic, st[0], fb, wb, source_sha(st[1])))


def dispatch_rows(d, trace=False):
    """[(dispatch id, kernel, {name: value})] in dispatch order: from a kernel
    trace (name "ns": the duration) or from a counter run."""
    if trace:
        return [(i, k, {"ns": float(ns)}) for i, k, ns in trace_dispatches(d)]
    rows = collections.defaultdict(dict)
    kern = {}
    for p in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(p) as f:
            for r in csv.DictReader(f):
                i = int(r["Dispatch_Id"])
                rows[i][r["Counter_Name"]] = rows[i].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
                kern[i] = r["Kernel_Name"]
    return [(i, kern[i], rows[i]) for i in sorted(rows)]


def by_frame(rows, leg):
    """Split dispatch rows into the frames of leg `leg`: [[(kernel family, values)]]."""
    frames, cur_leg, seen = [], 0, False
    for _, k, v in rows:
        fam = family(k)
        if fam == "rn::k_fill_u32":
            if seen:                 # a cache reset after frames: the next leg
                cur_leg += 1
                seen = False
            continue
        if fam == "rn::k_hist_key":
            seen = True
        if cur_leg != leg or stage_of(k) is None:
            continue
        if fam == "rn::k_hist_key":
            frames.append([])
        if frames:
            frames[-1].append((fam, v))
    return frames


def span(a):
    lo, hi = a.warmup, a.warmup + a.steps
    legs = [int(x) for x in str(a.leg).split(",")]

    def select(d, trace=False):
        rows = dispatch_rows(d, trace)
        out = []
        for g in legs:
            fr = by_frame(rows, g)
            if len(fr) < hi:
                raise SystemExit("leg %d of %s holds %d frames, fewer than %d" % (g, d, len(fr), hi))
            out.append(fr[lo:hi])
        return out          # [leg][frame] -> [(kernel family, values)]

    runs = {"ns": select(a.trace, trace=True)}
    for key, d in (("fetch", a.fetch), ("write", a.write), ("mfma", a.mfma)):
        if d:
            runs[key] = select(d)
    scale = {"FETCH_SIZE": a.fetch_scale or 0.0, "WRITE_SIZE": a.write_scale or 0.0}
    per = collections.defaultdict(lambda: collections.defaultdict(list))
    for key, by_leg in runs.items():
        for fr in by_leg:
            for f in fr:
                for fam, v in f:
                    for c, x in v.items():
                        per[fam][c].append(x * scale.get(c, 1.0))
    mean = lambda v: sum(v) / len(v) if v else float("nan")
    print("# frames %d..%d of leg %s (%d frames%s)" % (lo, hi - 1, a.leg, hi - lo,
                                                     ", means over the legs" if len(legs) > 1 else ""))
    cols = sorted({c for v in per.values() for c in v if c != "ns"})
    print("%-24s %8s %10s " % ("kernel", "launches", "avg_us") + " ".join("%16s" % c for c in cols))
    for fam in sorted(per, key=lambda f: -sum(per[f]["ns"])):
        print("%-24s %8d %10.2f " % (fam, len(per[fam]["ns"]), mean(per[fam]["ns"]) / 1e3)
              + " ".join("%16.1f" % mean(per[fam][c]) if per[fam].get(c) else "%16s" % "-" for c in cols))
    print("# per frame, rn::k_gru (bytes: counter units times the calibration scales)")
    print("%6s %10s %14s %14s %10s %12s %12s" % ("frame", "us", "MfmaFlopsF32", "MfmaFlopsBF16", "MfmaUtil",
                                                  "fetch_MB", "write_MB"))
    for i in range(lo, hi):
        def val(key, c):
            if key not in runs:
                return float("nan")
            per_leg = []
            for fr in runs[key]:
                xs = [v.get(c, 0.0) for fam, v in fr[i - lo] if fam == "rn::k_gru"]
                per_leg.append(sum(xs) if c != "MfmaUtil" else mean(xs))
            return mean(per_leg)
        print("%6d %10.2f %14.0f %14.0f %10.1f %12.2f %12.2f" % (
            i, val("ns", "ns") / 1e3, val("mfma", "MfmaFlopsF32"), val("mfma", "MfmaFlopsBF16"),
            val("mfma", "MfmaUtil"), val("fetch", "FETCH_SIZE") * scale["FETCH_SIZE"] / 1e6,
            val("write", "WRITE_SIZE") * scale["WRITE_SIZE"] / 1e6))
    if a.fetch and a.write:
        for fam in sorted(per):
            st = KERNELS.get(fam)
            if st and per[fam].get("FETCH_SIZE") and per[fam].get("WRITE_SIZE"):
                print("traffic %s:frames%d-%d %s fetch_bytes=%d write_bytes=%d source_sha256=%s"
                      % (a.span, lo, hi - 1, st[0], mean(per[fam]["FETCH_SIZE"]), mean(per[fam]["WRITE_SIZE"]),
                         source_sha(st[1])))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("dir", nargs="?")
    ap.add_argument("--copy-bytes", type=float, default=None)
    ap.add_argument("--dispatches", default=None, help="list every dispatch of the kernels matching this name")
    ap.add_argument("--traffic", default=None, help="workload name for traffic lines")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--fetch-scale", type=float, default=None)
    ap.add_argument("--write-scale", type=float, default=None)
    ap.add_argument("--sweep-trace", default=None, help="saturation sweep: the kernel-trace run's directory")
    ap.add_argument("--mfma", default=None, help="saturation sweep: an MfmaUtil counter run's directory")
    ap.add_argument("--group", type=int, default=6, help="saturation sweep: launches per size")
    ap.add_argument("--sizes", type=int, default=4, help="saturation sweep: number of sizes")
    ap.add_argument("--span", default=None, help="bench frames: the workload name for traffic lines")
    ap.add_argument("--trace", default=None, help="bench frames: the kernel-trace run's directory")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--leg", default="0", help="leg index, or several joined by commas")
    a = ap.parse_args()
    if a.span:
        return span(a)
    if a.sweep_trace:
        return sweep(a)
    if a.traffic:
        return traffic(a)
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
    if a.dispatches:
        rows = dispatches(a.dir, a.dispatches)
        names = sorted({c for _, _, v in rows for c in v})
        print("%10s %-40s " % ("dispatch", "kernel") + " ".join("%16s" % n for n in names))
        for i, k, v in rows:
            print("%10d %-40s " % (i, short(k, 40)) + " ".join("%16.1f" % v.get(c, float("nan")) for c in names))


if __name__ == "__main__":
    main()
