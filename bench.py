"""Benchmark: frame-wise RNNLM query scoring on one MI355X.

Workload (default): Large fp32 -- V=200,000, E=512, H=1024, one GRU layer,
2^26-entry MaxEnt table with 2-, 3- and 4-gram features, 2,048 queries per
frame from 512 fresh histories plus 30% repeated (history, word) pairs of the
previous frame; sign-only history compression. A step is one frame through
the whole path (quantise, hash, de-duplicate, cache probes, GRU GEMM, NCE +
MaxEnt scoring, cache admission, h' output). Inputs are resident in HBM
before timing starts; caches start empty at frame 0 and the first `warmup`
frames are untimed.

Prints one JSON line (see the keys below). Per-stage kernel times are the
mean of three replays of the timed frames (caches reset, the warm-up frames
run again, so every launch does the same work as in the timed pass), in which
the library records a HIP event pair around every stage's launches, on the
stream its kernels run on (rnnlm_profile). The events lengthen the gaps
between launches (ms_per_step_replay), not the kernels, which is why the
timed pass runs without them.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

REPLAYS = 3   # stamped replays of the timed frames; stage times are their mean
PEAK = {"hbm_GBs": 8000.0, "fp32_mfma_TFs": 157.3, "bf16_mfma_TFs": 2500.0}
METRIC = "RNNLM queries/sec (GRU+NCE+MaxEnt), H=1024 V=200k; % of MFMA/HBM roofline"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed frames (default: all but the warm-up)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed frames (default 50; check config 5)")
    ap.add_argument("--config", default="large")
    ap.add_argument("--qmode", default=None, help="sign | sigdig1 | sigdig2 | sigdig3 | exact")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="time budget of the oracle sample (whole frames from frame 0)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the cpu_baseline leg")
    ap.add_argument("--no-replay", action="store_true", help="skip the per-stage timing replay")
    ap.add_argument("--sessions", type=int, default=1,
                    help="independent decode sessions scored one frame each per launch (the workload's "
                         "frames split into that many consecutive streams)")
    ap.add_argument("--maxent", action="store_true",
                    help="check config: normalise the full output (NCE + MaxEnt logits of every word)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 256 MiB device copy (counter calibration)")
    ap.add_argument("--io-frames", type=int, default=400,
                    help="frames of the per-frame latency and PCIe-inclusive legs (0: skip both)")
    ap.add_argument("--sweep", action="store_true",
                    help="saturation sweep: the key and scoring kernels at 1..8 maximal frames per launch")
    return ap.parse_args()


def qmode_of(arg, cfg):
    from paper_1801_09866_amd import rnnlm as R
    if arg is None:
        return cfg.qmodes[0]
    if arg == "sign":
        return (R.Q_SIGN, 0)
    if arg == "exact":
        return (R.Q_EXACT, 0)
    if arg.startswith("sigdig"):
        return (R.Q_SIGDIG, int(arg[6:]))
    raise SystemExit("unknown qmode " + arg)


def qmode_name(qm, k):
    return {0: "exact", 1: "sign", 2: "sigdig%d" % k}[qm]


def counter_traffic(workload, stage, lo, hi):
    """HBM bytes per launch of `stage` (FETCH_SIZE + WRITE_SIZE, scaled by the
    plain-copy calibration) over frames lo..hi of the first leg, from the
    committed counter summaries under profiles/, or None when none covers this
    workload and frame span or the kernel's sources have changed since the
    counters were taken."""
    import glob

    from paper_1801_09866_amd.profsum import KERNELS, source_sha
    files = next((f for st, f in KERNELS.values() if st == stage), None)
    if files is None:
        return None
    sha = source_sha(files)
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.txt"))):
        with open(path) as fh:
            for line in fh:
                parts = line.split()
                if len(parts) == 6 and parts[0] == "traffic" and parts[2] == stage \
                        and parts[1] == "%s:frames%d-%d" % (workload, lo, hi):
                    kv = dict(x.split("=", 1) for x in parts[3:])
                    if kv.get("source_sha256") == sha:
                        return int(kv["fetch_bytes"]) + int(kv["write_bytes"])
    return None


def algorithmic_work(cfg, st, qm, frames):
    """Algorithmic FLOPs / bytes of each stage over a span with stats `st`.

    The GRU step is a contraction: FLOPs = 2 * 3H * (Kx + H) per row and
    layer. With few rows per frame its weights dominate instead (every frame
    must read all 3H x (Kx + H) weights once), so it is priced against
    whichever roofline is slower for the measured row count.
    """
    m = cfg.model
    wb = 2 if m.wdtype == 1 else 4
    LH, H, E = m.L * m.H, m.H, m.E
    cw_bytes = {0: LH * 4, 1: LH // 8, 2: LH * 2}[qm]
    K = [(E if l == 0 else H) + H for l in range(m.L)]
    flop_row = sum(2 * 3 * H * k for k in K)
    w_bytes = sum(3 * H * k * wb for k in K)
    row_bytes = sum(k * 4 + 2 * H * 4 for k in K)
    gru_flops = st["gru_rows"] * flop_row
    gru_bytes = frames * w_bytes + st["gru_rows"] * row_bytes
    mfma_peak = PEAK["bf16_mfma_TFs"] if m.wdtype == 1 else PEAK["fp32_mfma_TFs"]
    gru = ("mfma", gru_flops) if gru_flops / (mfma_peak * 1e12) >= gru_bytes / (PEAK["hbm_GBs"] * 1e9) \
        else ("hbm", gru_bytes)
    orders = max(0, m.maxent_order - 1)
    computed = st["computed"] + st["query_dups"]
    per_q = H * wb + 4 + 4 * orders + 32 + 4         # row, bias, MaxEnt, words + work record, score
    return {
        "gru_gemm": gru,
        # scores (row gathers, h' reads, MaxEnt) + h' copy-out + history-cache inserts
        "score_finish": ("hbm", computed * per_q + st["score_hits"] * 16 + st["hists"] * H * 4
                         + 2 * st["hists"] * LH * 4 + st["hist_inserted"] * cw_bytes),
        # history vectors and words in, codes and 16 B records out, cache-hit code comparisons;
        # query ids in, planner key and scorer words out
        "hist_key": ("hbm", st["hists"] * (LH * 4 + 12 + cw_bytes + 16) + st["hist_hits"] * cw_bytes
                     + st["queries"] * (8 + 16 + 16)),
        # the plan: per history its 16 B record in, status/slot/h' address out; per query its key
        # in and a 16 B work record out; per GRU row its word, source and destination
        "frame_plan": ("hbm", st["hists"] * (16 + 4 + 4 + 8) + st["queries"] * (16 + 16)
                       + st["gru_rows"] * (4 + 8 + 8)),
    }


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the scoring path here has no multi-GPU launch",
              file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_1801_09866_amd import rnnlm as R
    from paper_1801_09866_amd.workload import CONFIGS, make_workload

    cfg = CONFIGS[args.config]
    if args.warmup is None:
        args.warmup = 5 if cfg.queries == 0 else 50
    if args.steps is None:
        args.steps = cfg.frames - args.warmup
    if args.sweep:
        return main_sweep(args, cfg)
    if cfg.queries == 0:
        return main_check(args, cfg)
    if args.sessions > 1:
        return main_sessions(args, cfg)
    qm, qk = qmode_of(args.qmode, cfg)
    n_frames = min(cfg.frames, args.warmup + args.steps)
    W, K = min(args.warmup, n_frames - 1), n_frames - min(args.warmup, n_frames - 1)
    t0 = time.time()
    wl = make_workload(args.config, n_frames=n_frames)
    log("workload %s generated in %.1fs: %d frames" % (args.config, time.time() - t0, n_frames))
    m = cfg.model
    LH = m.L * m.H
    dev = torch.device("cuda:0")
    sc = R.Scorer(m, wl.weights, qm, qk, max_hist=cfg.max_hist, max_query=max(cfg.queries, 1),
                  cap_hist=cfg.cap_hist, cap_query=cfg.cap_query, device="cuda:0")

    # ---- inputs resident in HBM: all frames, back to back ----------------
    pool = torch.from_numpy(wl.pool.vec).to(dev)
    nh = np.array([f.n_hist for f in wl.frames])
    nq = np.array([f.n_query for f in wl.frames])
    ho = np.concatenate([[0], np.cumsum(nh)])
    qo = np.concatenate([[0], np.cumsum(nq)])
    hv = pool.index_select(0, torch.from_numpy(np.concatenate([f.pool_idx for f in wl.frames])).to(dev))
    hw = torch.from_numpy(np.concatenate([f.hist_words for f in wl.frames]).astype(np.int32)).to(dev)
    qh = torch.from_numpy(np.concatenate([f.q_hist for f in wl.frames]).astype(np.int32)).to(dev)
    qt = torch.from_numpy(np.concatenate([f.q_tgt for f in wl.frames]).astype(np.int32)).to(dev)
    scores = torch.empty(max(int(qo[-1]), 1), dtype=torch.float32, device=dev)
    hnew = torch.empty((int(ho[-1]), LH), dtype=torch.float32, device=dev)
    del pool
    fsz, hsz = hv.element_size() * LH, 4
    frames, outs = [], []
    for i in range(n_frames):
        frames.append(R.Frame(int(nh[i]), int(nq[i]), hv.data_ptr() + int(ho[i]) * fsz,
                              hw.data_ptr() + int(ho[i]) * 12, qh.data_ptr() + int(qo[i]) * 4,
                              qt.data_ptr() + int(qo[i]) * 4))
        outs.append(R.Out(scores.data_ptr() + int(qo[i]) * 4, hnew.data_ptr() + int(ho[i]) * LH * hsz,
                          None, None, None, None, None))
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    L = R.load()
    ctx = sc.ctx

    def run(lo, hi):
        for i in range(lo, hi):
            rc = L.rnnlm_score_frame(ctx, ctypes.byref(frames[i]), ctypes.byref(outs[i]), sp)
            if rc:
                raise R.RnnlmError(rc, L.rnnlm_last_error().decode())

    # ---- warmup + timed region -------------------------------------------
    sc.reset()
    run(0, W)
    torch.cuda.synchronize()
    st0 = sc.stats()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    ev0.record(stream)
    run(W, n_frames)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    gpu_ms = ev0.elapsed_time(ev1)
    st1 = sc.stats()
    span = {k: st1[k] - st0[k] for k in st1 if k not in ("hist_cache_size", "score_cache_size", "device_error")}
    secs = gpu_ms / 1e3
    queries = int(qo[n_frames] - qo[W])
    value = queries / secs
    log("timed %d frames: %.3f ms GPU (%.3f ms wall), %.0f queries/s" % (K, gpu_ms, wall * 1e3, value))

    # ---- per-stage kernel times: replay the same frames with events ------
    stages, roofline, stamped_ms = {}, None, None
    if not args.no_replay:
        prof, stamped_ms = {}, 0.0
        for _ in range(REPLAYS):
            sc.reset()
            run(0, W)
            sc.profile(R.STAGES[:4])
            torch.cuda.synchronize()
            ev0.record(stream)
            run(W, n_frames)
            ev1.record(stream)
            torch.cuda.synchronize()
            stamped_ms += ev0.elapsed_time(ev1) / REPLAYS
            for name, (ms, launches) in sc.profile_read().items():
                prof[name] = (prof.get(name, (0.0, 0))[0] + ms / REPLAYS, launches)
            sc.profile(())
        work = algorithmic_work(cfg, span, qm, K)
        for name, (ms, launches) in prof.items():
            entry = {"ms_total": round(ms, 4), "launches": launches, "us_per_launch": round(1e3 * ms / launches, 2)}
            if name in work:
                bound, amount = work[name]
                if bound == "mfma":
                    peak = PEAK["bf16_mfma_TFs"] if m.wdtype == 1 else PEAK["fp32_mfma_TFs"]
                    ach = amount / (ms / 1e3) / 1e12 if ms > 0 else 0.0
                    entry.update(bound="mfma", achieved=round(ach, 2), peak=peak, unit="TFLOP/s",
                                 frac=round(ach / peak, 4), algorithmic=amount)
                else:
                    ach = amount / (ms / 1e3) / 1e9 if ms > 0 else 0.0
                    entry.update(bound="hbm", achieved=round(ach, 1), peak=PEAK["hbm_GBs"], unit="GB/s",
                                 frac=round(ach / PEAK["hbm_GBs"], 4), algorithmic=amount)
            stages[name] = entry
        dom = max(stages, key=lambda n: stages[n]["ms_total"])
        e = stages[dom]
        roofline = {"kernel": dom, "bound": e["bound"], "achieved": e["achieved"], "peak": e["peak"],
                    "unit": e["unit"], "frac": e["frac"],
                    "traffic": counter_traffic("%s_%s" % (cfg.name, qmode_name(qm, qk)), dom, W, n_frames - 1),
                    "algorithmic_per_launch": round(e["algorithmic"] / e["launches"]),
                    "us_per_launch": e["us_per_launch"]}
        if dom == "gru_gemm":
            roofline["gru_rows_per_launch"] = round(span["gru_rows"] / K, 2)
        rows = rows_by_frame(sc, run, W, n_frames)
        log("gru rows by frame %d..%d: %s" % (W, n_frames - 1, rows))
        log("stages:", json.dumps(stages))

    # ---- per-frame latency, and the rate with each frame's block over PCIe --
    io = None
    if args.io_frames > 0 and K > 1:
        P = min(args.io_frames, K)
        io = {"frames": P}
        io.update(latency_leg(sc, run, W, P, stream))
        io.update(pcie_leg(sc, L, ctx, run, W, P, hv, hw, qh, qt, ho, qo, LH, dev))
        io["resident_queries_per_s_same_frames"] = io.pop("resident_rate")
        log("io:", json.dumps(io))

    if args.copy_calibration:
        a = torch.empty(64 << 20, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()

    # ---- cpu baseline: the oracle on a bounded prefix of the same frames --
    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(args, wl, qm, qk, sc, run, frames)

    hit = lambda a, b: round(a / b, 4) if b else None
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "queries/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(gpu_ms / K, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16-weights/f32-accumulate" if m.wdtype == 1 else "f32", "data": "synthetic",
        "ms_per_step_replay": round(stamped_ms / K, 5) if stamped_ms else None,
        "config": {"workload": "%s_%s: V=%d E=%d H=%d L=%d MaxEnt 2^%d orders 2..%d, %d queries/frame"
                               % (cfg.name, qmode_name(qm, qk), m.V, m.E, m.H, m.L, m.maxent_log2,
                                  m.maxent_order, cfg.queries),
                   "frames_timed": K, "queries_timed": queries, "qmode": qmode_name(qm, qk)},
        "frames_per_s": round(K / secs, 1),
        "computed_queries_per_s": round(span["computed"] / secs, 1),
        "gru_rows_per_s": round(span["gru_rows"] / secs, 1),
        "score_hit_ratio": hit(span["score_hits"], span["queries"]),
        "hist_hit_ratio": hit(span["hist_hits"], span["hists"]),
        "wall_ms": round(wall * 1e3, 3),
        "roofline": roofline,
        "gru_rows_by_frame": rows if roofline else None,
        "stages": stages,
        "frame_io": io,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def rows_by_frame(sc, run, W, n):
    """GRU rows of each of frames W..n-1 (one frame at a time, the statistics
    read after each), at most 200 frames."""
    import torch
    sc.reset()
    run(0, W)
    torch.cuda.synchronize()
    prev = sc.stats()["gru_rows"]
    out = []
    for i in range(W, min(n, W + 200)):
        run(i, i + 1)
        cur = sc.stats()["gru_rows"]
        out.append(cur - prev)
        prev = cur
    return out


def hip_runtime():
    """The HIP runtime torch has loaded (same soname as the library's), for
    copies and events on streams of our own."""
    H = ctypes.CDLL("libamdhip64.so.7")
    vp, P = ctypes.c_void_p, ctypes.POINTER
    H.hipMemcpyAsync.argtypes = [vp, vp, ctypes.c_size_t, ctypes.c_int, vp]
    H.hipEventCreateWithFlags.argtypes = [P(vp), ctypes.c_uint]
    H.hipEventRecord.argtypes = [vp, vp]
    H.hipEventDestroy.argtypes = [vp]
    H.hipStreamWaitEvent.argtypes = [vp, vp, ctypes.c_uint]
    H.hipStreamSynchronize.argtypes = [vp]
    H.hipEventElapsedTime.argtypes = [P(ctypes.c_float), vp, vp]
    return H


def _hip_ok(rc, what):
    if rc != 0:
        raise RuntimeError("%s failed: hip error %d" % (what, rc))


def latency_leg(sc, run, W, P, stream):
    """Frames W .. W+P-1 one at a time, the host waiting for each: host-observed
    latency from the launch call to the frame's results being complete."""
    import torch
    sc.reset()
    run(0, W)
    torch.cuda.synchronize()
    lat = []
    for i in range(W, W + P):
        t = time.perf_counter()
        run(i, i + 1)
        stream.synchronize()
        lat.append(time.perf_counter() - t)
    lat = np.array(lat) * 1e6
    return {"latency_us_p50": round(float(np.percentile(lat, 50)), 2),
            "latency_us_p99": round(float(np.percentile(lat, 99)), 2),
            "latency_us_max": round(float(lat.max()), 2)}


def pcie_leg(sc, L, ctx, run, W, P, hv, hw, qh, qt, ho, qo, LH, dev):
    """Frames W .. W+P-1 with their inputs starting in pinned host memory, as
    a decoder on the host would hand them over: per frame, one copy of the
    frame's block (history vectors, words, query ids) into device memory, the
    frame scored, and its scores copied back to pinned host memory, all in
    stream order on the library's stream. (Copies on a second stream, ordered
    by events, per frame or per 8 frames, measured no faster here: the copies
    and the frame's kernels did not overlap.) Returns the rate with transfers,
    the rate of one large copy from the same pinned buffer, and the resident
    rate on the same frames (inputs already in HBM)."""
    import torch

    from paper_1801_09866_amd import rnnlm as R
    H = hip_runtime()
    al = lambda n: (n + 255) // 256 * 256
    nh = [int(ho[i + 1] - ho[i]) for i in range(W, W + P)]
    nq = [int(qo[i + 1] - qo[i]) for i in range(W, W + P)]
    lay = [(0, al(a * LH * 4), al(a * LH * 4) + al(a * 12), al(a * LH * 4) + al(a * 12) + al(b * 4))
           for a, b in zip(nh, nq)]
    size = [l[3] + al(b * 4) for l, b in zip(lay, nq)]
    host_off = np.concatenate([[0], np.cumsum(size)]).astype(np.int64)
    host = torch.empty(int(host_off[-1]), dtype=torch.uint8, pin_memory=True)
    for j, i in enumerate(range(W, W + P)):
        base = int(host_off[j])
        o = lay[j]
        for off, t in ((o[0], hv[int(ho[i]):int(ho[i + 1])]), (o[1], hw[int(ho[i]):int(ho[i + 1])]),
                       (o[2], qh[int(qo[i]):int(qo[i + 1])]), (o[3], qt[int(qo[i]):int(qo[i + 1])])):
            b = t.contiguous().view(torch.uint8).reshape(-1).cpu()
            host[base + off: base + off + b.numel()].copy_(b)
    qoff = np.concatenate([[0], np.cumsum(nq)]).astype(np.int64)
    host_scores = torch.empty(int(qoff[-1]), dtype=torch.float32, pin_memory=True)
    slot = torch.empty(max(size), dtype=torch.uint8, device=dev)
    dscore = torch.empty(max(nq), dtype=torch.float32, device=dev)
    dh = torch.empty((max(nh), LH), dtype=torch.float32, device=dev)
    frames = [R.Frame(nh[j], nq[j], slot.data_ptr() + lay[j][0], slot.data_ptr() + lay[j][1],
                      slot.data_ptr() + lay[j][2], slot.data_ptr() + lay[j][3], None) for j in range(P)]
    out = R.Out(dscore.data_ptr(), dh.data_ptr(), None, None, None, None, None)
    comp = torch.cuda.current_stream()
    sp = ctypes.c_void_p(comp.cuda_stream)

    def event():
        e = ctypes.c_void_p()
        _hip_ok(H.hipEventCreateWithFlags(ctypes.byref(e), 0), "hipEventCreateWithFlags")
        return e
    t0, t1 = event(), event()

    def elapsed():
        _hip_ok(H.hipStreamSynchronize(sp), "hipStreamSynchronize")
        ms = ctypes.c_float()
        _hip_ok(H.hipEventElapsedTime(ctypes.byref(ms), t0, t1), "hipEventElapsedTime")
        return ms.value / 1e3

    sc.reset()
    run(0, W)
    torch.cuda.synchronize()
    _hip_ok(H.hipEventRecord(t0, sp), "hipEventRecord")
    for j in range(P):
        _hip_ok(H.hipMemcpyAsync(ctypes.c_void_p(slot.data_ptr()), ctypes.c_void_p(host.data_ptr() + int(host_off[j])),
                                 size[j], 1, sp), "hipMemcpyAsync")
        rc = L.rnnlm_score_frame(ctx, ctypes.byref(frames[j]), ctypes.byref(out), sp)
        if rc:
            raise R.RnnlmError(rc, L.rnnlm_last_error().decode())
        _hip_ok(H.hipMemcpyAsync(ctypes.c_void_p(host_scores.data_ptr() + int(qoff[j]) * 4),
                                 ctypes.c_void_p(dscore.data_ptr()), nq[j] * 4, 2, sp), "hipMemcpyAsync")
    _hip_ok(H.hipEventRecord(t1, sp), "hipEventRecord")
    secs = elapsed()
    # the link itself: one large copy from the same pinned buffer
    big = min(int(host_off[-1]), 256 << 20)
    dbig = torch.empty(big, dtype=torch.uint8, device=dev)
    _hip_ok(H.hipEventRecord(t0, sp), "hipEventRecord")
    _hip_ok(H.hipMemcpyAsync(ctypes.c_void_p(dbig.data_ptr()), ctypes.c_void_p(host.data_ptr()), big, 1, sp),
            "hipMemcpyAsync")
    _hip_ok(H.hipEventRecord(t1, sp), "hipEventRecord")
    big_secs = elapsed()
    # the same frames with inputs resident, for the comparison
    sc.reset()
    run(0, W)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(comp)
    run(W, W + P)
    e1.record(comp)
    torch.cuda.synchronize()
    rsecs = e0.elapsed_time(e1) / 1e3
    for e in (t0, t1):
        H.hipEventDestroy(e)
    h2d = int(sum(size))
    return {"pcie_queries_per_s": round(sum(nq) / secs, 1),
            "pcie_h2d_bytes_per_frame": h2d // P,
            "pcie_h2d_GBs": round(h2d / secs / 1e9, 2),
            "pcie_h2d_GBs_one_copy_of_%d_MiB" % (big >> 20): round(big / big_secs / 1e9, 2),
            "resident_rate": round(sum(nq) / rsecs, 1)}


def cpu_baseline(args, wl, qm, qk, sc, run, frames):
    import torch
    from threadpoolctl import threadpool_info

    from threadpoolctl import threadpool_limits

    from oracle import Oracle
    cfg, m = wl.cfg, wl.cfg.model

    def sample(budget):
        """Whole frames from frame 0 and empty caches until the budget is
        spent; when every frame is done first, the pass starts again from a
        new oracle (empty caches). Returns (frames of the longest pass, passes
        begun, queries, seconds)."""
        t = time.perf_counter()
        nq = S = passes = 0
        while time.perf_counter() - t < budget:
            o = Oracle(m.V, m.E, m.H, m.L, m.maxent_log2, m.maxent_order, wl.weights, qm, qk,
                       cap_hist=cfg.cap_hist, cap_query=cfg.cap_query)
            passes += 1
            for i, fr in enumerate(wl.frames):
                o.score_frame(wl.pool.vec[fr.pool_idx], fr.hist_words, fr.q_hist, fr.q_tgt)
                nq += fr.n_query
                S = max(S, i + 1)
                if time.perf_counter() - t >= budget:
                    break
        return S, passes, nq, time.perf_counter() - t

    S, passes, nq, secs = sample(args.cpu_seconds)
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    with threadpool_limits(limits=1):   # the same oracle on one thread, over a shorter budget
        S1, passes1, nq1, secs1 = sample(args.cpu_seconds / 3)
    what = lambda S, p: "frames 0..%d" % (S - 1) + (" x %d passes" % p if p > 1 else "")
    frames_q = wl.frames
    # the GPU on the same frames (cold caches, frame 0 on)
    sc.reset()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    run(0, S)
    e1.record()
    torch.cuda.synchronize()
    gsec = e0.elapsed_time(e1) / 1e3
    log("oracle: %s, %d queries in %.1fs" % (what(S, passes), nq, secs))
    return {"value": round(nq / secs, 1), "unit": "queries/s", "cores": int(threads), "kind": "oracle",
            "sample": "%s of the same workload from empty caches (%d queries, %.1f s)"
                      % (what(S, passes), nq, secs),
            "gpu_value_same_frames": round(sum(f.n_query for f in frames_q[:S]) / gsec, 1),
            "value_1_thread": round(nq1 / secs1, 1),
            "sample_1_thread": "%s (%d queries, %.1f s)" % (what(S1, passes1), nq1, secs1)}


METRIC_CHECK = "full-vocabulary log-normalisers/sec (GRU step + logsumexp over V), H=1024 V=200k; % of fp32 MFMA roofline"


def main_check(args, cfg):
    """Check config: each frame's histories go through the GRU step (EXACT
    keys, no queries), then the full-vocabulary log-normaliser of every
    resulting h' (a [n x H] . [H x V] GEMM plus logsumexp). One step is one
    frame; the value is log-normalisers (histories) per second."""
    import torch

    from paper_1801_09866_amd import rnnlm as R
    from paper_1801_09866_amd.workload import make_workload

    qm, qk = qmode_of(args.qmode, cfg)
    n_frames = min(cfg.frames, args.warmup + args.steps)
    W, K = min(args.warmup, n_frames - 1), n_frames - min(args.warmup, n_frames - 1)
    t0 = time.time()
    wl = make_workload(args.config, n_frames=n_frames)
    log("workload %s generated in %.1fs: %d frames" % (args.config, time.time() - t0, n_frames))
    m = cfg.model
    LH = m.L * m.H
    dev = torch.device("cuda:0")
    sc = R.Scorer(m, wl.weights, qm, qk, max_hist=cfg.max_hist, max_query=1,
                  cap_hist=cfg.cap_hist, cap_query=cfg.cap_query, device="cuda:0")
    pool = torch.from_numpy(wl.pool.vec).to(dev)
    nh = np.array([f.n_hist for f in wl.frames])
    ho = np.concatenate([[0], np.cumsum(nh)])
    hv = pool.index_select(0, torch.from_numpy(np.concatenate([f.pool_idx for f in wl.frames])).to(dev))
    hw = torch.from_numpy(np.concatenate([f.hist_words for f in wl.frames]).astype(np.int32)).to(dev)
    hnew = torch.empty((int(ho[-1]), LH), dtype=torch.float32, device=dev)
    logz = torch.empty(int(ho[-1]), dtype=torch.float32, device=dev)
    dummy = torch.empty(1, dtype=torch.float32, device=dev)
    del pool
    frames, outs = [], []
    for i in range(n_frames):
        frames.append(R.Frame(int(nh[i]), 0, hv.data_ptr() + int(ho[i]) * LH * 4, hw.data_ptr() + int(ho[i]) * 12,
                              None, None))
        outs.append(R.Out(dummy.data_ptr(), hnew.data_ptr() + int(ho[i]) * LH * 4, None, None, None, None, None))
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    L = R.load()
    ctx = sc.ctx
    top = (m.L - 1) * m.H

    def run(lo, hi):
        for i in range(lo, hi):
            rc = L.rnnlm_score_frame(ctx, ctypes.byref(frames[i]), ctypes.byref(outs[i]), sp)
            if rc == 0:
                hp = ctypes.c_void_p(hnew.data_ptr() + (int(ho[i]) * LH + top) * 4)
                zp = ctypes.c_void_p(logz.data_ptr() + int(ho[i]) * 4)
                if args.maxent:   # the context of the next word after each h' is its history's words
                    rc = L.rnnlm_log_normalizer_maxent(ctx, hp, ctypes.c_void_p(hw.data_ptr() + int(ho[i]) * 12),
                                                       int(nh[i]), zp, sp)
                else:
                    rc = L.rnnlm_log_normalizer(ctx, hp, int(nh[i]), zp, sp)
            if rc:
                raise R.RnnlmError(rc, L.rnnlm_last_error().decode())

    if m.L != 1:
        raise SystemExit("the check config has one layer (the normaliser reads h' rows back to back)")
    sc.reset()
    run(0, W)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_start = time.perf_counter()
    ev0.record(stream)
    run(W, n_frames)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    gpu_ms = ev0.elapsed_time(ev1)
    sc.stats()   # raises on a device error
    nlog = int(ho[n_frames] - ho[W])
    value = nlog / (gpu_ms / 1e3)
    z = logz[int(ho[W]):int(ho[n_frames])].double().cpu().numpy()
    log("timed %d frames: %.3f ms GPU, %.0f log-normalisers/s" % (K, gpu_ms, value))

    stages, roofline = {}, None
    if not args.no_replay:
        sc.reset()
        run(0, W)
        sc.profile(R.STAGES[:4] + ("lognorm_gemm", "lognorm_combine"))
        run(W, n_frames)
        torch.cuda.synchronize()
        prof = sc.profile_read()
        sc.profile(())
        flops = 2.0 * m.H * m.V * nlog
        for name, (ms, launches) in prof.items():
            e = {"ms_total": round(ms, 4), "launches": launches, "us_per_launch": round(1e3 * ms / launches, 2)}
            if name == "lognorm_gemm":
                ach = flops / (ms / 1e3) / 1e12
                e.update(bound="mfma", achieved=round(ach, 2), peak=PEAK["fp32_mfma_TFs"], unit="TFLOP/s",
                         frac=round(ach / PEAK["fp32_mfma_TFs"], 4), algorithmic=flops)
            stages[name] = e
        g = stages["lognorm_gemm"]
        roofline = {"kernel": "lognorm_gemm", "bound": "mfma", "achieved": g["achieved"], "peak": g["peak"],
                    "unit": "TFLOP/s", "frac": g["frac"],
                    "traffic": counter_traffic("%s_%s" % (cfg.name, qmode_name(qm, qk)), "lognorm_gemm",
                                               W, n_frames - 1),
                    "us_per_launch": g["us_per_launch"]}
        log("stages:", json.dumps(stages))

    cpu = None
    if not args.no_cpu:
        from threadpoolctl import threadpool_info

        from oracle import Oracle, log_normalizer, log_normalizer_maxent
        o = Oracle(m.V, m.E, m.H, m.L, m.maxent_log2, m.maxent_order, wl.weights, qm, qk,
                   cap_hist=cfg.cap_hist, cap_query=cfg.cap_query)
        t = time.perf_counter()
        S = cnt = 0
        for fr in wl.frames:
            res = o.score_frame(wl.pool.vec[fr.pool_idx], fr.hist_words, fr.q_hist, fr.q_tgt)
            if args.maxent:
                log_normalizer_maxent(res.hnew[:, top:top + m.H], wl.weights["U_out"], wl.weights["b_out"],
                                      wl.weights["maxent"], fr.hist_words, m.maxent_order, m.maxent_log2)
            else:
                log_normalizer(res.hnew[:, top:top + m.H], wl.weights["U_out"], wl.weights["b_out"])
            cnt += fr.n_hist
            S += 1
            if time.perf_counter() - t >= args.cpu_seconds:
                break
        secs = time.perf_counter() - t
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
        cpu = {"value": round(cnt / secs, 2), "unit": "log-normalisers/s", "cores": int(threads), "kind": "oracle",
               "sample": "frames 0..%d of the same workload (%d histories, %.1f s)" % (S - 1, cnt, secs)}
        log("oracle: %d frames, %d log-normalisers in %.1fs" % (S, cnt, secs))

    line = {
        "metric": METRIC_CHECK, "value": round(value, 1), "unit": "log-normalisers/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(gpu_ms / K, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "check: V=%d E=%d H=%d L=%d, %d histories/frame, EXACT keys, logsumexp over V%s"
                               % (m.V, m.E, m.H, m.L, cfg.hists,
                                  " of NCE + MaxEnt (orders 2..%d) logits" % m.maxent_order if args.maxent else ""),
                   "frames_timed": K, "maxent": bool(args.maxent)},
        "wall_ms": round(wall * 1e3, 3),
        # NCE self-normalisation: how far log Z is from 0 over the timed histories
        "logz": {"mean": round(float(z.mean()), 6), "sd": round(float(z.std()), 6),
                 "min": round(float(z.min()), 6), "max": round(float(z.max()), 6)},
        "roofline": roofline,
        "stages": stages,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def main_sessions(args, cfg):
    """S independent decode sessions: the workload's frames are split into S
    consecutive streams (session k gets frames k*F .. k*F + F - 1, its cache
    starting empty at its first frame), and one launch set scores one frame
    of every session. A step is one such block of S frames; the value is the
    queries of all sessions per second."""
    import torch

    from paper_1801_09866_amd import rnnlm as R
    from paper_1801_09866_amd.workload import make_workload

    S = args.sessions
    qm, qk = qmode_of(args.qmode, cfg)
    F = cfg.frames // S                      # frames per session
    W = min(args.warmup // S if args.warmup else 0, F - 1)
    wl = make_workload(args.config, n_frames=F * S)
    m = cfg.model
    LH = m.L * m.H
    dev = torch.device("cuda:0")
    sc = R.Scorer(m, wl.weights, qm, qk, max_hist=cfg.max_hist, max_query=max(cfg.queries, 1),
                  cap_hist=cfg.cap_hist, cap_query=cfg.cap_query, device="cuda:0", sessions=S)
    pool = torch.from_numpy(wl.pool.vec).to(dev)
    nh = np.array([f.n_hist for f in wl.frames])
    nq = np.array([f.n_query for f in wl.frames])
    ho = np.concatenate([[0], np.cumsum(nh)])
    qo = np.concatenate([[0], np.cumsum(nq)])
    hv = pool.index_select(0, torch.from_numpy(np.concatenate([f.pool_idx for f in wl.frames])).to(dev))
    hw = torch.from_numpy(np.concatenate([f.hist_words for f in wl.frames]).astype(np.int32)).to(dev)
    qh = torch.from_numpy(np.concatenate([f.q_hist for f in wl.frames]).astype(np.int32)).to(dev)
    qt = torch.from_numpy(np.concatenate([f.q_tgt for f in wl.frames]).astype(np.int32)).to(dev)
    scores = torch.empty(int(qo[-1]), dtype=torch.float32, device=dev)
    hnew = torch.empty((int(ho[-1]), LH), dtype=torch.float32, device=dev)
    del pool
    blocks = []
    for j in range(F):                       # block j: frame j of every session
        fa, oa = (R.Frame * S)(), (R.Out * S)()
        for k in range(S):
            i = k * F + j
            fa[k] = R.Frame(int(nh[i]), int(nq[i]), hv.data_ptr() + int(ho[i]) * LH * 4, hw.data_ptr() + int(ho[i]) * 12,
                            qh.data_ptr() + int(qo[i]) * 4, qt.data_ptr() + int(qo[i]) * 4, None)
            oa[k] = R.Out(scores.data_ptr() + int(qo[i]) * 4, hnew.data_ptr() + int(ho[i]) * LH * 4,
                          None, None, None, None, None)
        blocks.append((fa, oa))
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    L = R.load()
    ctx = sc.ctx

    def run(lo, hi):
        for j in range(lo, hi):
            rc = L.rnnlm_score_frames(ctx, blocks[j][0], blocks[j][1], S, sp)
            if rc:
                raise R.RnnlmError(rc, L.rnnlm_last_error().decode())

    sc.reset()
    run(0, W)
    torch.cuda.synchronize()
    st0 = sc.stats()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    run(W, F)
    ev1.record(stream)
    torch.cuda.synchronize()
    gpu_ms = ev0.elapsed_time(ev1)
    st1 = sc.stats()
    span = {k: st1[k] - st0[k] for k in st1 if k not in ("hist_cache_size", "score_cache_size", "device_error")}
    secs = gpu_ms / 1e3
    queries = span["queries"]
    value = queries / secs
    log("timed %d blocks of %d frames: %.3f ms GPU, %.0f queries/s" % (F - W, S, gpu_ms, value))
    stages = {}
    if not args.no_replay:
        sc.reset()
        run(0, W)
        sc.profile(R.STAGES[:4])
        run(W, F)
        torch.cuda.synchronize()
        for name, (ms, launches) in sc.profile_read().items():
            stages[name] = {"ms_total": round(ms, 4), "launches": launches, "us_per_launch": round(1e3 * ms / launches, 2)}
        sc.profile(())
        log("stages:", json.dumps(stages))
    hit = lambda a, b: round(a / b, 4) if b else None
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "queries/s", "n_gpus": 1,
        "steps": F - W, "warmup": W, "ms_per_step": round(gpu_ms / (F - W), 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32" if m.wdtype == 0 else "bf16-weights/f32-accumulate",
        "data": "synthetic",
        "config": {"workload": "%s_%s split into %d independent sessions of %d frames, one frame of each per launch"
                               % (cfg.name, qmode_name(qm, qk), S, F), "sessions": S, "qmode": qmode_name(qm, qk)},
        "frames_per_s": round(span["frames"] / secs, 1),
        "computed_queries_per_s": round(span["computed"] / secs, 1),
        "score_hit_ratio": hit(span["score_hits"], span["queries"]),
        "hist_hit_ratio": hit(span["hists"] and span["hist_hits"], span["hists"]),
        "stages": stages, "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


def main_sweep(args, cfg):
    """Saturation sweep. A frame is at most 2048 histories and 8192 queries
    (the planner's one-block limits), so one frame's key and scoring launches
    last a few microseconds and mostly show latency. Here S = 1, 2, 4, 8
    independent sessions each bring one maximal frame to one set of launches
    (up to 16,384 histories and 65,536 queries per launch), with fresh random
    histories, uniform target words and empty caches, so that every query is
    scored and every history key is new. Each point is the median of 5
    launches; the value per stage is its algorithmic bytes (or FLOPs) over its
    kernel time, against the HBM (or MFMA) peak. Prints one JSON line per
    point."""
    import torch

    from paper_1801_09866_amd import rnnlm as R
    from paper_1801_09866_amd.workload import make_weights

    m = cfg.model
    qm, qk = qmode_of(args.qmode, cfg)
    S_max, n_h, n_q = 8, 2048, 8192
    t0 = time.time()
    w = make_weights(m, 99)
    log("weights generated in %.1fs" % (time.time() - t0))
    LH = m.L * m.H
    dev = torch.device("cuda:0")
    sc = R.Scorer(m, w, qm, qk, max_hist=n_h, max_query=n_q, cap_hist=1 << 14, cap_query=1 << 16,
                  device="cuda:0", sessions=S_max)
    del w
    g = torch.Generator(device=dev)
    g.manual_seed(180109866)
    hv = torch.tanh(torch.randn((S_max, n_h, LH), generator=g, device=dev)) * 0.9
    hw = torch.randint(1, m.V, (S_max, n_h, 3), generator=g, device=dev, dtype=torch.int32)
    qh = torch.randint(0, n_h, (S_max, n_q), generator=g, device=dev, dtype=torch.int32)
    qt = torch.randint(0, m.V, (S_max, n_q), generator=g, device=dev, dtype=torch.int32)
    frames = [(hv[k], hw[k], qh[k], qt[k]) for k in range(S_max)]
    outs = [sc.alloc_out(n_h, n_q, hnew=True, debug=False) for _ in range(S_max)]
    mfma_peak = PEAK["bf16_mfma_TFs"] if m.wdtype == 1 else PEAK["fp32_mfma_TFs"]
    for S in (1, 2, 4, 8):
        reps = []
        for r in range(6):
            sc.reset()
            sc.profile(R.STAGES[:4])
            sc.score_frames(frames[:S], outs[:S], hnew=True, debug=False)
            torch.cuda.synchronize()
            prof = sc.profile_read()
            st = sc.stats()
            if r > 0:   # the first launch at each size is a warm-up
                reps.append({k: v[0] for k, v in prof.items()})
        sc.profile(())
        work = algorithmic_work(cfg, st, qm, 1)
        point = {"sweep": "saturation", "sessions": S, "histories_per_launch": st["hists"],
                 "queries_per_launch": st["queries"], "computed": st["computed"], "gru_rows": st["gru_rows"],
                 "qmode": qmode_name(qm, qk), "stages": {}}
        for name in R.STAGES[:4]:
            ms = float(np.median([rp[name] for rp in reps]))
            bound, amount = work[name]
            e = {"us": round(ms * 1e3, 2), "bound": bound}
            if bound == "mfma":
                ach = amount / (ms / 1e3) / 1e12
                e.update(TFLOPs=round(ach, 2), frac=round(ach / mfma_peak, 4))
            else:
                ach = amount / (ms / 1e3) / 1e9
                e.update(MB=round(amount / 1e6, 2), GBs=round(ach, 1), frac=round(ach / PEAK["hbm_GBs"], 4))
            point["stages"][name] = e
        print(json.dumps(point), flush=True)
    assert sc.stats()["device_error"] == 0


if __name__ == "__main__":
    main()
