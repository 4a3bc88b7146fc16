"""Synthetic redundancy sweep in the shape of the paper's Table 1.

    python -m paper_1801_09866_amd.table1 [--config large] [--beam 512]
        [--fanout 4] [--frames 200] [--stay 0.5] [--shared 12] [--focus 0.8]
        [--wx 0.5] [--wh 0.01] [--bz -2] [--seed 1]

Runs one seeded decode loop (workload.decode_plan: a beam whose hypotheses
either stay, repeating their queries, or advance by one of their candidate
words, the new history being the h' just produced) through the library once
per history compression: exact, 3, 2 and 1 significant digits, and sign
(Sec. 3). Histories are device-resident handles throughout. Prints, per
mode, the unique LM queries (scores computed), unique GRU rows, the cache
hit ratios, the reduction against exact, and how far the scores move from
the exact run's on the same queries; ends with one JSON line.

History compression only merges states that have come close, which a
trained language model's do once paths share their recent words (it
forgets). The random-weight model of the workload configs hardly forgets, so
the sweep rescales it into a forgetful one: input weights of scale --wx,
recurrent weights of scale --wh, and --bz added to the update-gate bias (a
small update gate: the new state follows the new word). The decode plan
shares each frame's candidate words across the beam and sends a fraction
--focus of the extensions through the frame's spoken word, so paths that
differ in older words continue on the same recent words.

The absolute counts depend on that synthetic model and beam: only the shape
of Table 1 (how much each compression merges, and in which order) is
comparable, not its numbers.
"""
from __future__ import annotations

import argparse
import json
import sys
import time

import numpy as np

MODES = (("exact", 0, 0), ("sigdig3", 2, 3), ("sigdig2", 2, 2), ("sigdig1", 2, 1), ("sign", 1, 0))


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", default="large")
    ap.add_argument("--beam", type=int, default=512)
    ap.add_argument("--fanout", type=int, default=4)
    ap.add_argument("--frames", type=int, default=200)
    ap.add_argument("--stay", type=float, default=0.5)
    ap.add_argument("--shared", type=int, default=12,
                    help="candidate words shared by the whole beam in a frame (0: independent draws)")
    ap.add_argument("--focus", type=float, default=0.8)
    ap.add_argument("--wx", type=float, default=0.5, help="input-weight scale of the swept model")
    ap.add_argument("--wh", type=float, default=0.01, help="recurrent-weight scale of the swept model")
    ap.add_argument("--bz", type=float, default=-2.0, help="added to the update-gate bias")
    ap.add_argument("--seed", type=int, default=1)
    a = ap.parse_args(argv)
    import torch

    from . import rnnlm as R
    from .decode import DeviceDecodeLoop
    from .workload import CONFIGS, decode_plan, make_workload

    cfg = CONFIGS[a.config]
    m = cfg.model
    wl = make_workload(a.config, n_frames=1, pool_size=max(a.beam, 64))
    rng = np.random.default_rng(a.seed)
    pick = rng.choice(len(wl.pool.vec), a.beam, replace=False)
    plan = decode_plan(m.V, a.beam, a.fanout, a.frames, a.stay, cfg.zipf_s, a.seed, wl.pool.words[pick],
                       shared=a.shared, focus=a.focus)
    w = dict(wl.weights)   # the workload weights use scale 0.05
    w["W_ih"] = [(x * (a.wx / 0.05)).astype(np.float32) for x in w["W_ih"]]
    w["W_hh"] = [(x * (a.wh / 0.05)).astype(np.float32) for x in w["W_hh"]]
    b = [x.copy() for x in w["b_ih"]]
    for x in b:
        x[m.H:2 * m.H] += np.float32(a.bz)   # gate order r, z, n
    w["b_ih"] = b
    dev = torch.device("cuda:0")
    init = torch.from_numpy(np.ascontiguousarray(wl.pool.vec[pick])).to(dev)
    nq = a.beam * a.fanout
    rows, ref = [], None
    for name, qm, qk in MODES:
        sc = R.Scorer(m, w, qm, qk, max_hist=a.beam, max_query=nq,
                      cap_hist=a.beam * a.frames + 1, cap_query=nq * a.frames + 1)
        loop = DeviceDecodeLoop(sc, init)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        outs = loop.run(plan, debug=False)
        torch.cuda.synchronize()
        secs = time.perf_counter() - t0
        st = sc.stats()
        scores = torch.cat([o["scores"][:nq] for o in outs]).double().cpu().numpy()
        if ref is None:
            ref = scores
        dev_abs = np.abs(scores - ref)
        rows.append({"mode": name, "queries": st["queries"], "unique_queries": st["computed"],
                     "unique_gru_rows": st["gru_rows"], "score_hit_ratio": round(st["score_hits"] / st["queries"], 4),
                     "hist_hit_ratio": round(st["hist_hits"] / st["hists"], 4),
                     "score_dev_mean": float(dev_abs.mean()), "score_dev_max": float(dev_abs.max()),
                     "frames_per_s": round(a.frames / secs, 1)})
        sc.close()
        del loop, outs
    base = rows[0]["unique_queries"]
    print("%-8s %10s %14s %9s %12s %10s %10s %12s %12s" % (
        "mode", "queries", "unique_LMq", "vs_exact", "unique_GRU", "score_hit", "hist_hit", "|ds| mean", "|ds| max"),
        file=sys.stderr)
    for r in rows:
        r["reduction_vs_exact"] = round(1.0 - r["unique_queries"] / base, 4)
        print("%-8s %10d %14d %8.2f%% %12d %10.4f %10.4f %12.3g %12.3g" % (
            r["mode"], r["queries"], r["unique_queries"], 100 * r["reduction_vs_exact"], r["unique_gru_rows"],
            r["score_hit_ratio"], r["hist_hit_ratio"], r["score_dev_mean"], r["score_dev_max"]), file=sys.stderr)
    print(json.dumps({"config": a.config, "beam": a.beam, "fanout": a.fanout, "frames": a.frames,
                      "stay": a.stay, "shared": a.shared, "focus": a.focus, "wx": a.wx, "wh": a.wh,
                      "bz": a.bz, "seed": a.seed, "rows": rows}))


if __name__ == "__main__":
    main()
