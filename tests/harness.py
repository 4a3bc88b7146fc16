"""Runs the HIP library and the CPU oracle side by side on the same seeded
frames and compares every output (tests only)."""
from __future__ import annotations

import dataclasses
import sys

import numpy as np
import torch

from oracle import Oracle
from paper_1801_09866_amd import rnnlm as R
from paper_1801_09866_amd.workload import make_workload

# fp32 scores and GRU outputs: |gpu - oracle| <= ATOL + RTOL * |oracle|
ATOL, RTOL = 1e-6, 1e-5
# bf16 weights (fp32 accumulation) against the fp32-master oracle
BF16_ATOL = 2e-2


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def close(got, want, atol, rtol):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    err = np.abs(got - want)
    ok = err <= atol + rtol * np.abs(want)
    return bool(ok.all()), float(err.max(initial=0.0))


@dataclasses.dataclass
class Pair:
    wl: object
    oracle: Oracle
    scorer: R.Scorer
    pool_dev: torch.Tensor
    atol: float
    rtol: float


def make_pair(name, qmode, qdigits, n_frames, pool_size=None, model=None, cap_hist=None,
              cap_query=None, weights=None):
    wl = make_workload(name, n_frames=n_frames, pool_size=pool_size, model=model,
                       with_weights=weights is None)
    if weights is not None:
        wl.weights = weights
    m = wl.cfg.model
    ch = wl.cfg.cap_hist if cap_hist is None else cap_hist
    cq = wl.cfg.cap_query if cap_query is None else cap_query
    oracle = Oracle(m.V, m.E, m.H, m.L, m.maxent_log2, m.maxent_order, wl.weights, qmode,
                    qdigits, cap_hist=ch, cap_query=cq, seed=R.DEFAULT_SEED)
    scorer = R.Scorer(m, wl.weights, qmode, qdigits, max_hist=wl.cfg.max_hist,
                      max_query=max(wl.cfg.queries, 1), cap_hist=ch, cap_query=cq)
    pool_dev = torch.from_numpy(wl.pool.vec).to("cuda")
    bf16 = m.wdtype == R.BF16
    return Pair(wl, oracle, scorer, pool_dev, BF16_ATOL if bf16 else ATOL, 0.0 if bf16 else RTOL)


def device_frame(p: Pair, fr):
    idx = torch.from_numpy(fr.pool_idx).to("cuda")
    hv = p.pool_dev.index_select(0, idx).contiguous()
    hw = torch.from_numpy(np.ascontiguousarray(fr.hist_words, np.int32)).to("cuda")
    qh = torch.from_numpy(fr.q_hist).to("cuda")
    qt = torch.from_numpy(fr.q_tgt).to("cuda")
    return hv, hw, qh, qt


def compare_frame(p: Pair, fi, fr, out, res, check_hnew=True):
    n_h, n_q = fr.n_hist, fr.n_query
    tag = "%s frame %d" % (p.wl.cfg.name, fi)
    g_hash = out["h_hash"][:n_h].cpu().numpy().view(np.uint64)
    assert np.array_equal(g_hash, res.h_hash), tag + ": history key hashes differ"
    assert np.array_equal(out["h_rep"][:n_h].cpu().numpy(), res.h_rep), tag + ": h_rep differs"
    assert np.array_equal(out["h_status"][:n_h].cpu().numpy(), res.h_status), tag + ": h_status differs"
    if n_q:
        assert np.array_equal(out["q_rep"][:n_q].cpu().numpy(), res.q_rep), tag + ": q_rep differs"
        gs = out["q_status"][:n_q].cpu().numpy()
        assert np.array_equal(gs, res.q_status), tag + ": q_status differs"
        ok, err = close(out["scores"][:n_q].cpu().numpy(), res.scores, p.atol, p.rtol)
        assert ok, "%s: scores differ (max abs err %.3g)" % (tag, err)
    if check_hnew:
        ok, err = close(out["hnew"][:n_h].cpu().numpy(), res.hnew,
                        p.atol if p.rtol else 2e-2, p.rtol)
        assert ok, "%s: GRU outputs differ (max abs err %.3g)" % (tag, err)


def run_frames(p: Pair, frames=None, check_hnew=True, log_every=10):
    frames = p.wl.frames if frames is None else frames
    tot = dict(gru_rows=0, hist_inserted=0, hist_rejected=0, score_inserted=0, score_rejected=0)
    for fi, fr in enumerate(frames):
        if fi % log_every == 0:
            log("  [%s] frame %d/%d" % (p.wl.cfg.name, fi, len(frames)))
        hv, hw, qh, qt = device_frame(p, fr)
        out = p.scorer.score_frame(hv, hw, qh, qt)
        res = p.oracle.score_frame(p.wl.pool.vec[fr.pool_idx], fr.hist_words, fr.q_hist, fr.q_tgt)
        torch.cuda.synchronize()
        compare_frame(p, fi, fr, out, res, check_hnew)
        for k in tot:
            tot[k] += getattr(res, k)
    st = p.scorer.stats()
    for k, v in tot.items():
        assert st[k] == v, "stat %s: gpu %d oracle %d" % (k, st[k], v)
    assert st["frames"] == len(frames)
    assert st["hist_cache_size"] == len(p.oracle.hist_cache)
    assert st["score_cache_size"] == len(p.oracle.score_cache)
    return st
