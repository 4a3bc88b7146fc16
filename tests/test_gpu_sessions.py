"""Independent decode sessions scored in one set of launches: each session's
keys, statuses and representatives must be bit-identical to a context of its
own fed the same frames, and its scores and h' equal to the fp32 tolerance
(the GRU rows of all sessions share one launch, whose path, and so its
summation order, follows the total row count), whatever the mix of frame
sizes, with a session missing a frame, and with caches small enough that
admission runs in order; each session must also match the oracle."""
import numpy as np
import pytest
import torch

from harness import ATOL, BF16_ATOL, RTOL, close, log
from oracle import Q_SIGDIG, Q_SIGN, Oracle
from paper_1801_09866_amd import rnnlm as R
from paper_1801_09866_amd.workload import BF16, F32, ModelCfg

pytestmark = pytest.mark.gpu

M = ModelCfg(V=4000, E=64, H=128, L=2, wdtype=F32, maxent_log2=12, maxent_order=4)
KEYS = ("scores", "hnew", "q_status", "q_rep", "h_status", "h_rep", "h_hash")


def weights(m, rng, scale=0.08):
    H, E = m.H, m.E
    return {"emb": (rng.standard_normal((m.V, E)) * scale).astype(np.float32),
            "W_ih": [(rng.standard_normal((3 * H, E if l == 0 else H)) * scale).astype(np.float32) for l in range(m.L)],
            "W_hh": [(rng.standard_normal((3 * H, H)) * scale).astype(np.float32) for l in range(m.L)],
            "b_ih": [(rng.standard_normal(3 * H) * scale).astype(np.float32) for l in range(m.L)],
            "U_out": (rng.standard_normal((m.V, H)) * scale).astype(np.float32),
            "b_out": (rng.standard_normal(m.V) * scale).astype(np.float32),
            "maxent": (rng.standard_normal(1 << m.maxent_log2) * 0.01).astype(np.float32)}


def frame(rng, pool, n_h, n_q):
    idx = rng.integers(0, len(pool), n_h)
    vec = pool[idx]
    words = rng.integers(0, M.V, (n_h, 3)).astype(np.int32)
    words[:, 0] = (idx * 7) % M.V   # repeated pool rows repeat their key
    qh = rng.integers(0, n_h, n_q).astype(np.int32)
    qt = rng.integers(0, M.V, n_q).astype(np.int32)
    return vec, words, qh, qt


@pytest.mark.parametrize("sizes,caps,qm", [
    ((6, 9, 12), (1 << 12, 1 << 14), (Q_SIGN, 0)),        # rows of all sessions <= 32: narrow path
    ((40, 25, 60), (1 << 12, 1 << 14), (Q_SIGN, 0)),      # medium path
    ((150, 120, 200), (1 << 12, 1 << 14), (Q_SIGN, 0)),   # 64 x 32 tiles
    ((30, 20, 50), (40, 90), (Q_SIGN, 0)),                # small caches: in-order admission per session
    ((33, 7, 52), (1 << 12, 1 << 14), (Q_SIGDIG, 2)),     # one key block per history
])
def test_sessions_match_independent_contexts_and_the_oracle(sizes, caps, qm):
    rng = np.random.default_rng(sum(sizes))
    w = weights(M, rng)
    S = len(sizes)
    pools = [(np.tanh(rng.standard_normal((3 * n, M.L * M.H))) * 0.9).astype(np.float32) for n in sizes]
    kw = dict(max_hist=256, max_query=1024, cap_hist=caps[0], cap_query=caps[1])
    multi = R.Scorer(M, w, qm[0], qm[1], sessions=S, **kw)
    solo = [R.Scorer(M, w, qm[0], qm[1], **kw) for _ in range(S)]
    orc = [Oracle(M.V, M.E, M.H, M.L, M.maxent_log2, M.maxent_order, w, qm[0], qm[1],
                  cap_hist=caps[0], cap_query=caps[1], seed=R.DEFAULT_SEED) for _ in range(S)]
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    for t in range(4):
        frs = [frame(rng, pools[k], sizes[k], 3 * sizes[k]) for k in range(S)]
        present = [not (t == 2 and k == 1) for k in range(S)]   # session 1 has no frame at t = 2
        log("  block", t, "sizes", sizes, "present", present)
        outs = multi.score_frames([tuple(d(a) for a in fr) if present[k] else None for k, fr in enumerate(frs)])
        for k in range(S):
            if not present[k]:
                continue
            vec, words, qh, qt = frs[k]
            o1 = solo[k].score_frame(d(vec), d(words), d(qh), d(qt))
            res = orc[k].score_frame(vec, words, qh, qt)
            torch.cuda.synchronize()
            n_h, n_q = len(vec), len(qh)
            for key in KEYS:
                n = n_q if key in ("scores", "q_status", "q_rep") else n_h
                a, b = outs[k][key][:n], o1[key][:n]
                if key in ("scores", "hnew"):
                    assert close(a.cpu().numpy(), b.cpu().numpy(), ATOL, RTOL)[0], (t, k, key)
                else:
                    assert torch.equal(a, b), (t, k, key)
            assert np.array_equal(outs[k]["h_status"][:n_h].cpu().numpy(), res.h_status), (t, k)
            assert np.array_equal(outs[k]["q_status"][:n_q].cpu().numpy(), res.q_status), (t, k)
            assert np.array_equal(outs[k]["q_rep"][:n_q].cpu().numpy(), res.q_rep), (t, k)
            assert close(outs[k]["scores"][:n_q].cpu().numpy(), res.scores, ATOL, RTOL)[0], (t, k)
            assert close(outs[k]["hnew"][:n_h].cpu().numpy(), res.hnew, ATOL, RTOL)[0], (t, k)
    total = {key: 0 for key in ("frames", "queries", "computed", "gru_rows", "hist_cache_size")}
    for k in range(S):
        a, b = multi.session_stats(k), solo[k].stats()
        assert a == b, (k, a, b)
        for key in total:
            total[key] += a[key]
    agg = multi.stats()
    for key in total:
        assert agg[key] == total[key]
    if caps[1] < 1000:
        assert agg["score_rejected"] > 0 and agg["hist_rejected"] > 0


def test_a_device_error_in_one_session_is_sticky_for_the_context():
    rng = np.random.default_rng(7)
    g = R.Scorer(M, weights(M, rng), Q_SIGN, 0, sessions=2, max_hist=32, max_query=64)
    pool = np.zeros((8, M.L * M.H), np.float32)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    good = tuple(d(a) for a in frame(rng, pool, 8, 16))
    vec, words, qh, qt = frame(rng, pool, 8, 16)
    words[2, 1] = M.V + 1
    g.score_frames([good, tuple(d(a) for a in (vec, words, qh, qt))])
    assert g.session_stats(0, check=False)["device_error"] == 0
    with pytest.raises(R.RnnlmError):
        g.stats()
    with pytest.raises(R.RnnlmError):
        g.score_frames([good])
    g.reset()
    g.score_frames([good, good])
    assert g.stats()["device_error"] == 0


@pytest.mark.parametrize("wd", [F32, BF16], ids=["fp32", "bf16"])
def test_eight_sessions_of_maximal_frames(wd):
    """The largest launch the API allows: 8 sessions, each frame at the
    planner's maxima (2048 histories, 8192 queries), with uniform targets and
    a second block that repeats half of each session's histories and many of
    its queries (cache hits). Every session must equal a context of its own,
    and one session the oracle. At H = 128 the 8-session launches run the
    64-unit tiles (fp32: both blocks, 16384 and 8192 GRU rows; bf16: the
    first block) and the 32-unit bf16 tiles (the second block), while a
    context of its own runs the 16-unit tiles on at most 2048 rows; bf16
    results are compared at the bf16 tolerance, since the tiles' summation
    orders differ."""
    m = ModelCfg(V=M.V, E=M.E, H=M.H, L=M.L, wdtype=wd, maxent_log2=M.maxent_log2, maxent_order=M.maxent_order)
    tol = (BF16_ATOL, 0.0) if wd == BF16 else (ATOL, RTOL)
    rng = np.random.default_rng(88)
    w = weights(m, rng)
    S, n_h, n_q = 8, 2048, 8192
    caps = (1 << 14, 1 << 16)
    kw = dict(max_hist=n_h, max_query=n_q, cap_hist=caps[0], cap_query=caps[1])
    multi = R.Scorer(m, w, Q_SIGN, 0, sessions=S, **kw)
    solo = R.Scorer(m, w, Q_SIGN, 0, **kw)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    blocks = []
    for t in range(2):
        frs = []
        for k in range(S):
            vec = (np.tanh(rng.standard_normal((n_h, m.L * m.H))) * 0.9).astype(np.float32)
            words = rng.integers(0, m.V, (n_h, 3)).astype(np.int32)
            qh = rng.integers(0, n_h, n_q).astype(np.int32)
            qt = rng.integers(0, m.V, n_q).astype(np.int32)
            if t == 1:   # the previous frame's first half of histories, and their queries, again
                pv, pw, pqh, pqt = blocks[0][k]
                vec[: n_h // 2], words[: n_h // 2] = pv[: n_h // 2], pw[: n_h // 2]
                sel = np.nonzero(pqh < n_h // 2)[0][: n_q // 2]
                qh[: len(sel)], qt[: len(sel)] = pqh[sel], pqt[sel]
            frs.append((vec, words, qh, qt))
        blocks.append(frs)
        log("  block", t, "of", S, "maximal frames")
        outs = multi.score_frames([tuple(d(a) for a in fr) for fr in frs])
        for k in range(S):
            solo.reset()
            for u in range(t + 1):
                o1 = solo.score_frame(*(d(a) for a in blocks[u][k]))
            torch.cuda.synchronize()
            for key in KEYS:
                a, b = outs[k][key], o1[key]
                if key in ("scores", "hnew"):
                    assert close(a.cpu().numpy(), b.cpu().numpy(), *tol)[0], (t, k, key)
                else:
                    assert torch.equal(a, b), (t, k, key)
            if t == 1:
                assert (outs[k]["q_status"] == R.Q_SCORE_HIT).sum().item() > n_q // 4, k
    assert multi.stats()["device_error"] == 0
    o = Oracle(m.V, m.E, m.H, m.L, m.maxent_log2, m.maxent_order, w, Q_SIGN, 0,
               cap_hist=caps[0], cap_query=caps[1], seed=R.DEFAULT_SEED)
    o.score_frame(*blocks[0][3])
    res = o.score_frame(*blocks[1][3])
    for key, want in (("q_status", res.q_status), ("q_rep", res.q_rep), ("h_status", res.h_status),
                      ("h_rep", res.h_rep)):
        assert np.array_equal(outs[3][key].cpu().numpy(), want), key
    assert close(outs[3]["scores"].cpu().numpy(), res.scores, *tol)[0]
    assert close(outs[3]["hnew"].cpu().numpy(), res.hnew, *tol)[0]
