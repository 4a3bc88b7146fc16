"""Every GRU path at the Large model's shapes, against the oracle.

A warm Large run has few new history keys per frame (Sec. 3: the history
cache absorbs the rest), so most frames run the narrow path (at most 32
rows) and the others the tiled path, whose row tiles shrink with the row
count. fp32 tiles are 16 hidden units wide, and 64 wide once the 16-unit
tiles would need more than one per CU (above 512 rows at H = 1024); bf16
tiles are 16 wide up to 256 rows, 32 wide up to 1024 and 64 wide above.
Here each path runs at E = 512, H = 1024: one fp32 layer (K = 1536), and two
bf16 layers (K = 1536, then 2048). A first frame puts some keys in the
history cache; the frame under test then has exactly M new history keys,
plus cached keys (HC_HIT), in-frame copies (H_DUP) and repeated queries of
the first frame (SCORE_HIT). It runs as a one-frame launch (whose narrow path
loads its operands before the row count arrives) and as a two-session launch
(one GRU launch over both sessions' rows). Keys, statuses and representatives
must be bit-exact; fp32 h' and scores within 1e-6 + 1e-5 |ref|; bf16 within
2e-2 of the fp32-master oracle (Sec. 2.1 GRU step, Sec. 2.2-2.3 scores)."""
import numpy as np
import pytest
import torch

from harness import ATOL, BF16_ATOL, RTOL, close, log
from oracle import HC_HIT, H_DUP, Q_SCORE_HIT, Q_SIGN, Oracle
from paper_1801_09866_amd import rnnlm as R
from paper_1801_09866_amd.workload import BF16, F32, ModelCfg

pytestmark = pytest.mark.gpu

V = 5000   # the GRU path does not depend on the vocabulary size
MODELS = {
    "fp32": ModelCfg(V=V, E=512, H=1024, L=1, wdtype=F32, maxent_log2=16, maxent_order=4),
    "bf16": ModelCfg(V=V, E=512, H=1024, L=2, wdtype=BF16, maxent_log2=16, maxent_order=4),
}
ROWS = (1, 15, 16, 17, 32, 33, 100, 256, 257)
ROWS_WIDE = {"fp32": (513, 1100), "bf16": (1025, 1600)}   # 64-unit tiles
N_WARM = 24      # keys of the first frame
N_CACHED = 8     # first-frame histories repeated in the frame under test
KEYS = ("h_hash", "h_status", "h_rep", "q_status", "q_rep")


def path_of(name, M, one):
    if M <= 16 and one:
        return "narrow_preloaded"
    if M <= 32:
        return "narrow"
    if name == "bf16":
        return "tiled64" if M > 1024 else "tiled32" if M > 256 else "tiled16"
    return "tiled64" if M > 512 else "tiled16"


def cases():
    for name in MODELS:
        for M in ROWS + ROWS_WIDE[name]:
            for sessions in (1, 2):
                # two sessions split the rows: session 0 has M - M // 3, session 1 has M // 3
                yield pytest.param(name, M, sessions,
                                   id="%s-%s-M%d-s%d" % (name, path_of(name, M, sessions == 1), M, sessions))


_W = {}


def weights(name):
    if name not in _W:
        m = MODELS[name]
        rng = np.random.default_rng(1024 + m.L)
        H, E, s = m.H, m.E, 0.05
        _W[name] = {
            "emb": (rng.standard_normal((m.V, E)) * s).astype(np.float32),
            "W_ih": [(rng.standard_normal((3 * H, E if l == 0 else H)) * s).astype(np.float32) for l in range(m.L)],
            "W_hh": [(rng.standard_normal((3 * H, H)) * s).astype(np.float32) for l in range(m.L)],
            "b_ih": [(rng.standard_normal(3 * H) * s).astype(np.float32) for l in range(m.L)],
            "U_out": (rng.standard_normal((m.V, H)) * s).astype(np.float32),
            "b_out": (rng.standard_normal(m.V) * s).astype(np.float32),
            "maxent": (rng.standard_normal(1 << m.maxent_log2) * 0.01).astype(np.float32)}
    return _W[name]


def rand_hist(rng, m, n):
    return (np.tanh(rng.standard_normal((n, m.L * m.H)) * 0.8) * 0.95).astype(np.float32)


def warm_frame(rng, m):
    vec = rand_hist(rng, m, N_WARM)
    words = rng.integers(1, m.V, (N_WARM, 3)).astype(np.int32)
    qh = np.repeat(np.arange(N_WARM, dtype=np.int32), 3)
    qt = rng.integers(1, m.V, len(qh)).astype(np.int32)
    return vec, words, qh, qt


def frame_under_test(rng, m, warm, M):
    """M new keys (every fifth of them also copied later in the frame), then
    N_CACHED histories of the warm frame; queries: two per history plus
    repeats of warm-frame queries on the cached histories."""
    wv, ww, wqh, wqt = warm
    new = rand_hist(rng, m, M)
    new_w = rng.integers(1, m.V, (M, 3)).astype(np.int32)
    dup = np.arange(0, M, 5)
    cached = rng.choice(N_WARM, N_CACHED, replace=False)
    vec = np.concatenate([new, new[dup], wv[cached]])
    words = np.concatenate([new_w, new_w[dup], ww[cached]])
    n_h = len(vec)
    qh = np.repeat(np.arange(n_h, dtype=np.int32), 2)
    qt = rng.integers(1, m.V, len(qh)).astype(np.int32)
    # a warm-frame query (same history key and target) again: a score hit
    base = M + len(dup)
    rep_q = np.array([np.nonzero(wqh == c)[0][0] for c in cached])
    qh = np.concatenate([qh, base + np.arange(N_CACHED, dtype=np.int32)])
    qt = np.concatenate([qt, wqt[rep_q]])
    perm = rng.permutation(len(qh))
    return vec, words, qh[perm].astype(np.int32), qt[perm].astype(np.int32)


def to_dev(fr):
    return tuple(torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in fr)


def compare(out, res, fr, bf16, tag):
    vec, words, qh, qt = fr
    n_h, n_q = len(vec), len(qh)
    got = {k: out[k][:n_q if k.startswith("q_") else n_h].cpu().numpy() for k in KEYS}
    assert np.array_equal(got["h_hash"].view(np.uint64), res.h_hash), tag + ": history key hashes"
    for k in KEYS[1:]:
        assert np.array_equal(got[k], getattr(res, k)), tag + ": " + k
    atol, rtol = (BF16_ATOL, 0.0) if bf16 else (ATOL, RTOL)
    ok, err = close(out["hnew"][:n_h].cpu().numpy(), res.hnew, atol, rtol)
    assert ok, "%s: GRU outputs differ by %.3g" % (tag, err)
    ok, err = close(out["scores"][:n_q].cpu().numpy(), res.scores, atol, rtol)
    assert ok, "%s: scores differ by %.3g" % (tag, err)


@pytest.mark.parametrize("name,M,sessions", list(cases()))
def test_gru_path_at_large_dims(name, M, sessions):
    m = MODELS[name]
    w = weights(name)
    rng = np.random.default_rng(M * 7 + sessions)
    split = [M] if sessions == 1 else [M - M // 3, M // 3]
    kw = dict(max_hist=2048, max_query=4096, cap_hist=1 << 12, cap_query=1 << 14)
    g = R.Scorer(m, w, Q_SIGN, 0, sessions=sessions, **kw)
    orc = [Oracle(m.V, m.E, m.H, m.L, m.maxent_log2, m.maxent_order, w, Q_SIGN, 0,
                  cap_hist=kw["cap_hist"], cap_query=kw["cap_query"], seed=R.DEFAULT_SEED)
           for _ in range(sessions)]
    warm = [warm_frame(rng, m) for _ in range(sessions)]
    log("  %s M=%d sessions=%d: warm frame" % (name, M, sessions))
    if sessions == 1:
        outs = [g.score_frame(*to_dev(warm[0]))]
    else:
        outs = g.score_frames([to_dev(f) for f in warm])
    for k in range(sessions):
        res = orc[k].score_frame(*warm[k])
        torch.cuda.synchronize()
        assert res.gru_rows == N_WARM
        compare(outs[k], res, warm[k], m.wdtype == BF16, "%s warm s%d" % (name, k))
    frames = [frame_under_test(rng, m, warm[k], split[k]) for k in range(sessions)]
    log("  %s M=%d sessions=%d: frame under test, path %s" % (name, M, sessions, path_of(name, M, sessions == 1)))
    if sessions == 1:
        outs = [g.score_frame(*to_dev(frames[0]))]
    else:
        outs = g.score_frames([to_dev(f) for f in frames])
    rows = 0
    for k in range(sessions):
        res = orc[k].score_frame(*frames[k])
        torch.cuda.synchronize()
        assert res.gru_rows == split[k]
        assert (res.h_status == HC_HIT).sum() == N_CACHED
        assert (res.h_status == H_DUP).sum() == len(np.arange(0, split[k], 5))
        assert (res.q_status == Q_SCORE_HIT).sum() >= N_CACHED
        compare(outs[k], res, frames[k], m.wdtype == BF16, "%s M=%d s%d" % (name, M, k))
        rows += res.gru_rows
    assert rows == M
    st = g.stats()
    assert st["gru_rows"] == M + N_WARM * sessions and st["device_error"] == 0
