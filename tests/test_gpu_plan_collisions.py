"""White-box cases for the frame planner's rare paths. The planner finds
equal keys with a race over hash tables whose slots hold a fingerprint (the
key hash's high bits) and an index; two distinct keys that reach the same slot
of the first table with the same fingerprint settle on one index, and the
exact key check then sends the other key to the exact scan. These frames are
built so that this happens, by searching on the CPU for such key pairs with
the planner's placement rule (first table of 64 slots for frames of at most
16 keys, addressed by the top 6 bits of the hash's low word; fingerprint =
the high word above the 11 (histories) or 13 (queries) index bits).
Statuses and representatives must still match the oracle bit for bit.

The last two cases build linear-probe chains longer than the 16 records a
cache probe reads per round trip, in the history-cache index and in the
LM-query cache, from the placement hashes the library uses."""
import numpy as np
import pytest
import torch

from harness import ATOL, RTOL, close, log
from oracle import HC_HIT, Q_EXACT, Q_SCORE_HIT, Oracle
from oracle.rnnlm_oracle import code_words, hist_key_hash, mix64, quantize
from paper_1801_09866_amd import rnnlm as R
from paper_1801_09866_amd.workload import F32, ModelCfg

pytestmark = pytest.mark.gpu

M = ModelCfg(V=60_000, E=64, H=64, L=1, wdtype=F32, maxent_log2=12, maxent_order=4)
PHI = np.uint64(0x9E3779B97F4A7C15)
M32 = np.uint64(0xFFFFFFFF)


def weights(rng, scale=0.08):
    H, E = M.H, M.E
    return {"emb": (rng.standard_normal((M.V, E)) * scale).astype(np.float32),
            "W_ih": [(rng.standard_normal((3 * H, E)) * scale).astype(np.float32)],
            "W_hh": [(rng.standard_normal((3 * H, H)) * scale).astype(np.float32)],
            "b_ih": [(rng.standard_normal(3 * H) * scale).astype(np.float32)],
            "U_out": (rng.standard_normal((M.V, H)) * scale).astype(np.float32),
            "b_out": (rng.standard_normal(M.V) * scale).astype(np.float32),
            "maxent": (rng.standard_normal(1 << M.maxent_log2) * 0.01).astype(np.float32)}


def hist_hashes(vec, w1):
    """Key hashes of history vector `vec` with each input word in `w1`."""
    words = code_words(quantize(vec[None, :], Q_EXACT), Q_EXACT)
    return hist_key_hash(np.repeat(words, len(w1), axis=0), w1, R.DEFAULT_SEED)


def query_place_hash(hh, w2, w3, t):
    """The planner's in-frame placement hash of a query key (history hash
    folded to 32 bits, context words, target)."""
    with np.errstate(over="ignore"):
        x = ((np.uint64(hh) << np.uint64(32)) | ((t.astype(np.uint64) + np.uint64(1)) & M32)) \
            + (np.uint64(w2 + 2) & M32) * PHI + (np.uint64(w3 + 2) & M32) * np.uint64(0xD6E8FEB86659FD93)
    return mix64(x)


def slot_key(h, index_bits):
    """(fingerprint, first-table slot) of 64-bit hashes, as one integer."""
    h = np.asarray(h, np.uint64)
    fp = (h >> np.uint64(32 + index_bits)).astype(np.int64)
    pos = ((h & M32) >> np.uint64(26)).astype(np.int64)
    return (fp << 6) | pos


def first_pair(keys_a, keys_b, same):
    seen = {}
    for i, k in enumerate(keys_a.tolist()):
        seen.setdefault(k, i)
    for j, k in enumerate(keys_b.tolist()):
        i = seen.get(k)
        if i is not None and not (same and i == j):
            return i, j
    return None


def run_frame(vec, words, qh, qt, rng_w):
    w = weights(rng_w)
    g = R.Scorer(M, w, Q_EXACT, 0, max_hist=16, max_query=16)
    o = Oracle(M.V, M.E, M.H, M.L, M.maxent_log2, M.maxent_order, w, Q_EXACT, 0,
               cap_hist=1 << 12, cap_query=1 << 14, seed=R.DEFAULT_SEED)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    for t in range(2):   # second pass: everything is a cache hit
        out = g.score_frame(d(vec), d(words), d(qh), d(qt))
        res = o.score_frame(vec, words, qh, qt)
        torch.cuda.synchronize()
        n, nq = len(vec), len(qh)
        for key, want in (("h_status", res.h_status), ("h_rep", res.h_rep), ("q_status", res.q_status),
                          ("q_rep", res.q_rep)):
            m = n if key.startswith("h") else nq
            assert np.array_equal(out[key][:m].cpu().numpy(), want), (t, key)
        assert close(out["scores"][:nq].cpu().numpy(), res.scores, ATOL, RTOL)[0], t
    assert g.stats()["device_error"] == 0


def test_two_history_keys_that_share_slot_and_fingerprint():
    rng = np.random.default_rng(11)
    vec = (np.tanh(rng.standard_normal(M.H)) * 0.9).astype(np.float32)
    w1 = np.arange(M.V, dtype=np.int64)
    keys = slot_key(hist_hashes(vec, w1), 11)
    pair = first_pair(keys, keys, same=True)
    assert pair is not None, "no colliding pair in the search range"
    a, b = pair
    log("  history keys w1 =", a, b, "share slot and fingerprint")
    vecs = np.stack([vec, vec])
    words = np.array([[a, 5, 6], [b, 7, 8]], np.int32)
    run_frame(vecs, words, np.array([0, 1, 1, 0], np.int32), np.array([3, 4, 3, 3], np.int32),
              np.random.default_rng(12))


def test_two_query_keys_that_share_slot_and_fingerprint():
    rng = np.random.default_rng(21)
    vecs = (np.tanh(rng.standard_normal((2, M.H))) * 0.9).astype(np.float32)
    words = np.array([[10, 11, 12], [20, 21, 22]], np.int32)
    hh = []
    for x in range(2):
        h = int(hist_hashes(vecs[x], np.array([words[x, 0]], np.int64))[0])
        hh.append((h ^ (h >> 32)) & 0xFFFFFFFF)
    t = np.arange(M.V, dtype=np.int64)
    ka = slot_key(query_place_hash(hh[0], int(words[0, 1]), int(words[0, 2]), t), 13)
    kb = slot_key(query_place_hash(hh[1], int(words[1, 1]), int(words[1, 2]), t), 13)
    pair = first_pair(ka, kb, same=False)
    assert pair is not None, "no colliding pair in the search range"
    ta, tb = pair
    log("  query keys (0, %d) and (1, %d) share slot and fingerprint" % (ta, tb))
    run_frame(vecs, words, np.array([0, 1], np.int32), np.array([ta, tb], np.int32), np.random.default_rng(22))


def test_history_cache_chain_longer_than_a_probe_window():
    """24 distinct history keys whose hashes share a position of a 64-slot
    history-cache index (capacity 32): their records form one linear-probe
    chain, and the keys at its end are found only in the second window of
    16 records. The repeat frame must hit on every key."""
    rng = np.random.default_rng(31)
    vec = (np.tanh(rng.standard_normal(M.H)) * 0.9).astype(np.float32)
    w1 = np.arange(1, M.V, dtype=np.int64)
    pos = (hist_hashes(vec, w1) & np.uint64(63)).astype(np.int64)
    target = np.bincount(pos).argmax()
    picks = w1[pos == target][:24]
    assert len(picks) == 24
    log("  24 keys at index position", int(target))
    n = len(picks)
    vecs = np.repeat(vec[None, :], n, axis=0)
    words = np.stack([picks, rng.integers(0, M.V, n), rng.integers(0, M.V, n)], axis=1).astype(np.int32)
    qh = np.arange(n, dtype=np.int32)
    qt = rng.integers(0, M.V, n).astype(np.int32)
    w = weights(np.random.default_rng(32))
    g = R.Scorer(M, w, Q_EXACT, 0, max_hist=32, max_query=64, cap_hist=32, cap_query=1 << 10)
    o = Oracle(M.V, M.E, M.H, M.L, M.maxent_log2, M.maxent_order, w, Q_EXACT, 0,
               cap_hist=32, cap_query=1 << 10, seed=R.DEFAULT_SEED)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    for t in range(2):
        out = g.score_frame(d(vecs), d(words), d(qh), d(qt))
        res = o.score_frame(vecs, words, qh, qt)
        torch.cuda.synchronize()
        for key, want in (("h_status", res.h_status), ("h_rep", res.h_rep), ("q_status", res.q_status)):
            assert np.array_equal(out[key][:n].cpu().numpy(), want), (t, key)
        assert close(out["scores"][:n].cpu().numpy(), res.scores, ATOL, RTOL)[0], t
    assert (res.h_status == HC_HIT).all()   # every key of the repeat frame is a history-cache hit
    assert g.stats()["device_error"] == 0


def lm_cache_hash(hs, w2, w3, t):
    """The LM-query cache's placement hash of a key (history-cache slot,
    context words, target), as the library computes it."""
    m32 = lambda x: np.asarray(x, np.int64).astype(np.uint64) & M32
    g = mix64(np.uint64(hs) + PHI)
    g = mix64(g ^ m32(w2 + 2))
    g = mix64(g ^ m32(w3 + 2))
    return mix64(g ^ m32(np.asarray(t, np.int64) + 1))


def test_lm_cache_chain_longer_than_a_probe_window():
    """24 queries of one history whose LM-query cache keys share a position
    of a 64-slot table (capacity 32): admitted after the first frame, they
    form one linear-probe chain, and the repeat frame finds the last of them
    only in the second window of 16 records."""
    rng = np.random.default_rng(41)
    vec = (np.tanh(rng.standard_normal((1, M.H))) * 0.9).astype(np.float32)
    words = np.array([[11, 12, 13]], np.int32)
    t = np.arange(M.V, dtype=np.int64)
    pos = (lm_cache_hash(0, 12, 13, t) & np.uint64(63)).astype(np.int64)
    target = np.bincount(pos).argmax()
    qt = t[pos == target][:24].astype(np.int32)
    assert len(qt) == 24
    log("  24 query keys at LM-cache position", int(target))
    qh = np.zeros(len(qt), np.int32)
    w = weights(np.random.default_rng(42))
    g = R.Scorer(M, w, Q_EXACT, 0, max_hist=4, max_query=64, cap_hist=16, cap_query=32)
    o = Oracle(M.V, M.E, M.H, M.L, M.maxent_log2, M.maxent_order, w, Q_EXACT, 0,
               cap_hist=16, cap_query=32, seed=R.DEFAULT_SEED)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    for k in range(2):
        out = g.score_frame(d(vec), d(words), d(qh), d(qt))
        res = o.score_frame(vec, words, qh, qt)
        torch.cuda.synchronize()
        assert np.array_equal(out["q_status"][:len(qt)].cpu().numpy(), res.q_status), k
        got = out["scores"][:len(qt)].cpu().numpy()
        assert close(got, res.scores, ATOL, RTOL)[0], k
        if k == 0:
            first = got.copy()
    assert (res.q_status == Q_SCORE_HIT).all()
    assert np.array_equal(got.view(np.uint32), first.view(np.uint32))   # hits return the stored bits
    assert g.stats()["device_error"] == 0
