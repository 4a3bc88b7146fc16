"""Pins of the oracle's frame semantics: keys, de-duplication and the caches.

Sec. 2.4 (LM-query cache: same history and next word) and Sec. 3 (history
cache: key = GRU input pair, value = GRU output; quantised histories) on
hand-built frames whose outcome is known without running the oracle:
merges below the quantisation grid, splits on one flipped sign, repeat
frames that must hit both caches with bit-identical scores, admission order
under a tiny capacity, and scores that reduce to closed forms.
"""
import numpy as np
import pytest

from oracle import (H_DUP, H_REP, HC_HIT, Q_COMPUTED, Q_DUP, Q_EXACT, Q_SCORE_HIT,
                    Q_SIGDIG, Q_SIGN, Oracle, gru_step, maxent_index)

V, E, H = 50, 8, 64


def weights(rng, L=1, zero_out=False, lam=None, me_log2=10):
    w = {
        "emb": (rng.standard_normal((V, E)) * 0.3).astype(np.float32),
        "W_ih": [(rng.standard_normal((3 * H, E if l == 0 else H)) * 0.2).astype(np.float32) for l in range(L)],
        "W_hh": [(rng.standard_normal((3 * H, H)) * 0.2).astype(np.float32) for l in range(L)],
        "b_ih": [(rng.standard_normal(3 * H) * 0.1).astype(np.float32) for l in range(L)],
        "U_out": (rng.standard_normal((V, H)) * 0.1).astype(np.float32),
        "b_out": (rng.standard_normal(V) * 0.1).astype(np.float32),
        "maxent": (rng.standard_normal(1 << me_log2) * 0.01).astype(np.float32),
    }
    if zero_out:
        w["U_out"][:] = 0
        w["b_out"][:] = 0
    if lam is not None:
        w["maxent"] = lam
    return w


def make(w, qmode, k=0, L=1, order=3, me_log2=10, **kw):
    return Oracle(V, E, H, L, me_log2, order, w, qmode, k, **kw)


def base_hist(rng, n):
    return (np.tanh(rng.standard_normal((n, H))) * 0.9).astype(np.float32)


def test_sign_merge_and_split():
    rng = np.random.default_rng(0)
    o = make(weights(rng), Q_SIGN)
    h = base_hist(rng, 1)[0]
    same_signs = (h * 0.5).astype(np.float32)          # different values, same signs
    flipped = h.copy()
    flipped[7] = -flipped[7]                             # one sign differs
    vec = np.stack([h, same_signs, flipped, h])
    words = np.array([[3, 2, 1], [3, 9, 9], [3, 2, 1], [4, 2, 1]], np.int32)
    r = o.score_frame(vec, words, np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert list(r.h_rep) == [0, 0, 2, 3]
    assert list(r.h_status) == [H_REP, H_DUP, H_REP, H_REP]
    assert r.gru_rows == 3
    # the merged history uses its representative's own full-precision vector
    emb = np.asarray(o.w["emb"], np.float64)
    want0 = gru_step(emb[[3]], vec[[0]], o.W_ih[0], o.W_hh[0], o.b_ih[0])[0]
    np.testing.assert_allclose(r.hnew[0], want0, rtol=1e-13, atol=1e-15)
    assert np.array_equal(r.hnew[1], r.hnew[0])
    assert r.h_hash[0] == r.h_hash[1] and r.h_hash[0] != r.h_hash[2] != r.h_hash[3]


def test_sigdig_merges_below_grid_and_splits_across_it():
    rng = np.random.default_rng(1)
    o = make(weights(rng), Q_SIGDIG, 2)
    h = np.full(H, 0.4321, np.float32)
    close = np.full(H, 0.4349, np.float32)              # both round to 0.43
    across = h.copy()
    across[5] = np.float32(0.4351)                       # rounds to 0.44
    vec = np.stack([h, close, across])
    words = np.array([[1, 0, 0]] * 3, np.int32)
    r = o.score_frame(vec, words, np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert list(r.h_rep) == [0, 0, 2]
    assert list(r.h_status) == [H_REP, H_DUP, H_REP]


def test_exact_mode_distinguishes_one_ulp():
    rng = np.random.default_rng(2)
    o = make(weights(rng), Q_EXACT)
    h = base_hist(rng, 1)[0]
    g = h.copy()
    g[0] = np.nextafter(g[0], np.float32(2))
    z = np.zeros(H, np.float32)
    nz = z.copy()
    nz[:] = -0.0
    vec = np.stack([h, g, h, z, nz])
    r = o.score_frame(vec, np.ones((5, 3), np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert list(r.h_rep) == [0, 1, 0, 3, 3]


def _frame(rng, n_h=6, n_q=20):
    vec = base_hist(rng, n_h)
    words = rng.integers(1, V, size=(n_h, 3)).astype(np.int32)
    q_hist = rng.integers(0, n_h, n_q).astype(np.int32)
    q_tgt = rng.integers(1, V, n_q).astype(np.int32)
    q_hist[-1], q_tgt[-1] = q_hist[0], q_tgt[0]          # an in-frame duplicate query
    return vec, words, q_hist, q_tgt


def test_repeat_frame_hits_both_caches_bit_identically():
    rng = np.random.default_rng(3)
    o = make(weights(rng), Q_SIGN)
    f = _frame(rng)
    r1 = o.score_frame(*f)
    assert set(r1.h_status) <= {H_REP, H_DUP}
    assert r1.q_status[-1] == Q_DUP and r1.q_rep[-1] == 0
    assert r1.scores[-1] == r1.scores[0]
    r2 = o.score_frame(*f)
    assert np.all(r2.h_status == HC_HIT)
    assert np.all(r2.q_status == Q_SCORE_HIT)
    assert r2.gru_rows == 0
    assert np.array_equal(r1.scores.view(np.uint32), r2.scores.view(np.uint32))
    np.testing.assert_array_equal(r1.hnew, r2.hnew)
    o.reset()
    r3 = o.score_frame(*f)
    assert np.array_equal(r3.h_status, r1.h_status) and np.array_equal(r3.q_status, r1.q_status)


def test_history_admission_order_under_tiny_capacity():
    rng = np.random.default_rng(4)
    o = make(weights(rng), Q_SIGN, cap_hist=2, cap_query=100)
    vec = base_hist(rng, 4)
    words = np.array([[1, 0, 0], [2, 0, 0], [3, 0, 0], [4, 0, 0]], np.int32)
    q_hist = np.arange(4, dtype=np.int32)
    q_tgt = np.full(4, 7, np.int32)
    r1 = o.score_frame(vec, words, q_hist, q_tgt)
    assert (r1.hist_inserted, r1.hist_rejected) == (2, 2)
    # scores are only cached under a cached history key
    assert (r1.score_inserted, r1.score_rejected) == (2, 0)
    r2 = o.score_frame(vec, words, q_hist, q_tgt)
    assert list(r2.h_status) == [HC_HIT, HC_HIT, H_REP, H_REP]
    assert list(r2.q_status) == [Q_SCORE_HIT, Q_SCORE_HIT, Q_COMPUTED, Q_COMPUTED]
    assert r2.hist_inserted == 0 and r2.hist_rejected == 2


def test_score_cache_admission_order_under_tiny_capacity():
    rng = np.random.default_rng(5)
    o = make(weights(rng), Q_SIGN, cap_hist=100, cap_query=3)
    vec = base_hist(rng, 1)
    words = np.array([[1, 2, 3]], np.int32)
    q_hist = np.zeros(5, np.int32)
    q_tgt = np.array([9, 8, 9, 7, 6], np.int32)
    r1 = o.score_frame(vec, words, q_hist, q_tgt)
    assert list(r1.q_status) == [Q_COMPUTED, Q_COMPUTED, Q_DUP, Q_COMPUTED, Q_COMPUTED]
    assert (r1.score_inserted, r1.score_rejected) == (3, 1)
    r2 = o.score_frame(vec, words, q_hist, q_tgt)
    assert list(r2.q_status) == [Q_SCORE_HIT, Q_SCORE_HIT, Q_SCORE_HIT, Q_SCORE_HIT, Q_COMPUTED]


def test_query_key_includes_maxent_context_words():
    rng = np.random.default_rng(6)
    o = make(weights(rng), Q_SIGN, order=3)
    h = base_hist(rng, 1)
    vec = np.concatenate([h, h, h])
    words = np.array([[5, 1, 1], [5, 2, 1], [5, 1, 2]], np.int32)   # w-3 unused at order 3
    r = o.score_frame(vec, words, np.arange(3, dtype=np.int32), np.full(3, 4, np.int32))
    assert list(r.h_status) == [H_REP, H_DUP, H_DUP]
    assert list(r.q_rep) == [0, 1, 0]
    assert list(r.q_status) == [Q_COMPUTED, Q_COMPUTED, Q_DUP]


def test_scores_reduce_to_closed_forms():
    rng = np.random.default_rng(7)
    # zero output layer, index-revealing MaxEnt table, bigram only:
    # score == slot of (w-1, target)
    lam = np.arange(1 << 12, dtype=np.float32)
    o = make(weights(rng, zero_out=True, lam=lam, me_log2=12), Q_SIGN, order=2, me_log2=12)
    vec, words, q_hist, q_tgt = _frame(rng)
    r = o.score_frame(vec, words, q_hist, q_tgt)
    want = maxent_index(2, [words[q_hist, 0]], q_tgt, 12)
    assert np.array_equal(r.scores, want.astype(np.float32))
    # zero MaxEnt: score = u_t . h' + b_t with h' from the GRU step
    w = weights(rng)
    w["maxent"][:] = 0
    o = make(w, Q_SIGN)
    r = o.score_frame(vec, words, q_hist, q_tgt)
    want = (r.hnew[q_hist] * w["U_out"][q_tgt].astype(np.float64)).sum(1) + w["b_out"][q_tgt]
    np.testing.assert_allclose(r.scores, want.astype(np.float32), rtol=1e-6)


def test_two_layer_history_and_output():
    rng = np.random.default_rng(8)
    w = weights(rng, L=2)
    o = make(w, Q_SIGN, L=2)
    vec = np.concatenate([base_hist(rng, 3), base_hist(rng, 3)], axis=1)
    words = np.array([[1, 0, 0], [2, 0, 0], [3, 0, 0]], np.int32)
    r = o.score_frame(vec, words, np.array([0, 1, 2], np.int32), np.array([4, 5, 6], np.int32))
    x = np.asarray(w["emb"][[1, 2, 3]], np.float64)
    h1 = gru_step(x, vec[:, :H], o.W_ih[0], o.W_hh[0], o.b_ih[0])
    h2 = gru_step(h1, vec[:, H:], o.W_ih[1], o.W_hh[1], o.b_ih[1])
    np.testing.assert_allclose(r.hnew, np.concatenate([h1, h2], axis=1), rtol=1e-13, atol=1e-15)


def test_rejects_bad_frames():
    rng = np.random.default_rng(9)
    o = make(weights(rng), Q_SIGDIG, 2)
    vec, words, q_hist, q_tgt = _frame(rng)
    bad = words.copy()
    bad[0, 0] = V
    with pytest.raises(ValueError):
        o.score_frame(vec, bad, q_hist, q_tgt)
    v2 = vec.copy()
    v2[1, 1] = 1.5
    with pytest.raises(ValueError):
        o.score_frame(v2, words, q_hist, q_tgt)
    with pytest.raises(ValueError):
        o.score_frame(vec, words, q_hist + 100, q_tgt)
