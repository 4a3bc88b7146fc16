"""GPU edge cases against the oracle: empty and ragged frames, frames at the
configured maxima, duplicates, tiny cache capacities, repeated frames, the
saturated-update-gate invariant, the sticky device error path, and MaxEnt
slots revealed exactly by an index-valued table."""
import numpy as np
import pytest
import torch

from harness import ATOL, RTOL, close, log
from oracle import (H_DUP, H_REP, HC_HIT, Q_DUP, Q_EXACT, Q_SCORE_HIT, Q_SIGDIG, Q_SIGN, Oracle)
from paper_1801_09866_amd import rnnlm as R
from paper_1801_09866_amd.workload import F32, ModelCfg

pytestmark = pytest.mark.gpu

M = ModelCfg(V=5000, E=64, H=128, L=1, wdtype=F32, maxent_log2=16, maxent_order=4)


def weights(m, rng, scale=0.05):
    H, E = m.H, m.E
    return {"emb": (rng.standard_normal((m.V, E)) * scale).astype(np.float32),
            "W_ih": [(rng.standard_normal((3 * H, E if l == 0 else H)) * scale).astype(np.float32) for l in range(m.L)],
            "W_hh": [(rng.standard_normal((3 * H, H)) * scale).astype(np.float32) for l in range(m.L)],
            "b_ih": [(rng.standard_normal(3 * H) * scale).astype(np.float32) for l in range(m.L)],
            "U_out": (rng.standard_normal((m.V, H)) * scale).astype(np.float32),
            "b_out": (rng.standard_normal(m.V) * scale).astype(np.float32),
            "maxent": (rng.standard_normal(1 << m.maxent_log2) * 0.01).astype(np.float32)}


class Both:
    def __init__(self, m, w, qmode, k=0, max_hist=300, max_query=3000, cap_hist=1 << 12, cap_query=1 << 14):
        # h' is a GRU step over K = E + H terms in fp32; the fixed bar holds
        # for the configurations' K <= 1536, and the rounding error of a
        # K-term sum grows with K, so longer sums scale the absolute bar
        self.hatol = ATOL * max(1.0, max(m.E + m.H, 2 * m.H if m.L == 2 else 0) / 1536)
        self.o = Oracle(m.V, m.E, m.H, m.L, m.maxent_log2, m.maxent_order, w, qmode, k,
                        cap_hist=cap_hist, cap_query=cap_query, seed=R.DEFAULT_SEED)
        self.g = R.Scorer(m, w, qmode, k, max_hist=max_hist, max_query=max_query,
                          cap_hist=cap_hist, cap_query=cap_query)

    def frame(self, vec, words, qh, qt, tag=""):
        log("  frame", tag, "n_hist", len(vec), "n_query", len(qh))
        d = lambda a, t: torch.from_numpy(np.ascontiguousarray(a, t)).cuda()
        out = self.g.score_frame(d(vec, np.float32), d(words, np.int32),
                                 d(qh, np.int32) if len(qh) else None, d(qt, np.int32) if len(qt) else None)
        res = self.o.score_frame(vec, words, qh, qt)
        torch.cuda.synchronize()
        n_h, n_q = len(vec), len(qh)
        assert np.array_equal(out["h_hash"][:n_h].cpu().numpy().view(np.uint64), res.h_hash), tag
        assert np.array_equal(out["h_status"][:n_h].cpu().numpy(), res.h_status), tag
        assert np.array_equal(out["h_rep"][:n_h].cpu().numpy(), res.h_rep), tag
        g, w = out["hnew"][:n_h].cpu().numpy().astype(np.float64), res.hnew
        ok, emax = close(g, w, self.hatol, RTOL)
        assert ok, (tag, "h' max error %.3g, %.3f of the tolerance" % (emax, (np.abs(g - w) / (self.hatol + RTOL * np.abs(w))).max()))
        if n_q:
            assert np.array_equal(out["q_status"][:n_q].cpu().numpy(), res.q_status), tag
            assert np.array_equal(out["q_rep"][:n_q].cpu().numpy(), res.q_rep), tag
            assert close(out["scores"][:n_q].cpu().numpy(), res.scores, ATOL, RTOL)[0], tag
        return out, res


def rand_frame(rng, m, n_h, n_q, dup_every=0):
    vec = (np.tanh(rng.standard_normal((n_h, m.L * m.H))) * 0.9).astype(np.float32)
    words = rng.integers(0, m.V, (n_h, 3)).astype(np.int32)
    if dup_every:
        for i in range(dup_every, n_h, dup_every):
            vec[i] = vec[i - dup_every]
            words[i, 0] = words[i - dup_every, 0]
    qh = rng.integers(0, max(n_h, 1), n_q).astype(np.int32)
    qt = rng.integers(0, m.V, n_q).astype(np.int32)
    return vec, words, qh, qt


def test_ragged_sizes_empty_and_maximal():
    rng = np.random.default_rng(0)
    b = Both(M, weights(M, rng), Q_SIGN)
    # nothing to do
    out = b.g.score_frame(torch.empty((0, M.H), device="cuda"), torch.empty((0, 3), dtype=torch.int32, device="cuda"), None, None)
    for n_h, n_q in [(1, 0), (1, 1), (63, 5), (65, 1000), (130, 0), (300, 3000), (257, 2999)]:
        b.frame(*rand_frame(rng, M, n_h, n_q, dup_every=7), tag="%d/%d" % (n_h, n_q))
    st = b.g.stats()
    assert st["frames"] == 7


def test_planner_maximal_frame():
    """The planner's largest frame (2048 histories, 8192 queries): query keys
    not staged in LDS, the query race table at load 1/2, keys left after the
    race tables, and many equal keys of both kinds."""
    rng = np.random.default_rng(17)
    b = Both(M, weights(M, rng), Q_SIGN, max_hist=2048, max_query=8192, cap_hist=1 << 13, cap_query=1 << 15)
    for t in range(2):
        vec, words, qh, qt = rand_frame(rng, M, 2048, 8192, dup_every=5)
        qt = rng.integers(0, 40, 8192).astype(np.int32)   # few targets: many equal query keys
        b.frame(vec, words, qh, qt, tag="max %d" % t)


def test_planner_round_boundaries():
    """Frames on each side of the planner's per-thread round counts (1024
    histories or queries per round of its 1024 threads; the launch sizes its
    rounds to the frame): 1024 and 1025 histories, 1024, 1025, 2048, 2049,
    4096 and 4097 queries, many equal keys of both kinds, the second frame
    of each pair repeating the first's histories and queries."""
    rng = np.random.default_rng(23)
    b = Both(M, weights(M, rng), Q_SIGN, max_hist=1100, max_query=4200, cap_hist=1 << 13, cap_query=1 << 15)
    for n_h, n_q in [(1024, 1024), (1025, 1025), (1024, 2048), (1025, 2049), (600, 4096), (1025, 4097)]:
        vec, words, qh, qt = rand_frame(rng, M, n_h, n_q, dup_every=6)
        qt = rng.integers(0, 60, n_q).astype(np.int32)   # few targets: many equal query keys
        b.frame(vec, words, qh, qt, tag="%d/%d" % (n_h, n_q))
        o2, r2 = b.frame(vec, words, qh, qt, tag="%d/%d again" % (n_h, n_q))
        assert np.all(r2.h_status == HC_HIT), (n_h, n_q)


def test_repeat_frame_hits_with_identical_bits():
    rng = np.random.default_rng(1)
    b = Both(M, weights(M, rng), Q_SIGDIG, 2)
    f = rand_frame(rng, M, 100, 900, dup_every=5)
    o1, r1 = b.frame(*f, tag="first")
    s1 = o1["scores"][:900].clone()
    o2, r2 = b.frame(*f, tag="repeat")
    assert np.all(r2.h_status == HC_HIT) and np.all(r2.q_status == Q_SCORE_HIT)
    assert torch.equal(o2["scores"][:900].view(torch.int32), s1.view(torch.int32))
    assert (r1.q_status == Q_DUP).any() and (r1.h_status == H_DUP).any()


def test_tiny_capacities_admission_order():
    rng = np.random.default_rng(2)
    b = Both(M, weights(M, rng), Q_SIGN, cap_hist=5, cap_query=7)
    f = rand_frame(rng, M, 20, 60)
    for t in range(3):
        b.frame(*f, tag="cap %d" % t)
    st = b.g.stats()
    assert st["hist_cache_size"] == 5 and st["score_cache_size"] == 7
    assert st["hist_rejected"] > 0


def test_zero_capacities():
    rng = np.random.default_rng(3)
    b = Both(M, weights(M, rng), Q_SIGN, cap_hist=0, cap_query=0)
    f = rand_frame(rng, M, 40, 200, dup_every=3)
    b.frame(*f, tag="a")
    b.frame(*f, tag="b")
    assert b.g.stats()["hist_cache_size"] == 0


def test_saturated_update_gate_keeps_history_bitwise():
    rng = np.random.default_rng(4)
    w = weights(M, rng)
    w["b_ih"][0][M.H:2 * M.H] = 100.0    # z = 1 exactly in fp32 and double
    b = Both(M, w, Q_SIGN)
    vec, words, qh, qt = rand_frame(rng, M, 50, 10)
    out, res = b.frame(vec, words, qh, qt, tag="z=1")
    assert torch.equal(out["hnew"][:50].cpu(), torch.from_numpy(vec))


def test_two_layer_fp32_and_exact_mode():
    m = ModelCfg(V=3000, E=64, H=128, L=2, wdtype=F32, maxent_log2=12, maxent_order=3)
    rng = np.random.default_rng(5)

    b = Both(m, weights(m, rng), Q_EXACT)
    for t in range(3):
        b.frame(*rand_frame(rng, m, 70, 400, dup_every=4), tag="L2 %d" % t)


@pytest.mark.parametrize("L,H,qmode,k", [(1, 512, Q_SIGN, 0), (1, 1024, Q_SIGDIG, 2), (1, 1024, Q_EXACT, 0),
                                         (2, 576, Q_SIGN, 0), (2, 576, Q_SIGDIG, 2), (2, 1024, Q_EXACT, 0),
                                         (1, 1088, Q_SIGN, 0), (1, 2048, Q_SIGN, 0)],
                         ids=["LH512-sign", "LH1024-sigdig2-cw256", "LH1024-exact-cw512", "LH1152-sign",
                              "LH1152-sigdig2-cw288", "LH2048-exact-cw1024", "H1088-sign", "H2048-sign"])
def test_scorer_register_sizes(L, H, qmode, k):
    """The scoring kernel holds a row of at most 1024 elements and a key of
    at most 256 code words in fewer registers; every combination of short or
    long rows and keys, at both limits, against the oracle. Output rows
    longer than 1024 elements (H = 1088: only some lanes of the fifth step
    are inside the row; H = 2048: every step) take the upper load steps."""
    m = ModelCfg(V=3000, E=64, H=H, L=L, wdtype=F32, maxent_log2=12, maxent_order=4)
    rng = np.random.default_rng(40 + L * 7 + H + qmode)
    b = Both(m, weights(m, rng), qmode, k, max_hist=64, max_query=512)
    frames = [rand_frame(rng, m, 48, 300, dup_every=5) for _ in range(2)]
    for t, f in enumerate(frames + frames[:1]):   # the repeat: cache hits and stored scores
        b.frame(*f, tag="L%d H%d %d" % (L, H, t))


def test_device_errors_are_sticky_until_reset():
    rng = np.random.default_rng(6)
    g = R.Scorer(M, weights(M, rng), Q_SIGDIG, 2, max_hist=64, max_query=64)
    vec, words, qh, qt = rand_frame(rng, M, 10, 20)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    bad_words = words.copy()
    bad_words[3, 1] = M.V + 5
    g.score_frame(d(vec), d(bad_words), d(qh), d(qt))
    with pytest.raises(R.RnnlmError) as e:
        g.stats()
    assert e.value.code == R.EDEVICE
    with pytest.raises(R.RnnlmError):
        g.score_frame(d(vec), d(words), d(qh), d(qt))
    g.reset()
    g.score_frame(d(vec), d(words), d(qh), d(qt))
    assert g.stats()["device_error"] == 0
    v2 = vec.copy()
    v2[2, 5] = 1.5          # outside [-1, 1] under decimal rounding
    bq = qh.copy()
    bq[0] = 99              # history index outside the frame
    g.score_frame(d(v2), d(words), d(bq), d(qt))
    s = g.stats(check=False)
    assert s["device_error"] == R.DERR_VALUE | R.DERR_QHIST
    g.reset()


def test_host_rejects_oversized_frames():
    rng = np.random.default_rng(7)
    g = R.Scorer(M, weights(M, rng), Q_SIGN, max_hist=8, max_query=8)
    vec, words, qh, qt = rand_frame(rng, M, 9, 4)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    with pytest.raises(R.RnnlmError) as e:
        g.score_frame(d(vec), d(words), d(qh), d(qt))
    assert e.value.code == R.EINVAL


@pytest.mark.parametrize("L,wd,E,H", [(1, F32, 128, 256), (2, F32, 128, 256), (1, 1, 128, 256), (2, 1, 192, 320),
                                       (2, 1, 64, 128), (2, F32, 64, 128)])
def test_gru_paths_by_row_count(L, wd, E, H):
    """Row counts on each side of the narrow path (<= 32 rows) and across the
    tiled path's row-tile heights, all new keys, against the oracle. H = 320
    gives unit tiles (20 fp32 tiles of 16 units, 10 bf16 tiles of 32) that do
    not split evenly over the 8 XCDs, with input sizes (192, then 320) that
    are not multiples of 128; E = 64 gives a first layer whose input part is
    a single K step."""
    m = ModelCfg(V=3000, E=E, H=H, L=L, wdtype=wd, maxent_log2=12, maxent_order=4)
    rng = np.random.default_rng(10 + L + 3 * wd)
    w = weights(m, rng, scale=0.08)
    tol = (2e-2, 0.0) if wd == 1 else (ATOL, RTOL)
    for n_h in (1, 15, 16, 17, 32, 33, 64, 200, 256, 257, 512):
        b = Both(m, w, Q_EXACT, max_hist=512, max_query=1024)
        vec, words, qh, qt = rand_frame(rng, m, n_h, min(2 * n_h, 1024))
        log("  GRU rows", n_h, "L", L, "wdtype", wd)
        d = lambda a, t: torch.from_numpy(np.ascontiguousarray(a, t)).cuda()
        out = b.g.score_frame(d(vec, np.float32), d(words, np.int32), d(qh, np.int32), d(qt, np.int32))
        res = b.o.score_frame(vec, words, qh, qt)
        torch.cuda.synchronize()
        assert res.gru_rows == n_h
        ok, err = close(out["hnew"][:n_h].cpu().numpy(), res.hnew, *tol)
        assert ok, "rows %d: GRU outputs differ by %.3g" % (n_h, err)
        ok, err = close(out["scores"][:len(qh)].cpu().numpy(), res.scores, *tol)
        assert ok, "rows %d: scores differ by %.3g" % (n_h, err)


@pytest.mark.parametrize("order", [2, 3, 4])
def test_maxent_slots_revealed_by_an_index_table(order):
    """Zero output layer and lambda[i] = i (exact in fp32 for 2^16 slots),
    one n-gram order at a time: each computed score is the slot the device's
    MaxEnt hash picks, which must equal the oracle's index of the n-gram
    (orders 2..order all add; subtracting the lower orders isolates the top
    one)."""
    from oracle.rnnlm_oracle import maxent_index
    m = ModelCfg(V=5000, E=64, H=128, L=1, wdtype=F32, maxent_log2=16, maxent_order=order)
    rng = np.random.default_rng(70 + order)
    w = weights(m, rng)
    w["U_out"][:] = 0
    w["b_out"][:] = 0
    w["maxent"] = np.arange(1 << 16, dtype=np.float32)
    b = Both(m, w, Q_SIGN)
    vec, words, qh, qt = rand_frame(rng, m, 40, 300)
    out, res = b.frame(vec, words, qh, qt, "index table, order %d" % order)
    comp = res.q_status == 0   # computed queries carry their own sum
    want = np.zeros(len(qt))
    for o in range(2, order + 1):
        ctx = [words[qh, c] for c in range(o - 1)]
        want += maxent_index(o, ctx, qt, 16).astype(np.float64)
    got = out["scores"][:len(qt)].cpu().numpy().astype(np.float64)
    assert np.array_equal(got[comp], want[comp])
