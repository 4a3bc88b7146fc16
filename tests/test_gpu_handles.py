"""History handles (device addresses of history rows) and the decode loop they
close: a frame read through handles gives the same bits as the same rows
passed contiguously; a bad handle is a sticky device error; and a seeded
decode loop whose histories are the library's own h' outputs matches the
oracle running the same plan on its own h'."""
import numpy as np
import pytest
import torch

from harness import ATOL, RTOL, close, log
from oracle import Q_EXACT, Q_SIGDIG, Q_SIGN, Oracle
from paper_1801_09866_amd import rnnlm as R
from paper_1801_09866_amd.decode import DeviceDecodeLoop
from paper_1801_09866_amd.workload import F32, ModelCfg, decode_plan

pytestmark = pytest.mark.gpu


def weights(m, rng, scale=0.08):
    H, E = m.H, m.E
    return {"emb": (rng.standard_normal((m.V, E)) * scale).astype(np.float32),
            "W_ih": [(rng.standard_normal((3 * H, E if l == 0 else H)) * scale).astype(np.float32) for l in range(m.L)],
            "W_hh": [(rng.standard_normal((3 * H, H)) * scale).astype(np.float32) for l in range(m.L)],
            "b_ih": [(rng.standard_normal(3 * H) * scale).astype(np.float32) for l in range(m.L)],
            "U_out": (rng.standard_normal((m.V, H)) * scale).astype(np.float32),
            "b_out": (rng.standard_normal(m.V) * scale).astype(np.float32),
            "maxent": (rng.standard_normal(1 << m.maxent_log2) * 0.01).astype(np.float32)}


KEYS = ("scores", "hnew", "q_status", "q_rep", "h_status", "h_rep", "h_hash")


@pytest.mark.parametrize("qmode,k", [(Q_EXACT, 0), (Q_SIGN, 0), (Q_SIGDIG, 2)])
def test_handles_give_the_same_bits_as_contiguous_rows(qmode, k):
    m = ModelCfg(V=3000, E=64, H=128, L=2, wdtype=F32, maxent_log2=12, maxent_order=4)
    rng = np.random.default_rng(20 + qmode)
    w = weights(m, rng)
    LH = m.L * m.H
    src = torch.from_numpy((np.tanh(rng.standard_normal((50, LH))) * 0.9).astype(np.float32)).cuda()
    a = R.Scorer(m, w, qmode, k, max_hist=128, max_query=512)
    b = R.Scorer(m, w, qmode, k, max_hist=128, max_query=512)
    for t in range(3):
        idx = rng.integers(0, 50, 100)                       # shuffled, with repeats
        words = torch.from_numpy(rng.integers(0, m.V, (100, 3)).astype(np.int32)).cuda()
        qh = torch.from_numpy(rng.integers(0, 100, 400).astype(np.int32)).cuda()
        qt = torch.from_numpy(rng.integers(0, m.V, 400).astype(np.int32)).cuda()
        hp = torch.tensor([src.data_ptr() + int(i) * LH * 4 for i in idx], dtype=torch.int64).cuda()
        log("  frame", t, "qmode", qmode)
        oa = a.score_frame(None, words, qh, qt, hist_ptr=hp)
        ob = b.score_frame(src[torch.from_numpy(idx).cuda()].contiguous(), words, qh, qt)
        torch.cuda.synchronize()
        for key in KEYS:
            n = 400 if key in ("scores", "q_status", "q_rep") else 100
            assert torch.equal(oa[key][:n].view(torch.uint8), ob[key][:n].view(torch.uint8)), (t, key)
    assert a.stats()["device_error"] == 0


def test_null_handle_is_a_sticky_device_error():
    m = ModelCfg(V=1000, E=64, H=64, L=1, wdtype=F32, maxent_log2=10, maxent_order=3)
    rng = np.random.default_rng(3)
    g = R.Scorer(m, weights(m, rng), Q_SIGN, 0, max_hist=16, max_query=16)
    src = torch.zeros((4, m.H), dtype=torch.float32, device="cuda")
    hp = torch.tensor([src.data_ptr(), 0, src.data_ptr() + 256, src.data_ptr()], dtype=torch.int64).cuda()
    words = torch.ones((4, 3), dtype=torch.int32, device="cuda")
    q = torch.zeros(2, dtype=torch.int32, device="cuda")
    g.score_frame(None, words, q, q + 1, hist_ptr=hp)
    s = g.stats(check=False)
    assert s["device_error"] == R.DERR_HANDLE
    with pytest.raises(R.RnnlmError):
        g.score_frame(None, words, q, q + 1, hist_ptr=hp)
    g.reset()
    g.score_frame(None, words, q, q + 1, hist_ptr=hp[[0, 0, 2, 3]].contiguous())
    assert g.stats()["device_error"] == 0


def test_decode_loop_matches_the_oracle_on_its_own_outputs():
    """Exact keys: equal keys arise on both sides exactly where the plan
    re-uses a history, so statuses and representatives must agree bit for
    bit, while scores and h' agree to the fp32 tolerance."""
    m = ModelCfg(V=4000, E=64, H=128, L=2, wdtype=F32, maxent_log2=12, maxent_order=4)
    rng = np.random.default_rng(31)
    w = weights(m, rng)
    beam, fan, nfr = 40, 3, 8
    LH = m.L * m.H
    init = (np.tanh(rng.standard_normal((beam, LH))) * 0.9).astype(np.float32)
    init_words = rng.integers(1, m.V, (beam, 3)).astype(np.int32)
    plan = decode_plan(m.V, beam, fan, nfr, 0.5, 1.0, 5, init_words)
    g = R.Scorer(m, w, Q_EXACT, 0, max_hist=beam, max_query=beam * fan)
    outs = DeviceDecodeLoop(g, torch.from_numpy(init).cuda()).run(plan)
    o = Oracle(m.V, m.E, m.H, m.L, m.maxent_log2, m.maxent_order, w, Q_EXACT, 0,
               cap_hist=1 << 12, cap_query=1 << 14, seed=R.DEFAULT_SEED)
    vec = init
    torch.cuda.synchronize()
    hits = 0
    for t, (fr, out) in enumerate(zip(plan, outs)):
        if t > 0:
            vec = np.stack([prev_h[p] if a else vec[p] for p, a in zip(fr.prev, fr.advanced)])
        res = o.score_frame(vec, fr.words, fr.q_hist, fr.q_tgt)
        nq = len(fr.q_hist)
        log("  decode frame", t, "score hits", int((res.q_status == 2).sum()))
        assert np.array_equal(out["h_status"][:beam].cpu().numpy(), res.h_status), t
        assert np.array_equal(out["h_rep"][:beam].cpu().numpy(), res.h_rep), t
        assert np.array_equal(out["q_status"][:nq].cpu().numpy(), res.q_status), t
        assert np.array_equal(out["q_rep"][:nq].cpu().numpy(), res.q_rep), t
        assert close(out["scores"][:nq].cpu().numpy(), res.scores, ATOL, RTOL)[0], t
        assert close(out["hnew"][:beam].cpu().numpy(), res.hnew, ATOL, RTOL)[0], t
        hits += int((res.q_status == 2).sum())
        prev_h = res.hnew.astype(np.float32)   # the next frame's histories, on the oracle side
    assert hits > 0   # staying hypotheses repeat their queries
    assert g.stats()["device_error"] == 0


def forgetful(w, m, wx=0.5, wh=0.01, bz=-2.0, scale=0.08):
    """The Table-1 sweep's model: strong input weights, weak recurrent ones and
    a small update gate, so that paths on the same recent words come close
    enough for lossy keys to merge them (Sec. 3)."""
    w = dict(w)
    w["W_ih"] = [(x * (wx / scale)).astype(np.float32) for x in w["W_ih"]]
    w["W_hh"] = [(x * (wh / scale)).astype(np.float32) for x in w["W_hh"]]
    b = [x.copy() for x in w["b_ih"]]
    for x in b:
        x[m.H:2 * m.H] += np.float32(bz)   # gate order r, z, n
    w["b_ih"] = b
    return w


@pytest.mark.parametrize("qmode,k", [(Q_SIGN, 0), (Q_SIGDIG, 1), (Q_SIGDIG, 2), (Q_SIGDIG, 3)],
                         ids=["sign", "sigdig1", "sigdig2", "sigdig3"])
def test_lossy_decode_loop_matches_the_oracle(qmode, k):
    """The Table-1 decode loop in each lossy mode (Sec. 3, Table 1). Both
    sides quantise the same vectors: the oracle's next-frame histories are
    the library's own h' (a last-bit difference in a double-precision h'
    could otherwise cross a rounding boundary or flip a sign). Statuses and
    representatives must agree bit for bit, so the unique LM queries and GRU
    rows per frame equal the oracle's; scores and h' agree to the fp32
    tolerance. The loop shares candidate words across the beam, so lossy keys
    do merge histories that exact keys keep apart."""
    m = ModelCfg(V=4000, E=64, H=128, L=1, wdtype=F32, maxent_log2=12, maxent_order=4)
    rng = np.random.default_rng(41 + 3 * qmode + k)
    w = forgetful(weights(m, rng), m)
    beam, fan, nfr = 96, 4, 10
    LH = m.L * m.H
    init = (np.tanh(rng.standard_normal((beam, LH))) * 0.9).astype(np.float32)
    init_words = rng.integers(1, m.V, (beam, 3)).astype(np.int32)
    plan = decode_plan(m.V, beam, fan, nfr, 0.5, 1.0, 9, init_words, shared=6, focus=0.8)
    g = R.Scorer(m, w, qmode, k, max_hist=beam, max_query=beam * fan)
    outs = DeviceDecodeLoop(g, torch.from_numpy(init).cuda()).run(plan)
    o = Oracle(m.V, m.E, m.H, m.L, m.maxent_log2, m.maxent_order, w, qmode, k,
               cap_hist=1 << 12, cap_query=1 << 14, seed=R.DEFAULT_SEED)
    torch.cuda.synchronize()
    vec = init
    computed = rows = exact_rows = 0
    seen = set()
    for t, (fr, out) in enumerate(zip(plan, outs)):
        if t > 0:
            vec = np.stack([prev_h[p] if a else vec[p] for p, a in zip(fr.prev, fr.advanced)])
        res = o.score_frame(vec, fr.words, fr.q_hist, fr.q_tgt)
        nq = len(fr.q_hist)
        log("  %s decode frame %d: GRU rows %d, computed %d" % (qmode, t, res.gru_rows, (res.q_status == 0).sum()))
        assert np.array_equal(out["h_hash"][:beam].cpu().numpy().view(np.uint64), res.h_hash), t
        assert np.array_equal(out["h_status"][:beam].cpu().numpy(), res.h_status), t
        assert np.array_equal(out["h_rep"][:beam].cpu().numpy(), res.h_rep), t
        assert np.array_equal(out["q_status"][:nq].cpu().numpy(), res.q_status), t
        assert np.array_equal(out["q_rep"][:nq].cpu().numpy(), res.q_rep), t
        assert close(out["scores"][:nq].cpu().numpy(), res.scores, ATOL, RTOL)[0], t
        assert close(out["hnew"][:beam].cpu().numpy(), res.hnew, ATOL, RTOL)[0], t
        computed += int((res.q_status == 0).sum())
        rows += res.gru_rows
        # GRU rows exact keys would need: (vector bits, input word) pairs not seen before
        for i in range(beam):
            key = (vec[i].tobytes(), int(fr.words[i, 0]))
            if key not in seen:
                seen.add(key)
                exact_rows += 1
        prev_h = out["hnew"][:beam].cpu().numpy()   # the next frame's histories, for both sides
    st = g.stats()
    assert st["computed"] == computed and st["gru_rows"] == rows
    log("  %s/%d: %d unique LM queries, %d GRU rows (exact keys: %d)" % (qmode, k, computed, rows, exact_rows))
    assert rows <= exact_rows
    if qmode == Q_SIGN:
        assert rows < exact_rows   # sign keys merge histories that exact keys keep apart
