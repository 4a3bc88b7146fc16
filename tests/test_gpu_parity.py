"""GPU parity: the HIP library against the CPU oracle on seeded frames of every
config. Keys, hashes, representatives, statuses and cache decisions must be
bit-exact; fp32 scores and GRU outputs within 1e-6 + 1e-5 |ref|; bf16-weight
scores within 2e-2 absolute of the fp32-master oracle."""
import dataclasses

import numpy as np
import pytest
import torch

from harness import ATOL, RTOL, close, device_frame, log, make_pair, run_frames
from oracle import Q_EXACT, Q_SIGDIG, Q_SIGN, log_normalizer, log_normalizer_maxent
from paper_1801_09866_amd import rnnlm as R
from paper_1801_09866_amd.workload import CONFIGS, ModelCfg

pytestmark = pytest.mark.gpu


def test_tiny_all_frames():
    p = make_pair("tiny", Q_SIGN, 0, n_frames=None)
    st = run_frames(p)
    log("  tiny stats", st)
    assert st["hist_hits"] > 0 and st["score_hits"] >= 0


def test_medium_three_digits_prefix():
    p = make_pair("medium", Q_SIGDIG, 3, n_frames=40)
    st = run_frames(p)
    assert st["hist_hits"] > 0


@pytest.mark.parametrize("qmode,k,n", [(Q_SIGN, 0, 6), (Q_SIGDIG, 2, 6), (Q_SIGDIG, 1, 4)],
                         ids=["sign", "sigdig2", "sigdig1"])
def test_large_fp32_prefix(qmode, k, n):
    """Large fp32 frames end to end; sign and 2 digits are the config's runs,
    1 digit the coarsest decimal row of Table 1 (Sec. 3)."""
    p = make_pair("large", qmode, k, n_frames=n)
    st = run_frames(p, log_every=1)
    assert st["score_hits"] > 0      # 30% of each frame repeats the previous frame's pairs


def test_large_bf16_two_layers_prefix():
    p = make_pair("large_bf16", Q_SIGN, 0, n_frames=3)
    run_frames(p, log_every=1)


def test_check_config_normaliser():
    p = make_pair("check", Q_EXACT, 0, n_frames=2)
    for fi, fr in enumerate(p.wl.frames):
        hv, hw, qh, qt = device_frame(p, fr)
        out = p.scorer.score_frame(hv, hw, None, None)
        res = p.oracle.score_frame(p.wl.pool.vec[fr.pool_idx], fr.hist_words, fr.q_hist, fr.q_tgt)
        h_gpu = out["hnew"][:fr.n_hist]
        logz = p.scorer.log_normalizer(h_gpu).cpu().numpy()
        ok, err = close(h_gpu.cpu().numpy(), res.hnew, ATOL, RTOL)
        assert ok, "GRU outputs differ %.3g" % err
        # same h on both sides: the normaliser alone
        want_same = log_normalizer(h_gpu.cpu().numpy(), p.wl.weights["U_out"], p.wl.weights["b_out"])
        ok, err = close(logz, want_same, ATOL, RTOL)
        assert ok, "logZ differs from the oracle on identical h (max err %.3g)" % err
        # end to end: oracle h' from its own GRU step
        want = log_normalizer(res.hnew, p.wl.weights["U_out"], p.wl.weights["b_out"])
        ok, err = close(logz, want, ATOL, RTOL)
        assert ok, "logZ differs end to end (max err %.3g)" % err
        log("  check frame %d: mean logZ %.4f sd %.4f" % (fi, want.mean(), want.std()))


def test_normaliser_closed_form_and_ragged_rows():
    """U_out = 0, b = 0: logZ = ln V exactly; ragged row counts, > 256 rows."""
    m = ModelCfg(V=200_000, E=64, H=128, L=1, wdtype=R.F32, maxent_log2=10, maxent_order=2)
    rng = np.random.default_rng(1)
    w = {"emb": np.zeros((m.V, m.E), np.float32), "W_ih": [np.zeros((384, 64), np.float32)],
         "W_hh": [np.zeros((384, 128), np.float32)], "b_ih": [np.zeros(384, np.float32)],
         "U_out": np.zeros((m.V, m.H), np.float32), "b_out": np.zeros(m.V, np.float32),
         "maxent": np.zeros(1 << 10, np.float32)}
    sc = R.Scorer(m, w, Q_SIGN, max_hist=600, max_query=1)
    for n in (1, 37, 256, 300, 600):
        h = torch.from_numpy(np.tanh(rng.standard_normal((n, m.H))).astype(np.float32)).cuda()
        z = sc.log_normalizer(h).cpu().numpy()
        assert np.allclose(z, np.log(m.V), rtol=2e-7, atol=0), (n, z[:4])
    # random weights, ragged vocabulary tail (V not a multiple of the tile)
    m2 = dataclasses.replace(m, V=1000 + 37)
    w2 = dict(w, U_out=(rng.standard_normal((m2.V, m2.H)) * 0.3).astype(np.float32),
              b_out=rng.standard_normal(m2.V).astype(np.float32),
              emb=np.zeros((m2.V, m2.E), np.float32))
    sc2 = R.Scorer(m2, w2, Q_SIGN, max_hist=300, max_query=1)
    h = np.tanh(rng.standard_normal((300, m2.H))).astype(np.float32)
    z = sc2.log_normalizer(torch.from_numpy(h).cuda()).cpu().numpy()
    ok, err = close(z, log_normalizer(h, w2["U_out"], w2["b_out"]), ATOL, RTOL)
    assert ok, err


def test_maxent_normaliser_against_the_oracle():
    """Normaliser over the full output (NCE + MaxEnt for every word): ragged
    vocabulary tail, > 256 rows, orders 2..4; zero MaxEnt weights give the
    plain normaliser's bits; a word outside [0, V) is a sticky device error."""
    m = ModelCfg(V=3000 + 29, E=64, H=128, L=1, wdtype=R.F32, maxent_log2=12, maxent_order=4)
    rng = np.random.default_rng(12)
    w = {"emb": np.zeros((m.V, m.E), np.float32), "W_ih": [np.zeros((384, 64), np.float32)],
         "W_hh": [np.zeros((384, 128), np.float32)], "b_ih": [np.zeros(384, np.float32)],
         "U_out": (rng.standard_normal((m.V, m.H)) * 0.3).astype(np.float32),
         "b_out": rng.standard_normal(m.V).astype(np.float32),
         "maxent": (rng.standard_normal(1 << 12) * 0.5).astype(np.float32)}
    sc = R.Scorer(m, w, Q_SIGN, max_hist=300, max_query=1)
    h = np.tanh(rng.standard_normal((300, m.H))).astype(np.float32)
    words = rng.integers(0, m.V, (300, 3)).astype(np.int32)
    words[:5] = 0   # sentence start context
    z = sc.log_normalizer_maxent(torch.from_numpy(h).cuda(), torch.from_numpy(words).cuda()).cpu().numpy()
    want = log_normalizer_maxent(h, w["U_out"], w["b_out"], w["maxent"], words, 4, 12)
    ok, err = close(z, want, ATOL, RTOL)
    assert ok, "MaxEnt logZ differs (max err %.3g)" % err
    assert not np.allclose(z, sc.log_normalizer(torch.from_numpy(h).cuda()).cpu().numpy(), atol=1e-3)
    sc0 = R.Scorer(m, dict(w, maxent=np.zeros(1 << 12, np.float32)), Q_SIGN, max_hist=300, max_query=1)
    hd, wd = torch.from_numpy(h).cuda(), torch.from_numpy(words).cuda()
    assert torch.equal(sc0.log_normalizer_maxent(hd, wd), sc0.log_normalizer(hd))
    wd[7, 1] = m.V + 3
    sc0.log_normalizer_maxent(hd, wd)
    assert sc0.stats(check=False)["device_error"] == R.DERR_WORD


def test_check_config_maxent_normaliser_sample():
    """Check-config sizes (V = 200,000, H = 1024, 2^26-entry table), 24 rows."""
    p = make_pair("check", Q_EXACT, 0, n_frames=1)
    fr = p.wl.frames[0]
    rng = np.random.default_rng(4)
    h = np.tanh(rng.standard_normal((24, p.wl.cfg.model.H))).astype(np.float32)
    words = fr.hist_words[:24].astype(np.int32)
    z = p.scorer.log_normalizer_maxent(torch.from_numpy(h).cuda(), torch.from_numpy(words).cuda()).cpu().numpy()
    m = p.wl.cfg.model
    want = log_normalizer_maxent(h, p.wl.weights["U_out"], p.wl.weights["b_out"], p.wl.weights["maxent"],
                                 words, m.maxent_order, m.maxent_log2)
    ok, err = close(z, want, ATOL, RTOL)
    assert ok, "MaxEnt logZ differs at check-config size (max err %.3g)" % err
