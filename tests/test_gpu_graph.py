"""A frame sequence captured into a HIP graph replays bit-identically to the
same frames launched eagerly. rnnlm_score_frame only enqueues kernels (no
allocation, synchronisation or memset on the stream), so a caller can capture
a decode loop's launches. Each replay starts from caches reset and refilled
by eagerly launched warm-up frames, with the host waiting between replays,
and every replay is checked (cold frames, which take the tiled GRU path, and
warm frames with cache hits)."""
import ctypes

import numpy as np
import pytest
import torch

from paper_1801_09866_amd import rnnlm as R
from paper_1801_09866_amd.workload import F32, ModelCfg

pytestmark = pytest.mark.gpu

M = ModelCfg(V=5000, E=128, H=256, L=1, wdtype=F32, maxent_log2=14, maxent_order=4)


def weights(m, rng, scale=0.08):
    H, E = m.H, m.E
    return {"emb": (rng.standard_normal((m.V, E)) * scale).astype(np.float32),
            "W_ih": [(rng.standard_normal((3 * H, E)) * scale).astype(np.float32)],
            "W_hh": [(rng.standard_normal((3 * H, H)) * scale).astype(np.float32)],
            "b_ih": [(rng.standard_normal(3 * H) * scale).astype(np.float32)],
            "U_out": (rng.standard_normal((m.V, H)) * scale).astype(np.float32),
            "b_out": (rng.standard_normal(m.V) * scale).astype(np.float32),
            "maxent": (rng.standard_normal(1 << m.maxent_log2) * 0.01).astype(np.float32)}


def test_graph_replay_matches_eager_frames():
    rng = np.random.default_rng(77)
    n_frames, warm = 8, 3
    pool = np.tanh(rng.standard_normal((600, M.H))).astype(np.float32)
    dev = torch.device("cuda:0")
    frames = []
    for f in range(n_frames):
        if f >= 5:                            # frames 5..7 repeat frames 2..4: cache hits
            frames.append(frames[f - 3])
            continue
        n_h = 300 if f < 2 else 80            # two cold frames (tiled GRU path), then small ones
        idx = rng.integers(0, 600, n_h)
        words = rng.integers(0, M.V, (n_h, 3)).astype(np.int32)
        words[:, 0] = idx % M.V
        qh = rng.integers(0, n_h, 4 * n_h).astype(np.int32)
        qt = rng.integers(0, M.V, 4 * n_h).astype(np.int32)
        frames.append([torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in (pool[idx], words, qh, qt)])
    sc = R.Scorer(M, weights(M, rng), R.Q_SIGN, 0, max_hist=300, max_query=1200,
                  cap_hist=4096, cap_query=8192, device="cuda:0")
    L = R.load()
    st = torch.cuda.Stream()
    sp = ctypes.c_void_p(st.cuda_stream)

    def buffers():
        out = []
        for hv, hw, qh, qt in frames:
            out.append({"scores": torch.full((qh.numel(),), float("nan"), device=dev),
                        "hnew": torch.full((hv.shape[0], M.H), float("nan"), device=dev),
                        "q_status": torch.zeros(qh.numel(), dtype=torch.uint8, device=dev)})
        return out

    def launch(bufs, lo, hi):
        for i in range(lo, hi):
            hv, hw, qh, qt = frames[i]
            fr = R.Frame(hv.shape[0], qh.numel(), hv.data_ptr(), hw.data_ptr(), qh.data_ptr(), qt.data_ptr())
            o = bufs[i]
            out = R.Out(o["scores"].data_ptr(), o["hnew"].data_ptr(), o["q_status"].data_ptr(), None, None, None, None)
            rc = L.rnnlm_score_frame(sc.ctx, ctypes.byref(fr), ctypes.byref(out), sp)
            assert rc == 0, L.rnnlm_last_error()

    with torch.cuda.stream(st):
        eager = buffers()
        sc.reset(st)
        launch(eager, 0, n_frames)
        torch.cuda.synchronize()
        ref_stats = sc.stats(st)
        graphed = buffers()
        sc.reset(st)
        launch(graphed, 0, warm)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=st):
            launch(graphed, warm, n_frames)
        for rep in range(3):
            for o in graphed[warm:]:
                for t in o.values():
                    t.zero_()
            sc.reset(st)
            launch(graphed, 0, warm)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for i in range(warm, n_frames):
                for k in ("scores", "hnew", "q_status"):
                    assert torch.equal(eager[i][k], graphed[i][k]), "replay %d frame %d: %s differs" % (rep, i, k)
            st_r = sc.stats(st)
            for k in ("queries", "computed", "score_hits", "gru_rows", "hist_hits"):
                assert st_r[k] == ref_stats[k], (rep, k, st_r[k], ref_stats[k])
    hits = sum(int((o["q_status"] == R.Q_SCORE_HIT).sum()) for o in eager[warm:])
    assert hits > 0 and ref_stats["gru_rows"] > 300
