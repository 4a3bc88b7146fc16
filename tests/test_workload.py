"""The seeded generator: determinism, ranges, and the frame structure of each config."""
import numpy as np

from paper_1801_09866_amd.workload import CONFIGS, make_workload


def test_generator_is_deterministic():
    a = make_workload("tiny", n_frames=5)
    b = make_workload("tiny", n_frames=5)
    assert np.array_equal(a.pool.vec, b.pool.vec)
    assert np.array_equal(a.weights["U_out"], b.weights["U_out"])
    for fa, fb in zip(a.frames, b.frames):
        assert np.array_equal(fa.q_tgt, fb.q_tgt) and np.array_equal(fa.pool_idx, fb.pool_idx)


def test_tiny_frames_cover_all_histories():
    w = make_workload("tiny", n_frames=10)
    cfg = w.cfg
    assert np.all(np.abs(w.pool.vec) < 1)
    for f in w.frames:
        assert f.n_hist == cfg.hists and f.n_query == cfg.queries
        assert len(set(f.pool_idx.tolist())) == cfg.hists
        assert set(f.q_hist.tolist()) == set(range(cfg.hists))
        assert f.q_tgt.min() >= 1 and f.q_tgt.max() < cfg.model.V


def test_large_frames_repeat_thirty_percent_of_previous_pairs():
    w = make_workload("large", n_frames=4, pool_size=4096, with_weights=False)
    cfg = w.cfg
    prev = None
    for i, f in enumerate(w.frames):
        assert f.n_query == cfg.queries
        assert f.n_hist <= cfg.max_hist
        pairs = set(zip(f.pool_idx[f.q_hist].tolist(), f.q_tgt.tolist()))
        if prev is not None:
            assert len(pairs & prev) >= 0.25 * cfg.queries
        prev = pairs


def test_medium_fanout_sums_and_bounds():
    w = make_workload("medium", n_frames=3, pool_size=2048, with_weights=False)
    for f in w.frames:
        fan = np.bincount(f.q_hist, minlength=f.n_hist)
        assert fan.sum() == 512 and fan.min() >= 1 and fan.max() <= 8


def test_all_configs_are_well_formed():
    for name, c in CONFIGS.items():
        m = c.model
        assert m.H % 64 == 0 and m.E % 64 == 0
        assert 1 <= m.L <= 2 and 1 <= m.maxent_order <= 4
        assert c.max_hist >= c.hists
