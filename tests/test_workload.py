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


def test_decode_plan_is_seeded_and_well_formed():
    from paper_1801_09866_amd.workload import decode_plan
    init = np.arange(30, dtype=np.int32).reshape(10, 3) + 1
    a = decode_plan(500, 10, 4, 6, 0.6, 1.0, 9, init)
    b = decode_plan(500, 10, 4, 6, 0.6, 1.0, 9, init)
    assert len(a) == 6
    for fa, fb in zip(a, b):
        for key in ("words", "cand", "prev", "advanced"):
            assert np.array_equal(getattr(fa, key), getattr(fb, key))
    assert np.array_equal(a[0].words, init) and np.all(a[0].prev == -1)
    for t in range(1, 6):
        f, p = a[t], a[t - 1]
        assert f.words.shape == (10, 3) and f.cand.shape == (10, 4)
        assert f.advanced.sum() == 4 and np.all((0 <= f.prev) & (f.prev < 10))
        for j in range(10):
            i = f.prev[j]
            if f.advanced[j]:   # extended by one of its parent's candidates, words shifted
                assert f.words[j, 0] in p.cand[i] and f.words[j, 1] == p.words[i, 0] and f.words[j, 2] == p.words[i, 1]
            else:               # stays: same words and candidates, so its queries repeat
                assert np.array_equal(f.words[j], p.words[i]) and np.array_equal(f.cand[j], p.cand[i])
        ext = {(int(f.prev[j]), int(f.words[j, 0])) for j in range(10) if f.advanced[j]}
        assert len(ext) == 4   # distinct extensions
    assert np.array_equal(a[1].q_hist, np.repeat(np.arange(10), 4))
