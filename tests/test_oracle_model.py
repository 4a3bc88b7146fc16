"""Pins of the oracle's GRU step, NCE score, MaxEnt hash and normaliser.

GRU (Sec. 2.1) against torch.nn.GRUCell in float64 (with the recurrent bias
zeroed, which leaves exactly six matrices and three bias vectors), plus
closed forms and the gate invariants; NCE (Sec. 2.2) by brute force on a tiny
vocabulary; the normaliser against closed forms and scipy's logsumexp;
SplitMix64 against its published seed-0 outputs.
"""
import os

import numpy as np
import pytest
import scipy.special
import torch

from oracle import (gru_step, hist_key_hash, log_normalizer, log_normalizer_maxent, maxent_index,
                    mix64, nce_score)

PHI = 0x9E3779B97F4A7C15
M64 = (1 << 64) - 1


def test_mix64_published_splitmix64_vectors():
    """SplitMix64 seeded with 0 returns mix(PHI), mix(2 PHI), mix(3 PHI);
    the published outputs are in tests/golden/splitmix64.txt."""
    path = os.path.join(os.path.dirname(__file__), "golden", "splitmix64.txt")
    want = {}
    for line in open(path):
        if line.strip() and not line.startswith("#"):
            k, v = line.split()
            want[int(k)] = int(v, 16)
    assert sorted(want) == [1, 2, 3]
    got = mix64(np.array([(k * PHI) & M64 for k in sorted(want)], dtype=np.uint64))
    assert [int(v) for v in got] == [want[k] for k in sorted(want)]


def _mix_int(z):
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def test_hist_key_hash_against_python_integers():
    """numpy uint64 wrapping arithmetic vs unbounded Python ints + masks."""
    rng = np.random.default_rng(11)
    words = rng.integers(0, 2 ** 63, size=(6, 5), dtype=np.int64).astype(np.uint64) * np.uint64(2) + np.uint64(1)
    w1 = rng.integers(0, 200000, 6)
    seed = 0x1234_5678_9ABC_DEF0
    got = hist_key_hash(words, w1, seed)
    for i in range(6):
        s = 0
        for j in range(5):
            s = (s + _mix_int(int(words[i, j]) ^ (((j + 1) * PHI) & M64))) & M64
        want = _mix_int(seed ^ s ^ _mix_int(int(w1[i]) + 1))
        assert int(got[i]) == want


def test_hist_key_hash_depends_on_position_and_word():
    w = np.array([[1, 2], [2, 1]], dtype=np.uint64)
    h = hist_key_hash(w, np.array([5, 5]), 0)
    assert h[0] != h[1]
    h2 = hist_key_hash(w[:1], np.array([6]), 0)
    assert h2[0] != h[0]


def test_maxent_index_against_python_integers_and_range():
    rng = np.random.default_rng(5)
    ctx = [rng.integers(0, 200000, 50) for _ in range(3)]
    tgt = rng.integers(1, 200000, 50)
    for order in (2, 3, 4):
        idx = maxent_index(order, ctx, tgt, 26)
        assert idx.min() >= 0 and idx.max() < (1 << 26)
        for q in range(50):
            g = _mix_int((order * PHI) & M64)
            for c in range(order - 1):
                g = _mix_int(g ^ (int(ctx[c][q]) + 1))
            g = _mix_int(g ^ (int(tgt[q]) + 1))
            assert int(idx[q]) == g & ((1 << 26) - 1)
    # different orders of the same words land in different slots
    a = maxent_index(2, ctx, tgt, 26)
    b = maxent_index(3, ctx, tgt, 26)
    assert np.mean(a == b) < 0.05


def _rand_gru(rng, Kx, H, scale=0.3):
    return (rng.standard_normal((3 * H, Kx)) * scale, rng.standard_normal((3 * H, H)) * scale,
            rng.standard_normal(3 * H) * scale)


def test_gru_matches_torch_grucell_float64():
    rng = np.random.default_rng(0)
    Kx, H, M = 24, 16, 9
    W_ih, W_hh, b = _rand_gru(rng, Kx, H)
    x = rng.standard_normal((M, Kx))
    h = np.tanh(rng.standard_normal((M, H)))
    cell = torch.nn.GRUCell(Kx, H).double()
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(W_ih))
        cell.weight_hh.copy_(torch.from_numpy(W_hh))
        cell.bias_ih.copy_(torch.from_numpy(b))
        cell.bias_hh.zero_()
        want = cell(torch.from_numpy(x), torch.from_numpy(h)).numpy()
    got = gru_step(x, h, W_ih, W_hh, b)
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-14)


def test_gru_closed_forms_and_invariants():
    rng = np.random.default_rng(1)
    Kx, H, M = 8, 6, 5
    x = rng.standard_normal((M, Kx))
    h = np.tanh(rng.standard_normal((M, H)))
    z3 = np.zeros((3 * H, Kx)), np.zeros((3 * H, H)), np.zeros(3 * H)
    # all-zero parameters: r = z = 1/2, n = 0, h' = h/2 exactly
    assert np.array_equal(gru_step(x, h, *z3), h / 2)
    # saturated update gate: z == 1 exactly, h' == h bitwise
    W_ih, W_hh, b = _rand_gru(rng, Kx, H, 0.1)
    b = b.copy()
    b[H:2 * H] = 100.0
    assert np.array_equal(gru_step(x, h, W_ih, W_hh, b), h)
    # moderate pre-activations: output strictly inside (-1, 1)
    W_ih, W_hh, b = _rand_gru(rng, Kx, H, 0.5)
    out = gru_step(x, h, W_ih, W_hh, b)
    assert np.all(np.abs(out) < 1)
    # z = 0 (b_z = -100) and no recurrence: h' = tanh(W_in x + b_n)
    W_hh0 = np.zeros_like(W_hh)
    b2 = b.copy()
    b2[H:2 * H] = -100.0
    out = gru_step(x, h, W_ih, W_hh0, b2)
    np.testing.assert_allclose(out, np.tanh(x @ W_ih[2 * H:].T + b2[2 * H:]), rtol=1e-14)


def test_nce_score_brute_force_tiny_vocab():
    rng = np.random.default_rng(2)
    V, H = 16, 8
    U = rng.standard_normal((V, H)).astype(np.float32)
    b = rng.standard_normal(V).astype(np.float32)
    h = rng.standard_normal(H)
    for t in range(V):
        want = sum(float(U[t, j]) * h[j] for j in range(H)) + float(b[t])
        assert abs(nce_score(h, U, b, t) - want) < 1e-12
    # one-hot output row, zero bias: score is the selected element of h
    U1 = np.zeros((V, H), np.float32)
    U1[3, 5] = 1
    assert nce_score(h, U1, np.zeros(V, np.float32), 3) == h[5]


def test_log_normalizer_closed_forms_and_scipy():
    rng = np.random.default_rng(4)
    V, H, n = 1000, 16, 3
    h = np.tanh(rng.standard_normal((n, H)))
    # zero model: every logit 0, Z = V
    z = log_normalizer(h, np.zeros((V, H), np.float32), np.zeros(V, np.float32))
    np.testing.assert_allclose(z, np.log(V), rtol=0, atol=1e-12)
    assert abs(log_normalizer(h[:1, :2], np.zeros((200000, 2), np.float32),
                              np.zeros(200000, np.float32), chunk=65536)[0]
               - 12.206072645530174) < 1e-12
    # constant rows c*1: logits all equal c*sum(h)
    c = 0.25
    z = log_normalizer(h, np.full((V, H), c, np.float32), np.zeros(V, np.float32), chunk=300)
    np.testing.assert_allclose(z, c * h.sum(1) + np.log(V), rtol=1e-14)
    U = rng.standard_normal((V, H)).astype(np.float32)
    b = rng.standard_normal(V).astype(np.float32)
    want = scipy.special.logsumexp(h @ U.astype(np.float64).T + b.astype(np.float64), axis=1)
    np.testing.assert_allclose(log_normalizer(h, U, b, chunk=128), want, rtol=1e-14)


def test_log_normalizer_maxent_closed_forms_and_brute_force():
    """MaxEnt-inclusive normaliser: zero weights reduce it to the plain one, a
    constant table shifts every logit by (orders) * c, and a direct double
    loop over a tiny vocabulary (math.fsum of exp) agrees."""
    import math
    rng = np.random.default_rng(9)
    V, H, n, log2 = 40, 6, 5, 7
    h = np.tanh(rng.standard_normal((n, H)))
    U = rng.standard_normal((V, H)).astype(np.float32)
    b = rng.standard_normal(V).astype(np.float32)
    words = rng.integers(0, V, (n, 3))
    lam = (rng.standard_normal(1 << log2) * 0.5).astype(np.float32)
    plain = log_normalizer(h, U, b)
    np.testing.assert_allclose(log_normalizer_maxent(h, U, b, np.zeros(1 << log2, np.float32), words, 4, log2),
                               plain, rtol=0, atol=1e-13)
    np.testing.assert_allclose(log_normalizer_maxent(h, U, b, np.full(1 << log2, 0.25, np.float32), words, 4, log2),
                               plain + 3 * 0.25, rtol=1e-14)
    got = log_normalizer_maxent(h, U, b, lam, words, 4, log2)
    for i in range(n):
        terms = []
        for v in range(V):
            a = sum(float(U[v, j]) * h[i, j] for j in range(H)) + float(b[v])
            for o in range(2, 5):
                a += float(lam[int(maxent_index(o, [int(words[i, c]) for c in range(o - 1)], v, log2))])
            terms.append(a)
        m = max(terms)
        want = m + math.log(math.fsum(math.exp(t - m) for t in terms))
        assert abs(got[i] - want) < 1e-12
    with pytest.raises(ValueError):
        log_normalizer_maxent(h, U, b, lam, np.full((n, 3), V), 4, log2)
