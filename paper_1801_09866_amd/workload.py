"""Seeded synthetic workloads for frame-wise RNNLM query scoring.

This module only draws random numbers and arranges them into model weights
and per-frame query batches. It holds none of the scoring method's arithmetic
(no quantiser, hash, cache, GRU, NCE or MaxEnt code), so the CPU oracle and
the HIP library can both consume its output without sharing any computation.

What the paper's workloads look like (Sec. 2 and Sec. 3):
  * a decoder emits, per frame, LM queries = (history vector, next word);
    the history vector is a recurrent hidden state with elements in (-1, 1);
  * queries from one frame share histories (several candidate words per
    hypothesis), and the same histories recur over later frames;
  * the vocabulary is frequency-skewed (V = 200,000 in the experiments).

The history vectors here are produced by an elementwise softsign recurrence
over per-word random vectors, h <- softsign(alpha*h + u[word]), run over
Zipf-distributed word prefixes. It stands in for decoder GRU states: values
in (-1, 1), dominated by the most recent words, identical for identical
prefixes. Softsign needs only +,*,/ and abs, so the draws are bit-identical
on every machine (no libm transcendental is involved).

Everything is float32 on output; bf16 configs get their bf16 copies from the
library itself (round-to-nearest-even of these fp32 masters).
"""
from __future__ import annotations

import dataclasses
import numpy as np

ROOT_SEED = 180109866
BOS = 0  # word id 0 is the sentence start; never drawn as a word

# Quantisation modes (numbering shared with the C ABI header).
Q_EXACT, Q_SIGN, Q_SIGDIG = 0, 1, 2
F32, BF16 = 0, 1


@dataclasses.dataclass(frozen=True)
class ModelCfg:
    V: int
    E: int
    H: int
    L: int
    wdtype: int          # F32 or BF16 weights
    maxent_log2: int     # MaxEnt table has 2**maxent_log2 fp32 weights
    maxent_order: int    # n-gram orders 2..maxent_order feed the bypass


@dataclasses.dataclass(frozen=True)
class WorkloadCfg:
    name: str
    model: ModelCfg
    frames: int
    queries: int          # queries per frame
    hists: int            # distinct (fresh) histories per frame
    pool: int             # distinct prefixes in the history pool
    zipf_s: float
    layout: str           # 'cover', 'fanout', 'fanout_repeat', 'none'
    qmodes: tuple         # ((qmode, qdigits), ...) runs of this workload
    repeat_frac: float = 0.0
    max_hist: int = 0     # upper bound on history records in one frame
    cap_hist: int = 0     # history-cache capacity (entries)
    cap_query: int = 0    # score-cache capacity (entries)
    seed_index: int = 0


def _cfg(name, model, frames, queries, hists, pool, zipf_s, layout, qmodes,
         repeat_frac=0.0, max_hist=None, cap_hist=None, cap_query=None,
         seed_index=0):
    max_hist = max_hist or hists
    return WorkloadCfg(name, model, frames, queries, hists, pool, zipf_s,
                       layout, tuple(qmodes), repeat_frac, max_hist,
                       cap_hist or 2 * pool, cap_query or 4 * frames * max(queries, 1),
                       seed_index)


CONFIGS = {
    # V=10k, E=128, H=128, 3-gram MaxEnt (orders 2,3), 100 x 64 queries,
    # 16 distinct histories per frame, sign-only compression.
    "tiny": _cfg("tiny", ModelCfg(10_000, 128, 128, 1, F32, 20, 3),
                 100, 64, 16, 512, 1.0, "cover", [(Q_SIGN, 0)], seed_index=0),
    # V=100k, E=256, H=512, 2^24 MaxEnt, 1000 x 512 queries from 128
    # histories with fan-out U{1..8}; 3 significant digits.
    "medium": _cfg("medium", ModelCfg(100_000, 256, 512, 1, F32, 24, 4),
                   1000, 512, 128, 16_384, 1.0, "fanout", [(Q_SIGDIG, 3)],
                   cap_query=1 << 20, seed_index=1),
    # V=200k, E=512, H=1024, 2^26 MaxEnt with 2-,3-,4-grams; 2000 x 2048
    # queries; 30% of each frame's queries repeat the previous frame's
    # (history, word) pairs; run with sign and with 2 significant digits.
    "large": _cfg("large", ModelCfg(200_000, 512, 1024, 1, F32, 26, 4),
                  2000, 2048, 512, 32_768, 1.0, "fanout_repeat",
                  [(Q_SIGN, 0), (Q_SIGDIG, 2)], repeat_frac=0.30,
                  max_hist=1152, cap_query=1 << 22, seed_index=2),
    # Same vocabulary, 2-layer GRU with bf16 weights (fp32 accumulate);
    # 500 x 8192 queries from 1024 histories, Zipf s=1.1; sign-only.
    "large_bf16": _cfg("large_bf16", ModelCfg(200_000, 512, 1024, 2, BF16, 26, 4),
                       500, 8192, 1024, 32_768, 1.1, "cover", [(Q_SIGN, 0)],
                       cap_query=1 << 22, seed_index=3),
    # Full-vocabulary normaliser check: 200 frames of 256 distinct histories,
    # no queries; h' from the GRU step, then logsumexp over all V rows.
    "check": _cfg("check", ModelCfg(200_000, 512, 1024, 1, F32, 26, 4),
                  200, 0, 256, 8_192, 1.0, "none", [(Q_EXACT, 0)],
                  cap_query=1024, seed_index=4),
}


# --------------------------------------------------------------------------
# weights
# --------------------------------------------------------------------------

def _normal(rng, shape, sigma):
    return rng.standard_normal(shape, dtype=np.float32) * np.float32(sigma)


def make_weights(model: ModelCfg, seed_index: int, sigma_w=0.05, sigma_me=0.01):
    """fp32 master weights, all ~N(0, sigma^2), drawn from fixed child seeds.

    Layout (row-major): emb [V, E]; W_ih[l] [3H, Kx] with Kx = E for the first
    layer and H above; W_hh[l] [3H, H]; b_ih[l] [3H]; U_out [V, H];
    b_out [V]; maxent [2**maxent_log2]. Gate blocks of W_ih, W_hh and b_ih
    are ordered (reset, update, candidate).
    """
    ss = np.random.SeedSequence([ROOT_SEED, seed_index, 0])
    kids = ss.spawn(7)
    g = [np.random.default_rng(k) for k in kids]
    V, E, H, L = model.V, model.E, model.H, model.L
    w = {
        "emb": _normal(g[0], (V, E), sigma_w),
        "W_ih": [_normal(g[1], (3 * H, E if l == 0 else H), sigma_w) for l in range(L)],
        "W_hh": [_normal(g[2], (3 * H, H), sigma_w) for l in range(L)],
        "b_ih": [_normal(g[3], (3 * H,), sigma_w) for l in range(L)],
        "U_out": _normal(g[4], (V, H), sigma_w),
        "b_out": _normal(g[5], (V,), sigma_w),
        "maxent": _normal(g[6], (1 << model.maxent_log2,), sigma_me),
    }
    return w


# --------------------------------------------------------------------------
# words, history pool, frames
# --------------------------------------------------------------------------

class Zipf:
    """Word ids 1..V-1 with P(r) proportional to r^-s (id = frequency rank)."""

    def __init__(self, V, s):
        r = np.arange(1, V, dtype=np.float64)
        p = r ** (-s)
        self.cdf = np.cumsum(p) / p.sum()

    def draw(self, rng, n):
        u = rng.random(n)
        return (np.searchsorted(self.cdf, u, side="right") + 1).astype(np.int32)


@dataclasses.dataclass
class HistoryPool:
    vec: np.ndarray     # [P, L*H] fp32, layer-major
    words: np.ndarray   # [P, 3] int32: (w-1, w-2, w-3); w-1 is the GRU input


def make_pool(model: ModelCfg, n_prefix: int, zipf: Zipf, rng,
              alpha=0.5, sigma_u=0.6, table_rows=4096):
    """History pool from distinct Zipf prefixes (lengths U{1..20}).

    Prefix (w1..wl): the history is the recurrence state after consuming
    (BOS, w1, ..., w_{l-1}); the word about to be fed to the LM step is
    w-1 = w_l, with context w-2 = w_{l-1}, w-3 = w_{l-2} (BOS-padded).
    """
    H, L = model.H, model.L
    seen = set()
    prefixes = []
    while len(prefixes) < n_prefix:
        need = n_prefix - len(prefixes)
        lens = rng.integers(1, 21, size=need)
        words = zipf.draw(rng, int(lens.sum()))
        off = 0
        for ln in lens:
            p = tuple(int(x) for x in words[off:off + ln])
            off += ln
            if p not in seen:
                seen.add(p)
                prefixes.append(p)
    P = len(prefixes)
    maxlen = 20
    seq = np.zeros((P, maxlen), dtype=np.int64)   # consumed words, BOS first
    nsteps = np.zeros(P, dtype=np.int64)
    words3 = np.zeros((P, 3), dtype=np.int32)
    for i, p in enumerate(prefixes):
        consumed = (BOS,) + p[:-1]
        seq[i, :len(consumed)] = consumed
        nsteps[i] = len(consumed)
        full = (BOS, BOS) + p
        words3[i] = (full[-1], full[-2], full[-3])
    # per-word drive vectors (one table per layer), softsign recurrence
    tabs = [_normal(rng, (table_rows, H), sigma_u) for _ in range(L)]
    states = [np.zeros((P, H), dtype=np.float32) for _ in range(L)]
    a = np.float32(alpha)
    one = np.float32(1.0)
    for t in range(maxlen):
        act = nsteps > t
        if not act.any():
            break
        idx = np.nonzero(act)[0]
        rows = seq[idx, t] % table_rows
        below = None
        for l in range(L):
            s = a * states[l][idx] + tabs[l][rows]
            if below is not None:
                s = s + a * below
            s = s / (one + np.abs(s))
            states[l][idx] = s
            below = s
    vec = np.concatenate(states, axis=1) if L > 1 else states[0]
    return HistoryPool(np.ascontiguousarray(vec, dtype=np.float32), words3)


@dataclasses.dataclass
class Frame:
    pool_idx: np.ndarray   # [n_hist] int64 indices into the pool
    hist_words: np.ndarray  # [n_hist, 3] int32
    q_hist: np.ndarray     # [n_q] int32 indices into this frame's histories
    q_tgt: np.ndarray      # [n_q] int32 target word ids

    @property
    def n_hist(self):
        return len(self.pool_idx)

    @property
    def n_query(self):
        return len(self.q_hist)


def _repair(rng, f, total, lo=1, hi=8):
    """Adjust fan-outs f (each in [lo, hi]) until they sum to `total`."""
    d = int(f.sum()) - total
    if d > 0:
        units = np.repeat(np.arange(len(f)), f - lo)
        pick = rng.choice(len(units), d, replace=False)
        f = f - np.bincount(units[pick], minlength=len(f))
    elif d < 0:
        units = np.repeat(np.arange(len(f)), hi - f)
        pick = rng.choice(len(units), -d, replace=False)
        f = f + np.bincount(units[pick], minlength=len(f))
    return f


def make_frames(cfg: WorkloadCfg, pool: HistoryPool, zipf: Zipf, rng, n_frames=None):
    n_frames = cfg.frames if n_frames is None else min(n_frames, cfg.frames)
    P = len(pool.vec)
    frames = []
    prev = None
    for f in range(n_frames):
        fresh = rng.choice(P, cfg.hists, replace=False)
        if cfg.layout == "none":
            q_hist = np.zeros(0, np.int32)
            q_tgt = np.zeros(0, np.int32)
            pidx = fresh
        elif cfg.layout == "cover":
            nh = cfg.hists
            extra = rng.integers(0, nh, size=cfg.queries - nh)
            q_hist = np.concatenate([np.arange(nh), extra]).astype(np.int32)
            q_tgt = zipf.draw(rng, cfg.queries)
            perm = rng.permutation(cfg.queries)
            q_hist, q_tgt = q_hist[perm], q_tgt[perm]
            pidx = fresh
        else:
            R = 0
            if cfg.layout == "fanout_repeat" and prev is not None:
                R = int(round(cfg.repeat_frac * cfg.queries))
                R = min(R, prev[0].size)
            fan = rng.integers(1, 9, size=cfg.hists)
            fan = _repair(rng, fan, cfg.queries - R)
            q_hist = np.repeat(np.arange(cfg.hists), fan).astype(np.int32)
            q_tgt = zipf.draw(rng, len(q_hist))
            pidx = list(fresh)
            if R:
                ppool, ptgt = prev
                pick = rng.choice(ppool.size, R, replace=False)
                where = {int(p): i for i, p in enumerate(pidx)}
                rh = np.empty(R, np.int32)
                for j, p in enumerate(ppool[pick]):
                    p = int(p)
                    if p not in where:
                        where[p] = len(pidx)
                        pidx.append(p)
                    rh[j] = where[p]
                q_hist = np.concatenate([q_hist, rh])
                q_tgt = np.concatenate([q_tgt, ptgt[pick]])
            pidx = np.asarray(pidx, dtype=np.int64)
            perm = rng.permutation(len(q_hist))
            q_hist, q_tgt = q_hist[perm], q_tgt[perm]
        pidx = np.asarray(pidx, dtype=np.int64)
        frames.append(Frame(pidx, pool.words[pidx], q_hist.astype(np.int32),
                            q_tgt.astype(np.int32)))
        # (pool index, target) pairs of this frame, for next frame's repeats
        prev = (pidx[q_hist], q_tgt.copy())
    return frames


@dataclasses.dataclass
class Workload:
    cfg: WorkloadCfg
    weights: dict
    pool: HistoryPool
    frames: list

    def hist_vec(self, frame: Frame) -> np.ndarray:
        return self.pool.vec[frame.pool_idx]


def make_workload(name: str, n_frames=None, pool_size=None, model=None,
                  with_weights=True) -> Workload:
    """Build config `name` (weights, pool, first `n_frames` frames).

    `pool_size` and `model` override the config for reduced test cases.
    """
    cfg = CONFIGS[name]
    if model is not None:
        cfg = dataclasses.replace(cfg, model=model)
    if pool_size is not None:
        cfg = dataclasses.replace(cfg, pool=pool_size,
                                  hists=min(cfg.hists, pool_size),
                                  max_hist=max(min(cfg.max_hist, 2 * pool_size),
                                               min(cfg.hists, pool_size)))
    m = cfg.model
    ss = np.random.SeedSequence([ROOT_SEED, cfg.seed_index, 1])
    rpool, rframes = [np.random.default_rng(k) for k in ss.spawn(2)]
    zipf = Zipf(m.V, cfg.zipf_s)
    pool = make_pool(m, cfg.pool, zipf, rpool)
    frames = make_frames(cfg, pool, zipf, rframes, n_frames)
    w = make_weights(m, cfg.seed_index) if with_weights else None
    return Workload(cfg, w, pool, frames)


# --------------------------------------------------------------------------
# decode-loop plans: frames whose histories are the previous frames' outputs
# --------------------------------------------------------------------------
@dataclasses.dataclass
class DecodeFrame:
    """One frame of a decode loop over a beam of hypotheses.

    Hypothesis j of this frame has words (w-1, w-2, w-3) = words[j] and
    queries its `fanout` candidate next words cand[j]. Its history vector is,
    for frame 0, row j of the initial histories; later, if advanced[j], the
    GRU output (h') of hypothesis prev[j] of the previous frame, else the same
    history vector as hypothesis prev[j] of the previous frame (a hypothesis
    that stays, whose queries repeat, as between word ends in a decoder).
    """
    words: np.ndarray      # [B, 3] int32
    cand: np.ndarray       # [B, F] int32
    prev: np.ndarray       # [B] int64 index into the previous frame (-1 in frame 0)
    advanced: np.ndarray   # [B] bool

    @property
    def q_hist(self):
        return np.repeat(np.arange(len(self.words), dtype=np.int32), self.cand.shape[1])

    @property
    def q_tgt(self):
        return self.cand.reshape(-1).astype(np.int32)


def decode_plan(V, beam, fanout, n_frames, stay, zipf_s, seed, init_words, shared=0, focus=0.0):
    """Seeded beam evolution, independent of any score: each frame keeps
    round(stay * beam) hypotheses (chosen uniformly) and fills the rest of
    the beam with distinct (hypothesis, candidate slot) extensions (chosen
    uniformly); new hypotheses draw fresh Zipf candidates. init_words [beam, 3]
    are the words of the initial histories.

    shared > 0 models hypotheses that compete for the same stretch of speech:
    each frame draws `shared` Zipf words and every new hypothesis takes its
    candidates from them. The first of them is the frame's spoken word: it
    is every new hypothesis' first candidate, and a fraction `focus` of the
    frame's extensions take it (from distinct parents). Paths that differ
    only in older words then continue on the same recent words, as in a
    decoding lattice."""
    rng = np.random.default_rng(seed)
    zipf = Zipf(V, zipf_s)
    spoken = [None]

    def draw_cand(n):
        if shared <= 0:
            return zipf.draw(rng, n * fanout).reshape(n, fanout)
        pool = np.unique(zipf.draw(rng, shared))
        while len(pool) < fanout:
            pool = np.unique(np.concatenate([pool, zipf.draw(rng, shared)]))
        spoken[0] = int(pool[rng.integers(len(pool))])
        rest = pool[pool != spoken[0]]
        return np.stack([np.concatenate([[spoken[0]], rng.choice(rest, fanout - 1, replace=False)])
                         for _ in range(n)]).astype(np.int32)

    words = np.asarray(init_words, dtype=np.int32).copy()
    cand = draw_cand(beam)
    frames = [DecodeFrame(words, cand, np.full(beam, -1, np.int64), np.zeros(beam, bool))]
    n_keep = int(round(stay * beam))
    for _ in range(1, n_frames):
        keep = np.sort(rng.choice(beam, n_keep, replace=False))
        n_adv = beam - n_keep
        n_foc = int(round(focus * n_adv)) if shared > 0 else 0
        if n_foc:
            # extensions by the spoken word: distinct parents whose candidates hold it
            holders = np.nonzero((cand == spoken[0]).any(axis=1))[0]
            n_foc = min(n_foc, len(holders))
            fpar = np.sort(rng.choice(holders, n_foc, replace=False))
            fslot = np.array([int(np.nonzero(cand[i] == spoken[0])[0][0]) for i in fpar], dtype=np.int64)
            taken = set((fpar * fanout + fslot).tolist())
            free = np.array([e for e in range(beam * fanout) if e not in taken])
            ext = np.sort(np.concatenate([fpar * fanout + fslot, rng.choice(free, n_adv - n_foc, replace=False)]))
        else:
            ext = np.sort(rng.choice(beam * fanout, n_adv, replace=False))
        par, slot = ext // fanout, ext % fanout
        w_new = np.stack([cand[par, slot], words[par, 0], words[par, 1]], axis=1).astype(np.int32)
        c_new = draw_cand(len(par))
        words = np.concatenate([words[keep], w_new])
        cand = np.concatenate([cand[keep], c_new])
        prev = np.concatenate([keep, par]).astype(np.int64)
        adv = np.concatenate([np.zeros(n_keep, bool), np.ones(len(par), bool)])
        frames.append(DecodeFrame(words, cand, prev, adv))
    return frames
