"""Plain double-precision oracle of frame-wise RNNLM query scoring.

TEST INFRASTRUCTURE ONLY: used by tests/, the smoke check and the
cpu_baseline leg of the benchmark; the HIP library never imports it.

Paper: Lee et al., arXiv 1801.09866. The paper prints no equations; every
formula below is the reading of its prose that this project adopts, and each
reading is named where it is used.

Per frame, in order (one call of ``Oracle.score_frame``):
  1. quantise each history vector                      (Sec. 3, Table 1)
  2. history key = (quantised history, GRU input word)  (Sec. 3, Fig. 2)
  3. de-duplicate histories in the frame, probe the history cache
  4. query key = (history key, MaxEnt context words, target word),
     de-duplicate queries, probe the LM-query (score) cache (Sec. 2.4, Fig. 1)
  5. one GRU step per history key not in the cache       (Sec. 2.1)
  6. unnormalised NCE score + hashed n-gram MaxEnt terms  (Sec. 2.2, 2.3)
  7. insert the frame's new keys into the two caches     (Sec. 2.4, Sec. 3)

Parity unpinned: the compositions in ``hist_key_hash`` and ``maxent_index``
are this implementation's own definitions, because the paper leaves both
hashes unspecified (Sec. 2.3, Sec. 3). Only their building block, the
SplitMix64 finaliser ``mix64``, is pinned, by its published outputs; nothing
outside this file fixes how the finaliser is combined.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from fractions import Fraction

import numpy as np

Q_EXACT, Q_SIGN, Q_SIGDIG = 0, 1, 2
# history statuses
H_REP, H_DUP, HC_HIT = 0, 1, 2
# query statuses
Q_COMPUTED, Q_DUP, Q_SCORE_HIT = 0, 1, 2

MASK64 = (1 << 64) - 1
PHI = 0x9E3779B97F4A7C15  # 2^64 / golden ratio, the SplitMix64 increment

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "_sigdig.so")
_lib = None


def build_c(force=False):
    """Compile the oracle's C part (the exact decimal quantiser) with gcc."""
    src = os.path.join(_HERE, "sigdig.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-shared", "-fPIC",
                               src, "-o", tmp])
        os.replace(tmp, _SO)
    return _SO


def _sigdig_lib():
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(build_c())
        _lib.oracle_sigdig_codes.restype = ctypes.c_int
        _lib.oracle_sigdig_codes.argtypes = [ctypes.c_void_p, ctypes.c_int64,
                                             ctypes.c_int, ctypes.c_void_p]
    return _lib


# --------------------------------------------------------------------------
# hashing: SplitMix64 finaliser (Steele, Lea, Flood, OOPSLA 2014)
# --------------------------------------------------------------------------

def mix64(z):
    """SplitMix64 output mix of 64-bit words (numpy uint64, wrapping)."""
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        z = z ^ (z >> np.uint64(31))
    return z


def hist_key_hash(words, w1, seed):
    """64-bit hash of history keys (code words [n, W] uint64, input word [n]).

    t_j = mix64(c_j xor (j+1)*PHI); h = mix64(seed xor sum_j t_j xor
    mix64(w1 + 1)), sums mod 2^64. Only used to place keys in tables; key
    equality is always decided on the full codes.
    """
    words = np.asarray(words, dtype=np.uint64)
    n, W = words.shape
    with np.errstate(over="ignore"):
        j1 = (np.arange(1, W + 1, dtype=np.uint64) * np.uint64(PHI))
        t = mix64(words ^ j1[None, :])
        s = np.sum(t, axis=1, dtype=np.uint64)
        wterm = mix64(np.asarray(w1, dtype=np.int64).astype(np.uint64) + np.uint64(1))
        return mix64(np.uint64(seed) ^ s ^ wterm)


def maxent_index(order, ctx, tgt, log2):
    """Slot of the order-`order` n-gram (ctx[0]=w-1, ctx[1]=w-2, ...; tgt).

    Sec. 2.3 names a hash-based MaxEnt table without giving the hash; this
    project uses g = mix64(order*PHI), then g = mix64(g xor (w+1)) for the
    order-1 context words from the most recent back, then for the target,
    and keeps the low `log2` bits. Works on scalars or aligned arrays.
    """
    with np.errstate(over="ignore"):
        g = mix64(np.uint64(order) * np.uint64(PHI))
        for i in range(order - 1):
            c = np.asarray(ctx[i], dtype=np.int64).astype(np.uint64)
            g = mix64(g ^ (c + np.uint64(1)))
        t = np.asarray(tgt, dtype=np.int64).astype(np.uint64)
        g = mix64(g ^ (t + np.uint64(1)))
    return (g & np.uint64((1 << log2) - 1)).astype(np.int64)


# --------------------------------------------------------------------------
# quantisation (Sec. 3)
# --------------------------------------------------------------------------

def quantize(x, mode, k=0):
    """Quantise fp32 history elements; returns per-element codes.

    EXACT  (Table 1 "(baseline)"): the fp32 bit pattern, -0 made +0 -> uint32.
    SIGN   (Sec. 3 "only the signs"): 1 where x < 0, else 0 (+0, -0 -> +1)
           -> bool per element.
    SIGDIG (Sec. 3 rounding; k significant digits, ties away from zero)
           -> uint16 code, see sigdig.c for the layout.
    Raises ValueError for non-finite input, or |x| > 1 under SIGDIG.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    if not np.all(np.isfinite(x)):
        raise ValueError("non-finite history element")
    if mode == Q_EXACT:
        b = x.view(np.uint32).copy()
        b[b == np.uint32(0x80000000)] = 0
        return b
    if mode == Q_SIGN:
        return x < 0
    if mode == Q_SIGDIG:
        out = np.empty(x.shape, dtype=np.uint16)
        rc = _sigdig_lib().oracle_sigdig_codes(x.ctypes.data, x.size, int(k),
                                               out.ctypes.data)
        if rc:
            raise ValueError("history element outside [-1, 1] for decimal rounding")
        return out
    raise ValueError("bad quantisation mode")


def code_words(codes, mode):
    """Pack per-element codes of [n, D] into little-endian uint64 words.

    SIGN: element i -> bit i%64 of word i//64; SIGDIG: 4 codes per word,
    element 4w+t in bits 16t..16t+15; EXACT: 2 codes per word, 32t..32t+31.
    """
    codes = np.asarray(codes)
    n, D = codes.shape
    if mode == Q_SIGN:
        per, bits = 64, 1
    elif mode == Q_SIGDIG:
        per, bits = 4, 16
    else:
        per, bits = 2, 32
    if D % per:
        raise ValueError("vector length must be a multiple of %d" % per)
    c = codes.astype(np.uint64).reshape(n, D // per, per)
    shifts = (np.arange(per, dtype=np.uint64) * np.uint64(bits))
    return np.bitwise_or.reduce(c << shifts[None, None, :], axis=2)


def dequantize_exact(code, mode, k=0):
    """Exact rational value a single code stands for (tests only)."""
    if mode == Q_SIGN:
        return Fraction(-1 if code else 1)
    if mode == Q_EXACT:
        return Fraction(float(np.array(code, dtype=np.uint32).view(np.float32)))
    code = int(code)
    if code == 0:
        return Fraction(0)
    neg = code >> 15
    e = ((code >> 10) & 31) - 20
    m = code & 1023
    v = Fraction(m) * Fraction(10) ** (e - k + 1)
    return -v if neg else v


def dequantize(codes, mode, k=0):
    """fp32 value of each code: correctly rounded from the exact decimal."""
    codes = np.asarray(codes)
    if mode == Q_SIGN:
        return np.where(codes, np.float32(-1), np.float32(1)).astype(np.float32)
    if mode == Q_EXACT:
        return codes.astype(np.uint32).view(np.float32)
    out = np.empty(codes.shape, np.float32)
    flat = out.reshape(-1)
    for i, c in enumerate(codes.reshape(-1)):
        c = int(c)
        if c == 0:
            flat[i] = 0.0
            continue
        e = ((c >> 10) & 31) - 20
        s = "%s%de%d" % ("-" if c >> 15 else "", c & 1023, e - k + 1)
        flat[i] = np.float32(s)   # numpy parses decimal strings correctly rounded
    return out


# --------------------------------------------------------------------------
# GRU step, NCE score, normaliser (Sec. 2.1, 2.2)
# --------------------------------------------------------------------------

def _sigmoid(v):
    return 1.0 / (1.0 + np.exp(-v))


def gru_step(x, h, W_ih, W_hh, b_ih):
    """One GRU step in float64, rows of x [M, Kx] and h [M, H].

    Sec. 2.1: a GRU with update gate, reset gate and candidate, using six
    weight matrices and three bias vectors. Reading: the reset gate scales
    the recurrent product of the candidate, with zero recurrent bias:
        a = W_ih x + b_ih,  c = W_hh h       (gate blocks r, z, n)
        r = sigmoid(a_r + c_r),  z = sigmoid(a_z + c_z)
        n = tanh(a_n + r * c_n)
        h' = (1 - z) * n + z * h
    so z = 1 keeps the history unchanged.
    """
    x = np.asarray(x, dtype=np.float64)
    h = np.asarray(h, dtype=np.float64)
    H = h.shape[1]
    a = x @ np.asarray(W_ih, dtype=np.float64).T + np.asarray(b_ih, dtype=np.float64)
    c = h @ np.asarray(W_hh, dtype=np.float64).T
    r = _sigmoid(a[:, :H] + c[:, :H])
    z = _sigmoid(a[:, H:2 * H] + c[:, H:2 * H])
    n = np.tanh(a[:, 2 * H:] + r * c[:, 2 * H:])
    return (1.0 - z) * n + z * h


def nce_score(h_top, U_out, b_out, tgt):
    """Unnormalised NCE score u_tgt . h + b_tgt (Sec. 2.2), float64."""
    u = np.asarray(U_out[tgt], dtype=np.float64)
    return np.sum(u * np.asarray(h_top, dtype=np.float64), axis=-1) \
        + np.asarray(b_out[tgt], dtype=np.float64)


def log_normalizer(h_top, U_out, b_out, chunk=8192):
    """logZ_i = log sum_v exp(U_out[v] . h_i + b_out[v]) over the full vocabulary.

    The normalisation that NCE lets the decoder skip (Sec. 2.2); computed as
    m + log sum exp(a - m) with m = max_v a_v. All logits are formed first
    (in row blocks of U_out only to bound memory), then reduced.
    """
    h = np.asarray(h_top, dtype=np.float64)
    V = U_out.shape[0]
    a = np.empty((h.shape[0], V), dtype=np.float64)
    for v0 in range(0, V, chunk):
        u = np.asarray(U_out[v0:v0 + chunk], dtype=np.float64)
        a[:, v0:v0 + chunk] = h @ u.T + np.asarray(b_out[v0:v0 + chunk], np.float64)
    m = a.max(axis=1)
    return m + np.log(np.sum(np.exp(a - m[:, None]), axis=1))


def log_normalizer_maxent(h_top, U_out, b_out, maxent, words, max_order, log2, chunk=8192):
    """logZ_i over the full model output: every word v's logit is the NCE
    logit plus its hashed n-gram MaxEnt weights after history i's context
    words (Sec. 2.2 with the Sec. 2.3 bypass), orders 2..max_order, the same
    slots the scores use (maxent_index). words: [n, 3] (w-1, w-2, w-3)."""
    h = np.asarray(h_top, dtype=np.float64)
    words = np.asarray(words, dtype=np.int64)
    V = U_out.shape[0]
    if words.shape != (h.shape[0], 3) or words.min(initial=0) < 0 or words.max(initial=0) >= V:
        raise ValueError("words must be [n, 3] ids in [0, V)")
    a = np.empty((h.shape[0], V), dtype=np.float64)
    for v0 in range(0, V, chunk):
        u = np.asarray(U_out[v0:v0 + chunk], dtype=np.float64)
        a[:, v0:v0 + chunk] = h @ u.T + np.asarray(b_out[v0:v0 + chunk], np.float64)
    lam = np.asarray(maxent, dtype=np.float64)
    v = np.arange(V, dtype=np.int64)
    for i in range(h.shape[0]):
        for o in range(2, max_order + 1):
            ctx = [np.full(V, words[i, c], dtype=np.int64) for c in range(o - 1)]
            a[i] += lam[maxent_index(o, ctx, v, log2)]
    m = a.max(axis=1)
    return m + np.log(np.sum(np.exp(a - m[:, None]), axis=1))


# --------------------------------------------------------------------------
# frame-wise scoring with the two caches
# --------------------------------------------------------------------------

@dataclasses.dataclass
class FrameResult:
    scores: np.ndarray     # fp32 [n_q]
    q_status: np.ndarray   # uint8 [n_q]
    q_rep: np.ndarray      # int32 [n_q]
    h_status: np.ndarray   # uint8 [n_h]
    h_rep: np.ndarray      # int32 [n_h]
    h_hash: np.ndarray     # uint64 [n_h]
    hnew: np.ndarray       # float64 [n_h, L*H]
    gru_rows: int
    hist_inserted: int
    hist_rejected: int
    score_inserted: int
    score_rejected: int


class Oracle:
    """Frame-by-frame scorer with a history cache and an LM-query cache.

    weights: dict of fp32 arrays as produced by the workload generator
    (emb, W_ih[l], W_hh[l], b_ih[l], U_out, b_out, maxent).
    """

    def __init__(self, V, E, H, L, maxent_log2, maxent_order, weights,
                 qmode, qdigits=0, cap_hist=1 << 20, cap_query=1 << 22,
                 seed=0x5EED):
        self.V, self.E, self.H, self.L = V, E, H, L
        self.me_log2, self.me_order = maxent_log2, maxent_order
        self.qmode, self.qdigits = qmode, qdigits
        self.cap_hist, self.cap_query = cap_hist, cap_query
        self.seed = seed
        self.w = weights
        self.W_ih = [np.asarray(m, np.float64) for m in weights["W_ih"]]
        self.W_hh = [np.asarray(m, np.float64) for m in weights["W_hh"]]
        self.b_ih = [np.asarray(m, np.float64) for m in weights["b_ih"]]
        self.reset()

    def reset(self):
        self.hist_cache = {}    # history key -> h' (float64 [L*H])
        self.score_cache = {}   # query key -> fp32 score

    def n_ctx(self):
        """Context words beyond w-1 that the MaxEnt orders read."""
        return max(0, self.me_order - 2)

    def history_keys(self, hist_vec, hist_words):
        codes = quantize(hist_vec, self.qmode, self.qdigits)
        words = code_words(codes, self.qmode)
        h_hash = hist_key_hash(words, hist_words[:, 0], self.seed)
        keys = [(words[i].tobytes(), int(hist_words[i, 0])) for i in range(len(words))]
        return keys, h_hash

    def score_frame(self, hist_vec, hist_words, q_hist, q_tgt) -> FrameResult:
        H, L, V = self.H, self.L, self.V
        hist_vec = np.asarray(hist_vec, np.float32)
        hist_words = np.asarray(hist_words, np.int64)
        q_hist = np.asarray(q_hist, np.int64)
        q_tgt = np.asarray(q_tgt, np.int64)
        n_h, n_q = len(hist_vec), len(q_hist)
        if hist_vec.shape != (n_h, L * H) or hist_words.shape != (n_h, 3):
            raise ValueError("bad history shapes")
        if n_h and (hist_words.min() < 0 or hist_words.max() >= V):
            raise ValueError("word id out of range")
        if n_q and (q_tgt.min() < 0 or q_tgt.max() >= V
                    or q_hist.min() < 0 or q_hist.max() >= n_h):
            raise ValueError("query index out of range")

        # 1-3: keys, in-frame representatives (lowest index), cache probe
        keys, h_hash = self.history_keys(hist_vec, hist_words)
        first = {}
        h_rep = np.empty(n_h, np.int32)
        for i, kk in enumerate(keys):
            h_rep[i] = first.setdefault(kk, i)
        h_status = np.empty(n_h, np.uint8)
        for i, kk in enumerate(keys):
            if kk in self.hist_cache:
                h_status[i] = HC_HIT
            elif h_rep[i] == i:
                h_status[i] = H_REP
            else:
                h_status[i] = H_DUP

        # 5: GRU on each new key's own (full-precision) representative vector
        rows = np.nonzero(h_status == H_REP)[0]
        hnew = np.zeros((n_h, L * H), np.float64)
        if len(rows):
            x = np.asarray(self.w["emb"][hist_words[rows, 0]], np.float64)
            outs = []
            for l in range(L):
                h = hist_vec[rows, l * H:(l + 1) * H]
                x = gru_step(x, h, self.W_ih[l], self.W_hh[l], self.b_ih[l])
                outs.append(x)
            hnew[rows] = np.concatenate(outs, axis=1)
        for i in range(n_h):
            if h_status[i] == HC_HIT:
                hnew[i] = self.hist_cache[keys[i]]
            elif h_status[i] == H_DUP:
                hnew[i] = hnew[h_rep[i]]

        # 4: query keys, representatives, score-cache probe
        nc = self.n_ctx()
        qkeys = [(keys[q_hist[q]], tuple(int(hist_words[q_hist[q], 1 + c]) for c in range(nc)),
                  int(q_tgt[q])) for q in range(n_q)]
        qfirst = {}
        q_rep = np.empty(n_q, np.int32)
        q_status = np.empty(n_q, np.uint8)
        for q, kk in enumerate(qkeys):
            q_rep[q] = qfirst.setdefault(kk, q)
            if kk in self.score_cache:
                q_status[q] = Q_SCORE_HIT
            elif q_rep[q] < q:
                q_status[q] = Q_DUP
            else:
                q_status[q] = Q_COMPUTED

        # 6: unnormalised NCE + MaxEnt for computed queries; dups copy, hits reuse
        scores = np.zeros(n_q, np.float32)
        comp = np.nonzero(q_status == Q_COMPUTED)[0]
        if len(comp):
            hq = q_hist[comp]
            tg = q_tgt[comp]
            s = nce_score(hnew[hq, (L - 1) * H:], self.w["U_out"], self.w["b_out"], tg)
            ctx = [hist_words[hq, c] for c in range(3)]
            lam = np.asarray(self.w["maxent"])
            for order in range(2, self.me_order + 1):
                s = s + lam[maxent_index(order, ctx, tg, self.me_log2)].astype(np.float64)
            scores[comp] = s.astype(np.float32)     # round to nearest fp32
        for q in range(n_q):
            if q_status[q] == Q_DUP:
                scores[q] = scores[q_rep[q]]
            elif q_status[q] == Q_SCORE_HIT:
                scores[q] = self.score_cache[qkeys[q]]

        # 7: admissions, in ascending index, while below capacity
        hi = hr = 0
        for i in rows:
            if len(self.hist_cache) < self.cap_hist:
                self.hist_cache[keys[i]] = hnew[i].copy()
                hi += 1
            else:
                hr += 1
        si = sr = 0
        for q in comp:
            kk = qkeys[q]
            if kk[0] not in self.hist_cache:
                continue   # a score is cached only under a cached history key
            if len(self.score_cache) < self.cap_query:
                self.score_cache[kk] = scores[q]
                si += 1
            else:
                sr += 1
        return FrameResult(scores, q_status, q_rep, h_status, h_rep, h_hash,
                           hnew, len(rows), hi, hr, si, sr)
