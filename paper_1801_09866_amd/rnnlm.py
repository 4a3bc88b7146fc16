"""Python binding of librnnlm.so (include/rnnlm.h): argument marshalling only.

Device memory and streams come from PyTorch; every step of the scoring path
runs in the library's HIP kernels. Importing this module does not load the
library; the first call does, and it raises if the library has not been built
(``python -m paper_1801_09866_amd.build``). There is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librnnlm.so")

OK, EINVAL, ENOMEM, EHIP, EDEVICE = 0, -1, -2, -3, -4
Q_EXACT, Q_SIGN, Q_SIGDIG = 0, 1, 2
F32, BF16 = 0, 1
H_REP, H_DUP, HC_HIT = 0, 1, 2
Q_COMPUTED, Q_DUP, Q_SCORE_HIT = 0, 1, 2
DERR_WORD, DERR_QHIST, DERR_VALUE, DERR_HANDLE = 1, 2, 4, 8
DEFAULT_SEED = 0x5EED

c_i32, c_i64, c_u64, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p


class Config(ctypes.Structure):
    _fields_ = [("V", c_i32), ("E", c_i32), ("H", c_i32), ("L", c_i32), ("wdtype", c_i32),
                ("maxent_log2", c_i32), ("maxent_order", c_i32), ("qmode", c_i32),
                ("qdigits", c_i32), ("max_hist", c_i32), ("max_query", c_i32), ("sessions", c_i32),
                ("cap_hist", c_i64), ("cap_query", c_i64), ("seed", c_u64)]


class Weights(ctypes.Structure):
    _fields_ = [("emb", c_vp), ("W_ih", c_vp * 2), ("W_hh", c_vp * 2), ("b_ih", c_vp * 2),
                ("U_out", c_vp), ("b_out", c_vp), ("maxent", c_vp)]


class Frame(ctypes.Structure):
    _fields_ = [("n_hist", c_i32), ("n_query", c_i32), ("hist_vec", c_vp), ("hist_words", c_vp),
                ("q_hist", c_vp), ("q_tgt", c_vp), ("hist_ptr", c_vp)]


class Out(ctypes.Structure):
    _fields_ = [("scores", c_vp), ("hnew", c_vp), ("q_status", c_vp), ("q_rep", c_vp),
                ("h_status", c_vp), ("h_rep", c_vp), ("h_hash", c_vp)]


class Stats(ctypes.Structure):
    _fields_ = [(n, c_i64) for n in (
        "frames", "queries", "score_hits", "query_dups", "computed", "hists", "hist_hits",
        "hist_dups", "gru_rows", "hist_inserted", "hist_rejected", "score_inserted",
        "score_rejected", "hist_cache_size", "score_cache_size")] + [("device_error", c_i32), ("pad", c_i32)]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_ if n != "pad"}


EXPORTS = ("rnnlm_workspace_size", "rnnlm_create", "rnnlm_score_frame", "rnnlm_score_frames",
           "rnnlm_cache_reset", "rnnlm_log_normalizer", "rnnlm_log_normalizer_maxent",
           "rnnlm_log_normalizer_static", "rnnlm_get_stats",
           "rnnlm_get_session_stats", "rnnlm_debug_quantize", "rnnlm_profile", "rnnlm_profile_read",
           "rnnlm_destroy", "rnnlm_last_error")
NSTAGES = 10
STAGES = ("hist_key", "frame_plan", "gru_gemm", "score_finish", "unused4", "unused5",
          "unused6", "unused7", "lognorm_gemm", "lognorm_combine")

_lib = None


def load(path=LIB_PATH):
    """Load librnnlm.so (raises if it is missing: there is no CPU fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("librnnlm.so not built: run `python -m paper_1801_09866_amd.build`")
    L = ctypes.CDLL(path)
    P = ctypes.POINTER
    L.rnnlm_workspace_size.argtypes = [P(Config), P(ctypes.c_size_t)]
    L.rnnlm_create.argtypes = [P(Config), P(Weights), c_vp, ctypes.c_size_t, c_vp, P(c_vp)]
    L.rnnlm_score_frame.argtypes = [c_vp, P(Frame), P(Out), c_vp]
    L.rnnlm_score_frames.argtypes = [c_vp, P(Frame), P(Out), c_i32, c_vp]
    L.rnnlm_get_session_stats.argtypes = [c_vp, c_i32, P(Stats), c_vp]
    L.rnnlm_cache_reset.argtypes = [c_vp, c_vp]
    L.rnnlm_log_normalizer.argtypes = [c_vp, c_vp, c_i32, c_vp, c_vp]
    L.rnnlm_log_normalizer_maxent.argtypes = [c_vp, c_vp, c_vp, c_i32, c_vp, c_vp]
    L.rnnlm_log_normalizer_static.argtypes = [c_vp, c_vp, c_i32, c_i32, c_vp, c_i32, c_vp, c_vp]
    L.rnnlm_get_stats.argtypes = [c_vp, P(Stats), c_vp]
    L.rnnlm_debug_quantize.argtypes = [c_i32, c_i32, c_vp, c_i64, c_vp, c_vp, c_vp]
    L.rnnlm_profile.argtypes = [c_vp, ctypes.c_uint32]
    L.rnnlm_profile_read.argtypes = [c_vp, P(ctypes.c_double), P(c_i64)]
    L.rnnlm_destroy.argtypes = [c_vp]
    L.rnnlm_destroy.restype = None
    L.rnnlm_last_error.restype = ctypes.c_char_p
    for n in EXPORTS[:-2]:
        getattr(L, n).restype = ctypes.c_int
    _lib = L
    return L


class RnnlmError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("rnnlm error %d: %s" % (code, msg))
        self.code = code


def _check(rc):
    if rc != OK:
        raise RnnlmError(rc, load().rnnlm_last_error().decode())
    return rc


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(x, dtype, device):
    if isinstance(x, torch.Tensor):
        return x.to(device=device, dtype=dtype).contiguous()
    return torch.from_numpy(np.ascontiguousarray(x)).to(device=device, dtype=dtype).contiguous()


def make_config(model, qmode, qdigits=0, max_hist=1024, max_query=8192, cap_hist=1 << 16,
                cap_query=1 << 20, seed=DEFAULT_SEED, sessions=1):
    return Config(V=model.V, E=model.E, H=model.H, L=model.L, wdtype=model.wdtype,
                  maxent_log2=model.maxent_log2, maxent_order=model.maxent_order,
                  qmode=qmode, qdigits=qdigits, max_hist=max_hist, max_query=max_query, sessions=sessions,
                  cap_hist=cap_hist, cap_query=cap_query, seed=seed)


def workspace_size(cfg: Config) -> int:
    n = ctypes.c_size_t()
    _check(load().rnnlm_workspace_size(ctypes.byref(cfg), ctypes.byref(n)))
    return n.value


class Scorer:
    """One library context: device weights, workspace and both caches."""

    def __init__(self, model, weights, qmode, qdigits=0, max_hist=1024, max_query=8192,
                 cap_hist=1 << 16, cap_query=1 << 20, seed=DEFAULT_SEED, device="cuda:0",
                 stream=None, sessions=1):
        L = load()
        self.device = torch.device(device)
        self.model = model
        self.sessions = sessions
        self.cfg = make_config(model, qmode, qdigits, max_hist, max_query, cap_hist, cap_query, seed, sessions)
        wdt = torch.bfloat16 if model.wdtype == BF16 else torch.float32
        dev = self.device
        self.w = {
            "emb": _dev(weights["emb"], wdt, dev),
            "W_ih": [_dev(m, wdt, dev) for m in weights["W_ih"]],
            "W_hh": [_dev(m, wdt, dev) for m in weights["W_hh"]],
            "b_ih": [_dev(m, torch.float32, dev) for m in weights["b_ih"]],
            "U_out": _dev(weights["U_out"], wdt, dev),
            "b_out": _dev(weights["b_out"], torch.float32, dev),
            "maxent": _dev(weights["maxent"], torch.float32, dev),
        }
        cw = Weights()
        cw.emb = self.w["emb"].data_ptr()
        for l in range(model.L):
            cw.W_ih[l] = self.w["W_ih"][l].data_ptr()
            cw.W_hh[l] = self.w["W_hh"][l].data_ptr()
            cw.b_ih[l] = self.w["b_ih"][l].data_ptr()
        cw.U_out = self.w["U_out"].data_ptr()
        cw.b_out = self.w["b_out"].data_ptr()
        cw.maxent = self.w["maxent"].data_ptr()
        self._cw = cw
        nbytes = workspace_size(self.cfg)
        raw = torch.empty(nbytes + 256, dtype=torch.uint8, device=dev)
        off = (-raw.data_ptr()) % 256
        self.workspace = raw[off:off + nbytes]
        self._raw = raw
        ctx = ctypes.c_void_p()
        _check(L.rnnlm_create(ctypes.byref(self.cfg), ctypes.byref(cw),
                              ctypes.c_void_p(self.workspace.data_ptr()), nbytes,
                              _stream(stream), ctypes.byref(ctx)))
        self.ctx = ctx
        self.LH = model.L * model.H

    def alloc_out(self, n_hist, n_query, hnew=True, debug=True):
        d = self.device
        o = {"scores": torch.empty(max(n_query, 1), dtype=torch.float32, device=d)}
        if hnew:
            o["hnew"] = torch.empty((max(n_hist, 1), self.LH), dtype=torch.float32, device=d)
        if debug:
            o["q_status"] = torch.empty(max(n_query, 1), dtype=torch.uint8, device=d)
            o["q_rep"] = torch.empty(max(n_query, 1), dtype=torch.int32, device=d)
            o["h_status"] = torch.empty(max(n_hist, 1), dtype=torch.uint8, device=d)
            o["h_rep"] = torch.empty(max(n_hist, 1), dtype=torch.int32, device=d)
            o["h_hash"] = torch.empty(max(n_hist, 1), dtype=torch.int64, device=d)
        return o

    def score_frame(self, hist_vec, hist_words, q_hist, q_tgt, out=None, hnew=True, debug=True,
                    stream=None, hist_ptr=None):
        """Score one frame; all inputs are device tensors (fp32 / int32).

        hist_ptr (optional, int64 device tensor [n_hist]): device addresses of
        the histories' L*H rows (e.g. rows of an earlier frame's hnew), used
        instead of hist_vec, which may then be None."""
        if hist_ptr is not None:
            n_h = int(hist_ptr.shape[0])
        else:
            n_h = int(hist_vec.shape[0]) if hist_vec is not None else 0
        n_q = int(q_hist.shape[0]) if q_hist is not None else 0
        if out is None:
            out = self.alloc_out(n_h, n_q, hnew, debug)
        fr = Frame(n_h, n_q, _ptr(hist_vec), _ptr(hist_words), _ptr(q_hist), _ptr(q_tgt), _ptr(hist_ptr))
        co = Out(*[_ptr(out.get(k)) for k in ("scores", "hnew", "q_status", "q_rep",
                                               "h_status", "h_rep", "h_hash")])
        _check(load().rnnlm_score_frame(self.ctx, ctypes.byref(fr), ctypes.byref(co), _stream(stream)))
        return out

    def score_frames(self, frames, outs=None, hnew=True, debug=True, stream=None):
        """Score one frame per session in one set of launches: frames[k] =
        (hist_vec, hist_words, q_hist, q_tgt) device tensors of session k
        (or None for no frame). Returns one output dict per frame."""
        n = len(frames)
        fa, oa = (Frame * max(n, 1))(), (Out * max(n, 1))()
        res = []
        for k, fr in enumerate(frames):
            hv, hw, qh, qt = fr if fr is not None else (None, None, None, None)
            n_h = int(hv.shape[0]) if hv is not None else 0
            n_q = int(qh.shape[0]) if qh is not None else 0
            out = outs[k] if outs is not None else self.alloc_out(n_h, n_q, hnew, debug)
            fa[k] = Frame(n_h, n_q, _ptr(hv), _ptr(hw), _ptr(qh), _ptr(qt), None)
            oa[k] = Out(*[_ptr(out.get(key)) for key in ("scores", "hnew", "q_status", "q_rep",
                                                        "h_status", "h_rep", "h_hash")])
            res.append(out)
        _check(load().rnnlm_score_frames(self.ctx, fa, oa, n, _stream(stream)))
        return res

    def session_stats(self, session, stream=None, check=True):
        s = Stats()
        rc = load().rnnlm_get_session_stats(self.ctx, session, ctypes.byref(s), _stream(stream))
        if check:
            _check(rc)
        return s.as_dict()

    def score_frame_raw(self, frame: Frame, out: Out, stream_ptr: ctypes.c_void_p):
        """Pre-marshalled call (for timing loops)."""
        _check(load().rnnlm_score_frame(self.ctx, ctypes.byref(frame), ctypes.byref(out), stream_ptr))

    def reset(self, stream=None):
        _check(load().rnnlm_cache_reset(self.ctx, _stream(stream)))

    def stats(self, stream=None, check=True):
        s = Stats()
        rc = load().rnnlm_get_stats(self.ctx, ctypes.byref(s), _stream(stream))
        if check:
            _check(rc)
        return s.as_dict()

    def log_normalizer(self, h_top, out=None, stream=None):
        n = int(h_top.shape[0])
        if out is None:
            out = torch.empty(max(n, 1), dtype=torch.float32, device=self.device)
        _check(load().rnnlm_log_normalizer(self.ctx, _ptr(h_top), n, _ptr(out), _stream(stream)))
        return out[:n]

    def log_normalizer_maxent(self, h_top, words, out=None, stream=None):
        """Normaliser over the full output: NCE logit plus each word's MaxEnt
        weights after the row's context words ([n, 3] int32 device tensor)."""
        n = int(h_top.shape[0])
        if out is None:
            out = torch.empty(max(n, 1), dtype=torch.float32, device=self.device)
        _check(load().rnnlm_log_normalizer_maxent(self.ctx, _ptr(h_top), _ptr(words), n, _ptr(out),
                                                  _stream(stream)))
        return out[:n]

    def profile(self, stages=()):
        """Time the named stages with HIP events (empty: timing off)."""
        mask = 0
        for st in stages:
            mask |= 1 << STAGES.index(st)
        _check(load().rnnlm_profile(self.ctx, mask))

    def profile_read(self):
        ms = (ctypes.c_double * NSTAGES)()
        n = (c_i64 * NSTAGES)()
        _check(load().rnnlm_profile_read(self.ctx, ms, n))
        return {STAGES[i]: (ms[i], n[i]) for i in range(NSTAGES) if n[i]}

    def close(self):
        if getattr(self, "ctx", None):
            load().rnnlm_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def log_normalizer_static(U_out, b_out, h_top, out=None, stream=None):
    """Full-vocabulary log normaliser without a context or workspace
    (rnnlm_log_normalizer_static): U_out [V, H], b_out [V], h_top [n, H],
    fp32 device tensors; the library's static scratch holds the partials."""
    V, H = int(U_out.shape[0]), int(U_out.shape[1])
    n = int(h_top.shape[0])
    if out is None:
        out = torch.empty(max(n, 1), dtype=torch.float32, device=h_top.device)
    _check(load().rnnlm_log_normalizer_static(_ptr(U_out), _ptr(b_out), V, H, _ptr(h_top), n, _ptr(out),
                                              _stream(stream)))
    return out[:n]


def debug_quantize(x, qmode, qdigits=0, stream=None):
    """Quantise a flat fp32 device tensor with the library's kernel."""
    n = int(x.numel())
    if qmode == Q_SIGN:
        codes = torch.empty(max(n // 64, 1), dtype=torch.int64, device=x.device)
    elif qmode == Q_SIGDIG:
        codes = torch.empty(max(n, 1), dtype=torch.int16, device=x.device)
    else:
        codes = torch.empty(max(n, 1), dtype=torch.int32, device=x.device)
    err = torch.zeros(1, dtype=torch.int32, device=x.device)
    _check(load().rnnlm_debug_quantize(qmode, qdigits, _ptr(x), n, _ptr(codes), _ptr(err), _stream(stream)))
    return codes, err
