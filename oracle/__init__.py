"""CPU oracle for frame-wise RNNLM query scoring -- TEST INFRASTRUCTURE ONLY.

A plain, slow, double-precision implementation of what the scoring path of
Lee et al., "Accelerating recurrent neural network language model based online
speech recognition system" (arXiv 1801.09866) computes: history quantisation
(Sec. 3), cache keys and de-duplication (Sec. 2.4, Sec. 3), the GRU step
(Sec. 2.1), the unnormalised NCE score (Sec. 2.2), the hashed n-gram MaxEnt
bypass (Sec. 2.3), plus the full-vocabulary normaliser that NCE avoids
(Sec. 2.2).

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or run anything in this package. The HIP library and
its Python binding never touch it, and it shares no code with them.
"""
from .rnnlm_oracle import (  # noqa: F401
    Q_EXACT, Q_SIGN, Q_SIGDIG,
    H_REP, H_DUP, HC_HIT, Q_COMPUTED, Q_DUP, Q_SCORE_HIT,
    mix64, hist_key_hash, maxent_index, quantize, dequantize, code_words,
    gru_step, nce_score, log_normalizer, log_normalizer_maxent, Oracle, FrameResult,
)
