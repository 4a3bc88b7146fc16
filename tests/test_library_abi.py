"""Host-only checks of the C ABI: the library loads, exports every function the
header declares, and rejects bad configurations before touching a GPU."""
import ctypes
import os
import re

import pytest

from paper_1801_09866_amd import rnnlm as R
from paper_1801_09866_amd.workload import CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "rnnlm.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rnnlm_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(R.LIB_PATH):
        import paper_1801_09866_amd.build as b
        b.build()
    return R.load()


def test_header_declares_the_boundary():
    fns = header_functions()
    for name in ("rnnlm_create", "rnnlm_score_frame", "rnnlm_cache_reset"):
        assert name in fns
    assert set(fns) == set(R.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in header_functions():
        assert hasattr(lib, name), name


def test_workspace_sizes_for_every_config(lib):
    for name, c in CONFIGS.items():
        for qm, qd in c.qmodes:
            cfg = R.make_config(c.model, qm, qd, c.max_hist, max(c.queries, 1), c.cap_hist, c.cap_query)
            n = R.workspace_size(cfg)
            assert 0 < n < 8 << 30
            assert n % 256 == 0


@pytest.mark.parametrize("field,value", [
    ("H", 100), ("E", 32), ("L", 3), ("wdtype", 7), ("maxent_order", 5), ("maxent_log2", 0),
    ("qmode", 3), ("max_hist", 0), ("cap_hist", -1), ("V", 0)])
def test_bad_configs_are_rejected(lib, field, value):
    cfg = R.make_config(CONFIGS["tiny"].model, R.Q_SIGN, 0, 16, 64)
    setattr(cfg, field, value)
    n = ctypes.c_size_t()
    assert lib.rnnlm_workspace_size(ctypes.byref(cfg), ctypes.byref(n)) == R.EINVAL
    assert lib.rnnlm_last_error()


def test_sigdig_digits_checked(lib):
    cfg = R.make_config(CONFIGS["tiny"].model, R.Q_SIGDIG, 4, 16, 64)
    n = ctypes.c_size_t()
    assert lib.rnnlm_workspace_size(ctypes.byref(cfg), ctypes.byref(n)) == R.EINVAL


def test_host_argument_checks_need_no_gpu(lib):
    assert lib.rnnlm_score_frame(None, None, None, None) == R.EINVAL
    assert lib.rnnlm_cache_reset(None, None) == R.EINVAL
    assert lib.rnnlm_get_stats(None, None, None) == R.EINVAL
    assert lib.rnnlm_debug_quantize(9, 0, None, 64, None, None, None) == R.EINVAL
    assert lib.rnnlm_debug_quantize(R.Q_SIGN, 0, None, 63, None, None, None) == R.EINVAL
    assert lib.rnnlm_debug_quantize(R.Q_SIGN, 0, None, 0, None, None, None) == R.OK
    # the allocation-free normaliser checks its sizes before touching a device
    one = ctypes.c_void_p(256)
    assert lib.rnnlm_log_normalizer_static(one, one, 425_985, 64, one, 4, one, None) == R.EINVAL
    assert b"425984" in lib.rnnlm_last_error()
    assert lib.rnnlm_log_normalizer_static(one, one, 1000, 96, one, 4, one, None) == R.EINVAL
    assert lib.rnnlm_log_normalizer_static(None, one, 1000, 64, one, 4, one, None) == R.EINVAL
    assert lib.rnnlm_log_normalizer_static(one, one, 1000, 64, one, 0, one, None) == R.OK


def test_sessions_scale_the_per_session_state(lib):
    """Sessions share the packed weights and the normaliser scratch; caches,
    counters and per-frame scratch are repeated per session."""
    m = CONFIGS["medium"].model
    size = []
    for s in (0, 1, 2, 8):
        cfg = R.make_config(m, R.Q_SIGN, 0, 128, 512, sessions=s)
        n = ctypes.c_size_t()
        assert lib.rnnlm_workspace_size(ctypes.byref(cfg), ctypes.byref(n)) == R.OK
        size.append(n.value)
    assert size[0] == size[1]                      # 0 means one session
    per = size[2] - size[1]
    assert per > 0 and size[3] - size[1] == 7 * per
    packed = 3 * m.H * (m.E + m.H) * 4
    assert size[1] - per >= packed                  # the shared part holds the packed weights
    cfg = R.make_config(m, R.Q_SIGN, 0, 128, 512, sessions=9)
    assert lib.rnnlm_workspace_size(ctypes.byref(cfg), ctypes.byref(ctypes.c_size_t())) == R.EINVAL
    assert lib.rnnlm_score_frames(None, None, None, 1, None) == R.EINVAL
    assert lib.rnnlm_get_session_stats(None, 0, None, None) == R.EINVAL
