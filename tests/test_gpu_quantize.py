"""GPU quantiser (the frame kernels' own code, through the debug hook) against
the oracle, bit for bit: random values, every dyadic tie, both sides of every
decade boundary, and a strided sweep over all fp32 bit patterns in [-1, 1].
The exhaustive sweeps run by default (about 3.5 minutes); RNNLM_QUICK=1 skips
them."""
import os

import numpy as np
import pytest
import torch

from harness import log
from oracle import Q_EXACT, Q_SIGDIG, Q_SIGN, code_words, quantize
from paper_1801_09866_amd import rnnlm as R

pytestmark = pytest.mark.gpu


def gpu_codes(x, qmode, k=0):
    xd = torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda()
    codes, err = R.debug_quantize(xd, qmode, k)
    c = codes.cpu().numpy()
    return c, int(err.item())


def check_sigdig(x, k):
    got, err = gpu_codes(x, Q_SIGDIG, k)
    want = quantize(x, Q_SIGDIG, k)
    got = got[:len(x)].view(np.uint16)
    bad = np.nonzero(got != want)[0]
    assert len(bad) == 0, "k=%d: %d mismatches, first x=%r gpu=%d oracle=%d" % (
        k, len(bad), float(x[bad[0]]), got[bad[0]], want[bad[0]])
    assert err == 0


def decade_edges():
    out = []
    for j in range(0, 22):
        c = np.float32(10.0 ** -j)
        for t in (c, np.nextafter(c, np.float32(0)), np.nextafter(c, np.float32(2)),
                  np.nextafter(np.nextafter(c, np.float32(2)), np.float32(2))):
            out.append(t)
    return np.array(out, np.float32)


def ties(k):
    out = []
    for e in range(-8, 1):
        for m in range(10 ** (k - 1), 10 ** k):
            v = (m + 0.5) * 10.0 ** (e - k + 1)
            f = np.float32(v)
            out.extend([f, np.nextafter(f, np.float32(0)), np.nextafter(f, np.float32(2))])
    return np.array(out, np.float32)


@pytest.mark.parametrize("k", [1, 2, 3])
def test_sigdig_edges_ties_random(k):
    rng = np.random.default_rng(k)
    mag = np.concatenate([10.0 ** rng.uniform(-22, 0, 200_000), rng.uniform(0, 1, 200_000)])
    x = np.concatenate([decade_edges(), ties(k), mag.astype(np.float32),
                        np.array([0.0, -0.0, 1.0, -1.0], np.float32)])
    x = np.concatenate([x, -x])
    x = x[np.abs(x) <= 1]
    check_sigdig(x, k)


@pytest.mark.parametrize("k", [1, 2, 3])
def test_sigdig_strided_sweep_all_bit_patterns(k):
    bits = np.arange(0, 0x3F800001, 251, dtype=np.uint32)
    x = bits.view(np.float32)
    check_sigdig(np.concatenate([x, -x]), k)


@pytest.mark.skipif(os.environ.get("RNNLM_QUICK") == "1", reason="RNNLM_QUICK=1 skips the exhaustive sweeps")
@pytest.mark.parametrize("k", [1, 2, 3])
def test_sigdig_exhaustive(k):
    """Every fp32 value in [-1, 1] (2 x 1,065,353,217 bit patterns)."""
    chunk = 1 << 24
    for n, lo in enumerate(range(0, 0x3F800001, chunk)):
        bits = np.arange(lo, min(lo + chunk, 0x3F800001), dtype=np.uint32)
        x = bits.view(np.float32)
        check_sigdig(np.concatenate([x, -x]), k)
        if n % 16 == 15:
            log("  k=%d: bit patterns below %#x agree" % (k, lo + chunk))


@pytest.mark.skipif(os.environ.get("RNNLM_QUICK") == "1", reason="RNNLM_QUICK=1 skips the exhaustive sweeps")
def test_sign_exhaustive():
    """Sign codes of every fp32 bit pattern (NaNs and infinities excluded,
    since they raise the device flag)."""
    chunk = 1 << 26
    for lo in range(0, 1 << 32, chunk):
        bits = np.arange(lo, lo + chunk, dtype=np.uint64).astype(np.uint32)
        x = bits.view(np.float32)
        x = x[np.isfinite(x)]
        x = x[: len(x) // 64 * 64]
        got, err = gpu_codes(x, Q_SIGN)
        want = code_words(quantize(x.reshape(1, -1), Q_SIGN), Q_SIGN)[0]
        assert np.array_equal(got.view(np.uint64)[: len(want)], want) and err == 0, hex(lo)
        if (lo // chunk) % 16 == 15:
            log("  sign: bit patterns below %#x agree" % (lo + chunk))


def test_sigdig_flags_out_of_domain():
    x = np.zeros(256, np.float32)
    x[3] = 1.5
    _, err = gpu_codes(x, Q_SIGDIG, 2)
    assert err == R.DERR_VALUE
    x[3] = np.nan
    _, err = gpu_codes(x, Q_SIGDIG, 2)
    assert err == R.DERR_VALUE


def test_sign_and_exact_codes():
    rng = np.random.default_rng(9)
    x = rng.standard_normal(64 * 500).astype(np.float32)
    x[:4] = [0.0, -0.0, -1e-40, 1e-40]
    got, err = gpu_codes(x, Q_SIGN)
    want = code_words(quantize(x.reshape(1, -1), Q_SIGN), Q_SIGN)[0]
    assert np.array_equal(got.view(np.uint64), want) and err == 0
    got, err = gpu_codes(x, Q_EXACT)
    assert np.array_equal(got.view(np.uint32), quantize(x, Q_EXACT)) and err == 0
    x[7] = np.inf
    _, err = gpu_codes(x, Q_SIGN)
    assert err == R.DERR_VALUE
