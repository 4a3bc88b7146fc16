"""The allocation-free normaliser (rnnlm_log_normalizer_static, its partial
sums in the library's static device array) against the context normaliser
(rnnlm_log_normalizer, partial sums in the caller's workspace), which runs the
same kernels: two calls in a row through the C ABI, the second with fewer
rows, at the check config's sizes (V = 200,000, H = 1024) and at a ragged
vocabulary tail. The outputs must be identical bit for bit."""
import numpy as np
import pytest
import torch

from harness import log
from paper_1801_09866_amd import rnnlm as R
from paper_1801_09866_amd.workload import F32, ModelCfg

pytestmark = pytest.mark.gpu


def device_weights(m, g, dev):
    z = lambda *s: torch.zeros(*s, dtype=torch.float32, device=dev)
    return {"emb": z(m.V, m.E), "W_ih": [z(3 * m.H, m.E)], "W_hh": [z(3 * m.H, m.H)], "b_ih": [z(3 * m.H)],
            "U_out": torch.randn(m.V, m.H, generator=g, device=dev) * 0.05,
            "b_out": torch.randn(m.V, generator=g, device=dev) * 0.05,
            "maxent": z(1 << m.maxent_log2)}


@pytest.mark.parametrize("V,H", [(200_000, 1024), (1000 + 37, 128)])
def test_static_normaliser_matches_the_context_normaliser(V, H):
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(V + H)
    m = ModelCfg(V=V, E=64, H=H, L=1, wdtype=F32, maxent_log2=10, maxent_order=1)
    sc = R.Scorer(m, device_weights(m, g, dev), R.Q_SIGN, max_hist=300, max_query=1)
    U, b = sc.w["U_out"], sc.w["b_out"]
    for n in (300, 37):   # the second call is smaller: nothing of the first may leak into it
        log("  static normaliser V=%d H=%d n=%d" % (V, H, n))
        h = torch.tanh(torch.randn(n, H, generator=g, device=dev))
        got = R.log_normalizer_static(U, b, h)
        want = sc.log_normalizer(h)
        torch.cuda.synchronize()
        assert torch.isfinite(got).all()
        assert torch.equal(got, want), "max diff %.3g" % float((got - want).abs().max())


def test_static_normaliser_rejects_a_vocabulary_above_its_scratch():
    dev = torch.device("cuda:0")
    h = torch.zeros(4, 64, device=dev)
    U = torch.zeros(8, 64, device=dev)
    rc = R.load().rnnlm_log_normalizer_static(R._ptr(U), R._ptr(U), 425_985, 64, R._ptr(h), 4, R._ptr(h),
                                              R._stream(None))
    assert rc == R.EINVAL and b"425984" in R.load().rnnlm_last_error()
