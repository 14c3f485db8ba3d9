"""The MFMA throughput probes that bench.py reports as the measured peaks."""
import pytest

pytestmark = pytest.mark.gpu


def test_mfma_probe_rate_is_plausible():
    import torch

    import paper_2608_08751_amd as ivf

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ctx = ivf.Context(0)
    try:
        ms, tflops = ctx.mfma_probe(2000)
        # the published dense fp32 matrix peak of the MI355X is 157.3 TFLOP/s
        assert ms > 0.0
        assert 20.0 < tflops < 170.0
        with pytest.raises(ivf.IvfError):
            ctx.mfma_probe(0)
    finally:
        ctx.close()


def test_mfma_probe_i8_rate_is_plausible():
    import torch

    import paper_2608_08751_amd as ivf

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ctx = ivf.Context(0)
    try:
        ms, tops = ctx.mfma_probe_i8(2000)
        # the published dense int8 matrix peak of the MI355X is 5.0 POP/s
        assert ms > 0.0
        assert 500.0 < tops < 5100.0
        with pytest.raises(ivf.IvfError):
            ctx.mfma_probe_i8(0)
    finally:
        ctx.close()
