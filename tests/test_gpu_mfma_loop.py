"""The register-fed MFMA loop behind the bench's measured ceiling, through
the C ABI: its FLOP count, that every accumulator chain runs, and argument
checks.  The loop adds the same random product to each accumulator every
step, so two steps give twice the sums of one (up to fp32 rounding)."""
import numpy as np
import pytest
import torch

from paper_2103_03231_amd import binding as b
from paper_2103_03231_amd import inputs

pytestmark = pytest.mark.gpu

STEP_FLOP = {"fp32": 2 * 32 * 32 * 8, "bf16": 2 * 32 * 32 * 16, "fp8": 2 * 32 * 32 * 64}


def _renderer(precision):
    prec = {"fp32": b.FP32, "bf16": b.BF16, "fp8": b.FP8}[precision]
    return b.Renderer(b.Config(n_bins=128, n_max=4, precision=prec), inputs.make_weights(128, 0))


@pytest.mark.parametrize("precision", ["fp32", "bf16", "fp8"])
def test_mfma_loop_counts_and_scales(precision):
    r = _renderer(precision)
    wg = 7
    s1, f1 = r.mfma_peak(wg, 1)
    s2, f2 = r.mfma_peak(wg, 2)
    torch.cuda.synchronize()
    assert f1 == wg * 4 * 4 * 1 * STEP_FLOP[precision]
    assert f2 == 2 * f1
    a, c = s1.cpu().numpy(), s2.cpu().numpy()
    assert a.shape == (wg * 256,) and np.isfinite(a).all() and np.isfinite(c).all()
    assert np.count_nonzero(a) > 0.9 * a.size      # random operands: sums are nonzero
    np.testing.assert_allclose(c, 2 * a, rtol=1e-5, atol=1e-5 * np.abs(a).max())
    r.close()


def test_mfma_loop_rejects_bad_arguments():
    r = _renderer("bf16")
    sink = torch.empty(256, dtype=torch.float32, device="cuda")
    for wg, it, ptr in ((0, 1, sink.data_ptr()), (1, 0, sink.data_ptr()), (1 << 21, 1, sink.data_ptr()),
                        (1, 1 << 25, sink.data_ptr()), (1, 1, None)):
        with pytest.raises(b.DonerfError) as e:
            b.donerf_debug_mfma_peak(r.h, wg, it, ptr)
        assert e.value.status == b.E_INVALID_ARG, (wg, it)
    r.close()
