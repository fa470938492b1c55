"""donerf_render_static_scratch, the render for callers that cannot
allocate: through the C ABI it must give donerf_render's results bit for bit
(the same kernels; only the split tail's scratch lives in the library's
static device array), on two calls in a row, the second with a smaller
input, so the second reuses the array the first left behind.  The shapes
leave a partial last round of tiles, so the split tail and its scratch are
used."""
import numpy as np
import pytest
import torch

from paper_2103_03231_amd import binding as b
from paper_2103_03231_amd import inputs

pytestmark = pytest.mark.gpu


def _render(r, fn, poses, H, W, N):
    P = len(poses)
    rgb = torch.full((P, H, W, 3), -1.0, dtype=torch.float32, device="cuda")
    depth = torch.full((P, H, W), -1.0, dtype=torch.float32, device="cuda")
    fn(r.h, poses, P, H, W, N, rgb.data_ptr(), depth.data_ptr())
    torch.cuda.synchronize()
    return rgb.cpu().numpy(), depth.cpu().numpy()


@pytest.mark.parametrize("precision,N,B,select", [
    ("bf16", 4, 128, "topn"), ("fp32", 8, 128, "topn"), ("fp8", 16, 128, "topn"),
    # the two-sweep inverse-CDF kernel (the depth head streamed twice)
    ("bf16", 8, 256, "cdf"),
])
def test_static_scratch_matches_render(precision, N, B, select):
    prec = {"bf16": b.BF16, "fp32": b.FP32, "fp8": b.FP8}[precision]
    sel = b.SELECT_CDF if select == "cdf" else b.SELECT_TOPN
    r = b.Renderer(b.Config(n_bins=B, n_max=N, precision=prec, select=sel), inputs.make_weights(B, 0))
    # 2 x 96 x 80 rays: 60 (bf16, fp8) or 120 (fp32) tiles, a partial round
    # split by samples; then 1 x 33 x 29 rays: 4 or 8 tiles, split again
    for poses, H, W in ((inputs.make_poses([0, 3]), 96, 80), (inputs.make_poses([5]), 33, 29)):
        ref = _render(r, b.donerf_render, poses, H, W, N)
        got = _render(r, b.donerf_render_static_scratch, poses, H, W, N)
        assert np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1]), (H, W)
        assert np.isfinite(got[0]).all() and got[0].min() >= 0.0 and got[0].max() <= 1.0
    r.close()


def test_static_scratch_rejects_bad_arguments():
    r = b.Renderer(b.Config(n_bins=128, n_max=4), inputs.make_weights(128, 0))
    out = torch.empty((1, 8, 8, 3), dtype=torch.float32, device="cuda")
    poses = inputs.make_poses([0])
    for P, H, W, N in ((0, 8, 8, 4), (1, 8, 8, 5), (1, 8192, 8192, 4)):
        with pytest.raises(b.DonerfError) as e:
            b.donerf_render_static_scratch(r.h, poses, P, H, W, N, out.data_ptr())
        assert e.value.status == b.E_INVALID_ARG
    with pytest.raises(b.DonerfError) as e:
        b.donerf_render_static_scratch(None, poses, 1, 8, 8, 4, out.data_ptr())
    assert e.value.status == b.E_INVALID_ARG
    r.close()
