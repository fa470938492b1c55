"""donerf_render inside a captured HIP graph: the call issues kernel
launches only (poses travel by value in the kernel arguments, no memset, no
copy, no synchronisation, no allocation), so a caller can capture it on its
own stream and replay it.  Every replay must equal the eager render bit for
bit, with eager work of the same handle between the replays."""
import numpy as np
import pytest
import torch

from paper_2103_03231_amd import binding as b
from paper_2103_03231_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("precision,poses,H,W,N", [
    ("bf16", [0, 3], 96, 80, 4),          # few tiles: the split tail and its combine kernel
    ("bf16", [0, 1, 2, 3, 4], 400, 400, 4),
    ("fp8", [1], 61, 47, 8),
])
def test_render_replays_from_a_graph(precision, poses, H, W, N):
    prec = {"bf16": b.BF16, "fp8": b.FP8}[precision]
    r = b.Renderer(b.Config(n_bins=128, n_max=N, precision=prec), inputs.make_weights(128, 0))
    ps = inputs.make_poses(poses)
    eager = r.render(ps, H, W, N, depth=True)
    torch.cuda.synchronize()
    ref_rgb, ref_depth = eager["rgb"].clone(), eager["depth"].clone()

    out = r.alloc(len(poses), H, W, N, depth=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                       # warm-up on the capture's kind of stream
        b.donerf_set_stream(r.h, side.cuda_stream)
        r.render_into(ps, H, W, N, out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        b.donerf_set_stream(r.h, torch.cuda.current_stream().cuda_stream)
        r.render_into(ps, H, W, N, out)
    b.donerf_set_stream(r.h, torch.cuda.current_stream().cuda_stream)

    for i in range(3):
        out["rgb"].fill_(-1.0)
        out["depth"].fill_(-1.0)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out["rgb"], ref_rgb), i
        assert torch.equal(out["depth"], ref_depth), i
        other = r.render(inputs.make_poses([7]), 33, 29, N)   # eager work between replays
        torch.cuda.synchronize()
        assert np.isfinite(other["rgb"].cpu().numpy()).all()
    del g
    r.close()
