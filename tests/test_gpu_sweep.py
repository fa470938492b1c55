"""Randomized configurations through the C ABI, checked against the oracle
with the same per-ray rules as the fixed parity tests: precision, placement,
number of classes, samples per ray, frame shape, poses, weights and depth
input drawn from a seeded generator, so that combinations the fixed cases do
not name are covered too.  Frames of up to 2 x 90 x 90 rays span several
tiles and the split tail; the larger ones are checked on sampled rays."""
import numpy as np
import pytest

import test_gpu_parity as T
from paper_2103_03231_amd import binding as b
from paper_2103_03231_amd import inputs

pytestmark = pytest.mark.gpu


def _case(i):
    rng = np.random.default_rng(1000 + i)
    prec = str(rng.choice(["fp32", "bf16", "fp8"]))
    select = str(rng.choice(["topn", "cdf"]))
    B = int(rng.choice([64, 128, 192, 256]))
    din = str(rng.choice(["encoded", "positions"]))
    N = min(int(rng.integers(1, 17)), B)
    P = int(rng.integers(1, 3))
    H, W = int(rng.integers(12, 91)), int(rng.integers(12, 91))
    return dict(prec=prec, select=select, B=B, din=din, N=N, P=P, H=H, W=W,
                wseed=int(rng.integers(0, 1000)), pseeds=[int(x) for x in rng.integers(0, 1000, P)], rng=rng)


@pytest.mark.parametrize("i", range(24))
def test_random_configuration(i):
    c = _case(i)
    rng = c.pop("rng")
    T.log(f"[sweep {i}] {c}")
    sel = b.SELECT_CDF if c["select"] == "cdf" else b.SELECT_TOPN
    r, w = T.renderer(c["prec"], n_bins=c["B"], n_max=c["N"], select=sel, seed=c["wseed"], depth_input=c["din"])
    poses = inputs.make_poses(c["pseeds"])
    H, W, N = c["H"], c["W"], c["N"]
    g = T.gpu_render(r, poses, H, W, N)
    r.close()
    total = len(poses) * H * W
    sub = None if total <= 1500 else np.unique(np.concatenate([rng.integers(0, total, 500), [0, total - 1]]))
    label = f"sweep {i}"
    if c["select"] == "cdf":
        T.check_cdf(g, w, poses, H, W, N, c["prec"], n_bins=c["B"], subset=sub, label=label, depth_input=c["din"])
    else:
        T.check_against_oracle(g, w, poses, H, W, N, c["prec"], n_bins=c["B"], subset=sub, label=label,
                               max_flip_frac=T.FLIPS[c["prec"]] if sub is None or c["prec"] == "fp32" else 0.25,
                               depth_input=c["din"])
