"""CPU oracle for DONeRF's depth-oracle training targets and losses.
TEST INFRASTRUCTURE ONLY.

Only the test suite and the benchmark's CPU baseline may import this module;
the library never calls it and shares no code with it.

It follows DONeRF (Neff et al., EGSR 2021, arXiv 2103.03231), Sec. 5.1 and
Sec. 6.1, one step at a time:

  depth of the first surface per pixel -> one-hot class target (Eq. 6)
  -> radial neighbourhood filter in image space, size K (Eq. 7)
  -> triangle filter along the classes, size Z, clamped to 1 (Eq. 8)
  and the opacity loss and the weighted total loss (Eq. 9-10).

Readings where the paper is silent (the design document lists them):
  - classes are the logarithmic depth classes of Eq. 3 (``bin_table``); a
    depth outside [d_min, d_max), or not finite, has no class (background);
  - neighbours outside the image contribute nothing; with K = 1 the window is
    the pixel itself (weight 1);
  - classes outside [0, B) contribute nothing to the depth filter;
  - the opacity terms are the compositing weights of the ray's samples,
    whose sum is the accumulated opacity.
Computed in fp64 (class bounds taken as their fp32 values); targets are
returned as fp64 arrays.
"""
from __future__ import annotations

import math

import numpy as np

from oracle.donerf_oracle import bin_table

F32 = np.float32


def depth_classes(depth, near, far, n_bins):
    """Eq. 6's class of each depth value: the z with b_z <= d < b_{z+1} on
    the fp32 class bounds, or -1 for no class.  depth: any shape, fp32."""
    d = np.asarray(depth, dtype=F32)
    bounds, _, _ = bin_table(near, far, n_bins)
    z = np.searchsorted(bounds, d, side="right") - 1
    ok = np.isfinite(d) & (d >= bounds[0]) & (d < bounds[-1])
    return np.where(ok, z, -1).astype(np.int64)


def one_hot_targets(depth, near, far, n_bins):
    """Eq. 6: C(z) = 1 where the first surface's depth falls in class z.
    depth (H, W) -> (H, W, B)."""
    cls = depth_classes(depth, near, far, n_bins)
    C = np.zeros(cls.shape + (n_bins,))
    hit = cls >= 0
    C[hit, cls[hit]] = 1.0
    return C


def neighbourhood_weight(i, j, K):
    """The contribution 1 - sqrt(i^2 + j^2) / (sqrt(2) floor(K/2)) a surface
    at pixel offset (i, j) makes inside the K x K window (Eq. 7); 1 at the
    centre, also for K = 1."""
    h = K // 2
    if h == 0:
        return 1.0
    return 1.0 - math.sqrt(i * i + j * j) / (math.sqrt(2.0) * h)


def neighbourhood_filter(C, K):
    """Eq. 7: C^(z) = max over the K x K window of (C_{x+i,y+j}(z) - the
    distance term).  C (H, W, B); neighbours outside the image are left out.
    The centre's own term keeps the result >= C >= 0."""
    H, W, B = C.shape
    h = K // 2
    out = np.full_like(C, -np.inf)
    for i in range(-h, h + 1):
        for j in range(-h, h + 1):
            t = C - (1.0 - neighbourhood_weight(i, j, K))
            # shifted[y, x] = t[y + i, x + j] where inside the image
            y0, y1 = max(0, -i), min(H, H - i)
            x0, x1 = max(0, -j), min(W, W - j)
            if y0 >= y1 or x0 >= x1:
                continue   # the offset leaves the image for every pixel
            out[y0:y1, x0:x1] = np.maximum(out[y0:y1, x0:x1], t[y0 + i:y1 + i, x0 + j:x1 + j])
    return out


def depth_filter(Chat, Z):
    """Eq. 8: C`(z) = min(sum_i C^(z + i) (h + 1 - |i|) / (h + 1), 1) with
    h = floor(Z/2); classes outside [0, B) contribute nothing."""
    h = Z // 2
    B = Chat.shape[-1]
    out = np.zeros_like(Chat)
    for i in range(-h, h + 1):
        w = (h + 1 - abs(i)) / (h + 1)
        lo, hi = max(0, -i), min(B, B - i)
        out[..., lo:hi] += Chat[..., lo + i:hi + i] * w
    return np.minimum(out, 1.0)


def training_targets(depth, near, far, n_bins, K, Z):
    """The depth oracle's target (Sec. 5.1): Eq. 6, then Eq. 7, then Eq. 8."""
    return depth_filter(neighbourhood_filter(one_hot_targets(depth, near, far, n_bins), K), Z)


def opacity_loss(weights):
    """Eq. 9: with the accumulated opacity a = sum of the ray's sample
    opacities (rays, N) -> 0 where a >= 1, (a - 1)^2 otherwise; per ray."""
    a = np.sum(np.asarray(weights, dtype=np.float64), axis=-1)
    return np.where(a >= 1.0, 0.0, (a - 1.0) ** 2)


def total_loss(rgb, rgb_ref, weights, alpha=1.0, beta=10.0):
    """Eq. 10: alpha * MSE(rgb) + beta * mean opacity loss, the paper's
    alpha = 1 and beta = 10 by default (Sec. 6.1)."""
    mse = np.mean((np.asarray(rgb, dtype=np.float64) - np.asarray(rgb_ref, dtype=np.float64)) ** 2)
    return alpha * mse + beta * float(np.mean(opacity_loss(weights)))
