"""Seeded synthetic inputs shared by the HIP path's tests/bench and the CPU oracle.

This module holds no step of the rendering method: it only draws numbers.
It produces

* network weights: He-uniform, drawn from a SplitMix64 stream in blob order
  (the flat fp32 layout the C ABI takes, documented in ``include/donerf.h``);
* camera poses: camera-to-world 3x4 matrices of a pinhole camera placed at a
  seeded point of a sphere around the origin and looking at the origin
  (OpenGL axes: the camera looks down its -z axis, +y is up);
* the named workloads (image size, poses, samples per ray, bins, precision).

The paper's scenes and trained weights are not available; these generators
stand in for them with the paper's resolutions (400x400 renders, Fig. 1 and
Sec. 6; a 1440x1600-per-eye headset, Sec. 1) and random-init networks of the
paper's architecture (8 layers of 256 units, App. D).  Timing does not depend
on weight values.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

MASK64 = (1 << 64) - 1

# Network shapes (out, in) in blob order, from the architecture of App. D:
# 8 linear layers of 256 units, the depth network reads the positional
# encodings of the unified origin (63) and the direction (27), the shading
# network reads the encoded warped sample (63) and takes the encoded
# direction (27) again as a skip into its last layer.
HIDDEN = 256
D_IN = 90
S_IN = 63
DIR_SKIP = 27
S_OUT = 4


def depth_inputs(n_bins: int, depth_input: str = "encoded") -> int:
    """Width of the depth network's first layer: 90 encoded inputs, or
    6 + 3 n_bins for the unencoded origin, direction and class positions."""
    return {"encoded": D_IN, "positions": 6 + 3 * n_bins}[depth_input]


def layer_shapes(n_bins: int, depth_input: str = "encoded"):
    """(out, in) of the 16 linear layers: depth network 0..7, then shading 0..7."""
    d = ([(HIDDEN, depth_inputs(n_bins, depth_input))] + [(HIDDEN, HIDDEN)] * 6
         + [(n_bins, HIDDEN)])
    s = [(HIDDEN, S_IN)] + [(HIDDEN, HIDDEN)] * 6 + [(S_OUT, HIDDEN + DIR_SKIP)]
    return d + s


def n_weights(n_bins: int, depth_input: str = "encoded") -> int:
    return sum(o * i + o for o, i in layer_shapes(n_bins, depth_input))


class SplitMix64:
    """SplitMix64 (Steele, Lea, Flood, OOPSLA 2014), the 64-bit output mixer
    of Java's SplittableRandom.  Vectorised: ``next(n)`` returns the next n
    outputs of the single sequential stream."""

    GAMMA = 0x9E3779B97F4A7C15

    def __init__(self, seed: int):
        self.state = np.uint64(seed & MASK64)

    def next(self, n: int) -> np.ndarray:
        with np.errstate(over="ignore"):
            idx = np.arange(1, n + 1, dtype=np.uint64)
            z = self.state + idx * np.uint64(self.GAMMA)
            self.state = np.uint64((int(self.state) + n * self.GAMMA) & MASK64)
            z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
            z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
            z = z ^ (z >> np.uint64(31))
        return z

    def uniform(self, n: int) -> np.ndarray:
        """n floats in [0, 1): the top 24 bits of each output times 2^-24."""
        return (self.next(n) >> np.uint64(40)).astype(np.float64) * (2.0 ** -24)


def make_weights(n_bins: int = 128, seed: int = 0, depth_input: str = "encoded") -> np.ndarray:
    """Flat fp32 weight blob: for each layer W[out][in] row-major, then b[out].

    W ~ U(-a, a) with a = sqrt(6 / fan_in) (He-uniform), b ~ U(-1/sqrt(fan_in),
    1/sqrt(fan_in)) so that the bias path is exercised.  Values are drawn in
    blob order from one SplitMix64 stream."""
    rng = SplitMix64(seed)
    parts = []
    for out_f, in_f in layer_shapes(n_bins, depth_input):
        a = math.sqrt(6.0 / in_f)
        parts.append((a * (2.0 * rng.uniform(out_f * in_f) - 1.0)).astype(np.float32))
        bb = 1.0 / math.sqrt(in_f)
        parts.append((bb * (2.0 * rng.uniform(out_f) - 1.0)).astype(np.float32))
    blob = np.concatenate(parts)
    assert blob.size == n_weights(n_bins, depth_input)
    return blob


def _look_at(eye: np.ndarray, target: np.ndarray) -> np.ndarray:
    fwd = target - eye
    fwd = fwd / np.linalg.norm(fwd)
    up = np.array([0.0, 0.0, 1.0])
    right = np.cross(fwd, up)
    if np.linalg.norm(right) < 1e-6:
        up = np.array([0.0, 1.0, 0.0])
        right = np.cross(fwd, up)
    right = right / np.linalg.norm(right)
    cam_up = np.cross(right, fwd)
    m = np.zeros((3, 4))
    m[:, 0] = right
    m[:, 1] = cam_up
    m[:, 2] = -fwd
    m[:, 3] = eye
    return m


def make_pose(seed: int, radius: float = 1.5) -> np.ndarray:
    """Camera-to-world 3x4 (fp32) at a seeded point of the sphere |x| = radius,
    looking at the origin: z ~ U(-1, 1), phi ~ U(0, 2 pi)."""
    u = SplitMix64(0xD0E5 + 7919 * seed).uniform(2)
    z = 2.0 * u[0] - 1.0
    phi = 2.0 * math.pi * u[1]
    s = math.sqrt(max(0.0, 1.0 - z * z))
    eye = radius * np.array([s * math.cos(phi), s * math.sin(phi), z])
    return _look_at(eye, np.zeros(3)).astype(np.float32)


def make_stereo_pose(seed: int, ipd: float = 0.064, radius: float = 1.5) -> np.ndarray:
    """Two parallel-axis eye poses (left, right) offset by -/+ ipd/2 along the
    camera's right axis: shape (2, 3, 4)."""
    c = make_pose(seed, radius).astype(np.float64)
    left, right = c.copy(), c.copy()
    left[:, 3] -= 0.5 * ipd * c[:, 0]
    right[:, 3] += 0.5 * ipd * c[:, 0]
    return np.stack([left, right]).astype(np.float32)


def make_poses(seeds, radius: float = 1.5) -> np.ndarray:
    return np.stack([make_pose(s, radius) for s in seeds])


def make_depth_maps(P: int, H: int, W: int, seed: int, near: float = 0.1, far: float = 10.0,
                    shapes: int = 12) -> np.ndarray:
    """Seeded synthetic first-surface depth maps (P, H, W) fp32 with the
    structure of rendered scenes: a background without surface (+inf), and
    front-most of `shapes` discs and rectangles, each a tilted plane patch
    whose depth is log-uniform in [near, far] (z-buffered, so objects occlude
    and depth jumps at their edges).  A few pixels fall outside [near, far)
    or are NaN (invalid samples)."""
    rng = SplitMix64(0xDE97 + 104729 * seed)
    out = np.full((P, H, W), np.inf, dtype=np.float64)
    yy, xx = np.mgrid[0:H, 0:W].astype(np.float64)
    for p in range(P):
        for _ in range(shapes):
            u = rng.uniform(8)
            cx, cy = u[0] * W, u[1] * H
            rad = (0.08 + 0.3 * u[2]) * min(H, W)
            d0 = near * (far / near) ** u[3]
            gx, gy = (u[4] - 0.5) * 4.0 * d0 / W, (u[5] - 0.5) * 4.0 * d0 / H
            if u[6] < 0.5:
                inside = (xx - cx) ** 2 + (yy - cy) ** 2 <= rad * rad
            else:
                inside = (np.abs(xx - cx) <= rad) & (np.abs(yy - cy) <= rad * (0.5 + u[7]))
            d = np.maximum(d0 + gx * (xx - cx) + gy * (yy - cy), 0.5 * near)
            out[p] = np.where(inside, np.minimum(out[p], d), out[p])
        u = rng.uniform(2 * H * W).reshape(2, H, W)
        out[p][u[0] < 0.002] = np.nan
        out[p][u[1] < 0.002] = far * 1.5
    return out.astype(np.float32)


def random_logits(rays: int, n_bins: int, seed: int, mode: str = "normal") -> np.ndarray:
    """Seeded logit rows for selection tests.

    mode 'normal' - Gaussian-like values (sum of uniforms)
    mode 'ties'   - values quantised to a few levels, so rows hold many ties,
                    including +0 and -0
    mode 'const'  - every value of a row equal
    mode 'special' - the 'ties' levels mixed with NaN, +inf and -inf (about
                    one value in eight each)
    """
    rng = SplitMix64(0x70F + seed)
    if mode == "normal":
        u = rng.uniform(rays * n_bins * 4).reshape(rays, n_bins, 4).sum(-1) - 2.0
        return u.astype(np.float32)
    if mode == "ties":
        u = rng.uniform(rays * n_bins).reshape(rays, n_bins)
        q = np.floor(u * 7.0) - 3.0  # levels -3..3
        out = (q * 0.25).astype(np.float32)
        signs = rng.uniform(rays * n_bins).reshape(rays, n_bins) < 0.5
        out[(out == 0) & signs] = np.float32(-0.0)
        return out
    if mode == "special":
        out = random_logits(rays, n_bins, seed, "ties")
        pick = SplitMix64(0x5EC1A1 + seed).uniform(rays * n_bins).reshape(rays, n_bins)
        out[pick < 0.125] = np.float32(np.nan)
        out[(pick >= 0.125) & (pick < 0.25)] = np.float32(np.inf)
        out[(pick >= 0.25) & (pick < 0.375)] = np.float32(-np.inf)
        return out
    if mode == "const":
        v = (rng.uniform(rays) * 4.0 - 2.0).astype(np.float32)
        return np.repeat(v[:, None], n_bins, axis=1)
    raise ValueError(mode)


@dataclass(frozen=True)
class Workload:
    """A named rendering workload: P poses of H x W rays, N samples per ray,
    n_bins depth classes, arithmetic precision of the networks."""

    name: str
    H: int
    W: int
    pose_seeds: tuple
    N: int
    n_bins: int = 128
    fov_deg: float = 60.0
    precision: str = "bf16"          # 'fp32', 'bf16' or 'fp8' (the mixed network)
    select: str = "topn"              # 'topn', 'topn_softmax' or 'cdf'
    depth_input: str = "encoded"      # 'encoded' (90 inputs) or 'positions' (6 + 3 B)
    want_depth: bool = False
    stereo: bool = False
    near: float = 0.1
    far: float = 10.0
    radius: float = 1.5
    extra: dict = field(default_factory=dict, hash=False, compare=False)

    @property
    def n_poses(self) -> int:
        return len(self.pose_seeds) * (2 if self.stereo else 1)

    def poses(self) -> np.ndarray:
        if self.stereo:
            return np.concatenate([make_stereo_pose(s, radius=self.radius)
                                   for s in self.pose_seeds])
        return make_poses(self.pose_seeds, self.radius)

    @property
    def rays(self) -> int:
        return self.n_poses * self.H * self.W


WORKLOADS = {
    "tiny32_fp32": Workload("tiny32_fp32", 32, 32, (0,), 4, precision="fp32"),
    "frame400_n4_bf16": Workload("frame400_n4_bf16", 400, 400, (0, 1, 2, 3, 4), 4),
    "frame400_n4_cdf_bf16": Workload("frame400_n4_cdf_bf16", 400, 400, (0, 1, 2, 3, 4), 4,
                                     select="cdf", want_depth=True),
    "frame400_n4_positions_bf16": Workload("frame400_n4_positions_bf16", 400, 400, (0, 1, 2, 3, 4), 4,
                                           depth_input="positions"),
    "frame400_n4_fp8": Workload("frame400_n4_fp8", 400, 400, (0, 1, 2, 3, 4), 4, precision="fp8"),
    "frame800_n8_depth_bf16": Workload("frame800_n8_depth_bf16", 800, 800, (0, 1, 2, 3, 4), 8,
                                       want_depth=True),
    "hd1080_n4_softmax_bf16": Workload("hd1080_n4_softmax_bf16", 1080, 1920, tuple(range(10)), 4,
                                       fov_deg=90.0, select="topn_softmax"),
    "stereo1440x1600_n16_b256_bf16": Workload("stereo1440x1600_n16_b256_bf16", 1600, 1440,
                                              tuple(range(60)), 16, n_bins=256, stereo=True),
    "stereo1440x1600_n16_b256_cdf_bf16": Workload("stereo1440x1600_n16_b256_cdf_bf16", 1600, 1440,
                                                  tuple(range(60)), 16, n_bins=256, stereo=True, select="cdf"),
}


@dataclass(frozen=True)
class TargetWorkload:
    """Depth-oracle training targets for P synthetic depth maps of H x W."""

    name: str
    P: int
    H: int
    W: int
    n_bins: int
    K: int
    Z: int
    seed: int = 7

    @property
    def pixels(self) -> int:
        return self.P * self.H * self.W


TARGET_WORKLOADS = {
    # the paper's K-5 Z-5 configuration at its 400 x 400 resolution, 128 classes
    "targets400_b128_k5_z5": TargetWorkload("targets400_b128_k5_z5", 5, 400, 400, 128, 5, 5),
}
