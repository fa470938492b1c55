"""Pins for the oracle's inverse-CDF sample placement (Sec. 5.1, Fig. 7)."""
import math

import numpy as np

from oracle import donerf_oracle as O
from paper_2103_03231_amd import inputs

F32 = np.float32
NEAR, FAR = float(F32(0.1)), float(F32(10.0))
SPAN = FAR - NEAR


def to_depth(s):
    return NEAR + (SPAN + 1.0) ** np.asarray(s) - 1.0


def test_inverse_matches_np_interp():
    # np.interp of u over the (CDF, coordinate) knots is the inverse of the
    # piecewise-linear CDF of a piecewise-constant PDF.
    B, N = 128, 8
    lg = inputs.random_logits(200, B, seed=5).astype(np.float64) * 2.0
    t, delta, cls = O.cdf_samples(lg, N, NEAR, FAR)
    p = 1.0 / (1.0 + np.exp(-lg))
    for r in range(lg.shape[0]):
        cdf = np.concatenate([[0.0], np.cumsum(p[r])]) / p[r].sum()
        knots = np.arange(B + 1) / B
        s_mid = np.interp((np.arange(N) + 0.5) / N, cdf, knots)
        s_edge = np.interp(np.arange(N + 1) / N, cdf, knots)
        np.testing.assert_allclose(t[r], to_depth(s_mid), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(delta[r], np.diff(to_depth(s_edge)), rtol=1e-9, atol=1e-12)
        assert np.array_equal(cls[r], np.minimum((s_mid * B).astype(int), B - 1))


def test_uniform_scores_give_uniform_log_steps():
    B, N = 64, 4
    t, delta, cls = O.cdf_samples(np.zeros((3, B)), N, NEAR, FAR)
    s = (np.arange(N) + 0.5) / N
    np.testing.assert_allclose(t, np.tile(to_depth(s), (3, 1)), rtol=1e-12)
    # Eq. 3 maps the samples back onto the uniform midpoints of [near, far]
    np.testing.assert_allclose(O.log_depth(t[0], NEAR, FAR), NEAR + s * SPAN, rtol=1e-12)
    np.testing.assert_allclose(delta.sum(1), SPAN, rtol=1e-12)
    np.testing.assert_allclose(delta[0], np.diff(to_depth(np.arange(N + 1) / N)), rtol=1e-12)
    assert np.array_equal(cls[0], (s * B).astype(int))


def test_concentrated_mass_keeps_samples_in_the_class():
    B, N, k0 = 128, 4, 37
    lg = np.full((1, B), -40.0)
    lg[0, k0] = 40.0
    t, delta, cls = O.cdf_samples(lg, N, NEAR, FAR)
    b, _, _ = O.bin_table(NEAR, FAR, B)
    assert np.all(cls == k0)
    assert np.all((t >= float(b[k0]) - 1e-9) & (t <= float(b[k0 + 1]) + 1e-9))
    assert np.all(np.diff(t[0]) > 0)
    np.testing.assert_allclose(delta.sum(), SPAN, rtol=1e-12)


def test_samples_monotone_and_widths_tile_the_ray():
    lg = inputs.random_logits(500, 128, seed=8).astype(np.float64) * 3.0
    for N in (1, 2, 4, 16):
        t, delta, _ = O.cdf_samples(lg, N, NEAR, FAR)
        assert np.all(np.diff(t, axis=1) > 0)
        assert np.all((t > NEAR) & (t < FAR)) and np.all(delta > 0)
        np.testing.assert_allclose(delta.sum(1), SPAN, rtol=1e-9)


def test_cdf_render_wiring():
    # Uniform scores place the first of N samples at the closed-form depth;
    # an opaque pass-through shading network then reports the warp of that
    # sample (Eq. 1 with the camera origin, Eq. 4-5) and its depth.
    B, N = 128, 4
    d = [(np.zeros((256, 90)), np.zeros(256))] + [(np.zeros((256, 256)), np.zeros(256))] * 6 \
        + [(np.zeros((B, 256)), np.zeros(B))]
    W0 = np.zeros((256, 63)); W0[:3, :3] = np.eye(3)
    b0 = np.zeros(256); b0[:3] = 4.0
    s = [(W0, b0)] + [(np.eye(256), np.zeros(256))] * 6
    W7 = np.zeros((4, 283)); W7[:3, :3] = np.eye(3)
    b7 = np.array([-4.0, -4.0, -4.0, 1e4])
    s.append((W7, b7))
    blob = np.concatenate([np.concatenate([np.asarray(W, F32).ravel(), np.asarray(bb, F32)])
                           for W, bb in d + s])
    pose = inputs.make_pose(7)
    out = O.render(blob, pose[None], 3, 5, N, n_bins=B, near=NEAR, far=FAR, select="cdf")
    o, r = O.camera_rays(pose, 3, 5, 60.0)
    t0 = to_depth(0.5 / N)
    x = o.astype(np.float64) + t0 * r.astype(np.float64)
    w = x / np.sqrt(np.linalg.norm(x, axis=1, keepdims=True) * FAR)
    np.testing.assert_allclose(out["rgb"], 1 / (1 + np.exp(-w)), atol=1e-6)
    np.testing.assert_allclose(out["depth"], t0, rtol=1e-6)
    np.testing.assert_allclose(out["t"][:, 0], t0, rtol=1e-12)
