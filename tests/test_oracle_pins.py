"""Pins for the CPU oracle: each check is fixed by the paper, a closed form,
an invariant, an independent library routine or brute force on tiny inputs,
never by re-running the oracle's own formula."""
import math
import os

import numpy as np
import pytest
import torch

from oracle import donerf_oracle as O
from paper_2103_03231_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
F32 = np.float32


# ------------------------------------------------------------------ bf16 rounding

def test_round_bf16_matches_torch_rne():
    # torch's CPU float32 -> bfloat16 cast is an independent RNE implementation.
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000),
        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0, -0.0,
                  65504.0, 1e-30, 3.0e38]),
    ]).astype(F32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.round_bf16(x)
    assert np.array_equal(got, ref)
    # ties go to even: 1 + 2^-8 -> 1, 1 + 3*2^-8 -> 1 + 2^-6
    assert O.round_bf16(np.float32(1 + 2 ** -8)) == 1.0
    assert O.round_bf16(np.float32(1 + 3 * 2 ** -8)) == 1.0 + 2 ** -6


# ------------------------------------------------------------------ depth bins (Eq. 3)

@pytest.mark.parametrize("B", [16, 128, 256])
def test_bins_bounds_monotone_and_centres_inside(B):
    near, far = 0.1, 10.0
    b, c, w = O.bin_table(near, far, B)
    assert b[0] == F32(near) and b[-1] == F32(far)
    assert np.all(np.diff(b.astype(np.float64)) > 0)
    assert np.all(c > b[:-1]) and np.all(c < b[1:])
    assert np.all(np.diff(c.astype(np.float64)) > 0)
    assert np.all(w > 0)


@pytest.mark.parametrize("B", [128, 256])
def test_bins_are_uniform_in_eq3_coordinate(B):
    # Eq. 3 maps every class boundary onto a uniform grid of [near, far] and
    # every centre onto the grid's mid points.
    near, far = float(F32(0.1)), float(F32(10.0))
    b, c, _ = O.bin_table(near, far, B)
    span = far - near
    k = np.arange(B + 1)
    np.testing.assert_allclose(O.log_depth(b.astype(np.float64), near, far),
                               near + k * span / B, rtol=0, atol=4e-6)
    np.testing.assert_allclose(O.log_depth(c.astype(np.float64), near, far),
                               near + (k[:-1] + 0.5) * span / B, rtol=0, atol=4e-6)


def test_bin_widths_are_geometric():
    # Closed form of the inverted Eq. 3: width_k = (D+1)^(k/B) ((D+1)^(1/B) - 1).
    near, far, B = F32(0.1), F32(10.0), 128
    _, _, w = O.bin_table(near, far, B)
    D = float(far) - float(near)
    g = (D + 1.0) ** (1.0 / B)
    expect = (D + 1.0) ** (np.arange(B) / B) * (g - 1.0)
    np.testing.assert_allclose(w.astype(np.float64), expect, rtol=2e-6)
    assert abs(w.astype(np.float64).sum() - (float(far) - float(near))) < 1e-5


# ------------------------------------------------------------------ camera (Eq. 1)

def test_camera_rays_unit_and_centre_pixel_forward():
    pose = inputs.make_pose(3)
    H, W = 31, 33  # odd, so one pixel centre lies on the optical axis
    o, r = O.camera_rays(pose, H, W, 60.0)
    assert o.dtype == F32 and r.dtype == F32
    np.testing.assert_allclose(np.linalg.norm(r.astype(np.float64), axis=1), 1.0, atol=2e-7)
    mid = (H // 2) * W + W // 2
    fwd = -pose[:, 2].astype(np.float64)
    np.testing.assert_allclose(r[mid], fwd / np.linalg.norm(fwd), atol=1e-7)
    np.testing.assert_array_equal(o, np.broadcast_to(pose[:, 3], o.shape))


def test_camera_horizontal_field_of_view():
    # The outer edges of the image plane subtend fov_x: pixel centres at the
    # row through the axis make angle atan((W/2 - 0.5)/f) with the axis,
    # f = (W/2)/tan(fov/2).
    pose = np.eye(3, 4, dtype=F32)
    H, W, fov = 9, 64, 75.0
    _, r = O.camera_rays(pose, H, W, fov)
    row = r.reshape(H, W, 3)[H // 2].astype(np.float64)
    f = (W / 2) / math.tan(math.radians(fov) / 2)
    # camera frame = world frame here: looks down -z
    ang = np.arctan2(row[:, 0], -row[:, 2])
    expect = np.arctan(((np.arange(W) + 0.5) - W / 2) / f)
    np.testing.assert_allclose(ang, expect, atol=1e-6)
    # +y up: rows above the axis point up
    col = r.reshape(H, W, 3)[:, W // 2, 1]
    assert np.all(np.diff(col) < 0)


# ------------------------------------------------------------------ unification (Sec. 5.2)

def test_unify_lands_on_sphere_and_is_origin_invariant():
    rng = np.random.default_rng(1)
    n = 500
    c = np.array([0.2, -0.1, 0.3], dtype=F32)
    R = 1.5
    d = rng.standard_normal((n, 3))
    r = (d / np.linalg.norm(d, axis=1, keepdims=True)).astype(F32)
    o1 = (c + rng.uniform(-0.5, 0.5, (n, 3))).astype(F32)
    o2 = (o1 + rng.uniform(0.0, 0.4, (n, 1)) * r).astype(F32)  # same line, further along
    u1 = O.unify(o1, r, c, R).astype(np.float64)
    u2 = O.unify(o2, r, c, R).astype(np.float64)
    np.testing.assert_allclose(np.linalg.norm(u1 - c, axis=1), R, atol=2e-6)
    np.testing.assert_allclose(u1, u2, atol=4e-6)
    # it moves forward along r
    assert np.all(np.einsum("ij,ij->i", u1 - o1, r.astype(np.float64)) >= -1e-6)


def test_unify_origin_on_sphere_looking_out_is_fixed():
    o = np.array([[1.5, 0.0, 0.0]], dtype=F32)
    r = np.array([[1.0, 0.0, 0.0]], dtype=F32)
    np.testing.assert_array_equal(O.unify(o, r, (0, 0, 0), 1.5), o)


# ------------------------------------------------------------------ warp (Eq. 4-5)

def test_warp_closed_forms():
    rng = np.random.default_rng(2)
    dmax = 10.0
    p = rng.standard_normal((1000, 3)) * rng.uniform(0.01, 12, (1000, 1))
    w = O.warp(p.astype(F32), (0, 0, 0), dmax).astype(np.float64)
    n = np.linalg.norm(p, axis=1)
    np.testing.assert_allclose(np.linalg.norm(w, axis=1), np.sqrt(n / dmax), rtol=2e-6)
    cosang = np.einsum("ij,ij->i", w, p) / (np.linalg.norm(w, axis=1) * n)
    np.testing.assert_allclose(cosang, 1.0, atol=1e-6)
    unit = np.array([[dmax, 0, 0], [0, -dmax, 0]], dtype=F32)
    np.testing.assert_allclose(np.linalg.norm(O.warp(unit, (0, 0, 0), dmax), axis=1), 1.0, atol=1e-7)
    assert np.all(O.warp(np.zeros((1, 3), F32), (0, 0, 0), dmax) == 0)
    assert np.all(O.warp(np.full((1, 3), 2.0, F32), (2, 2, 2), dmax) == 0)


# ------------------------------------------------------------------ encoding

def test_encode_dims_identity_and_trig_identities():
    rng = np.random.default_rng(3)
    v = rng.uniform(-1.2, 1.2, (200, 3))
    for L in (4, 10):
        e = O.encode(v, L)
        assert e.shape == (200, 3 + 6 * L)
        np.testing.assert_array_equal(e[:, :3], v)
        for k in range(L):
            s = e[:, 3 + 6 * k: 6 + 6 * k]
            cc = e[:, 6 + 6 * k: 9 + 6 * k]
            np.testing.assert_allclose(s * s + cc * cc, 1.0, atol=1e-12)
            if k + 1 < L:
                s2 = e[:, 3 + 6 * (k + 1): 6 + 6 * (k + 1)]
                # double-angle: each frequency is twice the previous one
                np.testing.assert_allclose(s2, 2 * s * cc, atol=1e-9)
    e = O.encode(np.array([[0.5, 0.0, -0.5]]), 1)
    np.testing.assert_allclose(e[0, 3:], [1, 0, -1, 0, 1, 0], atol=1e-15)


# ------------------------------------------------------------------ networks

def _tiny_layers(rng, dims):
    return [(rng.standard_normal((o, i)), rng.standard_normal(o)) for i, o in zip(dims[:-1], dims[1:])]


def _brute_mlp(layers, x, bf16=False, skip=None):
    def rb(a):
        if not bf16:
            return float(a)
        return float(torch.tensor(float(a), dtype=torch.float32).to(torch.bfloat16).to(torch.float64))
    out = []
    for row in range(len(x)):
        h = [rb(a) for a in x[row]]
        for li, (W, b) in enumerate(layers):
            if li == len(layers) - 1 and skip is not None:
                h = h + [rb(a) for a in skip[row]]
            y = []
            for o in range(W.shape[0]):
                acc = 0.0
                for i in range(W.shape[1]):
                    acc += rb(W[o, i]) * h[i]
                y.append(acc + float(b[o]))
            h = y if li == len(layers) - 1 else [rb(max(a, 0.0)) for a in y]
        out.append(h)
    return np.array(out)


@pytest.mark.parametrize("bf16", [False, True])
def test_mlp_matches_triple_loop(bf16):
    rng = np.random.default_rng(4)
    layers = _tiny_layers(rng, [5, 8, 8, 8, 3])
    x = rng.standard_normal((4, 5))
    got = O.mlp(layers, x, "bf16" if bf16 else "fp64")
    ref = _brute_mlp(layers, x, bf16)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_mlp_skip_goes_into_last_layer():
    rng = np.random.default_rng(5)
    layers = _tiny_layers(rng, [4, 6, 6])
    W2, b2 = rng.standard_normal((2, 6 + 3)), rng.standard_normal(2)
    layers = layers[:1] + [(W2, b2)]
    x = rng.standard_normal((3, 4))
    skip = rng.standard_normal((3, 3))
    np.testing.assert_allclose(O.mlp(layers, x, skip=skip), _brute_mlp(layers, x, skip=skip), rtol=1e-12)


def test_mlp_zero_hidden_weights_gives_head_bias_closed_form():
    rng = np.random.default_rng(6)
    layers = _tiny_layers(rng, [7, 16, 16, 16, 5])
    layers = [(np.zeros_like(W), b) for W, b in layers]
    # every hidden unit = relu(b_l); head = W_last @ relu(b_prev) + b_last
    W, b = layers[-1]
    x = rng.standard_normal((3, 7))
    expect = np.zeros(5) + b
    np.testing.assert_allclose(O.mlp(layers, x), np.tile(expect, (3, 1)))
    layers2 = [(np.zeros((16, 7)), np.abs(rng.standard_normal(16)))] + [(np.eye(16), np.zeros(16))] * 2 \
        + [(np.ones((5, 16)), np.zeros(5))]
    np.testing.assert_allclose(O.mlp(layers2, x), np.full((3, 5), layers2[0][1].sum()))


def test_weight_blob_shapes_and_storage_pin():
    # Table 2: 3.6 MiB of fp32 parameters for both networks of DONeRF with
    # the paper's 390-input depth network (unified origin + direction + 128
    # positions); 3.2 MiB for NeRF's two shading-shaped networks.
    d = 390 * 256 + 256 + 6 * (256 * 256 + 256) + 256 * 128 + 128
    s = 63 * 256 + 256 + 6 * (256 * 256 + 256) + 283 * 4 + 4
    assert abs((d + s) * 4 / 2 ** 20 - 3.6) < 0.05
    # NeRF's networks are only described as slightly adapted: within 2 %.
    assert abs(2 * s * 4 / 2 ** 20 - 3.2) / 3.2 < 0.02
    blob = inputs.make_weights(128, 0)
    dl, sl = O.split_weights(blob, 128)
    assert [W.shape for W, _ in dl] == [(256, 90)] + [(256, 256)] * 6 + [(128, 256)]
    assert [W.shape for W, _ in sl] == [(256, 63)] + [(256, 256)] * 6 + [(4, 283)]
    with pytest.raises(ValueError):
        O.split_weights(blob[:-1], 128)


def test_flops_reproduce_paper_table2():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "table2_mflop_per_pixel.txt"))
            if l.strip() and not l.startswith("#")]
    for method, n, _storage, mflop in rows:
        n, mflop = int(n), float(mflop)
        if method == "donerf":
            # the paper's depth network: the unencoded input of Sec. 5.2
            got = 2 * O.mlp_macs_per_ray(n, n_bins=128, d_in=O.depth_in_dims(128, "positions")) / 1e6
        else:  # NeRF: n evaluations of the shading-shaped network
            per_eval = O.mlp_macs_per_ray(1) - O.mlp_macs_per_ray(0)
            got = 2 * n * per_eval / 1e6
        assert abs(got - mflop) / mflop < 0.012, (method, n, got, mflop)


# ------------------------------------------------------------------ selection

def test_topn_matches_sorted_brute_force():
    rng = np.random.default_rng(7)
    for mode in ("normal", "ties", "const", "special"):
        lg = inputs.random_logits(300, 16, seed=3, mode=mode)
        for N in (1, 2, 4, 8, 16):
            got = O.topn(lg, N)
            for r in range(lg.shape[0]):
                # NaN after every number (-inf included), then by index
                def rank(i):
                    x = float(lg[r, i])
                    return (1, 0.0, i) if math.isnan(x) else (0, -x, i)
                ref = sorted(sorted(range(16), key=rank)[:N])
                assert list(got[r]) == ref
    lg = rng.permutation(64).astype(F32)[None, :]
    assert list(O.topn(lg, 5)[0]) == sorted(np.argsort(-lg[0])[:5])
    assert list(O.topn(np.zeros((1, 32), F32), 4)[0]) == [0, 1, 2, 3]


def test_softmax_is_monotone_and_normalised():
    lg = inputs.random_logits(50, 128, seed=1)
    p = O.softmax_fp32(lg)
    np.testing.assert_allclose(p.sum(1), 1.0, atol=1e-5)
    distinct = np.array([len(set(row)) == len(row) for row in p])
    assert np.array_equal(O.topn(p[distinct], 4), O.topn(lg[distinct], 4))
    ref = torch.softmax(torch.from_numpy(lg).double(), dim=1).numpy()
    np.testing.assert_allclose(p, ref, rtol=2e-6, atol=1e-9)


# ------------------------------------------------------------------ compositing

def test_single_opaque_sample_reproduces_its_colour():
    raw = np.array([[[0.3, -1.2, 2.0, 0.0], [1.0, 0.5, -0.5, 1e4], [2.0, 2.0, 2.0, 5.0]]])
    t = np.array([[1.0, 2.0, 3.0]])
    delta = np.array([[0.1, 0.1, 0.1]])
    C, D, W = O.composite(raw, t, delta)
    sig = 1 / (1 + np.exp(-raw[0, 1, :3]))
    np.testing.assert_array_equal(C[0], sig)
    assert D[0] == 2.0 and W[0, 2] == 0.0


def test_weights_sum_at_most_one_and_closed_form():
    rng = np.random.default_rng(8)
    raw = rng.standard_normal((2000, 8, 4)) * 3
    t = np.sort(rng.uniform(0.1, 10, (2000, 8)), axis=1)
    delta = rng.uniform(0.01, 0.3, (2000, 8))
    C, D, W = O.composite(raw, t, delta)
    tau = np.maximum(raw[..., 3], 0) * delta
    np.testing.assert_allclose(W.sum(1), 1 - np.exp(-tau.sum(1)), atol=1e-12)
    assert np.all(W.sum(1) <= 1 + 1e-12)
    cum = np.concatenate([np.zeros((2000, 1)), np.cumsum(tau, 1)[:, :-1]], 1)
    np.testing.assert_allclose(W, np.exp(-cum) * (1 - np.exp(-tau)), atol=1e-12)
    assert np.all((C >= 0) & (C <= 1))
    z = raw.copy()
    z[..., 3] = -1.0
    C0, D0, _ = O.composite(z, t, delta)
    assert np.all(C0 == 0) and np.all(D0 == 0)


def test_one_sample_closed_form():
    raw = np.array([[[0.7, -0.2, 0.1, 2.5]]])
    C, D, _ = O.composite(raw, np.array([[4.0]]), np.array([[0.2]]))
    a = 1 - math.exp(-2.5 * 0.2)
    np.testing.assert_allclose(C[0], a / (1 + np.exp(-raw[0, 0, :3])), rtol=1e-14)
    np.testing.assert_allclose(D[0], a * 4.0, rtol=1e-14)
