"""Pins for the training-target and loss oracle (Sec. 5.1 Eq. 6-8, Sec. 6.1
Eq. 9-10): the paper's worked example of the neighbourhood filter, closed
forms of the two filters, brute force on tiny depth maps, invariants the
text states, and the class boundaries against Eq. 3 written out here."""
import math
import os

import numpy as np
import pytest

from oracle import targets_oracle as T

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
NEAR, FAR = 0.1, 10.0
F32 = np.float32


def _class_closed_form(d, B):
    # Eq. 3's coordinate of d, scaled to B classes (floor)
    near, far = float(F32(NEAR)), float(F32(FAR))
    return np.floor(B * np.log(d - near + 1.0) / np.log(far - near + 1.0)).astype(int)


def test_worked_example_of_the_neighbourhood_filter():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "eq7_neighbourhood_5x5.txt"))
            if l.strip() and not l.startswith("#")]
    B, H, W = 8, 9, 9
    depth = np.full((H, W), np.inf, F32)
    depth[4, 4] = 1.0                                   # one surface at the centre pixel
    z = int(T.depth_classes(np.array([1.0], F32), NEAR, FAR, B)[0])
    Chat = T.neighbourhood_filter(T.one_hot_targets(depth, NEAR, FAR, B), 5)
    for di, dj, want, tol in rows:
        got = Chat[4 + int(di), 4 + int(dj), z]
        assert abs(got - float(want)) <= float(tol), (di, dj, got)
    # outside the window nothing arrives; other classes stay 0
    assert Chat[4, 7, z] == 0.0 and Chat[1, 4, z] == 0.0
    assert np.all(np.delete(Chat, z, axis=2) == 0.0)


def _brute(depth, B, K, Z):
    H, W = depth.shape
    cls = T.depth_classes(depth, NEAR, FAR, B)
    h, hz = K // 2, Z // 2
    out = np.zeros((H, W, B))
    for y in range(H):
        for x in range(W):
            chat = []
            for z in range(B):
                best = -math.inf
                for i in range(-h, h + 1):
                    for j in range(-h, h + 1):
                        if 0 <= y + i < H and 0 <= x + j < W:
                            c = 1.0 if cls[y + i, x + j] == z else 0.0
                            dist = math.sqrt(i * i + j * j) / (math.sqrt(2) * h) if h else 0.0
                            best = max(best, c - dist)
                chat.append(best)
            for z in range(B):
                s = 0.0
                for i in range(-hz, hz + 1):
                    if 0 <= z + i < B:
                        s += chat[z + i] * (hz + 1 - abs(i)) / (hz + 1)
                out[y, x, z] = min(s, 1.0)
    return out


@pytest.mark.parametrize("K,Z", [(1, 1), (3, 3), (5, 5), (5, 1), (1, 5), (9, 3), (2, 4), (4, 2), (6, 6)])
def test_brute_force(K, Z):
    rng = np.random.default_rng(K * 10 + Z)
    depth = rng.uniform(0.05, 11.0, size=(6, 7)).astype(F32)   # some below near, some beyond far
    depth[0, 0] = np.inf
    depth[2, 3] = np.nan
    got = T.training_targets(depth, NEAR, FAR, 8, K, Z)
    np.testing.assert_allclose(got, _brute(depth, 8, K, Z), rtol=0, atol=1e-12)


def test_closed_forms():
    rng = np.random.default_rng(1)
    depth = rng.uniform(0.1, 9.9, size=(5, 6)).astype(F32)
    C = T.one_hot_targets(depth, NEAR, FAR, 16)
    assert np.all(C.sum(-1) == 1.0)                               # one class per surface
    np.testing.assert_array_equal(T.neighbourhood_filter(C, 1), C)  # K = 1: the pixel itself
    np.testing.assert_array_equal(T.depth_filter(C, 1), C)          # Z = 1: identity
    # a lone class far from the ends spreads as the triangle (h + 1 - |i|)/(h + 1)
    one = np.zeros((1, 1, 32))
    one[0, 0, 10] = 1.0
    np.testing.assert_allclose(T.depth_filter(one, 5)[0, 0, 8:13], [1 / 3, 2 / 3, 1, 2 / 3, 1 / 3])
    np.testing.assert_allclose(T.depth_filter(one, 3)[0, 0, 9:12], [0.5, 1, 0.5])
    # two neighbouring classes: the sum passes 1 and is clamped
    two = one.copy()
    two[0, 0, 11] = 1.0
    f = T.depth_filter(two, 5)[0, 0]
    assert f[10] == 1.0 and f[11] == 1.0 and abs(f[12] - 1.0) < 1e-12 and abs(f[9] - 1.0) < 1e-12


def test_invariants_stated_by_the_paper():
    rng = np.random.default_rng(2)
    depth = rng.uniform(0.1, 9.9, size=(12, 13)).astype(F32)
    depth[rng.uniform(size=depth.shape) < 0.1] = np.inf
    C = T.one_hot_targets(depth, NEAR, FAR, 32)
    Chat = T.neighbourhood_filter(C, 5)
    Cg = T.depth_filter(Chat, 5)
    assert np.all(Chat >= C) and np.all(Chat >= 0.0) and np.all(Chat <= 1.0)
    assert np.all((Cg >= 0.0) & (Cg <= 1.0))
    # the largest value sits at the actual surface (value 1 there)
    cls = T.depth_classes(depth, NEAR, FAR, 32)
    ys, xs = np.nonzero(cls >= 0)
    assert np.all(Chat[ys, xs, cls[ys, xs]] == 1.0)
    assert np.all(Cg[ys, xs, cls[ys, xs]] == 1.0)


def test_depth_classes_against_eq3():
    B = 64
    rng = np.random.default_rng(3)
    d = rng.uniform(0.1, 10.0, 5000).astype(F32)
    got = T.depth_classes(d, NEAR, FAR, B)
    ref = _class_closed_form(d.astype(np.float64), B)
    # equal except where d sits within rounding of a class bound
    assert np.mean(got == ref) > 0.999
    from oracle.donerf_oracle import bin_table
    bounds, _, _ = bin_table(NEAR, FAR, B)
    np.testing.assert_array_equal(T.depth_classes(bounds[:-1], NEAR, FAR, B), np.arange(B))   # b_k -> k
    below = np.nextafter(bounds[1:], np.float32(-np.inf))
    np.testing.assert_array_equal(T.depth_classes(below, NEAR, FAR, B), np.arange(B))        # just below b_{k+1}
    edge = np.array([bounds[-1], np.inf, np.nan, np.nextafter(bounds[0], np.float32(-1)), -1.0], F32)
    np.testing.assert_array_equal(T.depth_classes(edge, NEAR, FAR, B), [-1] * 5)            # far, inf, nan, < near


def test_opacity_and_total_loss():
    w = np.array([[0.2, 0.3], [0.6, 0.5], [0.0, 0.0], [1.0, 0.0]])
    np.testing.assert_allclose(T.opacity_loss(w), [0.25, 0.0, 1.0, 0.0])
    rgb = np.array([[0.5, 0.5, 0.5]] * 4)
    ref = np.array([[0.6, 0.5, 0.5]] * 4)
    # mse = 0.01 / 3; mean opacity loss = 0.3125; alpha 1, beta 10 (Sec. 6.1)
    assert abs(T.total_loss(rgb, ref, w) - (0.01 / 3 + 3.125)) < 1e-12
    assert abs(T.total_loss(rgb, ref, w, alpha=2.0, beta=0.0) - 2 * 0.01 / 3) < 1e-12


@pytest.mark.parametrize("K", [2, 4, 6, 14])
def test_even_window_is_the_next_odd_one(K):
    """Eq. 7 and Eq. 8 see K and Z only through floor(K/2) and floor(Z/2):
    an even size gives the targets of the odd size above it."""
    rng = np.random.default_rng(K)
    depth = rng.uniform(0.05, 11.0, size=(9, 11)).astype(F32)
    a = T.training_targets(depth, NEAR, FAR, 16, K, K)
    c = T.training_targets(depth, NEAR, FAR, 16, K + 1, K + 1)
    assert np.array_equal(a, c)
    # Eq. 7 alone: the window of K reaches a neighbour that the one of K - 1
    # (half width one less) does not, so the two differ
    C = T.one_hot_targets(depth, NEAR, FAR, 16)
    assert not np.array_equal(T.neighbourhood_filter(C, K), T.neighbourhood_filter(C, K - 1))


@pytest.mark.parametrize("H,W,K", [(2, 7, 9), (6, 1, 15), (1, 1, 5), (3, 2, 14)])
def test_window_larger_than_the_image(H, W, K):
    """Offsets that leave the image for every pixel contribute nothing."""
    rng = np.random.default_rng(H * 100 + W * 10 + K)
    depth = rng.uniform(0.05, 11.0, size=(H, W)).astype(F32)
    got = T.training_targets(depth, NEAR, FAR, 8, K, 3)
    np.testing.assert_allclose(got, _brute(depth, 8, K, 3), rtol=0, atol=1e-12)
