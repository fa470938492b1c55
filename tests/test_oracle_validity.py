"""Pins for the oracle's checking aids: the fp32 accumulation bound, the
interval of valid rounded outputs, the per-layer view of the networks and the
accumulation jitter.  These are not steps of the method; they let a test
tell a GPU result that rounded a near-tied value the other way from a wrong
one, so each is pinned against brute force or a hand-built case."""
import numpy as np

from oracle import donerf_oracle as O

F32 = np.float32


def _fp32_sum(terms, order, truncate=False):
    """Sum in fp32, one rounding per addition, in the given order; truncate
    rounds each partial sum toward zero instead of to nearest."""
    s = F32(0.0)
    for i in order:
        exact = np.float64(s) + np.float64(terms[i])
        r = F32(exact)
        if truncate and abs(np.float64(r)) > abs(exact):
            r = np.nextafter(r, F32(0.0))
        s = r
    return np.float64(s)


def test_accumulation_bound_covers_fp32_sums_in_any_order():
    rng = np.random.default_rng(0)
    for K, bf16 in ((8, True), (64, True), (256, True), (256, False), (96, True)):
        W = rng.uniform(-0.15, 0.15, size=(3, K))
        h = np.maximum(rng.normal(size=(2, K)), 0.0)
        b = rng.uniform(-0.1, 0.1, size=3)
        if bf16:
            W, h = O.round_bf16(W), O.round_bf16(h)
        else:
            W, h = W.astype(F32).astype(np.float64), h.astype(F32).astype(np.float64)
        beta = O.accumulation_bound(h, W, b.astype(F32).astype(np.float64))
        exact = h @ W.T + b.astype(F32)
        for r in range(2):
            for o in range(3):
                terms = [F32(h[r, k] * W[o, k]) for k in range(K)] + [F32(b[o])]
                n = len(terms)
                orders = [range(n), range(n - 1, -1, -1)] + [rng.permutation(n) for _ in range(10)]
                for order in orders:
                    for trunc in (False, True):
                        got = _fp32_sum(terms, order, trunc)
                        assert abs(got - exact[r, o]) <= beta[r, o], (K, bf16, trunc)
    # the closed form on a hand case: K = 2, |terms| = 1 + 2 + 0.5 -> (K + 2) u / (1 - (K + 2) u) * 3.5
    beta = O.accumulation_bound(np.array([[1.0, 2.0]]), np.array([[1.0, -1.0]]), np.array([0.5]))
    n = 4
    assert beta[0, 0] == n * 2.0 ** -23 / (1 - n * 2.0 ** -23) * 3.5


def test_valid_activations_on_a_midpoint_and_far_from_one():
    """A tiny layer built to put its pre-activation exactly on a bf16
    rounding midpoint (1 + 2^-8, between 1 and 1 + 2^-7) may round either
    way; one landing on a bf16 value far from every midpoint has a single
    valid output."""
    h = np.array([[1.0, 1.0]])
    on_mid = [(np.array([[0.5, 0.50390625]]), np.array([0.0]))]
    far = [(np.array([[0.5, 0.5]]), np.array([0.0]))]
    for layers, expect in ((on_mid, (1.0, 1.0078125)), (far, (1.0, 1.0))):
        y, beta, _ = O.layer_preactivation(layers + [(np.eye(1), np.zeros(1))], 0, h, "bf16")
        assert beta[0, 0] > 0
        lo, hi = O.valid_activations(y, beta, "bf16")
        assert (lo[0, 0], hi[0, 0]) == expect
        nominal = O.activation(y, "bf16")[0, 0]
        assert lo[0, 0] <= nominal <= hi[0, 0]
    # E4M3: 17 lies midway between 16 and 18, 20 on the grid; the clamp and
    # the ReLU flatten the ends
    small = np.full((1, 1), 1e-6)
    cases = {17.0: (16.0, 18.0), 20.0: (20.0, 20.0), 500.0: (448.0, 448.0), 440.0: (448.0, 448.0),
             -3.0: (0.0, 0.0)}
    for y, expect in cases.items():
        lo, hi = O.valid_activations(np.full((1, 1), y), small, "e4m3")
        assert (lo[0, 0], hi[0, 0]) == expect, y
    lo, hi = O.valid_activations(np.zeros((1, 1)), small, "bf16")
    assert lo[0, 0] == 0.0 and hi[0, 0] > 0.0            # the ReLU's edge is within reach
    lo, hi = O.valid_activations(np.full((1, 1), -2.0), small, None)   # a head: no ReLU
    assert lo[0, 0] == -2.0 - 1e-6 and hi[0, 0] == -2.0 + 1e-6


def test_layer_arithmetic_of_the_networks():
    n = 8
    kinds = [O.layer_arithmetic("fp8", li, n) for li in range(n)]
    assert [k[1] for k in kinds] == ["bf16"] + ["fp8"] * 6 + ["bf16"]
    assert [k[2] for k in kinds] == ["e4m3"] * 6 + ["bf16", None]
    assert [O.layer_arithmetic("bf16", li, n)[2] for li in range(n)] == ["bf16"] * 7 + [None]
    assert [O.layer_arithmetic("fp64", li, n)[2] for li in range(n)] == ["none"] * 7 + [None]
    W = np.array([[0.3, -0.1, 1e-6]])
    assert np.array_equal(kinds[3][0](W), O.quantize_fp8_weights(W))
    assert np.array_equal(kinds[0][0](W), O.round_bf16(W))


def _net(rng, dims):
    return [(rng.uniform(-0.3, 0.3, size=(o, i)), rng.uniform(-0.1, 0.1, size=o)) for i, o in zip(dims, dims[1:])]


def test_layers_fed_their_own_inputs_reproduce_the_network():
    """Teacher forcing with the oracle's own chain: each layer evaluated by
    layer_preactivation on the input mlp fed it gives mlp's pre-activation,
    and its activation is the next layer's input."""
    rng = np.random.default_rng(3)
    layers = _net(rng, [9, 16, 16, 16, 5])
    x = rng.uniform(-1, 1, size=(6, 9))
    for prec in ("fp64", "bf16", "fp8"):
        trace = []
        out = O.mlp(layers, x, prec, trace=trace)
        for li, (h, Wq, b, y, rnd) in enumerate(trace):
            y2, beta, rnd2 = O.layer_preactivation(layers, li, h, prec)
            assert np.array_equal(y, y2) and rnd == rnd2 and np.all(beta > 0)
            nxt = trace[li + 1][0] if li + 1 < len(trace) else out
            assert np.array_equal(O.activation(y, rnd), nxt)


def test_jitter_stays_within_the_bound_and_zero_jitter_is_nominal():
    rng = np.random.default_rng(5)
    layers = _net(rng, [9, 32, 32, 32, 4])
    x = rng.uniform(-1, 1, size=(50, 9))
    skip = rng.uniform(-1, 1, size=(50, 3))
    layers[-1] = (rng.uniform(-0.3, 0.3, size=(4, 35)), layers[-1][1])
    for prec in ("fp64", "bf16", "fp8"):
        nominal = O.mlp(layers, x, prec, skip=skip)
        zero = {"fp64": 0.0, "bf16": 0.0, "fp8": 0.0, "input": 0.0}
        assert np.array_equal(O.mlp(layers, x, prec, skip=skip, jitter=(np.random.default_rng(1), zero)), nominal)
        rho = {"fp64": 0.5, "bf16": 0.5, "fp8": 0.5}
        trace = []
        jit = O.mlp(layers, x, prec, skip=skip, jitter=(np.random.default_rng(2), rho), trace=trace)
        assert not np.array_equal(jit, nominal)
        for li, (h, Wq, b, y, rnd) in enumerate(trace):
            exact = h @ Wq.T + b
            beta = O.accumulation_bound(h, Wq, b)
            assert np.all(np.abs(y - exact) <= 0.5 * beta)
            assert np.any(y != exact)
