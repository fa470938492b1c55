"""Every layer of the depth-oracle network, teacher-forced, through the C ABI.

Probe networks read one layer's activations out of the production kernel:
layers 0..k carry the real weights, layers k+1..6 are identities and the head
(256 classes) is the identity, so the dumped scores are layer k's outputs
exactly (identity weights pass bf16 and E4M3 values unchanged; ReLU keeps
the non-negative activations; the E4M3 scale of an identity layer is 2^8,
exact).  Layer k is then evaluated by the oracle on the GPU's own output of
layer k - 1 (layer 0 on the GPU's encoded features, read out the same way):
every GPU activation must lie in the oracle's interval of valid outputs
(``O.valid_activations``: the rounded values an fp32 accumulation of that
sum in any order can produce), which is a single value, bit for bit, for
every unit whose exact pre-activation is not within the bound of a rounding
midpoint.  The real head is checked on the GPU's last hidden layer the same
way.  A variant scales one layer's weights so that a quarter of its
activations exceed the E4M3 range and take the clamp.

The shading network runs the same layer code (the same function templates,
fed from the sample encoding) and is checked end to end in the parity
tests."""
import numpy as np
import pytest
import torch

from oracle import donerf_oracle as O
from paper_2103_03231_amd import binding as b
from paper_2103_03231_amd import inputs

pytestmark = pytest.mark.gpu

PREC = {"fp32": b.FP32, "bf16": b.BF16, "fp8": b.FP8}
POSES = [0, 9]
H, W, N = 24, 40, 4


def _blob(d_layers, s_layers):
    return np.concatenate([np.concatenate([np.asarray(Wt, np.float32).ravel(), np.asarray(bt, np.float32)])
                           for Wt, bt in d_layers + s_layers])


def _identity():
    return np.eye(256, dtype=np.float32), np.zeros(256, np.float32)


def _scores(precision, blob, n_bins):
    r = b.Renderer(b.Config(n_bins=n_bins, n_max=N, precision=PREC[precision]), blob)
    out = r.render(inputs.make_poses(POSES), H, W, N, debug=True)
    torch.cuda.synchronize()
    s = out["scores"].cpu().numpy().reshape(-1, n_bins).astype(np.float64)
    r.close()
    return s


def _gpu_features(precision):
    """The 90 encoded inputs the kernel feeds the depth network: units 2f and
    2f + 1 of layer 0 hold ReLU(x_f) and ReLU(-x_f), the head subtracts them
    (one nonzero product per sum: exact).  An fp8 network encodes like a
    bf16 one (its first layer is bf16), so its features are read with bf16."""
    W0 = np.zeros((256, 90), np.float32)
    W7 = np.zeros((128, 256), np.float32)
    for f in range(90):
        W0[2 * f, f], W0[2 * f + 1, f] = 1.0, -1.0
        W7[f, 2 * f], W7[f, 2 * f + 1] = 1.0, -1.0
    d = [(W0, np.zeros(256, np.float32))] + [_identity()] * 6 + [(W7, np.zeros(128, np.float32))]
    s = O.split_weights(inputs.make_weights(128, 0), 128)[1]
    return _scores("bf16" if precision == "fp8" else precision, _blob(d, s), 128)[:, :90]


@pytest.mark.parametrize("precision,hot", [("fp32", False), ("bf16", False), ("fp8", False), ("fp8", True)])
def test_depth_layers_teacher_forced(precision, hot):
    d_real, s_real = O.split_weights(inputs.make_weights(256, 0), 256)
    d_real = [(Wt.astype(np.float32), bt.astype(np.float32)) for Wt, bt in d_real]
    if hot:
        # layer 1 scaled so that many of its outputs exceed 448 and clamp
        d_real[1] = (d_real[1][0] * np.float32(600.0), d_real[1][1] * np.float32(600.0))
    oracle_layers = [(Wt.astype(np.float64), bt.astype(np.float64)) for Wt, bt in d_real]
    h = _gpu_features(precision)
    for k in range(7):
        probe = d_real[:k + 1] + [_identity()] * (6 - k) + [_identity()]
        g = _scores(precision, _blob(probe, s_real), 256)
        y, beta, rounding = O.layer_preactivation(oracle_layers, k, h, precision)
        lo, hi = O.valid_activations(y, beta, rounding)
        inside = (g >= lo) & (g <= hi)
        single = lo == hi
        tag = f"[{precision}{' hot' if hot else ''} layer {k}] units {g.size}:"
        if rounding == "none":
            live = y > beta
            print(f"{tag} max |h - exact| / bound {np.max(np.abs(g - y)[live] / beta[live]):.3e}", flush=True)
        else:
            other = int(np.sum(g != O.activation(y, rounding)))
            print(f"{tag} single valid value {single.mean():.4f}, rounded the other way {other}, "
                  f"clamped {np.mean(g == 448.0):.4f}", flush=True)
        assert inside.all(), (k, np.argwhere(~inside)[:5])
        if hot and k == 1:
            assert np.mean(g == 448.0) > 0.1
        h = g
    # the real head on the GPU's last hidden layer
    g = _scores(precision, _blob(d_real, s_real), 256)
    y, beta, rounding = O.layer_preactivation(oracle_layers, 7, h, precision)
    lo, hi = O.valid_activations(y, beta, rounding)
    err = np.abs(g - y)
    print(f"[{precision}{' hot' if hot else ''} head] max |score - exact| {err.max():.3e}, "
          f"max share of the bound {np.max(err / beta):.3e}", flush=True)
    assert np.all((g >= lo) & (g <= hi))
