"""CPU oracle for DONeRF per-ray inference.  TEST INFRASTRUCTURE ONLY.

Only the test suite, the package's smoke check and the benchmark's CPU
baseline leg may import this module.  The rendering library never calls it.
The oracle shares no code with the HIP path.

It follows DONeRF (Neff et al., EGSR 2021, arXiv 2103.03231) one step at a time:

  ray through a pixel (Sec. 4, Eq. 1)
  -> ray unification onto the view-cell sphere (Sec. 5.2, Fig. 8)
  -> encoded depth-network input, normalised by d_max (Sec. 4, Eq. 2), or the
     paper's unencoded input: unified origin, direction and one position per
     depth-class centre (Sec. 5.2, App. D)
  -> depth-oracle network, 8 linear layers of 256 units (Sec. 5.3, App. D)
  -> log-discretised depth bins (Sec. 4, Eq. 3; Sec. 5.2) and top-N selection
  -> samples x = o + t r (Eq. 1) at the selected bin centres
  -> space warp (Sec. 4, Eq. 4-5) and encoding
  -> shading network with the encoded direction skipped into its last layer
     (App. D, Fig. 12)
  -> alpha compositing with a black background (Sec. 3, Sec. 6.1).

Precision.  Ray geometry (ray, unification, sample placement, warp) runs in
fp32 with the operation order written below, so that a fp32 implementation
with the same order reproduces it bit for bit.  Encodings, matrix products
(fp64 accumulation) and compositing run in fp64.  In ``precision='bf16'`` the
oracle rounds to bf16 (round-to-nearest-even) exactly where a bf16 network
does: weights, encoded features and each hidden activation after bias + ReLU
(the unencoded positions input is not rounded).
Values are first rounded to fp32 and then to bf16.  Logits and head outputs
stay unrounded.  ``precision='fp8'`` is the mixed network of ``mlp_fp8``.

Readings where the paper is silent are listed in the design document; each
function names the one it uses.

Every function is pinned by ``tests/test_oracle_pins.py`` (and the
``test_oracle_*.py`` files beside it) against closed forms, invariants, the
paper's Table 2 and brute force on tiny inputs.
"""
from __future__ import annotations

import math

import numpy as np

F32 = np.float32
HIDDEN = 256
L_POS = 10
L_DIR = 4


# ---------------------------------------------------------------- rounding

def round_bf16(x) -> np.ndarray:
    """Round to bf16 (round-to-nearest-even on the fp32 bit pattern), returned
    as float64 holding the bf16 value.  Values are first rounded to fp32."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(F32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    out = (r & np.uint64(0xFFFFFFFF)).astype(np.uint32).view(F32)
    nan = np.isnan(f)
    if nan.any():
        out = np.where(nan, f, out)
    return out.astype(np.float64)


E4M3_MAX = 448.0


def round_e4m3(x) -> np.ndarray:
    """Round to the OCP fp8 E4M3 grid (1 sign, 4 exponent bits with bias 7,
    3 mantissa bits; subnormals of quantum 2^-9; largest finite 448), round to
    nearest, ties to even.  Defined for |x| <= 448 (values are clamped before
    they are rounded).  Returned as float64 holding the fp8 value."""
    x = np.asarray(x, dtype=np.float64)
    if np.any(np.abs(x) > E4M3_MAX):
        raise ValueError("round_e4m3: |x| > 448")
    a = np.abs(x)
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    # quantum: 2^(e - 3) for normal values (e >= -6), 2^-9 below
    q = np.exp2(np.maximum(e, -6.0) - 3.0)
    # np.rint rounds half to even; an even multiple of the quantum is an even code
    return np.sign(x) * np.rint(a / q) * q


def fp8_weight_scale(W) -> int:
    """Per-layer power-of-two scale of the fp8 weights: the largest integer s
    with max|W| 2^s <= 448, or 0 for an all-zero layer."""
    m = float(np.max(np.abs(np.asarray(W, dtype=np.float64)))) if np.size(W) else 0.0
    if m == 0.0:
        return 0
    s = int(math.floor(math.log2(E4M3_MAX / m)))
    while m * 2.0 ** (s + 1) <= E4M3_MAX:
        s += 1
    while m * 2.0 ** s > E4M3_MAX:
        s -= 1
    return s


def quantize_fp8_weights(W) -> np.ndarray:
    """fp8 weights as the network uses them: W 2^s rounded to E4M3 (from the
    fp32 value), times 2^-s."""
    W32 = np.asarray(W, dtype=np.float64).astype(F32).astype(np.float64)
    s = fp8_weight_scale(W32)
    return round_e4m3(W32 * 2.0 ** s) * 2.0 ** -s


# ---------------------------------------------------------------- depth bins

def log_depth(d, near, far):
    """Eq. 3: the logarithmic depth map, depth -> network coordinate."""
    d = np.asarray(d, dtype=np.float64)
    span = far - near
    return near + np.log(d - near + 1.0) / np.log(span + 1.0) * span


def bin_table(near, far, n_bins):
    """Depth classes uniform in the log coordinate of Eq. 3 (Sec. 5.2 applies
    the same transform to the classification steps).

    Boundaries are the inverse of Eq. 3 at B+1 uniform coordinates,
    b_k = d_min + (D+1)^(k/B) - 1 with b_0 = d_min and b_B = d_max exactly;
    centres are the inverse at the mid coordinates (k+0.5)/B; widths are
    b_{k+1} - b_k.  Computed in fp64, returned as fp32.  near/far are taken as
    fp32 values first (the C ABI stores them as fp32)."""
    near = float(F32(near))
    far = float(F32(far))
    span = far - near
    k = np.arange(n_bins + 1, dtype=np.float64)
    b = near + np.power(span + 1.0, k / n_bins) - 1.0
    b[0] = near
    b[n_bins] = far
    kc = np.arange(n_bins, dtype=np.float64) + 0.5
    c = near + np.power(span + 1.0, kc / n_bins) - 1.0
    w = b[1:] - b[:-1]
    return b.astype(F32), c.astype(F32), w.astype(F32)


# ---------------------------------------------------------------- geometry (fp32)

def focal_px(W, fov_x_deg):
    """Pinhole focal length in pixels for a horizontal field of view (fp64,
    rounded to fp32)."""
    fov = float(F32(fov_x_deg))
    return F32((0.5 * W) / math.tan(fov * (math.pi / 180.0) * 0.5))


def camera_rays(pose, H, W, fov_x_deg):
    """Eq. 1's ray o + d r through each pixel centre.  OpenGL camera: the
    camera looks down its -z axis, +y up, pixel (i, j) with i along the width
    and j down the image.  Returns o (H*W, 3) and unit r (H*W, 3), fp32,
    rays in row-major pixel order."""
    pose = np.asarray(pose, dtype=F32)
    f = focal_px(W, fov_x_deg)
    i = np.arange(W, dtype=F32)
    j = np.arange(H, dtype=F32)
    u = ((i + F32(0.5)) - F32(0.5 * W)) / f
    v = -(((j + F32(0.5)) - F32(0.5 * H)) / f)
    U = np.broadcast_to(u[None, :], (H, W)).reshape(-1)
    V = np.broadcast_to(v[:, None], (H, W)).reshape(-1)
    R = pose[:, :3]
    d = [(R[a, 0] * U + R[a, 1] * V) + R[a, 2] * F32(-1.0) for a in range(3)]
    n = np.sqrt((d[0] * d[0] + d[1] * d[1]) + d[2] * d[2])
    r = np.stack([d[0] / n, d[1] / n, d[2] / n], axis=1)
    o = np.broadcast_to(pose[:, 3], r.shape).astype(F32)
    return o, r


def dot3(a, b):
    return (a[:, 0] * b[:, 0] + a[:, 1] * b[:, 1]) + a[:, 2] * b[:, 2]


def unify(o, r, centre, radius):
    """Sec. 5.2, Fig. 8: move each ray origin onto the sphere of the given
    radius around the view-cell centre, along the ray (the forward root of
    |o + t r - c| = R, clamped at t >= 0; the paper's case of rays looking out
    of the view cell)."""
    c = np.asarray(centre, dtype=F32)
    R = F32(radius)
    q = o - c
    b = dot3(r, q)
    k = dot3(q, q) - R * R
    disc = np.maximum(b * b - k, F32(0.0))
    t = np.maximum(-b + np.sqrt(disc), F32(0.0))
    return o + t[:, None] * r


def sample_points(o, r, t):
    """Eq. 1: x = o + t r for each ray (o, r: (n,3); t: (n, N)) -> (n, N, 3)."""
    return o[:, None, :] + t[:, :, None] * r[:, None, :]


def warp(x, centre, d_max):
    """Eq. 4-5: p = x - c scaled by W(p) = 1/sqrt(|p| d_max), evaluated as
    p / sqrt(|p| d_max); the warp of p = 0 is 0."""
    c = np.asarray(centre, dtype=F32)
    p = (x - c).astype(F32)
    n = np.sqrt((p[..., 0] * p[..., 0] + p[..., 1] * p[..., 1]) + p[..., 2] * p[..., 2])
    s = np.sqrt(n * F32(d_max))
    with np.errstate(divide="ignore", invalid="ignore"):
        w = p / s[..., None]
    return np.where((n == 0)[..., None], F32(0.0), w).astype(F32)


# ---------------------------------------------------------------- encoding (fp64)

def encode(v, L):
    """The paper's encode() (Eq. 2, Eq. 4), read as NeRF's Fourier features
    with the identity kept: [v, sin(2^0 pi v), cos(2^0 pi v), ...,
    sin(2^(L-1) pi v), cos(2^(L-1) pi v)], each block over x, y, z.
    Output 3 + 6L values in fp64."""
    v = np.asarray(v, dtype=np.float64)
    out = [v]
    for k in range(L):
        a = math.pi * (2.0 ** k) * v
        out.append(np.sin(a))
        out.append(np.cos(a))
    return np.concatenate(out, axis=-1)


# ---------------------------------------------------------------- networks

def depth_in_dims(n_bins, depth_input="encoded"):
    """Inputs of the depth network's first layer: 90 for the encoded unified
    origin and direction, 6 + 3 n_bins for the paper's unencoded input of
    Sec. 5.2 (unified origin, direction, one position per class centre)."""
    if depth_input == "encoded":
        return 3 + 6 * L_POS + 3 + 6 * L_DIR
    if depth_input == "positions":
        return 6 + 3 * n_bins
    raise ValueError(depth_input)


def split_weights(blob, n_bins, depth_input="encoded"):
    """Parse the flat fp32 blob (per layer W[out][in] row-major then b[out];
    depth network layers 0..7, then shading network layers 0..7) into two
    lists of (W, b) in fp64.  Shapes follow App. D: 8 layers of 256 units;
    the depth network maps its inputs (``depth_in_dims``) to n_bins classes;
    the shading network maps 63 encoded inputs to (r, g, b, sigma) and reads
    the 27 encoded direction values again in its last layer."""
    dims_in = depth_in_dims(n_bins, depth_input)
    shapes = ([(HIDDEN, dims_in)] + [(HIDDEN, HIDDEN)] * 6 + [(n_bins, HIDDEN)]
              + [(HIDDEN, 3 + 6 * L_POS)] + [(HIDDEN, HIDDEN)] * 6
              + [(4, HIDDEN + 3 + 6 * L_DIR)])
    blob = np.asarray(blob, dtype=F32)
    layers, off = [], 0
    for o, i in shapes:
        W = blob[off:off + o * i].reshape(o, i).astype(np.float64)
        off += o * i
        b = blob[off:off + o].astype(np.float64)
        off += o
        layers.append((W, b))
    if off != blob.size:
        raise ValueError(f"weight blob has {blob.size} values, expected {off}")
    return layers[:8], layers[8:]


def activation(y, rounding):
    """A hidden unit's output: ReLU of its pre-activation y, then the rounding
    point of the network ('bf16', 'e4m3' with the clamp at 448 the E4M3 range
    imposes, or 'none'); rounding None is a head's output, y itself.
    Monotone non-decreasing in y."""
    if rounding is None:
        return np.asarray(y, dtype=np.float64)
    r = np.maximum(y, 0.0)
    if rounding == "bf16":
        return round_bf16(r)
    if rounding == "e4m3":
        return round_e4m3(np.minimum(r, E4M3_MAX))
    return r


def layer_arithmetic(precision, li, n):
    """How layer li of an n-layer network of the given precision computes:
    (weights as the layer uses them, the arithmetic of its products - 'fp64',
    'bf16' or 'fp8' - and the rounding of its output for ``activation``).
    bf16: bf16 weights, outputs rounded to bf16.  fp8 (``mlp_fp8``): bf16
    first and last layers, fp8 weights elsewhere, outputs rounded to E4M3
    except the one the last layer reads (bf16).  The last layer's output is a
    head (no ReLU, no rounding)."""
    last = li == n - 1
    if precision == "fp8":
        bf16_layer = li in (0, n - 1)
        wq = round_bf16 if bf16_layer else quantize_fp8_weights
        kind = "bf16" if bf16_layer else "fp8"
        out = None if last else "bf16" if li == n - 2 else "e4m3"
    elif precision == "bf16":
        wq, kind, out = round_bf16, "bf16", (None if last else "bf16")
    else:
        wq, kind, out = (lambda a: np.asarray(a, dtype=np.float64)), "fp64", (None if last else "none")
    return wq, kind, out


def _jittered(y, h, Wq, b, kind, jitter):
    """y moved by an accumulation error the evaluation may make (see
    ``mlp``); y itself without jitter."""
    if jitter is None:
        return y
    rng, rho = jitter
    beta = accumulation_bound(h, Wq, b)
    return y + rho[kind] * beta * rng.uniform(-1.0, 1.0, size=y.shape)


def _jittered_input(x, jitter):
    """Encoded features moved by up to rho['input'] (absolute) before they are
    rounded: an evaluation of sine and cosine within that error (see ``mlp``)."""
    x = np.asarray(x, dtype=np.float64)
    if jitter is None or not jitter[1].get("input"):
        return x
    rng, rho = jitter
    return x + rho["input"] * rng.uniform(-1.0, 1.0, size=x.shape)


def mlp(layers, x, precision="fp64", skip=None, round_input=True, jitter=None, trace=None):
    """ReLU MLP: h = ReLU(W_l h + b_l) for every layer but the last, whose
    output is returned without activation.  ``skip`` (rows x s) is appended to
    the last layer's input (App. D's single direction skip).  x is (rows, in).
    In bf16 mode weights, inputs (unless ``round_input`` is false) and hidden
    activations are rounded to bf16; sums accumulate in fp64.  fp8 mode: the
    mixed network of ``mlp_fp8``.  Each layer computes as
    ``layer_arithmetic`` states.

    Checking aids, not part of the method: ``jitter = (rng, rho)`` moves every
    pre-activation by a uniform amount within rho[kind] times its
    ``accumulation_bound`` before the activation is taken (kind: 'fp64',
    'bf16' or 'fp8', the arithmetic of the layer's products), i.e. evaluates
    the network as an implementation whose sums carry that much error may;
    rho['input'] (optional) moves the rounded inputs (encoded features and
    the skip) by up to that absolute amount first, as an encoding whose sine
    and cosine carry that error may; ``trace`` (a list) receives (input,
    weights as used, bias, pre-activation, rounding of the output) per
    layer."""
    rb = round_bf16 if precision in ("bf16", "fp8") else (lambda a: np.asarray(a, dtype=np.float64))
    h = rb(_jittered_input(x, jitter)) if round_input else np.asarray(x, dtype=np.float64)
    n = len(layers)
    for li, (W, b) in enumerate(layers):
        if li == n - 1 and skip is not None:
            h = np.concatenate([h, rb(_jittered_input(skip, jitter))], axis=1)
        wq, kind, out_round = layer_arithmetic(precision, li, n)
        Wq = wq(W)
        y = _jittered(h @ Wq.T + b, h, Wq, b, kind, jitter)
        if trace is not None:
            trace.append((h, Wq, b, y, out_round))
        h = activation(y, out_round)
    return h


def mlp_fp8(layers, x, skip=None, round_input=True, jitter=None, trace=None):
    """The mixed fp8 network.  The paper leaves lower bit widths as future
    headroom (Sec. 6.1) and fixes no scheme; this one keeps the first and the
    last layer in bf16 (weights, inputs and skip rounded to bf16) and runs
    the hidden layers in fp8: weights by ``quantize_fp8_weights``, inputs in
    E4M3.  Each activation after bias and ReLU is clamped to 448 and rounded
    to E4M3 where an fp8 layer reads it; where the last layer reads it, it is
    rounded to bf16 (no clamp).  Sums accumulate in fp64.  ``jitter`` and
    ``trace`` as in ``mlp``."""
    return mlp(layers, x, "fp8", skip, round_input, jitter, trace)


def layer_preactivation(layers, li, h, precision):
    """Layer li of a network evaluated on a given input h (rows, in), as
    ``mlp`` evaluates it: returns the exact pre-activations (fp64), their
    ``accumulation_bound`` and the rounding of the layer's output.  A
    checking aid: it lets a test feed each layer the GPU's own output of the
    layer before ("teacher forcing")."""
    W, b = layers[li]
    wq, _, out_round = layer_arithmetic(precision, li, len(layers))
    Wq = wq(W)
    h = np.asarray(h, dtype=np.float64)
    return h @ Wq.T + b, accumulation_bound(h, Wq, b), out_round


def depth_positions_input(o, r, ou, centre, d_max, centres):
    """The depth network's input as Sec. 5.2 describes it, without encoding:
    the unified origin, the ray direction and one 3-D position along the ray
    at the centre of every depth class, positions and origin moved into the
    view cell's frame and divided by d_max as in Eq. 2.  The class centres are
    depths from the camera origin o (Eq. 1), so position k is o + c_k r.
    fp32 geometry in the written order; returns (n, 6 + 3 B) fp32 in the
    order [origin xyz, direction xyz, position 0 xyz, position 1 xyz, ...]."""
    c = np.asarray(centre, dtype=F32)
    d_max = F32(d_max)
    cen = np.asarray(centres, dtype=F32)
    v = ((ou - c) / d_max).astype(F32)
    x = sample_points(o, r, np.broadcast_to(cen[None, :], (o.shape[0], cen.size))).astype(F32)
    p = ((x - c) / d_max).astype(F32)
    return np.concatenate([v, r.astype(F32), p.reshape(o.shape[0], -1)], axis=1)


# ---------------------------------------------------------------- rounding validity (checking aids)

U_ACC = 2.0 ** -23


def accumulation_bound(h, Wq, b):
    """Bound on the error of the pre-activations Wq h + b when each is summed
    in fp32 in any order: for n terms, |fl(sum) - sum| <= gamma_(n-1) sum |terms|
    with gamma_k = k u / (1 - k u) (Higham, Accuracy and Stability of
    Numerical Algorithms, 2nd ed., Sec. 3.1).  n = K + 2 (K products, the
    bias, one spare rounding for fp32 products, which are not exact) and
    u = 2^-23, which covers round-to-nearest and truncating adders alike.
    A checking aid, not part of the method."""
    Wq = np.asarray(Wq, dtype=np.float64)
    n = Wq.shape[1] + 2
    gamma = n * U_ACC / (1.0 - n * U_ACC)
    return gamma * (np.abs(h) @ np.abs(Wq).T + np.abs(np.asarray(b, dtype=np.float64)))


def valid_activations(y, beta, rounding):
    """The outputs [lo, hi] a unit with exact pre-activation y may take when
    its sum carries an error of at most beta: ``activation`` is monotone, so
    every value it takes on [y - beta, y + beta] lies between its values at
    the ends; lo == hi where no rounding midpoint (and no ReLU or clamp edge)
    lies within beta of y.  A checking aid."""
    return activation(y - beta, rounding), activation(y + beta, rounding)


# ---------------------------------------------------------------- selection

def topn(logits, N):
    """The N highest-scoring depth classes per ray, ordered by (score desc,
    index asc), then returned in ascending index order (= depth order).  -0
    and +0 compare equal; NaN ranks below every number."""
    logits = np.asarray(logits, dtype=F32)
    nanmask = np.isnan(logits)
    key = np.where(nanmask, -np.inf, logits).astype(np.float64)
    # np.lexsort is stable: among equal scores the lower index stays first.
    # Primary key: descending score; secondary: NaN after every number.
    order = np.lexsort((nanmask, -key), axis=-1)
    return np.sort(order[:, :N], axis=1).astype(np.int32)


def softmax_fp32(logits):
    """Softmax over the classes in fp32: subtract the row maximum, exponentiate,
    sum in class order, divide.  Monotone in exact arithmetic; in fp32 it can
    map distinct logits to equal probabilities, so the selection of the
    softmax workload ranks the logits (``topn``) and this only transforms the
    scores it reports."""
    x = np.asarray(logits, dtype=F32)
    m = x.max(axis=1, keepdims=True)
    e = np.exp(x - m).astype(F32)
    s = np.zeros((x.shape[0], 1), dtype=F32)
    for k in range(x.shape[1]):
        s = (s + e[:, k:k + 1]).astype(F32)
    return (e / s).astype(F32)


# ---------------------------------------------------------------- inverse-CDF placement

def cdf_samples(logits, N, near, far):
    """Sample placement of Sec. 5.1 (Fig. 7): the depth network's class values,
    sigmoid(score) (the network is trained with binary cross-entropy), taken
    as a piecewise-constant PDF over the classes, which are uniform in the
    coordinate of Eq. 3; the CDF is inverted at the uniform steps
    u_i = (i + 0.5) / N.  Each sample stands for the probability slice
    [i/N, (i+1)/N]; its width is the depth extent of that slice.

    Returns t (rays, N), delta (rays, N) and the class of each sample, fp64.
    near/far are taken as fp32 values first."""
    near = float(F32(near))
    far = float(F32(far))
    x = np.asarray(logits, dtype=np.float64)
    p = 1.0 / (1.0 + np.exp(-x))
    rays, B = p.shape
    cdf = np.concatenate([np.zeros((rays, 1)), np.cumsum(p, axis=1)], axis=1)
    cdf /= cdf[:, -1:]

    def inverse(u):
        # class k with cdf[k] <= u < cdf[k+1], so that cdf[k+1] > cdf[k]; the
        # ends u = 0 and u = 1 map to the near and far ends by definition
        # (numerically empty trailing classes would make the last step 0/0)
        if u >= 1.0:
            return np.ones(rays), np.full(rays, B - 1, dtype=np.int64)
        k = np.empty(rays, dtype=np.int64)
        for r in range(rays):
            k[r] = np.searchsorted(cdf[r], u, side="right") - 1
        k = np.clip(k, 0, B - 1)
        lo = cdf[np.arange(rays), k]
        hi = cdf[np.arange(rays), k + 1]
        frac = np.clip((u - lo) / (hi - lo), 0.0, 1.0)
        return (k + frac) / B, k

    span = far - near
    to_depth = lambda s: near + np.power(span + 1.0, s) - 1.0   # inverse of Eq. 3
    t = np.empty((rays, N))
    cls = np.empty((rays, N), dtype=np.int32)
    edges = np.empty((rays, N + 1))
    for i in range(N):
        s_mid, k = inverse((i + 0.5) / N)
        t[:, i] = to_depth(s_mid)
        cls[:, i] = k
    for i in range(N + 1):
        s_edge, _ = inverse(i / N)
        edges[:, i] = to_depth(s_edge)
    return t, np.diff(edges, axis=1), cls


# ---------------------------------------------------------------- compositing

def composite(raw, t, delta):
    """NeRF-style accumulation with a black background (Sec. 3, Sec. 6.1).

    raw: (rays, N, 4) network outputs (r, g, b, sigma) in depth order;
    t, delta: (rays, N) sample depth and the width of its depth class.
    rgb = sigmoid, sigma = ReLU, tau = sigma * delta, alpha = 1 - exp(-tau),
    T_0 = 1, T_{i+1} = T_i exp(-tau_i), w_i = T_i alpha_i,
    C = sum w_i rgb_i, depth = sum w_i t_i.  fp64."""
    raw = np.asarray(raw, dtype=np.float64)
    rgb = 1.0 / (1.0 + np.exp(-raw[..., :3]))
    sigma = np.maximum(raw[..., 3], 0.0)
    tau = sigma * np.asarray(delta, dtype=np.float64)
    alpha = -np.expm1(-tau)
    T = np.ones(raw.shape[0])
    C = np.zeros((raw.shape[0], 3))
    D = np.zeros(raw.shape[0])
    W = np.zeros(raw.shape[:2])
    for i in range(raw.shape[1]):
        w = T * alpha[:, i]
        W[:, i] = w
        C += w[:, None] * rgb[:, i]
        D += w * np.asarray(t, dtype=np.float64)[:, i]
        T = T * np.exp(-tau[:, i])
    return C, D, W


# ---------------------------------------------------------------- full path

def render_rays(d_layers, s_layers, o, r, N, near, far, n_bins, centre, radius,
                precision="fp64", select="topn", forced_bins=None, forced_samples=None,
                depth_input="encoded", jitter=None):
    """Per-ray inference for rays (o, r) (fp32, (n, 3)).  Returns dict with
    rgb (n,3), depth (n,), bins (n,N) int32, logits (n,B) fp64, the sample
    depths t and widths delta (n,N) and, for select='topn_softmax', probs
    (n,B) fp32.  select='cdf' places samples by the inverse CDF (Sec. 5.1).
    forced_samples = (t, delta) overrides the placement (for comparisons).
    depth_input='positions' feeds the depth network the paper's unencoded
    input (``depth_positions_input``); in bf16 mode that input is not
    rounded (only the weights and hidden activations are).  ``jitter`` is
    passed to both networks (``mlp``)."""
    d_max = F32(far)
    c = np.asarray(centre, dtype=F32)
    # 1-2: unification and the depth-network input (Eq. 2 / Sec. 5.2).
    ou = unify(o, r, c, radius)
    enc_r = encode(r, L_DIR)
    if depth_input == "encoded":
        v = ((ou - c) / d_max).astype(F32)
        x0 = np.concatenate([encode(v, L_POS), enc_r], axis=1)
        round_in = True
    elif depth_input == "positions":
        _, centres, _ = bin_table(near, far, n_bins)
        x0 = depth_positions_input(o, r, ou, c, d_max, centres)
        round_in = False
    else:
        raise ValueError(depth_input)
    # 3: depth oracle network -> class scores.
    logits = mlp(d_layers, x0, precision, round_input=round_in, jitter=jitter)
    out = {"logits": logits}
    # 4: selection of N classes.
    lg32 = logits.astype(F32)
    if select == "topn_softmax":
        out["probs"] = softmax_fp32(lg32)
    elif select not in ("topn", "cdf"):
        raise ValueError(select)
    if select == "cdf":
        # 4-5: samples by the inverse CDF of the class values (Sec. 5.1).
        t, delta, bins = cdf_samples(lg32, N, near, far)
    else:
        bins = topn(lg32, N) if forced_bins is None else np.asarray(forced_bins, dtype=np.int32)
        # 5: samples at the selected class centres (Eq. 1, Eq. 3).
        _, centres, widths = bin_table(near, far, n_bins)
        t = centres[bins]
        delta = widths[bins]
    if forced_samples is not None:
        t, delta = (np.asarray(a) for a in forced_samples)
    out["bins"] = bins
    out["t"] = np.asarray(t, dtype=np.float64)
    out["delta"] = np.asarray(delta, dtype=np.float64)
    t = np.asarray(t, dtype=F32)
    x = sample_points(o, r, t).astype(F32)
    # 6: space warp (Eq. 4-5) and encoding.
    w = warp(x, c, d_max)
    n = o.shape[0]
    feats = encode(w.reshape(n * N, 3), L_POS)
    skip = np.repeat(enc_r, N, axis=0)
    raw = mlp(s_layers, feats, precision, skip=skip, jitter=jitter).reshape(n, N, 4)
    # 7: compositing.
    C, D, _ = composite(raw, t, delta)
    out["rgb"] = C
    out["depth"] = D
    return out


def render(weights, poses, H, W, N, n_bins=128, near=0.1, far=10.0, fov_x_deg=60.0,
           centre=(0.0, 0.0, 0.0), radius=1.5, precision="fp64", select="topn",
           forced_bins=None, ray_subset=None, chunk=8192, forced_samples=None,
           depth_input="encoded", jitter=None):
    """Render P poses (P, 3, 4) of H x W rays.  Returns rgb (P*H*W, 3), depth,
    bins and logits for every ray (or for ``ray_subset``, global ray ids)."""
    d_layers, s_layers = split_weights(weights, n_bins, depth_input)
    poses = np.asarray(poses, dtype=F32).reshape(-1, 3, 4)
    hw = H * W
    ids = np.arange(len(poses) * hw) if ray_subset is None else np.asarray(ray_subset, dtype=np.int64)
    o = np.empty((len(ids), 3), F32)
    r = np.empty((len(ids), 3), F32)
    for pi in np.unique(ids // hw):
        sel = np.nonzero(ids // hw == pi)[0]
        po, pr = camera_rays(poses[pi], H, W, fov_x_deg)
        o[sel] = po[ids[sel] - pi * hw]
        r[sel] = pr[ids[sel] - pi * hw]
    fb = None if forced_bins is None else np.asarray(forced_bins)
    fs = None if forced_samples is None else tuple(np.asarray(a) for a in forced_samples)
    res = {}
    for s in range(0, len(ids), chunk):
        sl = slice(s, s + chunk)
        part = render_rays(d_layers, s_layers, o[sl], r[sl], N, near, far, n_bins,
                           centre, radius, precision, select,
                           None if fb is None else fb[s:s + chunk],
                           None if fs is None else (fs[0][sl], fs[1][sl]), depth_input, jitter)
        for k, val in part.items():
            res.setdefault(k, []).append(val)
    return {k: np.concatenate(v) for k, v in res.items()}


# ---------------------------------------------------------------- analytic cost

def mlp_macs_per_ray(N, n_bins=128, d_in=90, s_in=63, skip=27, width=HIDDEN):
    """Multiply-adds of both networks for one ray with N samples (App. D's
    8-layer architecture): depth network once, shading network N times."""
    d = d_in * width + 6 * width * width + width * n_bins
    s = s_in * width + 6 * width * width + (width + skip) * 4
    return d + N * s
