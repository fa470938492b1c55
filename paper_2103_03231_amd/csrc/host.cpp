// host.cpp - the C ABI of include/donerf.h: validation, depth-class table,
// weight packing into the kernels' fragment stream, launches.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/donerf.h"
#include "internal.h"
#include "layout.h"

using namespace donerf;

struct donerf_handle {
    donerf_cfg cfg;
    int prec;            // layout.h Precision of the network
    int32_t wscale[16];  // per streamed layer: E8M0 scale of fp8 weights (127 - s), else 127
    int device;
    hipStream_t stream;
    void* d_frags;       // device: depth stream then shading stream
    float* bias;         // device
    float* bins;         // device: centres[B], widths[B], bounds[B + 1]
    int n_d_chunks, n_s_chunks, bias_len;
    int n_cu;            // compute units: workgroups of one full round
    float* partial;      // device: split-tail parts, n_cu * 256 rays * 5 floats
    float* static_scratch;         // device address of the static scratch (kernels.hip)
    hipError_t static_scratch_err; // why it could not be looked up, if it is NULL
    std::vector<float> h_bounds, h_centres, h_widths;
};

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(DONERF_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

bool finite(float x) { return std::isfinite(x); }

const int kKinds[16] = {kDFirst, kHiddenL, kHiddenL, kHiddenL, kHiddenL, kHiddenL, kHiddenL, kDHead,
                        kSFirst, kHiddenL, kHiddenL, kHiddenL, kHiddenL, kHiddenL, kHiddenL, kSHead};

// Inputs of the first depth layer in the weight blob.
int depth_in_cols(int n_bins, int depth_input) {
    return depth_input == DONERF_DEPTH_POSITIONS ? 6 + 3 * n_bins : kDIn;
}

// Values of layer l's W in the blob.
size_t blob_w_count(int l, int n_bins, int depth_input) {
    const LayerGeom lg = layer_geom(kKinds[l], n_bins);
    return (size_t)lg.out_rows * (l == 0 ? depth_in_cols(n_bins, depth_input) : lg.in_cols);
}

bool bins_supported(int B) { return B >= 64 && B <= 256 && B % 64 == 0; }

// Inverse-CDF placement over more classes than fit in registers: the kernel
// runs the depth head twice, and the depth stream carries its chunks twice.
bool wide_cdf(const donerf_cfg& c) { return c.select == DONERF_SELECT_CDF && c.n_bins > 128; }

int validate_cfg(const donerf_cfg* c) {
    if (!c) return fail(DONERF_E_INVALID_ARG, "cfg is NULL");
    const float fs[] = {c->near_dist, c->far_dist, c->fov_x_deg, c->centre[0], c->centre[1],
                        c->centre[2], c->radius};
    for (float f : fs)
        if (!finite(f)) return fail(DONERF_E_NONFINITE, "cfg holds a NaN or Inf");
    if (!(c->near_dist > 0.0f)) return fail(DONERF_E_INVALID_ARG, "near_dist must be > 0");
    if (!(c->far_dist > c->near_dist)) return fail(DONERF_E_INVALID_ARG, "far_dist must exceed near_dist");
    if (!(c->fov_x_deg > 0.0f && c->fov_x_deg < 180.0f))
        return fail(DONERF_E_INVALID_ARG, "fov_x_deg must lie in (0, 180)");
    if (!(c->radius > 0.0f)) return fail(DONERF_E_INVALID_ARG, "radius must be > 0");
    if (c->n_bins < 1) return fail(DONERF_E_INVALID_ARG, "n_bins must be >= 1");
    if (c->n_max < 1 || c->n_max > DONERF_MAX_SAMPLES)
        return fail(DONERF_E_INVALID_ARG, "n_max must lie in [1, 16]");
    if (c->n_max > c->n_bins) return fail(DONERF_E_INVALID_ARG, "n_max exceeds n_bins");
    if (c->precision != DONERF_FP32 && c->precision != DONERF_BF16 && c->precision != DONERF_FP8)
        return fail(DONERF_E_INVALID_ARG, "unknown precision");
    if (c->select != DONERF_SELECT_TOPN && c->select != DONERF_SELECT_TOPN_SOFTMAX &&
        c->select != DONERF_SELECT_CDF)
        return fail(DONERF_E_INVALID_ARG, "unknown select mode");
    if (c->depth_input != DONERF_DEPTH_ENCODED && c->depth_input != DONERF_DEPTH_POSITIONS)
        return fail(DONERF_E_INVALID_ARG, "unknown depth_input");
    if (!bins_supported(c->n_bins))
        return fail(DONERF_E_UNSUPPORTED, "n_bins must be 64, 128, 192 or 256");
    return DONERF_OK;
}

// Inverse of Eq. 3 on the uniform grid of the network coordinate, in fp64.
void make_bins(const donerf_cfg& c, std::vector<float>& bounds, std::vector<float>& centres,
               std::vector<float>& widths) {
    const int B = c.n_bins;
    const double near = c.near_dist, far = c.far_dist, span = far - near;
    std::vector<double> b(B + 1);
    for (int k = 0; k <= B; ++k) b[k] = near + std::pow(span + 1.0, (double)k / B) - 1.0;
    b[0] = near;
    b[B] = far;
    bounds.resize(B + 1);
    centres.resize(B);
    widths.resize(B);
    for (int k = 0; k <= B; ++k) bounds[k] = (float)b[k];
    for (int k = 0; k < B; ++k) {
        centres[k] = (float)(near + std::pow(span + 1.0, ((double)k + 0.5) / B) - 1.0);
        widths[k] = (float)(b[k + 1] - b[k]);
    }
}

uint16_t to_bf16(float x) {  // round to nearest even (inputs are finite)
    uint32_t u;
    std::memcpy(&u, &x, 4);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// OCP E4M3 code of x, |x| <= 448: round to nearest, ties to even, on the
// grid of 3 mantissa bits.  Code bits: sign, 4 exponent bits (bias 7),
// 3 mantissa bits; exponent field 0 holds the subnormals m 2^-9.
uint8_t to_e4m3(float x) {
    const double a = std::fabs((double)x);
    const uint8_t sign = std::signbit(x) ? 0x80 : 0x00;
    int E = 0;
    std::frexp(a, &E);                  // a = f 2^E, f in [0.5, 1): binade e = E - 1
    const int e = E - 1;
    if (a == 0.0 || e < -6) {
        // n 2^-9 with n = 0..8; n = 8 is 2^-6, whose code 0x08 is the
        // smallest normal, so the code is n itself
        return (uint8_t)(sign | (uint8_t)std::nearbyint(std::ldexp(a, 9)));
    }
    int n = (int)std::nearbyint(std::ldexp(a, 3 - e));   // 8..16, ties to even
    int ee = e;
    if (n == 16) {
        n = 8;
        ++ee;
    }
    return (uint8_t)(sign | (uint8_t)((ee + 7) << 3) | (uint8_t)(n - 8));
}

// Largest s with max|W| 2^s <= 448 (0 for an all-zero layer): the per-layer
// power-of-two scale of fp8 weights.
int fp8_scale(const float* W, size_t n) {
    double m = 0.0;
    for (size_t k = 0; k < n; ++k) m = std::fmax(m, std::fabs((double)W[k]));
    if (m == 0.0) return 0;
    int s = (int)std::floor(std::log2(448.0 / m));
    while (std::ldexp(m, s + 1) <= 448.0) ++s;
    while (std::ldexp(m, s) > 448.0) --s;
    return s;
}

float bf16_value(float x) {
    const uint32_t u = (uint32_t)to_bf16(x) << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

// Folds the first depth layer of the positions input (256 x (6 + 3 B) over
// [u', r, p_0, ..., p_{B-1}], p_k = u_c + (c_k / d_max) r) into 256 x 9 over
// [u', r, u_c]: the origin columns stay, the direction columns gain
// sum_k (c_k / d_max) W_k and the u_c columns are sum_k W_k.  Sums in fp64
// from the weights as the network uses them (bf16-rounded in bf16 mode),
// stored as fp32.
std::vector<float> fold_positions_layer(const float* W, int B, bool bf16, const std::vector<float>& centres,
                                        float d_max) {
    const int n_in = 6 + 3 * B;
    std::vector<float> out((size_t)kHidden * kPIn);
    for (int u = 0; u < kHidden; ++u) {
        auto w = [&](int col) -> double {
            const float v = W[(size_t)u * n_in + col];
            return bf16 ? (double)bf16_value(v) : (double)v;
        };
        double mo[3] = {0.0, 0.0, 0.0}, mr[3] = {0.0, 0.0, 0.0};
        for (int k = 0; k < B; ++k) {
            const double s = (double)centres[k] / (double)d_max;
            for (int j = 0; j < 3; ++j) {
                const double wk = w(6 + 3 * k + j);
                mo[j] += wk;
                mr[j] += s * wk;
            }
        }
        for (int j = 0; j < 3; ++j) {
            out[(size_t)u * kPIn + j] = (float)w(j);
            out[(size_t)u * kPIn + 3 + j] = (float)(w(3 + j) + mr[j]);
            out[(size_t)u * kPIn + 6 + j] = (float)mo[j];
        }
    }
    return out;
}

// Logical input column of the blob for K step ks, lane group g, element e of
// a layer whose steps have precision p, in a network of precision net; hidx:
// the layer's position among its network's hidden layers (-1 for others).
// In bf16 networks (hid16) the hidden layers take 16x16 steps, and the
// heads read the 32x32 layout the swap after the last hidden layer restores.
int in_col(int p, int net, int kind, int hidx, int ks, int g, int e) {
    const int E = elems(p);
    switch (kind) {
        case kDFirst: return d_feature(g, ks * E + e);
        case kDFirstPos: return p_feature(ks, g, e);
        case kSFirst: return s_feature(g, ks * E + e);
        case kHiddenL:
            if (hid16(net)) return hidx == 0 ? chained16_from32(ks, g, e) : chained16(ks, g, e);
            return chained_row(p, ks, g, e);
        case kDHead: return hid16(net) ? chained32_from16(ks, g, e) : chained_row(p, ks, g, e);
        default: {  // kSHead: chained hidden units, then the direction skip
            if (hid16(net)) {
                // 16x16 steps of 32: the last hidden layer's 16x16 output,
                // then the skip, swapped from its two 32x32 steps
                if (ks < 8) return chained16(ks, g, e);
                const int f = skip_feature(g / 2, (g % 2) * E + e);
                return f < 0 ? -1 : kHidden + f;
            }
            const int ksh = ksteps(p, kHidden);
            if (ks < ksh) return chained_row(p, ks, g, e);
            const int f = skip_feature(g, (ks - ksh) * E + e);
            return f < 0 ? -1 : kHidden + f;
        }
    }
}

// Append one layer's steps, in the order the kernel consumes them (pass,
// K step, row block within the pass), padded to whole chunks.  prec: the
// layer's step precision (layout.h frag_prec); net: the network's (for the
// chunk count and the hidden layers' step shape); hidx: the layer's position
// among the hidden layers (-1 for others); s: power-of-two scale of fp8
// weights (W 2^s is rounded).  A 16x16 hidden layer (hid16) streams passes
// of four 16-row tiles, each over its eight K steps of 32: lane l holds row
// 16 tile + l % 16 and lane group l / 16.
void pack_layer(int prec, int net, int kind, int hidx, int n_bins, const float* W, int s, std::vector<uint8_t>& dst) {
    const LayerGeom lg = layer_geom(kind, n_bins);
    const bool t16 = (kind == kHiddenL || kind == kSHead) && hid16(net);
    const int rows_per = t16 ? 16 : 32, groups = t16 ? 4 : 2;
    const int KS = t16 ? lg.kpad / 32 : ksteps(prec, lg.kpad);
    // row blocks or tiles per pass, passes (a 16x16 shading head is one tile)
    const int RPP = t16 ? (kind == kSHead ? 1 : 4) : lg.rbp;
    const int NP = t16 && kind == kSHead ? 1 : lg.rb * 32 / rows_per / RPP;
    const int E = elems(prec), EB = elem_bytes(prec), U = units(prec);
    const size_t start = dst.size();
    dst.resize(start + (size_t)layer_chunks(net, kind, n_bins) * kChunkBytes, 0);
    uint8_t* out = dst.data() + start;
    size_t f = 0;
    for (int p = 0; p < NP; ++p)
        for (int ks = 0; ks < KS; ++ks)
            for (int r = 0; r < RPP; ++r, ++f) {
                const int rb = p * RPP + r;
                uint8_t* step = out + f * U * kFragBytes;
                for (int lane = 0; lane < 64; ++lane) {
                    const int row = rows_per * rb + lane % rows_per, g = lane / (64 / groups);
                    for (int e = 0; e < E; ++e) {
                        const int colx = in_col(prec, net, kind, hidx, ks, g, e);
                        const float v = (row < lg.out_rows && colx >= 0) ? W[(size_t)row * lg.in_cols + colx] : 0.0f;
                        // element e: unit (e * EB) / 16, byte (e * EB) % 16 of the lane's 16
                        uint8_t* dstp = step + ((e * EB) / 16) * kFragBytes + lane * 16 + (e * EB) % 16;
                        if (prec == kFP8) {
                            *dstp = to_e4m3((float)std::ldexp((double)v, s));
                        } else if (prec == kBF16) {
                            const uint16_t h = to_bf16(v);
                            std::memcpy(dstp, &h, 2);
                        } else {
                            std::memcpy(dstp, &v, 4);
                        }
                    }
                }
            }
}

int check_device(int* dev_out) {
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || n < 1) {
        (void)hipGetLastError();
        return fail(DONERF_E_DEVICE, "no HIP device");
    }
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return fail(DONERF_E_DEVICE, "hipGetDevice failed");
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess)
        return fail(DONERF_E_DEVICE, "hipGetDeviceProperties failed");
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(DONERF_E_DEVICE, std::string("device is ") + prop.gcnArchName + ", need gfx950");
    *dev_out = dev;
    return DONERF_OK;
}

int validate_render(const donerf_t* h, const float* poses, int32_t P, int32_t H, int32_t W, int32_t N,
                    const float* out_rgb) {
    if (!h) return fail(DONERF_E_INVALID_ARG, "handle is NULL");
    if (!poses) return fail(DONERF_E_INVALID_ARG, "cam_poses is NULL");
    if (!out_rgb) return fail(DONERF_E_INVALID_ARG, "out_rgb is NULL");
    if (P < 1 || H < 1 || W < 1) return fail(DONERF_E_INVALID_ARG, "P, H and W must be >= 1");
    if (N < 1 || N > h->cfg.n_max || N > h->cfg.n_bins)
        return fail(DONERF_E_INVALID_ARG, "N must lie in [1, n_max]");
    if ((int64_t)P * H * W >= ((int64_t)1 << 31)) return fail(DONERF_E_INVALID_ARG, "P*H*W must be < 2^31");
    if ((int64_t)H * W > (1 << 24)) return fail(DONERF_E_INVALID_ARG, "H*W must be <= 2^24");
    for (int64_t k = 0; k < (int64_t)P * 12; ++k)
        if (!finite(poses[k])) return fail(DONERF_E_NONFINITE, "cam_poses holds a NaN or Inf");
    return DONERF_OK;
}

int ncap_for(int N) { return N <= 4 ? 4 : N <= 8 ? 8 : 16; }

// Split of the last, partial round of tiles: n_full tiles run whole, the
// remaining rem tiles are each split `split` ways by samples.
struct TailPlan {
    uint32_t n_full, rem, split;
};

TailPlan plan_tail(const donerf_t* h, uint32_t total_rays, int32_t N) {
    // Full rounds of one workgroup per CU run as they are.  The tiles of a
    // last, partial round are split by samples over up to n_cu / r
    // workgroups each (every part recomputes the depth network), and a
    // combine pass composites the parts.
    const uint32_t rpb = (uint32_t)rays_per_block(h->prec);
    const uint32_t tiles = (total_rays + rpb - 1) / rpb;
    const uint32_t round = (uint32_t)h->n_cu;
    const uint32_t full = tiles / round * round, rem = tiles - full;
    uint32_t split = rem ? round / rem : 1;
    if (split > (uint32_t)N) split = (uint32_t)N;
    if (split < 1) split = 1;
    return TailPlan{split > 1 ? full : tiles, split > 1 ? rem : 0, split};
}

// Floats of split-tail scratch a plan writes: 5 per ray and part.
size_t tail_floats(const donerf_t* h, const TailPlan& t) {
    return t.split > 1 ? (size_t)5 * t.rem * (size_t)rays_per_block(h->prec) * t.split : 0;
}

// partial: split-tail scratch of partial_cap floats (the handle's buffer, or
// the static scratch).
int render_impl(donerf_t* h, const float* poses, int32_t P, int32_t H, int32_t W, int32_t N, float* out_rgb,
                float* out_depth, int32_t* out_bins, float* out_scores, float* out_samples, float* partial,
                size_t partial_cap) {
    int rc = validate_render(h, poses, P, H, W, N, out_rgb);
    if (rc) return rc;
    const size_t hw = (size_t)H * W;
    // every launch's scratch need is known before the first one is enqueued
    for (int32_t p0 = 0; p0 < P; p0 += kMaxPosesPerLaunch) {
        const int np = P - p0 < kMaxPosesPerLaunch ? P - p0 : kMaxPosesPerLaunch;
        const size_t need = tail_floats(h, plan_tail(h, (uint32_t)(np * hw), N));
        if (need > partial_cap)
            return fail(DONERF_E_UNSUPPORTED, "the split tail needs " + std::to_string(need) +
                                                  " floats of scratch, " + std::to_string(partial_cap) +
                                                  " are available");
    }
    const donerf_cfg& c = h->cfg;
    RenderArgs a;
    std::memset(&a, 0, sizeof a);
    a.d_frags = static_cast<const uint4*>(h->d_frags);
    a.s_frags = static_cast<const uint4*>(h->d_frags) + (size_t)h->n_d_chunks * (kChunkBytes / 16);
    a.bias = h->bias;
    a.bins = h->bins;
    a.n_d_chunks = h->n_d_chunks;
    a.n_s_chunks = h->n_s_chunks;
    a.bias_len = h->bias_len;
    a.H = H;
    a.W = W;
    a.N = N;
    static_assert(kMaxSamples == DONERF_MAX_SAMPLES, "sample capacity");
    for (int i = 0; i < kMaxSamples; ++i) {
        a.cdf_u[i] = i < N ? ((float)i + 0.5f) / (float)N : 2.0f;
        a.cdf_u[kMaxSamples + i] = i + 1 < N ? (float)(i + 1) / (float)N : 2.0f;
    }
    a.B = c.n_bins;
    a.focal = (float)((0.5 * W) / std::tan((double)c.fov_x_deg * (M_PI / 180.0) * 0.5));
    a.half_w = 0.5f * (float)W;
    a.half_h = 0.5f * (float)H;
    a.cx = c.centre[0];
    a.cy = c.centre[1];
    a.cz = c.centre[2];
    a.radius = c.radius;
    a.near = c.near_dist;
    a.dmax = c.far_dist;
    a.log2_span1 = (float)std::log2((double)c.far_dist - (double)c.near_dist + 1.0);
    const int place = c.select != DONERF_SELECT_CDF ? kPlaceTopN : wide_cdf(c) ? kPlaceCdfWide : kPlaceCdf;
    for (int32_t p0 = 0; p0 < P; p0 += kMaxPosesPerLaunch) {
        const int np = P - p0 < kMaxPosesPerLaunch ? P - p0 : kMaxPosesPerLaunch;
        a.n_poses = np;
        a.total_rays = (uint32_t)(np * hw);
        std::memcpy(a.poses, poses + (size_t)p0 * 12, sizeof(float) * 12 * np);
        a.out_rgb = out_rgb + (size_t)p0 * hw * 3;
        a.out_depth = out_depth ? out_depth + (size_t)p0 * hw : nullptr;
        a.out_bins = out_bins ? out_bins + (size_t)p0 * hw * N : nullptr;
        a.out_scores = out_scores ? out_scores + (size_t)p0 * hw * c.n_bins : nullptr;
        a.out_samples = out_samples ? out_samples + (size_t)p0 * hw * N * 2 : nullptr;
        const TailPlan tp = plan_tail(h, a.total_rays, N);
        a.n_full = tp.n_full;
        a.split = (int32_t)tp.split;
        a.partial = partial;
        std::memcpy(a.wscale, h->wscale, sizeof a.wscale);
        hipError_t e = launch_render(h->prec, ncap_for(N), place,
                                     c.depth_input == DONERF_DEPTH_POSITIONS ? kDinPositions : kDinEncoded, a,
                                     tp.rem, h->stream);
        if (e != hipSuccess) return hip_fail(e, "render launch");
        if (tp.split > 1) {
            e = launch_combine(h->prec, a, h->stream);
            if (e != hipSuccess) return hip_fail(e, "combine launch");
        }
        if (out_scores && c.select == DONERF_SELECT_TOPN_SOFTMAX) {
            e = launch_softmax_rows(a.out_scores, a.total_rays, c.n_bins, h->stream);
            if (e != hipSuccess) return hip_fail(e, "softmax launch");
        }
    }
    return DONERF_OK;
}

}  // namespace

extern "C" {

size_t donerf_weight_count(int32_t n_bins, int32_t depth_input) {
    if (n_bins < 1) return 0;
    if (depth_input != DONERF_DEPTH_ENCODED && depth_input != DONERF_DEPTH_POSITIONS) return 0;
    size_t n = 0;
    for (int l = 0; l < 16; ++l)
        n += blob_w_count(l, n_bins, depth_input) + (size_t)layer_geom(kKinds[l], n_bins).out_rows;
    return n;
}

int donerf_create(const donerf_cfg* cfg, const float* weights, size_t n_weights, donerf_t** out) {
    g_err.clear();
    if (!out) return fail(DONERF_E_INVALID_ARG, "out is NULL");
    *out = nullptr;
    int rc = validate_cfg(cfg);
    if (rc) return rc;
    if (!weights) return fail(DONERF_E_INVALID_ARG, "weights is NULL");
    const size_t want = donerf_weight_count(cfg->n_bins, cfg->depth_input);
    if (n_weights != want)
        return fail(DONERF_E_SIZE, "weight count " + std::to_string(n_weights) + " != " + std::to_string(want));
    for (size_t k = 0; k < n_weights; ++k)
        if (!finite(weights[k])) return fail(DONERF_E_NONFINITE, "weights hold a NaN or Inf");
    int dev = 0;
    rc = check_device(&dev);
    if (rc) return rc;

    const int prec = cfg->precision == DONERF_FP8 ? kFP8 : cfg->precision == DONERF_BF16 ? kBF16 : kF32;
    const int B = cfg->n_bins;
    const bool positions = cfg->depth_input == DONERF_DEPTH_POSITIONS;
    std::vector<float> bounds, centres, widths;
    make_bins(*cfg, bounds, centres, widths);
    std::vector<uint8_t> frags;
    std::vector<float> bias, head_bias;
    int n_d_chunks = 0, n_s_chunks = 0;
    int32_t wscale[16];
    size_t off = 0;
    for (int l = 0; l < 16; ++l) {
        const int kind = (l == 0 && positions) ? kDFirstPos : kKinds[l];
        const LayerGeom lg = layer_geom(kind, B);
        const int fp = frag_prec(prec, kind);
        const int s = fp == kFP8 ? fp8_scale(weights + off, blob_w_count(l, B, cfg->depth_input)) : 0;
        wscale[l] = 127 - s;
        if (kind == kDFirstPos) {
            // the folded sums use the weights as the first layer of the
            // network uses them: bf16 in bf16 and fp8 networks
            const std::vector<float> folded =
                fold_positions_layer(weights + off, B, prec != kF32, centres, cfg->far_dist);
            pack_layer(fp, prec, kind, -1, B, folded.data(), 0, frags);
        } else {
            pack_layer(fp, prec, kind, kind == kHiddenL ? l % 8 - 1 : -1, B, weights + off, s, frags);
        }
        (l < 8 ? n_d_chunks : n_s_chunks) += layer_chunks(prec, kind, B);
        if (l == 7 && wide_cdf(*cfg)) {
            pack_layer(fp, prec, kind, -1, B, weights + off, s, frags);
            n_d_chunks += layer_chunks(prec, kind, B);
        }
        off += blob_w_count(l, B, cfg->depth_input);
        // the depth head's bias (B-dependent length) goes last
        std::vector<float>& dst = l == 7 ? head_bias : bias;
        const size_t b0 = dst.size();
        dst.resize(b0 + bias_len(kind, B), 0.0f);
        std::memcpy(dst.data() + b0, weights + off, sizeof(float) * lg.out_rows);
        off += lg.out_rows;
    }
    bias.insert(bias.end(), head_bias.begin(), head_bias.end());

    donerf_t* h = new (std::nothrow) donerf_handle();
    if (!h) return fail(DONERF_E_NOMEM, "host allocation failed");
    h->cfg = *cfg;
    h->prec = prec;
    std::memcpy(h->wscale, wscale, sizeof wscale);
    h->device = dev;
    h->stream = nullptr;
    h->n_d_chunks = n_d_chunks;
    h->n_s_chunks = n_s_chunks;
    h->bias_len = (int)bias.size();
    h->h_bounds = bounds;
    h->h_centres = centres;
    h->h_widths = widths;
    std::vector<float> bins(3 * B + 1);
    std::memcpy(bins.data(), h->h_centres.data(), sizeof(float) * B);
    std::memcpy(bins.data() + B, h->h_widths.data(), sizeof(float) * B);
    std::memcpy(bins.data() + 2 * B, h->h_bounds.data(), sizeof(float) * (B + 1));

    hipError_t e;
    if ((e = hipDeviceGetAttribute(&h->n_cu, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess ||
        h->n_cu < 1) {
        donerf_destroy(h);
        return hip_fail(e, "hipDeviceGetAttribute");
    }
    if ((e = hipMalloc(&h->d_frags, frags.size())) != hipSuccess ||
        (e = hipMalloc(&h->partial, sizeof(float) * 5 * 256 * (size_t)h->n_cu)) != hipSuccess ||
        (e = hipMalloc(&h->bias, sizeof(float) * bias.size())) != hipSuccess ||
        (e = hipMalloc(&h->bins, sizeof(float) * bins.size())) != hipSuccess) {
        donerf_destroy(h);
        return fail(DONERF_E_NOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
    }
    // the static scratch of donerf_render_static_scratch, looked up here
    // (with the handle's device current) so that entry point makes no HIP
    // call besides its launches; a failure surfaces there
    h->static_scratch_err = static_scratch_address(dev, &h->static_scratch);
    if (h->static_scratch_err != hipSuccess) {
        (void)hipGetLastError();
        h->static_scratch = nullptr;
    }
    if ((e = hipMemcpy(h->d_frags, frags.data(), frags.size(), hipMemcpyHostToDevice)) != hipSuccess ||
        (e = hipMemcpy(h->bias, bias.data(), sizeof(float) * bias.size(), hipMemcpyHostToDevice)) != hipSuccess ||
        (e = hipMemcpy(h->bins, bins.data(), sizeof(float) * bins.size(), hipMemcpyHostToDevice)) != hipSuccess) {
        donerf_destroy(h);
        return hip_fail(e, "hipMemcpy");
    }
    *out = h;
    return DONERF_OK;
}

void donerf_destroy(donerf_t* h) {
    if (!h) return;
    if (h->d_frags) (void)hipFree(h->d_frags);
    if (h->bias) (void)hipFree(h->bias);
    if (h->bins) (void)hipFree(h->bins);
    if (h->partial) (void)hipFree(h->partial);
    delete h;
}

int donerf_set_stream(donerf_t* h, void* stream) {
    if (!h) return fail(DONERF_E_INVALID_ARG, "handle is NULL");
    h->stream = static_cast<hipStream_t>(stream);
    return DONERF_OK;
}

int donerf_render(donerf_t* h, const float* cam_poses, int32_t P, int32_t H, int32_t W, int32_t N,
                  float* out_rgb, float* out_depth) {
    g_err.clear();
    return render_impl(h, cam_poses, P, H, W, N, out_rgb, out_depth, nullptr, nullptr, nullptr,
                       h ? h->partial : nullptr, h ? (size_t)5 * 256 * (size_t)h->n_cu : 0);
}

int donerf_render_static_scratch(donerf_t* h, const float* cam_poses, int32_t P, int32_t H, int32_t W,
                                 int32_t N, float* out_rgb, float* out_depth) {
    g_err.clear();
    if (h && !h->static_scratch)
        return hip_fail(h->static_scratch_err, "static scratch lookup at create");
    return render_impl(h, cam_poses, P, H, W, N, out_rgb, out_depth, nullptr, nullptr, nullptr,
                       h ? h->static_scratch : nullptr, kStaticScratchFloats);
}

int donerf_render_debug(donerf_t* h, const float* cam_poses, int32_t P, int32_t H, int32_t W, int32_t N,
                        float* out_rgb, float* out_depth, int32_t* out_bins, float* out_scores,
                        float* out_samples) {
    g_err.clear();
    return render_impl(h, cam_poses, P, H, W, N, out_rgb, out_depth, out_bins, out_scores, out_samples,
                       h ? h->partial : nullptr, h ? (size_t)5 * 256 * (size_t)h->n_cu : 0);
}

int donerf_debug_topn(donerf_t* h, const float* scores, int32_t rays, int32_t N, int32_t* out_idx) {
    g_err.clear();
    if (!h) return fail(DONERF_E_INVALID_ARG, "handle is NULL");
    if (!scores || !out_idx) return fail(DONERF_E_INVALID_ARG, "NULL buffer");
    if (rays < 1) return fail(DONERF_E_INVALID_ARG, "rays must be >= 1");
    if (N < 1 || N > h->cfg.n_max || N > h->cfg.n_bins) return fail(DONERF_E_INVALID_ARG, "N out of range");
    hipError_t e = launch_topn(h->prec != kF32, ncap_for(N), scores, rays, N, h->cfg.n_bins, out_idx, h->stream);
    if (e != hipSuccess) return hip_fail(e, "topn launch");
    return DONERF_OK;
}

int donerf_debug_mfma_peak(donerf_t* h, int32_t workgroups, int32_t iters, float* sink, double* flop) {
    g_err.clear();
    if (!h) return fail(DONERF_E_INVALID_ARG, "handle is NULL");
    if (!sink) return fail(DONERF_E_INVALID_ARG, "NULL buffer");
    if (workgroups < 1 || workgroups > (1 << 20)) return fail(DONERF_E_INVALID_ARG, "workgroups must lie in [1, 2^20]");
    if (iters < 1 || iters > (1 << 24)) return fail(DONERF_E_INVALID_ARG, "iters must lie in [1, 2^24]");
    if (flop) *flop = (double)workgroups * 4 * 4 * (double)iters * mfma_step_flop(h->prec);
    hipError_t e = launch_mfma_peak(h->prec, workgroups, iters, 0x5EED0u, sink, h->stream);
    if (e != hipSuccess) return hip_fail(e, "mfma peak launch");
    return DONERF_OK;
}

int donerf_targets(donerf_t* h, const float* depth, int32_t P, int32_t H, int32_t W, int32_t K, int32_t Z,
                   float* out) {
    g_err.clear();
    if (!h) return fail(DONERF_E_INVALID_ARG, "handle is NULL");
    if (!depth || !out) return fail(DONERF_E_INVALID_ARG, "NULL buffer");
    if (P < 1 || H < 1 || W < 1) return fail(DONERF_E_INVALID_ARG, "P, H and W must be >= 1");
    if (K < 1 || K > kTgtMaxK || Z < 1 || Z > kTgtMaxK)
        return fail(DONERF_E_INVALID_ARG, "K and Z must lie in [1, 15]");
    if ((int64_t)P * H * W >= ((int64_t)1 << 31)) return fail(DONERF_E_INVALID_ARG, "too many pixels");
    const int B = h->cfg.n_bins;
    const float inv_l2span =
        (float)(1.0 / std::log2((double)h->cfg.far_dist - (double)h->cfg.near_dist + 1.0));
    hipError_t e = launch_targets(depth, P, H, W, h->bins + 2 * B, B, K, Z, inv_l2span, out, h->stream);
    if (e != hipSuccess) return hip_fail(e, "targets launch");
    return DONERF_OK;
}

int donerf_debug_bins(const donerf_t* h, float* bounds, float* centres, float* widths) {
    g_err.clear();
    if (!h) return fail(DONERF_E_INVALID_ARG, "handle is NULL");
    if (!centres || !widths) return fail(DONERF_E_INVALID_ARG, "NULL buffer");
    const int B = h->cfg.n_bins;
    if (bounds) std::memcpy(bounds, h->h_bounds.data(), sizeof(float) * (B + 1));
    std::memcpy(centres, h->h_centres.data(), sizeof(float) * B);
    std::memcpy(widths, h->h_widths.data(), sizeof(float) * B);
    return DONERF_OK;
}

const char* donerf_status_str(int status) {
    switch (status) {
        case DONERF_OK: return "ok";
        case DONERF_E_INVALID_ARG: return "invalid argument";
        case DONERF_E_SIZE: return "weight count mismatch";
        case DONERF_E_NONFINITE: return "non-finite value";
        case DONERF_E_DEVICE: return "no gfx950 device";
        case DONERF_E_NOMEM: return "out of memory";
        case DONERF_E_HIP: return "HIP error";
        case DONERF_E_UNSUPPORTED: return "unsupported configuration";
        default: return "unknown status";
    }
}

const char* donerf_last_error(void) { return g_err.c_str(); }

}  // extern "C"
