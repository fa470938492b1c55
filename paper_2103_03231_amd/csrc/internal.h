// internal.h - interface between the host planner (host.cpp) and the kernels
// (kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "layout.h"

namespace donerf {

constexpr int kMaxSamples = 16;   // samples per ray (include/donerf.h DONERF_MAX_SAMPLES)

// Everything one render launch needs, passed by value as the kernel argument.
struct RenderArgs {
    const uint4* d_frags;   // depth network fragments, chunk-padded per layer
    const uint4* s_frags;   // shading network fragments, chunk-padded per layer
    const float* bias;      // all biases (layout.h bias_len); the depth head's last
    const float* bins;      // centres[B] then widths[B]
    float* out_rgb;         // rays x 3
    float* out_depth;       // rays, or null
    int32_t* out_bins;      // rays x N, or null
    float* out_scores;      // rays x B, or null
    float* out_samples;     // rays x N x (depth, width), or null
    int32_t n_d_chunks;
    int32_t n_s_chunks;
    int32_t bias_len;       // floats in bias
    int32_t H, W, n_poses, N, B;
    uint32_t total_rays;    // n_poses * H * W
    // Workgroups b < n_full render tile b whole.  Workgroups b >= n_full
    // split the remaining tiles by samples: with c = b - n_full, tile
    // n_full + c / split, samples [j N / split, (j + 1) N / split) for
    // j = c % split.  With split > 1 such a part writes its composite (C rgb,
    // depth, transmittance) to partial[(local_ray * split + j) * 5], local_ray
    // counted from the first ray of tile n_full, instead of the outputs.
    uint32_t n_full;
    int32_t split;
    float* partial;
    float focal, half_w, half_h;
    float cx, cy, cz;
    float radius;
    float near;             // d_min
    float dmax;             // d_max
    float log2_span1;       // log2(d_max - d_min + 1), for the inverse of Eq. 3
    // inverse-CDF targets (Sec. 5.1): cdf_u[i] = (i + 1/2) / N, the centre of
    // probability slice i < N, and cdf_u[kMaxSamples + i] = (i + 1) / N, the
    // inner end of slice i < N - 1; 2 elsewhere.  Each is the correctly
    // rounded fp32 quotient, as the kernel's own division would give.
    float cdf_u[2 * kMaxSamples];
    int32_t wscale[16];     // per streamed layer (depth 0-7, shading 8-15): E8M0 scale of
                            // its fp8 weights, 127 - s for weights stored as W 2^s
    float poses[kMaxPosesPerLaunch][12];
};

// Launch shape of the bf16 render kernel: 32-ray column blocks per wave and
// waves per workgroup, and waves per SIMD the register budget is sized for.
#ifndef DONERF_BF16_CB
#define DONERF_BF16_CB 1
#endif
#ifndef DONERF_BF16_NW
#define DONERF_BF16_NW 8
#endif
#ifndef DONERF_BF16_OCC
#define DONERF_BF16_OCC 2
#endif
constexpr int kBf16CB = DONERF_BF16_CB;
constexpr int kBf16NW = DONERF_BF16_NW;
constexpr int kBf16Occ = DONERF_BF16_OCC;

// Rays handled by one workgroup (prec: layout.h Precision of the network;
// the fp8 kernel has the bf16 kernel's launch shape).
inline int rays_per_block(int prec) { return prec != kF32 ? kBf16NW * 32 * kBf16CB : 4 * 32; }

// Launches a.n_full whole tiles plus n_split_tiles tiles split a.split ways.
// place: layout.h Placement; din: layout.h DepthInput.
hipError_t launch_render(int prec, int ncap, int place, int din, const RenderArgs& a, uint32_t n_split_tiles,
                         hipStream_t stream);
// The variants of one precision and placement (render_*.hip).
hipError_t launch_render_bf16_topn(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream);
hipError_t launch_render_bf16_cdf(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream);
hipError_t launch_render_fp32_topn(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream);
hipError_t launch_render_fp32_cdf(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream);
hipError_t launch_render_fp8_topn(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream);
hipError_t launch_render_fp8_cdf(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream);
hipError_t launch_render_bf16_cdf_wide(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream);
hipError_t launch_render_fp32_cdf_wide(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream);
hipError_t launch_render_fp8_cdf_wide(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream);
// Composites the split parts of rays [n_full * rays_per_block, total_rays)
// into out_rgb / out_depth.
hipError_t launch_combine(int prec, const RenderArgs& a, hipStream_t stream);
// Floats of the static device scratch behind donerf_render_static_scratch:
// the split tail's parts (5 floats per ray and part) of up to 256 compute
// units x 256 rays, 1.25 MiB per device.
constexpr size_t kStaticScratchFloats = (size_t)5 * 256 * 256;
constexpr int kMaxDevices = 64;
// Device address of that scratch on `device`, which must be the current
// device; looked up once per device, then cached.
hipError_t static_scratch_address(int device, float** out);
hipError_t launch_softmax_rows(float* scores, uint32_t rows, int B, hipStream_t stream);
hipError_t launch_topn(bool bf16_layout, int ncap, const float* scores, int32_t rays,
                       int32_t N, int32_t B, int32_t* out_idx, hipStream_t stream);

// Register-fed MFMA loop (kernels.hip): workgroups x 4 waves, four
// independent 32 x 32 chains of `iters` steps per wave in precision prec;
// sink holds workgroups x 256 floats.
hipError_t launch_mfma_peak(int prec, int workgroups, int iters, uint32_t seed, float* sink, hipStream_t stream);
// FLOP of one chain step: a 32 x 32 x 16 bf16, 32 x 32 x 64 E4M3 or four
// 32 x 32 x 2 fp32 MFMAs.
constexpr double mfma_step_flop(int prec) {
    return prec == kFP8 ? 2.0 * 32 * 32 * 64 : prec == kBF16 ? 2.0 * 32 * 32 * 16 : 2.0 * 32 * 32 * 8;
}

// Training targets (targets.hip): P depth maps of H x W, class bounds
// bounds[0..B], window sizes K and Z (1..kTgtMaxK), out P x H x W x B.
constexpr int kMaxBins = 256;
constexpr int kTgtMaxK = 15;
hipError_t launch_targets(const float* depth, int P, int H, int W, const float* bounds, int B, int K, int Z,
                          float inv_l2span, float* out, hipStream_t stream);

}  // namespace donerf
