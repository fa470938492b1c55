// targets.hip - training targets of the depth oracle (Sec. 5.1, Eq. 6-8) on
// gfx950: one-hot depth class of each pixel's first surface, the radial
// K x K neighbourhood filter (Eq. 7) and the triangle filter of size Z along
// the classes, clamped to 1 (Eq. 8).
//
// A workgroup renders one segment of kTgtSeg pixels of one image row.  It
// first classifies the window rows around the segment (the segment plus a
// halo of floor(K/2) pixels, floor(K/2) rows above and below) into LDS: the
// coordinate of Eq. 3 proposes a class and comparisons with the class bounds
// settle it.  Each wave then takes its pixels one
// at a time: one window entry per lane, each entry raises its class in a
// per-wave LDS row of B values to the entry's weight with an LDS max
// (Eq. 7's maximum; zeros stand for the centre term of classes without a
// surface), and the lanes, now over classes (CPL = B / 64 consecutive ones
// each), apply Eq. 8 from that row, whose zero margins stand for the classes
// outside [0, B), and write the pixel's B targets as coalesced rows.  The output (4 B bytes per
// pixel) is the only sizeable HBM traffic.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace donerf {
namespace {

constexpr int kTgtSeg = 64;                 // pixels per workgroup
constexpr int kTgtWaves = 4;
constexpr int kTgtMaxH = kTgtMaxK / 2;      // largest half window

// Class of depth d: k with b_k <= d < b_{k+1}, or -1 outside [b_0, b_B) or
// not finite (comparisons with NaN are false).  The coordinate of Eq. 3
// gives the class up to rounding; comparisons with the stored bounds settle
// it, so the result is defined by the bounds alone.  inv_l2span =
// 1 / log2(d_max - d_min + 1).
__device__ __forceinline__ int classify(float d, const float* bnd, int B, float inv_l2span) {
    if (!(d >= bnd[0] && d < bnd[B])) return -1;
    int k = (int)((float)B * (__log2f(d - bnd[0] + 1.0f) * inv_l2span));
    k = k < 0 ? 0 : (k > B - 1 ? B - 1 : k);
    while (k > 0 && d < bnd[k]) --k;
    while (k < B - 1 && d >= bnd[k + 1]) ++k;
    return k;
}

// CPL: classes per lane (B / 64), lanes own classes CPL lane .. CPL lane +
// CPL - 1, so each lane writes CPL consecutive targets.  HZ: floor(Z / 2).
template <int CPL, int HZ>
__global__ void __launch_bounds__(64 * kTgtWaves)
targets_kernel(const float* __restrict__ depth, int H, int W, const float* __restrict__ bounds, int K,
               float inv_l2span, float* __restrict__ out) {
    constexpr int B = 64 * CPL;
    constexpr int RW = B + 2 * kTgtMaxH;     // row with a zero margin of the largest HZ on each side
    __shared__ float bnd[kMaxBins + 1];
    __shared__ int cls[(2 * kTgtMaxH + 1) * (kTgtSeg + 2 * kTgtMaxH)];
    __shared__ int row[kTgtWaves][2][RW];    // fp32 bits of C^ (all >= 0); row[..][kTgtMaxH + z] holds class z

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = K / 2;
    const int segs = (W + kTgtSeg - 1) / kTgtSeg;
    const int seg = blockIdx.x % segs;
    const int y = (blockIdx.x / segs) % H;
    const size_t img = blockIdx.x / ((size_t)segs * H);
    const int x0 = seg * kTgtSeg;
    const float* dimg = depth + img * (size_t)H * W;

    for (int k = tid; k <= B; k += 64 * kTgtWaves) bnd[k] = bounds[k];
    for (int k = tid; k < kTgtWaves * 2 * RW; k += 64 * kTgtWaves) (&row[0][0][0])[k] = 0;   // margins stay 0
    __syncthreads();
    const int cw = kTgtSeg + 2 * h, nrow = 2 * h + 1;
    for (int e = tid; e < nrow * cw; e += 64 * kTgtWaves) {
        const int yy = y - h + e / cw, xx = x0 - h + e % cw;
        int c = -1;
        if (yy >= 0 && yy < H && xx >= 0 && xx < W) c = classify(dimg[(size_t)yy * W + xx], bnd, B, inv_l2span);
        cls[e] = c;
    }
    __syncthreads();

    // Window entries handled by this lane: e = lane + 64 m, offset (i, j).
    // Weights 1 - sqrt(i^2 + j^2) / (sqrt(2) h), in fp64, rounded to fp32
    // (>= 0 inside the window; 1 at the centre, also for K = 1).
    constexpr int NM = (kTgtMaxK * kTgtMaxK + 63) / 64;
    const int KK = K * K;
    const int nm = (KK + 63) / 64;
    float wgt[NM];
    int off[NM];
#pragma unroll
    for (int m = 0; m < NM; ++m) {
        const int e = lane + 64 * m;
        const int i = e / K - h, j = e % K - h;
        double w = 1.0;
        if (h > 0) w = 1.0 - sqrt((double)(i * i + j * j)) / (sqrt(2.0) * (double)h);
        wgt[m] = fmaxf((float)w, 0.0f);
        off[m] = (i + h) * cw + j + h;   // entry's class slot, relative to the pixel's column
    }
    // Eq. 8 taps (HZ + 1 - |i|) / (HZ + 1), i = -HZ .. HZ
    float tap[2 * HZ + 1];
#pragma unroll
    for (int i = -HZ; i <= HZ; ++i) tap[i + HZ] = (float)(HZ + 1 - (i < 0 ? -i : i)) / (float)(HZ + 1);

    // Two pixels of the wave at a time (xl, xl + 1), each on its own row, so
    // that the LDS round trips of one overlap the other's.
    constexpr int PPW = kTgtSeg / kTgtWaves;   // pixels per wave
    static_assert(PPW % 2 == 0, "pixel pairs");
    for (int q = 0; q < PPW; q += 2) {
        const int xb = wave * PPW + q;          // first pixel of the pair within the segment
        if (x0 + xb >= W) break;                // uniform per wave
        const bool two = x0 + xb + 1 < W;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int c = 0; c < CPL; ++c) row[wave][t][kTgtMaxH + CPL * lane + c] = 0;
        // the lane's window entries: classes of both pixels (-1: none)
        int cl[2][NM];
        int cc[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            cc[t] = cls[h * cw + h + xb + t];
#pragma unroll
            for (int m = 0; m < NM; ++m) {
                cl[t][m] = -1;
                if (m < nm) {
                    const int e = lane + 64 * m;
                    const int c = cls[(e < KK ? off[m] : 0) + xb + t];
                    cl[t][m] = e < KK ? c : -1;
                }
            }
        }
        // Where every surface in the window has the centre's class (flat
        // regions), C^ is 1 at that class alone and one lane writes it;
        // otherwise each entry raises its class with an LDS max.
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            bool mixed = false;
#pragma unroll
            for (int m = 0; m < NM; ++m) mixed |= cl[t][m] >= 0 && cl[t][m] != cc[t];
            if (__builtin_amdgcn_ballot_w64(mixed) == 0) {
                if (lane == 0 && cc[t] >= 0) row[wave][t][kTgtMaxH + cc[t]] = __float_as_int(1.0f);
            } else {
#pragma unroll
                for (int m = 0; m < NM; ++m)
                    if (m < nm && cl[t][m] >= 0) atomicMax(&row[wave][t][kTgtMaxH + cl[t][m]], __float_as_int(wgt[m]));
            }
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            if (t == 1 && !two) break;
            // this lane's classes and their HZ neighbours on both sides
            float v[CPL + 2 * HZ];
#pragma unroll
            for (int k = 0; k < CPL + 2 * HZ; ++k)
                v[k] = __int_as_float(row[wave][t][kTgtMaxH - HZ + CPL * lane + k]);
            float o[CPL];
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                float sum = 0.0f;
#pragma unroll
                for (int i = 0; i <= 2 * HZ; ++i) sum += v[c + i] * tap[i];
                o[c] = fminf(sum, 1.0f);
            }
            float* dst = out + ((img * H + y) * (size_t)W + x0 + xb + t) * (size_t)B + CPL * lane;
            // written once, read by a later consumer: stream past the caches
#pragma unroll
            for (int c = 0; c < CPL; ++c) __builtin_nontemporal_store(o[c], dst + c);
        }
    }
}

}  // namespace

namespace {
template <int CPL, int HZ>
void launch_cz(dim3 grid, hipStream_t stream, const float* depth, int H, int W, const float* bounds, int K,
               float inv_l2span, float* out) {
    hipLaunchKernelGGL((targets_kernel<CPL, HZ>), grid, dim3(64 * kTgtWaves), 0, stream, depth, H, W, bounds, K, inv_l2span, out);
}
template <int CPL>
void launch_c(int hz, dim3 grid, hipStream_t stream, const float* depth, int H, int W, const float* bounds, int K,
              float inv_l2span, float* out) {
    switch (hz) {
        case 0: launch_cz<CPL, 0>(grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        case 1: launch_cz<CPL, 1>(grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        case 2: launch_cz<CPL, 2>(grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        case 3: launch_cz<CPL, 3>(grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        case 4: launch_cz<CPL, 4>(grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        case 5: launch_cz<CPL, 5>(grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        case 6: launch_cz<CPL, 6>(grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        default: launch_cz<CPL, 7>(grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
    }
}
}  // namespace

hipError_t launch_targets(const float* depth, int P, int H, int W, const float* bounds, int B, int K, int Z,
                          float inv_l2span, float* out, hipStream_t stream) {
    const int segs = (W + kTgtSeg - 1) / kTgtSeg;
    const dim3 grid((uint32_t)((size_t)P * H * segs));
    const int hz = Z / 2;   // 0..7 (Z <= kTgtMaxK)
    switch (B / 64) {       // B in {64, 128, 192, 256}
        case 1: launch_c<1>(hz, grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        case 2: launch_c<2>(hz, grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        case 3: launch_c<3>(hz, grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        default: launch_c<4>(hz, grid, stream, depth, H, W, bounds, K, inv_l2span, out); break;
    }
    return hipGetLastError();
}

}  // namespace donerf
