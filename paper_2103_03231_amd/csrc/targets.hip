// targets.hip - training targets of the depth oracle (Sec. 5.1, Eq. 6-8) on
// gfx950: one-hot depth class of each pixel's first surface, the radial
// K x K neighbourhood filter (Eq. 7) and the triangle filter of size Z along
// the classes, clamped to 1 (Eq. 8).
//
// A workgroup renders a tile of kTgtRows image rows by kTgtSeg pixels.  It
// first classifies the window rows around the tile (the tile plus a halo of
// floor(K/2) pixels and rows on every side) into LDS: the coordinate of
// Eq. 3 proposes a class and comparisons with the class bounds settle it.
// Each wave then takes the pixels of one tile row two at a time, one window
// entry per lane.  Where every surface in a pixel's window has the centre's
// class (flat regions, most pixels), the targets are Eq. 8's taps around that
// class and the lanes, now over classes (CPL = B / 64 consecutive ones each),
// compute them in registers.  Otherwise each entry raises its class in a
// per-wave LDS row of B values to the entry's weight with an LDS max (Eq. 7's
// maximum; zeros stand for the centre term of classes without a surface),
// the lanes apply Eq. 8 from that row, whose zero margins stand for the
// classes outside [0, B), and clear it again.  Each pixel's B targets leave
// as one coalesced row; the output (4 B bytes per pixel) is the only sizeable
// HBM traffic.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace donerf {
namespace {

#ifndef DONERF_TGT_SEG
#define DONERF_TGT_SEG 64
#endif
constexpr int kTgtSeg = DONERF_TGT_SEG;     // pixels per row of a workgroup's tile
#ifndef DONERF_TGT_ROWS
#define DONERF_TGT_ROWS 1
#endif
constexpr int kTgtRows = DONERF_TGT_ROWS;   // rows per tile
constexpr int kTgtWaves = 4;
static_assert(kTgtWaves % kTgtRows == 0, "waves split evenly over the rows");
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
// Eq. 7's offsets run over -floor(K/2) .. floor(K/2), a window of side
// S = 2 floor(K/2) + 1 (K + 1 for an even K).  NM: window entries per lane,
// ceil(S^2 / 64); fixed at compile time so that a pixel's window reads issue
// together instead of one guarded read at a time.
template <int CPL, int HZ, int NM>
__global__ void __launch_bounds__(64 * kTgtWaves)
targets_kernel(const float* __restrict__ depth, int H, int W, const float* __restrict__ bounds, int K,
               float inv_l2span, float* __restrict__ out) {
    constexpr int B = 64 * CPL;
    // a row of C^ with a zero margin of HZ classes on each side, so that a
    // lane's window into it starts on an 8-byte boundary
    constexpr int RW = B + 2 * HZ;
    __shared__ float bnd[kMaxBins + 1];
    __shared__ int cls[(2 * kTgtMaxH + kTgtRows) * (kTgtSeg + 2 * kTgtMaxH)];
    __shared__ int row[kTgtWaves][2][RW];    // fp32 bits of C^ (all >= 0); row[..][HZ + z] holds class z

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = K / 2;
    const int segs = (W + kTgtSeg - 1) / kTgtSeg;
    const int tiles_y = (H + kTgtRows - 1) / kTgtRows;
    const int seg = blockIdx.x % segs;
    const int y0 = (blockIdx.x / segs) % tiles_y * kTgtRows;   // first row of the tile
    const size_t img = blockIdx.x / ((size_t)segs * tiles_y);
    const int x0 = seg * kTgtSeg;
    const float* dimg = depth + img * (size_t)H * W;

    for (int k = tid; k <= B; k += 64 * kTgtWaves) bnd[k] = bounds[k];
    for (int k = tid; k < kTgtWaves * 2 * RW; k += 64 * kTgtWaves) (&row[0][0][0])[k] = 0;   // margins stay 0
    __syncthreads();
    const int cw = kTgtSeg + 2 * h, nrow = 2 * h + kTgtRows;
    for (int e = tid; e < nrow * cw; e += 64 * kTgtWaves) {
        const int yy = y0 - h + e / cw, xx = x0 - h + e % cw;
        int c = -1;
        if (yy >= 0 && yy < H && xx >= 0 && xx < W) c = classify(dimg[(size_t)yy * W + xx], bnd, B, inv_l2span);
        cls[e] = c;
    }
    __syncthreads();

    // Window entries handled by this lane: e = lane + 64 m, offset (i, j).
    // Weights 1 - sqrt(i^2 + j^2) / (sqrt(2) h), in fp64, rounded to fp32
    // (>= 0 inside the window; 1 at the centre, also for K = 1).
    const int S = 2 * h + 1;
    const int KK = S * S;   // <= 64 NM
    float wgt[NM];
    int off[NM];
#pragma unroll
    for (int m = 0; m < NM; ++m) {
        const int e = lane + 64 * m;
        const int i = e / S - h, j = e % S - h;
        double w = 1.0;
        if (h > 0) w = 1.0 - sqrt((double)(i * i + j * j)) / (sqrt(2.0) * (double)h);
        wgt[m] = fmaxf((float)w, 0.0f);
        off[m] = (i + h) * cw + j + h;   // entry's class slot, relative to the pixel's column
    }
    // Eq. 8 taps (HZ + 1 - |i|) / (HZ + 1), i = -HZ .. HZ
    float tap[2 * HZ + 1];
#pragma unroll
    for (int i = -HZ; i <= HZ; ++i) tap[i + HZ] = (float)(HZ + 1 - (i < 0 ? -i : i)) / (float)(HZ + 1);

    // Each wave takes PPW pixels of one tile row, two at a time (xb, xb + 1),
    // each on its own LDS row, so that the LDS round trips of one overlap the
    // other's.
    constexpr int WPR = kTgtWaves / kTgtRows;  // waves per tile row
    constexpr int PPW = kTgtSeg / WPR;         // pixels per wave
    static_assert(PPW % 2 == 0, "pixel pairs");
    const int ty = wave / WPR;                 // the wave's row in the tile
    const int y = y0 + ty;
    if (y >= H) return;                        // uniform per wave; no barrier follows
    const int cbase = ty * cw;                 // its window's first class row
    for (int q = 0; q < PPW; q += 2) {
        const int xb = wave % WPR * PPW + q;    // first pixel of the pair within the segment
        if (x0 + xb >= W) break;                // uniform per wave
        const bool two = x0 + xb + 1 < W;
        const int np = two ? 2 : 1;
        // the lane's window entries: classes of both pixels (-1: none)
        int cl[2][NM];
        int cc[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            cc[t] = cls[cbase + h * cw + h + xb + t];
#pragma unroll
            for (int m = 0; m < NM; ++m) {
                const int e = lane + 64 * m;
                const int c = cls[cbase + (e < KK ? off[m] : 0) + xb + t];
                cl[t][m] = e < KK ? c : -1;
            }
        }
        // Where every surface in the window has the centre's class (flat
        // regions), C^ is 1 at that class alone (0 everywhere without a
        // surface) and Eq. 8 reduces to the taps around it, computed in
        // registers.  Otherwise each entry raises its class in the pixel's
        // LDS row with an LDS max.
        bool flat[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            bool mixed = false;
#pragma unroll
            for (int m = 0; m < NM; ++m) mixed |= cl[t][m] >= 0 && cl[t][m] != cc[t];
            flat[t] = __builtin_amdgcn_ballot_w64(mixed) == 0;
            if (!flat[t] && t < np) {
#pragma unroll
                for (int m = 0; m < NM; ++m)
                    if (cl[t][m] >= 0) atomicMax(&row[wave][t][HZ + cl[t][m]], __float_as_int(wgt[m]));
            }
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            if (t == 1 && !two) break;
            float o[CPL];
            if (flat[t]) {
                // the same sums as below with a single 1 among the zeros
#pragma unroll
                for (int c = 0; c < CPL; ++c) {
                    const int d = CPL * lane + c - cc[t];
                    float r = 0.0f;
#pragma unroll
                    for (int i = -HZ; i <= HZ; ++i) r = (cc[t] >= 0 && d == i) ? tap[i + HZ] : r;
                    o[c] = r;
                }
            } else {
                // this lane's classes and their HZ neighbours on both sides
                int* rw = &row[wave][t][CPL * lane];
                float v[CPL + 2 * HZ];
#pragma unroll
                for (int k = 0; k < CPL + 2 * HZ; ++k) v[k] = __int_as_float(rw[k]);
#pragma unroll
                for (int c = 0; c < CPL; ++c) {
                    float sum = 0.0f;
#pragma unroll
                    for (int i = 0; i <= 2 * HZ; ++i) sum += v[c + i] * tap[i];
                    o[c] = fminf(sum, 1.0f);
                }
                // back to zeros for the next pixel: every class is some
                // lane's own, and the wave's reads above precede these writes
#pragma unroll
                for (int c = 0; c < CPL; ++c) rw[HZ + c] = 0;
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
    const int S = 2 * (K / 2) + 1;   // the window's side, <= 15
    switch ((S * S + 63) / 64) {     // 1 .. 4
        case 1: hipLaunchKernelGGL((targets_kernel<CPL, HZ, 1>), grid, dim3(64 * kTgtWaves), 0, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        case 2: hipLaunchKernelGGL((targets_kernel<CPL, HZ, 2>), grid, dim3(64 * kTgtWaves), 0, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        case 3: hipLaunchKernelGGL((targets_kernel<CPL, HZ, 3>), grid, dim3(64 * kTgtWaves), 0, stream, depth, H, W, bounds, K, inv_l2span, out); break;
        default: hipLaunchKernelGGL((targets_kernel<CPL, HZ, 4>), grid, dim3(64 * kTgtWaves), 0, stream, depth, H, W, bounds, K, inv_l2span, out); break;
    }
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
    const dim3 grid((uint32_t)((size_t)P * ((H + kTgtRows - 1) / kTgtRows) * segs));
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
