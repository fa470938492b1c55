// targets.hip - training targets of the depth oracle (Sec. 5.1, Eq. 6-8) on
// gfx950: one-hot depth class of each pixel's first surface, the radial
// K x K neighbourhood filter (Eq. 7) and the triangle filter of size Z along
// the classes, clamped to 1 (Eq. 8).
//
// A workgroup renders one segment of kTgtSeg pixels of one image row.  It
// first classifies the window rows around the segment (the segment plus a
// halo of floor(K/2) pixels, floor(K/2) rows above and below) into LDS with a
// binary search over the class bounds.  Each wave then takes its pixels one
// at a time: one window entry per lane, each entry raises its class in a
// per-wave LDS row of B values to the entry's weight with an LDS max
// (Eq. 7's maximum; zeros stand for the centre term of classes without a
// surface), and the lanes, now over classes, apply Eq. 8 from that row and
// write the pixel's B targets as coalesced rows.  The output (4 B bytes per
// pixel) is the only sizeable HBM traffic.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace donerf {
namespace {

constexpr int kTgtSeg = 64;                 // pixels per workgroup
constexpr int kTgtWaves = 4;
constexpr int kTgtMaxH = kTgtMaxK / 2;      // largest half window

// Class of depth d: k with b_k <= d < b_{k+1}, or -1 outside [b_0, b_B) or
// not finite (comparisons with NaN are false).
__device__ __forceinline__ int classify(float d, const float* bnd, int B) {
    if (!(d >= bnd[0] && d < bnd[B])) return -1;
    int lo = 0, hi = B;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (d >= bnd[mid]) lo = mid;
        else hi = mid;
    }
    return lo;
}

__global__ void __launch_bounds__(64 * kTgtWaves)
targets_kernel(const float* __restrict__ depth, int H, int W, const float* __restrict__ bounds, int B, int K,
               int Z, float* __restrict__ out) {
    __shared__ float bnd[kMaxBins + 1];
    __shared__ int cls[(2 * kTgtMaxH + 1) * (kTgtSeg + 2 * kTgtMaxH)];
    __shared__ int row[kTgtWaves][kMaxBins];   // fp32 bits of the filtered values (all >= 0)

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = K / 2, hz = Z / 2;
    const int segs = (W + kTgtSeg - 1) / kTgtSeg;
    const int seg = blockIdx.x % segs;
    const int y = (blockIdx.x / segs) % H;
    const size_t img = blockIdx.x / ((size_t)segs * H);
    const int x0 = seg * kTgtSeg;
    const float* dimg = depth + img * (size_t)H * W;

    for (int k = tid; k <= B; k += 64 * kTgtWaves) bnd[k] = bounds[k];
    __syncthreads();
    const int cw = kTgtSeg + 2 * h, nrow = 2 * h + 1;
    for (int e = tid; e < nrow * cw; e += 64 * kTgtWaves) {
        const int yy = y - h + e / cw, xx = x0 - h + e % cw;
        int c = -1;
        if (yy >= 0 && yy < H && xx >= 0 && xx < W) c = classify(dimg[(size_t)yy * W + xx], bnd, B);
        cls[e] = c;
    }
    __syncthreads();

    // Window entries handled by this lane: e = lane + 64 m, offset (i, j).
    // Weights 1 - sqrt(i^2 + j^2) / (sqrt(2) h), in fp64, rounded to fp32
    // (>= 0 inside the window; 1 at the centre, also for K = 1).
    const int KK = K * K;
    const int nm = (KK + 63) / 64;
    float wgt[(kTgtMaxK * kTgtMaxK + 63) / 64];
    int off[(kTgtMaxK * kTgtMaxK + 63) / 64];
#pragma unroll
    for (int m = 0; m < (kTgtMaxK * kTgtMaxK + 63) / 64; ++m) {
        const int e = lane + 64 * m;
        const int i = e / K - h, j = e % K - h;
        double w = 1.0;
        if (h > 0) w = 1.0 - sqrt((double)(i * i + j * j)) / (sqrt(2.0) * (double)h);
        wgt[m] = fmaxf((float)w, 0.0f);
        off[m] = (i + h) * cw + j + h;   // entry's class slot, relative to the pixel's column
    }
    const float zden = (float)(hz + 1);

    for (int q = 0; q < kTgtSeg / kTgtWaves; ++q) {
        const int xl = wave * (kTgtSeg / kTgtWaves) + q;   // pixel within the segment (uniform per wave)
        if (x0 + xl >= W) break;
        for (int z = lane; z < B; z += 64) row[wave][z] = 0;
        for (int m = 0; m < nm; ++m) {
            const int e = lane + 64 * m;
            if (e < KK) {
                const int c = cls[off[m] + xl];
                if (c >= 0) atomicMax(&row[wave][c], __float_as_int(wgt[m]));
            }
        }
        float* o = out + ((img * H + y) * (size_t)W + x0 + xl) * (size_t)B;
        for (int z = lane; z < B; z += 64) {
            float s = 0.0f;
            for (int i = -hz; i <= hz; ++i) {
                const int zz = z + i;
                if (zz >= 0 && zz < B) s += __int_as_float(row[wave][zz]) * ((float)(hz + 1 - (i < 0 ? -i : i)) / zden);
            }
            o[z] = fminf(s, 1.0f);
        }
    }
}

}  // namespace

hipError_t launch_targets(const float* depth, int P, int H, int W, const float* bounds, int B, int K, int Z,
                          float* out, hipStream_t stream) {
    const int segs = (W + kTgtSeg - 1) / kTgtSeg;
    const dim3 grid((uint32_t)((size_t)P * H * segs));
    hipLaunchKernelGGL(targets_kernel, grid, dim3(64 * kTgtWaves), 0, stream, depth, H, W, bounds, B, K, Z, out);
    return hipGetLastError();
}

}  // namespace donerf
