// kernels.hip - the small kernels around the fused render kernel (split-tail
// combine, softmax of dumped scores, stand-alone top-N for testing), the
// static scratch of the allocation-free render, and the dispatch of render
// launches to the per-variant translation units.
#include <mutex>

#include "render_kernel.h"

namespace donerf {
namespace {

// Front-to-back composite of the split parts of a ray: C = C_0 + T_0 (C_1 +
// T_1 (C_2 + ...)), the same recurrence the render kernel runs per sample.
__global__ void combine_kernel(const float* partial, int split, uint32_t first_ray, uint32_t total_rays,
                               float* out_rgb, float* out_depth) {
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    const uint32_t ray = first_ray + i;
    if (ray >= total_rays) return;
    float T = 1.0f, c0 = 0.0f, c1 = 0.0f, c2 = 0.0f, d = 0.0f;
    for (int j = 0; j < split; ++j) {
        const float* q = partial + ((size_t)i * split + j) * 5;
        c0 += T * q[0];
        c1 += T * q[1];
        c2 += T * q[2];
        d += T * q[3];
        T *= q[4];
    }
    out_rgb[(size_t)ray * 3 + 0] = c0;
    out_rgb[(size_t)ray * 3 + 1] = c1;
    out_rgb[(size_t)ray * 3 + 2] = c2;
    if (out_depth) out_depth[ray] = d;
}

// Softmax of each score row in place (fp32: subtract the row maximum,
// exponentiate, sum in class order, divide).  Used for score dumps only: the
// softmax is strictly monotone, so it never changes the selection.
__global__ void softmax_rows_kernel(float* s, uint32_t rows, int B) {
    const uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= rows) return;
    float* x = s + (size_t)r * B;
    float m = x[0];
    for (int k = 1; k < B; ++k) m = fmaxf(m, x[k]);
    float sum = 0.0f;
    for (int k = 0; k < B; ++k) sum += expf(x[k] - m);
    for (int k = 0; k < B; ++k) x[k] = expf(x[k] - m) / sum;
}

// The render kernel's selection on given scores: each lane pushes its classes
// in the render kernel's register order, then merges with its partner lane.
template <int CB, int NCAP>
__global__ void __launch_bounds__(256) topn_kernel(const float* scores, int32_t rays, int32_t N, int32_t B,
                                                   int32_t* out) {
    const int lane = threadIdx.x & 63;
    const int g = lane >> 5;
    const int col = lane & 31;
    const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    sfor<CB>([&](auto C) {
        const int32_t r = wave * 32 * CB + 32 * CV(C) + col;
        const bool valid = r < rays;
        const float* row = scores + (size_t)(valid ? r : rays - 1) * B;
        TopList<NCAP> t;
        t.init();
        for (int p = 0; p < B / 64; ++p)
            for (int R = 0; R < 2; ++R)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int c = 64 * p + 32 * R + 8 * (i / 4) + (i % 4);
                    t.push(row[c + 4 * g], c);
                }
        t.rebase(4 * g);
        t.merge_partner();
        int s[NCAP];
        t.ascending(N, s);
        if (g == 0 && valid)
            for (int k = 0; k < N; ++k) out[(size_t)r * N + k] = pick<true>(s, k);
    });
}

}  // namespace

hipError_t launch_render(int prec, int ncap, int place, int din, const RenderArgs& a, uint32_t n_split_tiles,
                         hipStream_t stream) {
    const dim3 grid(a.n_full + n_split_tiles * (uint32_t)a.split);
    if (place == kPlaceCdfWide)
        return prec == kFP8    ? launch_render_fp8_cdf_wide(ncap, din, a, grid, stream)
               : prec == kBF16 ? launch_render_bf16_cdf_wide(ncap, din, a, grid, stream)
                               : launch_render_fp32_cdf_wide(ncap, din, a, grid, stream);
    if (prec == kFP8)
        return place == kPlaceCdf ? launch_render_fp8_cdf(ncap, din, a, grid, stream)
                                  : launch_render_fp8_topn(ncap, din, a, grid, stream);
    if (prec == kBF16)
        return place == kPlaceCdf ? launch_render_bf16_cdf(ncap, din, a, grid, stream)
                                  : launch_render_bf16_topn(ncap, din, a, grid, stream);
    return place == kPlaceCdf ? launch_render_fp32_cdf(ncap, din, a, grid, stream)
                              : launch_render_fp32_topn(ncap, din, a, grid, stream);
}

// ------------------------------------------------------------------ static scratch

// The split tail's partial results of donerf_render_static_scratch: a
// file-scope device array, so that entry point allocates nothing.  Each
// device holds its own copy, at its own address, until the process ends.
static __device__ __align__(256) float scratch[kStaticScratchFloats];

hipError_t static_scratch_address(int device, float** out) {
    static std::mutex mu;
    static float* ptr[kMaxDevices] = {};
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!ptr[device]) {
        // the array's name is a host-side stand-in; kernels need the
        // device address, which this call returns for the current device
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        ptr[device] = static_cast<float*>(p);
    }
    *out = ptr[device];
    return hipSuccess;
}

hipError_t launch_combine(int prec, const RenderArgs& a, hipStream_t stream) {
    const uint32_t first = a.n_full * (uint32_t)rays_per_block(prec);
    const uint32_t n = a.total_rays - first;
    hipLaunchKernelGGL(combine_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, a.partial, a.split, first,
                       a.total_rays, a.out_rgb, a.out_depth);
    return hipGetLastError();
}

hipError_t launch_softmax_rows(float* scores, uint32_t rows, int B, hipStream_t stream) {
    hipLaunchKernelGGL(softmax_rows_kernel, dim3((rows + 255) / 256), dim3(256), 0, stream, scores, rows, B);
    return hipGetLastError();
}

// ------------------------------------------------------------------ MFMA ceiling

// lowbias32 (C. Wellons' integer hash): operand bits for the loop below.
__device__ __forceinline__ uint32_t mix32(uint32_t x) {
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

// A uniform value in [-1, 1) and the next hash state.
__device__ __forceinline__ float rand_unit(uint32_t& st) {
    st = mix32(st + 0x9e3779b9u);
    return (float)(int32_t)st * 0x1p-31f;
}

// One u32x4 operand unit of random values in the precision's element format:
// uniform in [-1, 1) like the weights, or (RELU) their positive part like
// the activations a ReLU layer passes on, half of them zero.
template <int PR, bool RELU>
__device__ __forceinline__ u32x4 rand_operand(uint32_t& st) {
    auto next = [&]() { const float x = rand_unit(st); return RELU ? fmaxf(x, 0.0f) : x; };
    u32x4 v;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        if constexpr (PR == kBF16) {
            const float x = next(), y = next();
            v[w] = pack_bf16x2(x, y);
        } else if constexpr (PR == kFP8) {
            const float x0 = next(), x1 = next(), x2 = next(), x3 = next();
            uint32_t q = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(x0, x1, 0, false);
            v[w] = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(x2, x3, (int)q, true);
        } else {
            v[w] = __float_as_uint(next());
        }
    }
    return v;
}

// Register-fed MFMA loop: each wave runs four independent 32 x 32
// accumulator chains of `iters` steps on register operands drawn like the
// render kernel's (uniform weights as A, ReLU activations as B), so the
// matrix pipes never wait on memory or on a dependence.  What it sustains
// (the operands' data-dependent power included) is the practical ceiling of
// the render kernel's MFMA stream.  One value per thread keeps the work live.
template <int PR>
__global__ __launch_bounds__(256) void mfma_peak_kernel(int iters, uint32_t seed, float* sink) {
    using P = Prec<PR>;
    constexpr int U = PR == kFP8 ? 2 : 1;
    const uint32_t t = blockIdx.x * 256u + threadIdx.x;
    uint32_t st = mix32(seed ^ mix32(t));
    u32x4 a[2][U], b[2][U];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int u = 0; u < U; ++u) {
            a[m][u] = rand_operand<PR, false>(st);
            b[m][u] = rand_operand<PR, true>(st);
        }
    f32x16 acc[4];
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[c][e] = 0.0f;
    for (int i = 0; i < iters; ++i) {
        acc[0] = P::mma(a[0], b[0], acc[0], 127);
        acc[1] = P::mma(a[1], b[0], acc[1], 127);
        acc[2] = P::mma(a[0], b[1], acc[2], 127);
        acc[3] = P::mma(a[1], b[1], acc[3], 127);
    }
    float s = 0.0f;
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) s += acc[c][e];
    sink[t] = s;
}

hipError_t launch_mfma_peak(int prec, int workgroups, int iters, uint32_t seed, float* sink, hipStream_t stream) {
    const dim3 grid(workgroups), block(256);
    if (prec == kFP8) hipLaunchKernelGGL(mfma_peak_kernel<kFP8>, grid, block, 0, stream, iters, seed, sink);
    else if (prec == kBF16) hipLaunchKernelGGL(mfma_peak_kernel<kBF16>, grid, block, 0, stream, iters, seed, sink);
    else hipLaunchKernelGGL(mfma_peak_kernel<kF32>, grid, block, 0, stream, iters, seed, sink);
    return hipGetLastError();
}

hipError_t launch_topn(bool bf16_layout, int ncap, const float* scores, int32_t rays, int32_t N,
                       int32_t B, int32_t* out_idx, hipStream_t stream) {
    const int cb = bf16_layout ? 2 : 1;
    const int rays_per_block = 4 * 32 * cb;
    const dim3 grid((rays + rays_per_block - 1) / rays_per_block);
#define DN_TOPN(CB, NC) hipLaunchKernelGGL((topn_kernel<CB, NC>), grid, dim3(256), 0, stream, scores, rays, N, B, out_idx)
    if (cb == 2) {
        if (ncap == 4) DN_TOPN(2, 4);
        else if (ncap == 8) DN_TOPN(2, 8);
        else DN_TOPN(2, 16);
    } else {
        if (ncap == 4) DN_TOPN(1, 4);
        else if (ncap == 8) DN_TOPN(1, 8);
        else DN_TOPN(1, 16);
    }
#undef DN_TOPN
    return hipGetLastError();
}

}  // namespace donerf
