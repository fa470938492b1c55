// render_kernel.h - the fused DONeRF per-ray kernel for gfx950 (MI355X).
//
// One workgroup renders a tile of rays: ray generation and unification
// (Sec. 5.2), the depth-network input (encoded, Eq. 2, or the unencoded
// positions of Sec. 5.2), the depth-oracle network (App. D) on MFMA, the
// choice of samples (top-N classes in registers, or the inverse CDF of
// Sec. 5.1), the space warp (Eq. 4-5) and encoding, the shading network on
// MFMA with the encoded direction skipped into its last layer (App. D), and
// front-to-back compositing over black.  The only HBM traffic is the streamed
// weights (L2-resident after first touch) and the output pixels.
//
// Work split (bf16): 8 waves per workgroup, two per SIMD, one workgroup per
// CU.  Each wave owns 32 * CB rays (the MFMA columns); the workgroup shares
// one stream of weight fragments through two LDS chunk slots, so each
// weight byte read from L2 feeds every wave.  Activations never leave the
// registers: accumulators of layer l become, after bias, ReLU and rounding,
// the B operand of layer l+1 (layout.h explains the K permutation that makes
// this possible).
//
// Included by the render_*.hip translation units, each of which instantiates
// the variants of one precision and placement; everything here has internal
// linkage.
#pragma once

#include <hip/hip_runtime.h>

#include <utility>

#include "internal.h"

namespace donerf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

// ------------------------------------------------------------------ compile-time loops

template <class F, int... I>
__device__ __forceinline__ void sfor_impl(F& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void sfor(F&& f) {
    sfor_impl(f, std::make_integer_sequence<int, N>{});
}
#define CV(x) decltype(x)::value

// ------------------------------------------------------------------ precision traits

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    f32x2 v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

template <int PR>
struct Prec;

template <>
struct Prec<kBF16> {
    static constexpr int E = 8;      // K elements per lane per step
    static constexpr int U = 1;      // 1 KiB units (u32x4 per lane) per step, A and B alike
    static constexpr int KSPB = 2;   // K steps produced per 32-row block
    __device__ static __forceinline__ f32x16 mma(const u32x4* a, const u32x4* b, f32x16 c, int) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[0]),
                                                       __builtin_bit_cast(bf16x8, b[0]), c, 0, 0, 0);
    }
    __device__ static __forceinline__ u32x4 pack(const float* f) {
        return u32x4{pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]),
                     pack_bf16x2(f[4], f[5]), pack_bf16x2(f[6], f[7])};
    }
};

template <>
struct Prec<kF32> {
    static constexpr int E = 4;
    static constexpr int U = 1;
    static constexpr int KSPB = 4;
    __device__ static __forceinline__ f32x16 mma(const u32x4* a, const u32x4* b, f32x16 c, int) {
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[0].x), __uint_as_float(b[0].x), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[0].y), __uint_as_float(b[0].y), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[0].z), __uint_as_float(b[0].z), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[0].w), __uint_as_float(b[0].w), c, 0, 0, 0);
        return c;
    }
    __device__ static __forceinline__ u32x4 pack(const float* f) {
        return u32x4{__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                     __float_as_uint(f[3])};
    }
};

// E4M3 steps: A is 32 bytes per lane (two units), scaled by 2^(sa - 127)
// inside the MFMA (E8M0), which undoes the weights' per-layer 2^s; B is the
// 32 E4M3 activations of the lane (two u32x4 of the chained layout).
template <>
struct Prec<kFP8> {
    static constexpr int E = 32;
    static constexpr int U = 2;
    __device__ static __forceinline__ f32x16 mma(const u32x4* a, const u32x4* b, f32x16 c, int sa) {
        const i32x8 av = {(int)a[0].x, (int)a[0].y, (int)a[0].z, (int)a[0].w,
                          (int)a[1].x, (int)a[1].y, (int)a[1].z, (int)a[1].w};
        const i32x8 bv = {(int)b[0].x, (int)b[0].y, (int)b[0].z, (int)b[0].w,
                          (int)b[1].x, (int)b[1].y, (int)b[1].z, (int)b[1].w};
        return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, c, 0, 0, 0, sa, 0, 127);
    }
};

// ------------------------------------------------------------------ LDS weight stream

__device__ __forceinline__ void lds_barrier() {
    // Orders LDS traffic only; outstanding global prefetches stay in flight.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Orders one wave's LDS accesses across its lanes: LDS executes a wave's
// instructions in order, so only the compiler has to keep them in place.
__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}

constexpr int kChunkVec = kChunkBytes / 16;  // u32x4 per chunk
// LDS fragment reads in flight, in fragments: bf16 and fp32 fragments are
// one 1 KiB unit, fp8 steps two.  Measured on 5 x 400 x 400, N = 4: 12 bf16
// fragments ahead ran 2 % faster than 3 with 32x32 hidden layers; with the
// 16x16 hidden layers 10 runs 0.4 % faster than 12 and 14 0.6 % slower; fp8
// layers run best with 2 (of 2, 3, 4, 6).
#ifndef DONERF_FRAG_AHEAD
#define DONERF_FRAG_AHEAD 10
#endif
#ifndef DONERF_FRAG_AHEAD_FP8
#define DONERF_FRAG_AHEAD_FP8 2
#endif
constexpr int kFragAhead = DONERF_FRAG_AHEAD;
constexpr int kFragAheadFp8 = DONERF_FRAG_AHEAD_FP8;
#ifndef DONERF_FP8_OVERLAP
#define DONERF_FP8_OVERLAP 1
#endif
#ifndef DONERF_FP8_EPI_DELAY
#define DONERF_FP8_EPI_DELAY 2
#endif
#ifndef DONERF_FP8_BIAS_LEAD
#define DONERF_FP8_BIAS_LEAD 3
#endif

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int VM>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(VM >= 0 && VM < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4) | (15 << 8));
}

// The workgroup consumes one logical sequence of chunks: every depth-network
// chunk, then the shading-network chunks once per sample.  Chunks travel
// from L2 straight into LDS (global_load_lds, 16 bytes per lane) one chunk
// ahead of use, alternating between two LDS arrays.  The slot of every chunk
// is known at compile time (each layer is told the slot parity of its first
// chunk; layout.h layer_chunks), so every read and copy names its array
// statically: reads of one slot then carry a different alias scope from the
// copy in flight into the other, and need no wait for it.  Each wave copies
// kChunkFrags / NW fragments of every chunk; advancing to chunk c waits for
// the wave's own copies of c and then barriers, which both publishes c and
// retires every reader of chunk c - 1, whose slot the copy of c + 1 reuses.
// The copy count per step is constant (the stream index is clamped past its
// end) so the counter arithmetic holds at the tail.
template <int NW>
struct WeightStream {
    static constexpr int FPW = kChunkFrags / NW;  // fragments each wave copies per chunk
    static_assert(kChunkFrags % NW == 0, "chunk split");
    const u32x4* dsrc;
    const u32x4* ssrc;
    u32x4* ring0;
    u32x4* ring1;
    int nd, ns, total;
    int lane, wave;
    int src_k;   // stream index of the next chunk to copy (clamped to total - 1)
    int src_s;   // its position in the shading-network chunks (mod ns)

    // Branch-free (selects only), so chunk changes do not split the
    // scheduling region of the MFMA stream around them.
    template <int SLOT>
    __device__ __forceinline__ void issue() {
        const bool in_d = src_k < nd;
        const u32x4* base = in_d ? dsrc : ssrc;
        const int off = in_d ? src_k : src_s;
        const u32x4* sp = base + (size_t)off * kChunkVec + wave * FPW * 64 + lane;
        u32x4* dp = (SLOT ? ring1 : ring0) + wave * FPW * 64;
        // a scalar base and lane offset per four copies (the instruction
        // offset, below 4 KiB, moves both the global and the LDS address by
        // i KiB), so the copies hold no per-copy address registers
        sfor<FPW>([&](auto I) {
            constexpr int grp = CV(I) / 4, sub = CV(I) % 4;
            __builtin_amdgcn_global_load_lds(sp + grp * 4 * 64, dp + grp * 4 * 64, 16, sub * kFragBytes, 0);
        });
        const int nk = src_k + 1;
        const bool adv = nk < total;
        src_s = (adv && nk > nd) ? (src_s + 1 == ns ? 0 : src_s + 1) : src_s;
        src_k = adv ? nk : src_k;
    }
    __device__ __forceinline__ void start() {
        src_k = 0;
        src_s = 0;
        issue<0>();
    }
    // Begin the next chunk, which sits in slot PAR.
    template <int PAR>
    __device__ __forceinline__ void next() {
        wait_vmcnt<0>();
        lds_barrier();
        issue<1 - PAR>();
    }
    __device__ __forceinline__ void finish() { wait_vmcnt<0>(); }

    template <int PAR>
    __device__ __forceinline__ u32x4 frag(int i) const {
        return (PAR ? ring1 : ring0)[i * 64 + lane];
    }
};

// ------------------------------------------------------------------ MFMA layers

// A layer's biases: element off of the workgroup's LDS bias array.  Reads
// index the array itself with one integer offset: address arithmetic that
// passes through loop-carried pointers loses the array's identity, and the
// compiler then makes each such read wait for every LDS copy in flight.
struct BiasAt {
    const float* s;
    int off;
    __device__ __forceinline__ BiasAt operator+(int d) const { return BiasAt{s, off + d}; }
};

// Accumulator initialised with the bias of 32-row block r: lane group g holds
// rows 8q + 4g + j (q, j = 0..3) in register 4q + j.
__device__ __forceinline__ f32x16 bias_frag(BiasAt bias, int g) {
    f32x16 b;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(bias.s + (bias.off + 8 * q + 4 * g));
        b[4 * q + 0] = v[0];
        b[4 * q + 1] = v[1];
        b[4 * q + 2] = v[2];
        b[4 * q + 3] = v[3];
    }
    return b;
}

struct NoSide {
    template <class F>
    __device__ __forceinline__ void operator()(F) const {}
};

// One accumulator pass: RBP output row blocks x CB column blocks over KS K
// steps.  BASE is the index of the pass's first fragment within its layer;
// layers start on chunk boundaries, so chunk changes are known statically.
// D: LDS reads issued this many fragments ahead.  side(f) runs after the
// MFMAs of fragment f: register work that the matrix pipe can cover.
template <int PR, int CB, int KS, int RBP, int BASE, int D = kFragAhead, class WS, class GetB, class Epi,
          class Side = NoSide>
__device__ __forceinline__ void run_pass(WS& st, int g, BiasAt bias, GetB& getB, Epi&& epi, Side&& side = Side{}) {
    using P = Prec<PR>;
    static_assert(P::U == 1, "heads run single-unit steps");
    constexpr int NF = KS * RBP;   // fragments of the pass, in (K step, row block) order
    f32x16 acc[RBP][CB];
    sfor<RBP>([&](auto R) {
        const f32x16 b = bias_frag(bias + 32 * CV(R), g);
        sfor<CB>([&](auto C) { acc[CV(R)][CV(C)] = b; });
    });
    u32x4 a[NF];
    // Software pipeline: step s reads fragment s and multiplies fragment
    // s - D.  The scheduling barriers keep LDS reads and MFMAs in this order
    // (bounding the registers held by fragments in flight) while VALU and
    // SALU work may move across them.
    sfor<NF + D>([&](auto S) {
        constexpr int s = CV(S);
        if constexpr (s < NF) {
            constexpr int idx = BASE + s;   // BASE counts from an even chunk
            if constexpr (idx % kChunkFrags == 0) st.template next<(idx / kChunkFrags) & 1>();
            a[s] = st.template frag<(idx / kChunkFrags) & 1>(idx % kChunkFrags);
        }
        if constexpr (s >= D) {
            constexpr int f = s - D;
            constexpr int k = f / RBP, r = f % RBP;
            sfor<CB>([&](auto C) {
                const u32x4 bk = getB(std::integral_constant<int, k>{}, C);
                acc[r][CV(C)] = P::mma(&a[f], &bk, acc[r][CV(C)], 127);
            });
            side(std::integral_constant<int, f>{});
        }
        __builtin_amdgcn_sched_barrier(0x6);
    });
    sfor<RBP>([&](auto R) { sfor<CB>([&](auto C) { epi(R, C, acc[CV(R)][CV(C)]); }); });
}

// ReLU, round, and place a 32-row accumulator block as K steps
// [ks0, ks0 + KSPB) of the next layer's B operand.  bf16: round to nearest
// even, then ReLU on the packed pair as a signed 16-bit max with 0 (rounding
// preserves the sign, so this equals rounding the ReLU).
template <int PR, int NK, int CB>
__device__ __forceinline__ void emit_relu(const f32x16& acc, u32x4 (&out)[NK][CB], int ks0, int cb) {
    using P = Prec<PR>;
    if constexpr (PR == kBF16) {
        typedef short i16x2 __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int h = 0; h < P::KSPB; ++h) {
            u32x4 o;
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const i16x2 v = __builtin_bit_cast(i16x2, pack_bf16x2(acc[8 * h + 2 * w], acc[8 * h + 2 * w + 1]));
                o[w] = __builtin_bit_cast(uint32_t, __builtin_elementwise_max(v, i16x2{0, 0}));
            }
            out[ks0 + h][cb] = o;
        }
    } else {
        float v[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) v[i] = fmaxf(acc[i], 0.0f);
#pragma unroll
        for (int h = 0; h < P::KSPB; ++h) out[ks0 + h][cb] = P::pack(v + h * P::E);
    }
}

// ReLU, clamp to the E4M3 range and round (nearest even) the two 32-row
// blocks of a pass as K step ks of an fp8 layer's B operand: elements 0-15
// are block 0's registers, 16-31 block 1's (layout.h chained_row).
template <int NK, int CB>
__device__ __forceinline__ void emit_fp8(const f32x16& a0, const f32x16& a1, u32x4 (&out)[NK][CB], int ks,
                                         int cb) {
    uint32_t d[8];
#pragma unroll
    for (int w = 0; w < 8; ++w) {
        const f32x16& v = w < 4 ? a0 : a1;
        const int i = 4 * (w % 4);
        const float v0 = __builtin_amdgcn_fmed3f(v[i + 0], 0.0f, 448.0f);
        const float v1 = __builtin_amdgcn_fmed3f(v[i + 1], 0.0f, 448.0f);
        const float v2 = __builtin_amdgcn_fmed3f(v[i + 2], 0.0f, 448.0f);
        const float v3 = __builtin_amdgcn_fmed3f(v[i + 3], 0.0f, 448.0f);
        // The convert writes one half of its tied operand and keeps the
        // other; the second convert overwrites the half this one keeps, so
        // the operand may be any register: v0's, which dies here, rather
        // than a zero that costs a move per word.
        uint32_t x = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(v0, v1, __builtin_bit_cast(int, v0), false);
        x = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(v2, v3, (int)x, true);
        d[w] = x;
    }
    out[2 * ks][cb] = u32x4{d[0], d[1], d[2], d[3]};
    out[2 * ks + 1][cb] = u32x4{d[4], d[5], d[6], d[7]};
}

// Fully connected ReLU layer with 256 outputs (8 row blocks) as one software
// pipeline over its KS * 8 fragments: passes of kRbPerPass row blocks use
// alternating accumulator sets, so the bias/ReLU/rounding of pass p can
// overlap the MFMAs of pass p + 1, and LDS reads run kFragAhead fragments
// ahead across pass and chunk boundaries.  OUT is the precision of the
// output activations (the next layer's), MP that of the layer's own steps and
// input; sa is the E8M0 scale of fp8 weights.  getB(k, c) returns the u32x4
// k of the input (an fp8 step reads two).
template <int OUT, int CB, int KS, int MP, int PAR0 = 0, bool PADDED = true, class WS, class GetB, int NOUT>
__device__ __forceinline__ void hidden_layer(WS& st, int g, BiasAt bias, GetB&& getB,
                                             u32x4 (&out)[NOUT][CB], int sa = 127) {
    using M = Prec<MP>;
    constexpr int U = M::U;
    constexpr int RBP = kRbPerPass;
    constexpr int PF = KS * RBP;       // steps per pass
    constexpr int NF = 8 * KS;         // steps of the layer
    constexpr int SPC = kChunkFrags / U;  // steps per chunk
    constexpr int D = MP == kFP8 ? kFragAheadFp8 : kFragAhead;
    static_assert(OUT != kFP8 || RBP == 2, "an fp8 K step takes two row blocks");
    f32x16 acc[2][RBP][CB];
    u32x4 a[D + 1][U];
    constexpr int NP = 8 / RBP;        // passes
    // Overlapped passes (fp8 steps): the next pass's biases are read into its
    // accumulator set LEAD steps before the current pass ends, and a pass's
    // epilogue runs DEL steps into the next pass.
    constexpr bool OV = DONERF_FP8_OVERLAP && MP == kFP8;
    constexpr int DEL = DONERF_FP8_EPI_DELAY < PF - 2 ? DONERF_FP8_EPI_DELAY : PF - 2;
    constexpr int LEAD = DONERF_FP8_BIAS_LEAD < PF - DEL - 1 ? DONERF_FP8_BIAS_LEAD : PF - DEL - 1;
    static_assert(!OV || LEAD >= 1, "overlap needs room between the epilogue and the next biases");
    auto load_bias = [&](auto PP) {
        constexpr int q = CV(PP);
        sfor<RBP>([&](auto R) {
            const f32x16 b = bias_frag(bias + 32 * (RBP * q + CV(R)), g);
            sfor<CB>([&](auto C) { acc[q & 1][CV(R)][CV(C)] = b; });
        });
    };
    auto epilogue = [&](auto PP) {
        constexpr int p = CV(PP);
        if constexpr (OUT == kFP8) {
            sfor<CB>([&](auto C) { emit_fp8(acc[p & 1][0][CV(C)], acc[p & 1][1][CV(C)], out, p, CV(C)); });
            // Pin the pass's outputs here: layers outside a loop could
            // otherwise have their pure MFMA chains sunk past the later chunk
            // barriers to the blocks that use them, holding every fragment of
            // those chunks in registers.
            sfor<CB>([&](auto C) {
                const u32x4 o0 = out[2 * p][CV(C)], o1 = out[2 * p + 1][CV(C)];
                asm volatile("" ::"v"(o0), "v"(o1));
            });
        } else if constexpr (MP == kFP8) {
            sfor<RBP>([&](auto R) {
                sfor<CB>([&](auto C) {
                    emit_relu<OUT>(acc[p & 1][CV(R)][CV(C)], out, (p * RBP + CV(R)) * Prec<OUT>::KSPB, CV(C));
                    sfor<Prec<OUT>::KSPB>([&](auto H) {
                        const u32x4 o = out[(p * RBP + CV(R)) * Prec<OUT>::KSPB + CV(H)][CV(C)];
                        asm volatile("" ::"v"(o));
                    });
                });
            });
        } else {
            sfor<RBP>([&](auto R) {
                sfor<CB>([&](auto C) {
                    emit_relu<OUT>(acc[p & 1][CV(R)][CV(C)], out, (p * RBP + CV(R)) * Prec<OUT>::KSPB, CV(C));
                });
            });
        }
    };
    sfor<NF + D>([&](auto S) {
        constexpr int s = CV(S);
        if constexpr (s < NF) {
            if constexpr (s % SPC == 0) st.template next<(s / SPC + PAR0) & 1>();
#pragma unroll
            for (int u = 0; u < U; ++u)
                a[s % (D + 1)][u] = st.template frag<(s / SPC + PAR0) & 1>((s % SPC) * U + u);
        }
        if constexpr (s >= D) {
            constexpr int f = s - D;
            constexpr int p = f / PF, w = f % PF, k = w / RBP, r = w % RBP;
            if constexpr (!OV) {
                if constexpr (w == 0) load_bias(std::integral_constant<int, p>{});
            } else {
                if constexpr (p == 0 && w == 0) load_bias(std::integral_constant<int, 0>{});
                if constexpr (p + 1 < NP && w == PF - LEAD) load_bias(std::integral_constant<int, p + 1>{});
            }
            sfor<CB>([&](auto C) {
                u32x4 bk[U];
                sfor<U>([&](auto V) { bk[CV(V)] = getB(std::integral_constant<int, k * U + CV(V)>{}, C); });
                acc[p & 1][r][CV(C)] = M::mma(a[f % (D + 1)], bk, acc[p & 1][r][CV(C)], sa);
            });
            if constexpr (!OV) {
                if constexpr (w == PF - 1) epilogue(std::integral_constant<int, p>{});
            } else {
                if constexpr (p >= 1 && w == DEL) epilogue(std::integral_constant<int, p - 1>{});
                if constexpr (p == NP - 1 && w == PF - 1) epilogue(std::integral_constant<int, p>{});
            }
        }
        __builtin_amdgcn_sched_barrier(0x6);
    });
    // a layer of an odd number of chunks is padded to an even one (unless
    // the stream omits that padding)
    constexpr int CH = (NF * U + kChunkFrags - 1) / kChunkFrags;
    if constexpr (PADDED && (CH & 1)) st.template next<(CH + PAR0) & 1>();
}

// ------------------------------------------------------------------ 16x16 hidden layers (bf16)

// One v_mfma_f32_16x16x32_bf16 step (layout.h hid16).
__device__ __forceinline__ f32x4 mma16(const u32x4& a, const u32x4& b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
}

// Exchanges lane quadrant 1 of x with quadrant 0 of y and quadrant 3 of x
// with quadrant 2 of y (v_permlane16_swap_b32, per register).
__device__ __forceinline__ void swap16(u32x4& x, u32x4& y) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const auto r = __builtin_amdgcn_permlane16_swap(x[w], y[w], false, false);
        x[w] = r[0];
        y[w] = r[1];
    }
}

// The 16 K steps of a 32x32 B operand of one 32-ray block become the eight
// 16x16 K steps of its two 16-column tiles (step u, tile t in entry 2 u + t),
// and back: the swap is its own inverse.
template <int NK, int CB>
__device__ __forceinline__ void swap_layouts(u32x4 (&h)[NK][CB]) {
    static_assert(NK >= 16 && CB == 1, "one 32-ray block of 16 bf16 K steps");
#pragma unroll
    for (int u = 0; u < 8; ++u) swap16(h[2 * u][0], h[2 * u + 1][0]);
}

// ReLU and bf16 rounding of a pair (rounding keeps the sign, so a signed
// 16-bit max with 0 on the packed pair equals rounding the ReLU).
__device__ __forceinline__ uint32_t relu_bf16x2(float lo, float hi) {
    typedef short i16x2 __attribute__((ext_vector_type(2)));
    const i16x2 v = __builtin_bit_cast(i16x2, pack_bf16x2(lo, hi));
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(v, i16x2{0, 0}));
}

// A 256 -> 256 bf16 ReLU layer on 16x16x32 steps: four passes of four 16-row
// tiles (one 32 KiB chunk each), each over eight K steps of 32, for the two
// 16-column tiles, so a pass runs eight independent accumulation chains.  As
// in hidden_layer, passes alternate between two accumulator sets and the LDS
// reads run kFragAhead fragments ahead.  G: the lane group (lane / 16).
// getB(e, 0) returns entry e (16x16 step e / 2, tile e % 2) of the input;
// out receives the output in the same form.
template <int PAR0 = 0, class WS, class GetB, int NOUT, int CB>
__device__ __forceinline__ void hidden_layer16(WS& st, int G, BiasAt bias, GetB&& getB, u32x4 (&out)[NOUT][CB]) {
    constexpr int KS = 8;            // K steps of 32
    constexpr int RT = 4;            // 16-row tiles per pass
    constexpr int PF = KS * RT;      // fragments per pass
    constexpr int NF = 4 * PF;       // fragments of the layer
    constexpr int SPC = kChunkFrags; // fragments per chunk
    constexpr int D = kFragAhead;
    static_assert(PF == SPC, "a pass is one chunk");
    f32x4 acc[2][RT][2];
    u32x4 a[D + 1];
    auto load_bias = [&](auto PP) {
        constexpr int q = CV(PP);
        sfor<RT>([&](auto R) {
            const f32x4 b = *reinterpret_cast<const f32x4*>(bias.s + (bias.off + 16 * (RT * q + CV(R)) + 4 * G));
            acc[q & 1][CV(R)][0] = b;
            acc[q & 1][CV(R)][1] = b;
        });
    };
    // row tiles 2 j and 2 j + 1 of pass p become K step 2 p + j of the next
    // layer (layout.h chained16)
    auto epilogue = [&](auto PP) {
        constexpr int p = CV(PP);
        sfor<2>([&](auto J) {
            sfor<2>([&](auto T) {
                const f32x4& x = acc[p & 1][2 * CV(J)][CV(T)];
                const f32x4& y = acc[p & 1][2 * CV(J) + 1][CV(T)];
                out[2 * (2 * p + CV(J)) + CV(T)][0] =
                    u32x4{relu_bf16x2(x[0], x[1]), relu_bf16x2(x[2], x[3]), relu_bf16x2(y[0], y[1]),
                          relu_bf16x2(y[2], y[3])};
            });
        });
    };
    sfor<NF + D>([&](auto S) {
        constexpr int s = CV(S);
        if constexpr (s < NF) {
            if constexpr (s % SPC == 0) st.template next<(s / SPC + PAR0) & 1>();
            a[s % (D + 1)] = st.template frag<(s / SPC + PAR0) & 1>(s % SPC);
        }
        if constexpr (s >= D) {
            constexpr int f = s - D;
            constexpr int p = f / PF, w = f % PF, k = w / RT, r = w % RT;
            if constexpr (w == 0) load_bias(std::integral_constant<int, p>{});
            sfor<2>([&](auto T) {
                const u32x4 bk = getB(std::integral_constant<int, 2 * k + CV(T)>{}, std::integral_constant<int, 0>{});
                acc[p & 1][r][CV(T)] = mma16(a[f % (D + 1)], bk, acc[p & 1][r][CV(T)]);
            });
            if constexpr (w == PF - 1) epilogue(std::integral_constant<int, p>{});
        }
        __builtin_amdgcn_sched_barrier(0x6);
    });
}

// The shading head of a 16x16 network: one 16-row tile (rows 0..3 = r, g,
// b, sigma; the rest zero) over nine K steps of 32, the eight of the last
// hidden layer's 16x16 output h (entries 2 u + t) and the direction skip sk
// (entries t, swapped into the 16x16 layout), for the two 16-column tiles.
// A swap of the two tiles' accumulators then puts rows 0..3 of rays 0..31 in
// registers 0..3 of lanes 0..31, the lanes and registers the 32x32 head left
// them in.  BASE: 32 times the slot parity of the head's chunk.
template <int BASE, class WS, int NK, int NS, int CB, class Epi>
__device__ __forceinline__ void head16(WS& st, int G, BiasAt bias, u32x4 (&h)[NK][CB], u32x4 (&sk)[NS][CB],
                                       Epi&& epi) {
    static_assert(NK >= 16 && NS >= 2 && CB == 1, "one 32-ray block");
    constexpr int KS = 9;
    constexpr int D = kFragAhead;
    const f32x4 b = *reinterpret_cast<const f32x4*>(bias.s + (bias.off + 4 * G));
    f32x4 acc[2] = {b, b};
    u32x4 a[KS];
    sfor<KS + D>([&](auto S) {
        constexpr int s = CV(S);
        if constexpr (s < KS) {
            constexpr int idx = BASE + s;
            if constexpr (idx % kChunkFrags == 0) st.template next<(idx / kChunkFrags) & 1>();
            a[s] = st.template frag<(idx / kChunkFrags) & 1>(idx % kChunkFrags);
        }
        if constexpr (s >= D && s - D < KS) {
            constexpr int f = s - D;
            sfor<2>([&](auto T) {
                if constexpr (f < 8) acc[CV(T)] = mma16(a[f], h[2 * f + CV(T)][0], acc[CV(T)]);
                else acc[CV(T)] = mma16(a[f], sk[CV(T)][0], acc[CV(T)]);
            });
        }
        __builtin_amdgcn_sched_barrier(0x6);
    });
    f32x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(acc[0][i]), __float_as_uint(acc[1][i]), false,
                                                        false);
        o[i] = __uint_as_float(r[0]);
    }
    epi(o);
}

// ------------------------------------------------------------------ selection

// Best-first list of (score, class) under the order: higher score first,
// lower class index first among equal scores, -0 equal to +0, NaN below
// every number.  Each entry is one 64-bit key that orders exactly like that:
// the score's bits mapped to an unsigned order (the sign bit flipped for
// numbers >= +0, every bit flipped below), then 20 bits of 0xFFFFF - class.
// With the exponent of 1.0 above them the keys are doubles in [1, 2) whose
// numeric order is the key order, so an insertion is a max/min chain of
// v_max_f64 / v_min_f64: no compare masks and no branches, where a
// compare-and-select list needs four masks per insertion.  The list starts
// with keys of 1.0, below every real key.
template <int NCAP>
struct TopList {
    static constexpr uint32_t kIdx = 0xFFFFFu;
    double v[NCAP];
    __device__ __forceinline__ void init() {
#pragma unroll
        for (int k = 0; k < NCAP; ++k) v[k] = 1.0;
    }
    __device__ static __forceinline__ double key(float x, uint32_t cidx) {
        const uint32_t u = __float_as_uint(x + 0.0f);   // -0 becomes +0; NaN stays NaN
        uint32_t ord = u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
        ord = x != x ? 0u : ord;
        const uint32_t hi = __builtin_amdgcn_alignbit(0x3FFu, ord, 12);   // 0x3FF00000 | ord >> 12
        const uint32_t lo = (ord << 20) | cidx;
        return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
    }
    // v_max_f64 / v_min_f64 written out: keys are never NaN, where the
    // library fmax and fmin would first canonicalise their operands (one
    // more f64 instruction per operand not known to be canonical).
    __device__ static __forceinline__ double kmax(double a, double b) {
        double r;
        asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
        return r;
    }
    __device__ static __forceinline__ double kmin(double a, double b) {
        double r;
        asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
        return r;
    }
    __device__ __forceinline__ void insert(double t) {
#pragma unroll
        for (int k = 0; k < NCAP; ++k) {
            const double hi = kmax(v[k], t);
            if (k + 1 < NCAP) t = kmin(v[k], t);
            v[k] = hi;
        }
    }
    // Insert class ix - off of score x: callers pass the wave-uniform part
    // of the class index here and its lane part (off) to rebase() once all
    // classes are in; the order within the lane is the same.
    __device__ __forceinline__ void push(float x, int ix) { insert(key(x, kIdx - (uint32_t)ix)); }
    // Classes become ix + off.  Every key is a real one by then (each lane
    // pushes at least NCAP classes), so the index field does not wrap.
    __device__ __forceinline__ void rebase(int off) {
#pragma unroll
        for (int k = 0; k < NCAP; ++k)
            v[k] = __builtin_bit_cast(double, __builtin_bit_cast(uint64_t, v[k]) - (uint64_t)(uint32_t)off);
    }
    __device__ __forceinline__ int index(int k) const {
        return (int)(kIdx - ((uint32_t)__builtin_bit_cast(uint64_t, v[k]) & kIdx));
    }
    // Merge with the list of lane l ^ 32 (the other half of the same ray's
    // classes); both lanes end with the same list.
    __device__ __forceinline__ void merge_partner() {
        double pv[NCAP];
#pragma unroll
        for (int k = 0; k < NCAP; ++k) pv[k] = __shfl_xor(v[k], 32);
#pragma unroll
        for (int k = 0; k < NCAP; ++k) insert(pv[k]);
    }
    // The first N classes in ascending index order in s[0..N), padding after.
    __device__ __forceinline__ void ascending(int N, int (&s)[NCAP]) const {
#pragma unroll
        for (int k = 0; k < NCAP; ++k) s[k] = k < N ? index(k) : 0x7fff;
#pragma unroll
        for (int round = 0; round < NCAP; ++round) {
#pragma unroll
            for (int k = round & 1; k + 1 < NCAP; k += 2) {
                const int a = s[k], b = s[k + 1];
                s[k] = min(a, b);
                s[k + 1] = max(a, b);
            }
        }
    }
};

// Element k of a per-lane array, as a select chain.  PIN: each element
// first passes through an empty asm that pins it in a VGPR.  Otherwise the
// compiler folds the selects of array loads into one load at a computed
// index, the array becomes a per-thread LDS block, and placing each
// thread's block makes every wave read the workgroup size from the dispatch
// packet, a scalar load from host memory: pinning the top-N classes took
// 8,800 cycles off the 5 x 400 x 400 kernel's step from the depth head to
// the first sample.  The inverse-CDF arrays (pick_f, and the classes there)
// are left to the compiler: pinned in registers they spill, and those
// kernels ran 1 % (N = 4) to 5-10 % (N = 16) slower.
template <bool PIN, int NCAP>
__device__ __forceinline__ int pick(const int (&s)[NCAP], int k) {
    int r = s[0];
#pragma unroll
    for (int q = 1; q < NCAP; ++q) {
        if constexpr (PIN) {
            int v = s[q];
            asm("" : "+v"(v));
            r = k == q ? v : r;
        } else {
            r = k == q ? s[q] : r;
        }
    }
    return r;
}

__device__ __forceinline__ float pick_f(const float* v, int n, int k) {
    float r = v[0];
    for (int q = 1; q < n; ++q) r = k == q ? v[q] : r;
    return r;
}

// ------------------------------------------------------------------ inverse-CDF placement

// Sample placement of Sec. 5.1 (Fig. 7): the class values sigmoid(score)
// form a piecewise-constant PDF over the classes (uniform in the coordinate
// of Eq. 3); the CDF is inverted at u_i = (i + 0.5) / N, and each sample's
// width is the depth extent of its probability slice [i/N, (i+1)/N].
//
// v[P][R][i] holds this lane's class values for class 32 (P * RBP + R) +
// 8 (i/4) + 4 g + i%4, i.e. lane-local blocks of four consecutive classes;
// global block b = 2 * local + g alternates between the lane pair.  Both
// lanes build the same prefix over the blocks (the partner's block sums
// arrive by a lane swap), locate each target's block by counting the blocks
// that end at or below it, and take the block's four values from the lane
// that owns it.  Everything is fp32.
template <int NPM, int NCAP>
__device__ __forceinline__ void cdf_place(const float (&v)[NPM][kRbPerPass][16], int g, int N, int B,
                                          const float* u, float near, float far, float log2_span1, float (&ts)[NCAP],
                                          float (&ds)[NCAP], int (&cls)[NCAP]) {
    constexpr int NLB = NPM * kRbPerPass * 4;  // lane-local blocks
    constexpr int NB = 2 * NLB;                // blocks in class order
    float bs[NLB], pbs[NLB];
#pragma unroll
    for (int P = 0; P < NPM; ++P)
#pragma unroll
        for (int R = 0; R < kRbPerPass; ++R)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                bs[(P * kRbPerPass + R) * 4 + q] =
                    ((v[P][R][4 * q] + v[P][R][4 * q + 1]) + v[P][R][4 * q + 2]) + v[P][R][4 * q + 3];
#pragma unroll
    for (int lb = 0; lb < NLB; ++lb) pbs[lb] = __shfl_xor(bs[lb], 32);
    float pre[NB + 1];
    pre[0] = 0.0f;
#pragma unroll
    for (int b = 0; b < NB; ++b) pre[b + 1] = pre[b] + (((b & 1) == g) ? bs[b >> 1] : pbs[b >> 1]);
    const float total = pre[NB];

    // coordinate s in [0, 1] of the target fraction u; k: its class
    auto inverse = [&](float u, int& k) {
        const float m = u * total;
        int b = 0;
#pragma unroll
        for (int bb = 0; bb < NB; ++bb) b += pre[bb + 1] <= m ? 1 : 0;
        b = min(b, NB - 1);
        const int lb = b >> 1;
        float w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float r = 0.0f;
#pragma unroll
            for (int P = 0; P < NPM; ++P)
#pragma unroll
                for (int R = 0; R < kRbPerPass; ++R)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        r = lb == (P * kRbPerPass + R) * 4 + q ? v[P][R][4 * q + j] : r;
            w[j] = r;
        }
        const bool own = (b & 1) == g;
        float a4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float pw = __shfl_xor(w[j], 32);
            a4[j] = own ? w[j] : pw;
        }
        float lo = pre[0];
#pragma unroll
        for (int bb = 1; bb < NB; ++bb) lo = b == bb ? pre[bb] : lo;
        const float c1 = lo + a4[0], c2 = c1 + a4[1], c3 = c2 + a4[2];
        const int j = (m >= c1 ? 1 : 0) + (m >= c2 ? 1 : 0) + (m >= c3 ? 1 : 0);
        const float base = j == 0 ? lo : j == 1 ? c1 : j == 2 ? c2 : c3;
        const float aj = j == 0 ? a4[0] : j == 1 ? a4[1] : j == 2 ? a4[2] : a4[3];
        const float frac = aj > 0.0f ? fminf(fmaxf((m - base) / aj, 0.0f), 1.0f) : 0.0f;
        k = 4 * b + j;
        return ((float)k + frac) / (float)B;
    };
    auto to_depth = [&](float s) { return near + exp2f(s * log2_span1) - 1.0f; };  // inverse of Eq. 3
    float edge[NCAP + 1];
    edge[0] = near;
#pragma unroll
    for (int i = 0; i < NCAP; ++i) {
        if (i < N) {
            int k;
            ts[i] = to_depth(inverse(u[i], k));
            cls[i] = k;
            int kk;
            edge[i + 1] = i + 1 < N ? to_depth(inverse(u[kMaxSamples + i], kk)) : far;
        } else {
            ts[i] = far;
            cls[i] = B - 1;
            edge[i + 1] = far;
        }
    }
#pragma unroll
    for (int i = 0; i < NCAP; ++i) ds[i] = edge[i + 1] - edge[i];
}

// ------------------------------------------------------------------ geometry (fp32, fixed order)
// Built with -ffp-contract=off: every operation below rounds to fp32 in the
// written order.  Divides and sqrtf are correctly rounded (hipcc's default
// expansions); __fsqrt_rn is not used because it lowers to the bare hardware
// square root, which can be one ulp off, and the encoding multiplies an ulp
// of the ray geometry by up to 2^9 pi.

struct Ray {
    float o[3], r[3];
};

__device__ __forceinline__ Ray camera_ray(const RenderArgs& a, uint32_t ray) {
    const uint32_t hw = (uint32_t)a.H * (uint32_t)a.W;
    const uint32_t p = ray / hw;
    const uint32_t pix = ray - p * hw;
    const uint32_t j = pix / (uint32_t)a.W;
    const uint32_t i = pix - j * (uint32_t)a.W;
    const float u = (((float)i + 0.5f) - a.half_w) / a.focal;
    const float v = -((((float)j + 0.5f) - a.half_h) / a.focal);
    const float* M = a.poses[p];
    float d[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) d[k] = (M[4 * k + 0] * u + M[4 * k + 1] * v) + M[4 * k + 2] * -1.0f;
    const float n = sqrtf((d[0] * d[0] + d[1] * d[1]) + d[2] * d[2]);
    Ray out;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        out.r[k] = d[k] / n;
        out.o[k] = M[4 * k + 3];
    }
    return out;
}

// Sec. 5.2: the forward intersection with the sphere |x - c| = R, t >= 0.
__device__ __forceinline__ void unify(const RenderArgs& a, const Ray& ray, float (&ou)[3]) {
    const float q0 = ray.o[0] - a.cx, q1 = ray.o[1] - a.cy, q2 = ray.o[2] - a.cz;
    const float b = (ray.r[0] * q0 + ray.r[1] * q1) + ray.r[2] * q2;
    const float k = ((q0 * q0 + q1 * q1) + q2 * q2) - a.radius * a.radius;
    const float disc = fmaxf(b * b - k, 0.0f);
    const float t = fmaxf(-b + sqrtf(disc), 0.0f);
#pragma unroll
    for (int c = 0; c < 3; ++c) ou[c] = ray.o[c] + t * ray.r[c];
}

// Eq. 4-5: w = p / sqrt(|p| d_max), p = x - c, w = 0 at p = 0.
__device__ __forceinline__ void warp(const RenderArgs& a, const float (&x)[3], float (&w)[3]) {
    const float p0 = x[0] - a.cx, p1 = x[1] - a.cy, p2 = x[2] - a.cz;
    const float n = sqrtf((p0 * p0 + p1 * p1) + p2 * p2);
    const float s = sqrtf(n * a.dmax);
    const bool z = n == 0.0f;
    w[0] = z ? 0.0f : p0 / s;
    w[1] = z ? 0.0f : p1 / s;
    w[2] = z ? 0.0f : p2 / s;
}

// Encoding slots: T frequency pairs 2t + g (t < T) of v, written as
// [sin x, sin y, sin z, cos x, cos y, cos z] per frequency.  The scale 2^k is
// exact in fp32.  EXACT (fp32 networks): sincospif at every frequency, which
// avoids multiplying by a rounded pi.  Otherwise (bf16 features) the
// hardware sine and cosine, which take revolutions: y = v 2^(k-1) and its
// distance to the nearest integer r = y - rint(y) are exact, so sin(pi v 2^k)
// = sin(2 pi r) with r in [-1/2, 1/2], the range the hardware is accurate on.
// Measured against fp64 over that range and the encodings' arguments (up to
// about 280 revolutions before reduction): at most 1.3e-7 absolute error,
// far below the bf16 rounding the features then undergo.
#ifndef DONERF_PE_EXACT
#define DONERF_PE_EXACT 0
#endif
template <int T, bool EXACT>
__device__ __forceinline__ void fourier(const float (&v)[3], int g, float* f) {
    const float gs = g ? 2.0f : 1.0f;
#pragma unroll
    for (int c = 0; c < 3; ++c) {
#pragma unroll
        for (int t = 0; t < T; ++t) {
            float s, co;
            if (EXACT || DONERF_PE_EXACT) {
                const float sc = (float)(1u << (2 * t)) * gs;
                sincospif(v[c] * sc, &s, &co);
            } else {
                const float y = v[c] * ((float)(1u << (2 * t)) * 0.5f * gs);
                const float r = y - __builtin_rintf(y);
                s = __builtin_amdgcn_sinf(r);
                co = __builtin_amdgcn_cosf(r);
            }
            f[6 * t + c] = s;
            f[6 * t + 3 + c] = co;
        }
    }
}

// ------------------------------------------------------------------ scalar functions

// exp(-x), 1 / (1 + exp(-x)) and 1 - exp(-x): correctly rounded library
// functions for the fp32 network; for bf16 and fp8 networks the hardware
// exponential (v_exp_f32 on x log2 e) and reciprocal (v_rcp_f32), each within
// about an ulp, far inside what those networks' roundings already move.
template <bool EXACT>
__device__ __forceinline__ float exp_neg(float x) {
    if constexpr (EXACT) return expf(-x);
    else return __builtin_amdgcn_exp2f(x * -1.4426950408889634f);
}
template <bool EXACT>
__device__ __forceinline__ float sigmoid(float x) {
    if constexpr (EXACT) return 1.0f / (1.0f + expf(-x));
    else return __builtin_amdgcn_rcpf(1.0f + exp_neg<false>(x));
}
template <bool EXACT>
__device__ __forceinline__ float one_minus_exp_neg(float x) {
    if constexpr (EXACT) return -expm1f(-x);
    else return 1.0f - exp_neg<false>(x);
}

// ------------------------------------------------------------------ fused kernel

// LDS bias table: the seven depth layers, the seven shading layers and the
// shading head (32 floats), then the depth head (B <= 256): every offset the
// layer loops index is a compile-time constant.
constexpr int kDepthHeadBias = 7 * 256 + 7 * 256 + 32;
constexpr int kBiasMax = kDepthHeadBias + 256;

// LDS table of the wide inverse-CDF placement, one region per wave: first a
// ray's prefix over its 64 4-class blocks (stride 65 floats, odd so that the
// rays of a wave spread over the banks), later one head pass's class values
// (8 x 64 lanes x 16 bytes).
#ifndef DONERF_CDFW_AHEAD
#define DONERF_CDFW_AHEAD 4
#endif
constexpr int kCdfRayStride = 65;
constexpr int kCdfWaveFloats = 32 * kCdfRayStride;
constexpr int kCdfClass = 2 * 16;   // a ray's sample classes follow its (depth, width) pairs
static_assert(kCdfClass + 16 <= kCdfRayStride, "a ray's samples fit its row");
static_assert(kCdfWaveFloats >= 8 * 64 * 4 && kCdfWaveFloats % 4 == 0, "a pass's values fit a wave's region");

// PR: network precision (layout.h Precision; an fp8 network keeps its first
// layers and heads in bf16).  CB: 32-ray column blocks per wave.  NW: waves
// per workgroup.  OCC: waves per SIMD the register budget is sized for (with
// OCC * 4 > NW several workgroups share a CU).  NCAP: capacity of the top-N
// list (top-N) or of the sample arrays (CDF).  PLACE: sample placement.
// DIN: depth-network input (layout.h DepthInput).
template <int PR, int CB, int NW, int OCC, int NCAP, int PLACE, int DIN>
__global__ void __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(OCC, OCC)))
render_kernel(const RenderArgs a) {
    constexpr int FP = PR == kFP8 ? kBF16 : PR;   // first layers, heads, features
    using P = Prec<FP>;
    constexpr int E = P::E;
    // first depth layer: K steps of the encoded input or of the folded
    // positions input (always fp32 steps, 8 K each)
    constexpr int KS_D0 = DIN == kDinEncoded ? kDKPad / (2 * E) : kPKPad / (2 * Prec<kF32>::E);
    constexpr int KS_H = kHidden / (2 * E);       // heads: 16 | 32
    constexpr int KS_HID = ksteps(PR, kHidden);   // hidden layers: 16 | 32 | 4
    constexpr int KS_S0 = kSKPad / (2 * E);       // 4 | 8
    constexpr int KS_SK = kSkipKPad / (2 * E);    // 2 | 4

    __shared__ u32x4 ring0[kChunkVec];
    __shared__ u32x4 ring1[kChunkVec];
    __shared__ float bias_s[kBiasMax];
    __shared__ float bins_s[2 * 256];
    __shared__ __align__(16) float cdf_s[PLACE == kPlaceCdfWide ? NW * kCdfWaveFloats : 4];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: lets the stream address one chunk from scalars
    const int g = lane >> 5;
    const int col = lane & 31;

    for (int k = tid; k < a.bias_len; k += 64 * NW) bias_s[k] = a.bias[k];
    for (int k = tid; k < 2 * a.B; k += 64 * NW) bins_s[k] = a.bins[k];

    WeightStream<NW> st;
    st.dsrc = reinterpret_cast<const u32x4*>(a.d_frags);
    st.ssrc = reinterpret_cast<const u32x4*>(a.s_frags);
    st.ring0 = ring0;
    st.ring1 = ring1;
    st.nd = a.n_d_chunks;
    st.ns = a.n_s_chunks;
    // this workgroup's tile and its share of the samples
    const bool split_part = blockIdx.x >= a.n_full;
    const uint32_t cpart = blockIdx.x - a.n_full;
    const int nsplit = split_part ? a.split : 1;
    const int part = split_part ? (int)(cpart % (uint32_t)a.split) : 0;
    const uint32_t tile_local = split_part ? cpart / (uint32_t)a.split : 0;
    const uint32_t tile = split_part ? a.n_full + tile_local : blockIdx.x;
    const int k_begin = part * a.N / nsplit;
    const int k_end = (part + 1) * a.N / nsplit;
    st.total = a.n_d_chunks + (k_end - k_begin) * a.n_s_chunks;
    st.lane = lane;
    st.wave = wave;
    st.start();

    // ---- rays of this wave: column col of block cb
    const uint32_t ray0 = (tile * NW + wave) * (32 * CB);
    uint32_t rid[CB];
    bool valid[CB];
    Ray ray[CB];
    u32x4 din[KS_D0][CB];
    u32x4 skip[KS_SK][CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
        const uint32_t r = ray0 + 32 * cb + col;
        valid[cb] = r < a.total_rays;
        rid[cb] = valid[cb] ? r : a.total_rays - 1;
        ray[cb] = camera_ray(a, rid[cb]);
        float ou[3], v[3];
        unify(a, ray[cb], ou);
        v[0] = (ou[0] - a.cx) / a.dmax;
        v[1] = (ou[1] - a.cy) / a.dmax;
        v[2] = (ou[2] - a.cz) / a.dmax;
        float f[kDSlots];
        if constexpr (DIN == kDinEncoded) {
            fourier<5, FP == kF32>(v, g, f);
            fourier<2, FP == kF32>(ray[cb].r, g, f + 30);
            f[42] = g ? ray[cb].r[0] : v[0];
            f[43] = g ? ray[cb].r[1] : v[1];
            f[44] = g ? ray[cb].r[2] : v[2];
            f[45] = f[46] = f[47] = 0.0f;
#pragma unroll
            for (int ks = 0; ks < KS_D0; ++ks) din[ks][cb] = P::pack(f + E * ks);
        } else {
            // Sec. 5.2's unencoded input: position k is ((o - c) + c_k r) / d_max,
            // so its weight columns fold into those of u_c = (o - c) / d_max and
            // of r (done once at create).  The folded layer reads
            // [u', r, u_c] (layout.h p_feature) as fp32 fragments.
            const float q9[9] = {v[0], v[1], v[2], ray[cb].r[0], ray[cb].r[1], ray[cb].r[2],
                                 (ray[cb].o[0] - a.cx) / a.dmax, (ray[cb].o[1] - a.cy) / a.dmax,
                                 (ray[cb].o[2] - a.cz) / a.dmax};
            float q[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                q[e] = g ? q9[2 * e + 1] : q9[2 * e];
                q[4 + e] = (e == 0 && g == 0) ? q9[8] : 0.0f;
            }
            din[0][cb] = Prec<kF32>::pack(q);
            din[1][cb] = Prec<kF32>::pack(q + 4);
            fourier<2, FP == kF32>(ray[cb].r, g, f + 30);
        }
        // the direction skip of the last shading layer: the same direction
        // encoding plus the identity
        float fs[kSkipSlots];
#pragma unroll
        for (int k = 0; k < 12; ++k) fs[k] = f[30 + k];
        fs[12] = g ? 0.0f : ray[cb].r[0];
        fs[13] = g ? 0.0f : ray[cb].r[1];
        fs[14] = g ? 0.0f : ray[cb].r[2];
        fs[15] = 0.0f;
#pragma unroll
        for (int ks = 0; ks < KS_SK; ++ks) skip[ks][cb] = P::pack(fs + E * ks);
    }
    // a 16x16 shading head reads the skip as one K step of its two tiles
    if constexpr (hid16(PR)) swap16(skip[0][0], skip[1][0]);
    lds_barrier();  // bias_s and bins_s visible

    // ---- depth-oracle network
    // Layers alternate h0 -> h1 -> h0; h0 holds the input of the next layer
    // (an fp8 layer's input takes the first 2 KS_HID entries).
    u32x4 h0[KS_H][CB], h1[KS_H][CB];
    auto g0 = [&](auto K, auto C) { return h0[CV(K)][CV(C)]; };
    auto g1 = [&](auto K, auto C) { return h1[CV(K)][CV(C)]; };
    // six 256 -> 256 ReLU layers whose biases start at bias_l0 and whose fp8
    // weight scales start at ws; the last one feeds a head in FP
    // (PAR: slot parity of the first chunk; every hidden layer streams an
    // even number of chunks, so it holds for all six)
    // BACK: whether the output returns to the 32x32 layout (the depth head
    // needs it; the shading head of a 16x16 network reads the 16x16 one)
    auto hidden6 = [&](auto PAR, BiasAt bias_l0, const int32_t* ws, auto BACK) {
        constexpr int Q = CV(PAR);
        if constexpr (PR == kFP8) {
            for (int l = 0; l < 2; ++l) {
                hidden_layer<kFP8, CB, KS_HID, kFP8, Q>(st, g, bias_l0 + 256 * (2 * l), g0, h1, ws[2 * l]);
                hidden_layer<kFP8, CB, KS_HID, kFP8, Q>(st, g, bias_l0 + 256 * (2 * l + 1), g1, h0, ws[2 * l + 1]);
            }
            hidden_layer<kFP8, CB, KS_HID, kFP8, Q>(st, g, bias_l0 + 256 * 4, g0, h1, ws[4]);
            hidden_layer<FP, CB, KS_HID, kFP8, Q>(st, g, bias_l0 + 256 * 5, g1, h0, ws[5]);
        } else if constexpr (hid16(PR)) {
            // 16x16 steps: the first layer's output changes layout on the way
            // in, the last hidden layer's on the way out to a 32x32 head
            const int G = lane >> 4;
            swap_layouts(h0);
            for (int l = 0; l < 3; ++l) {
                hidden_layer16<Q>(st, G, bias_l0 + 256 * (2 * l), g0, h1);
                hidden_layer16<Q>(st, G, bias_l0 + 256 * (2 * l + 1), g1, h0);
            }
            if constexpr (CV(BACK)) swap_layouts(h0);
        } else {
            for (int l = 0; l < 3; ++l) {
                hidden_layer<PR, CB, KS_HID, PR, Q>(st, g, bias_l0 + 256 * (2 * l), g0, h1);
                hidden_layer<PR, CB, KS_HID, PR, Q>(st, g, bias_l0 + 256 * (2 * l + 1), g1, h0);
            }
        }
    };
    static_assert(layer_chunks(PR, kHiddenL, 128) % 2 == 0, "hidden layers keep the slot parity");
    {
        auto gin = [&](auto K, auto C) { return din[CV(K)][CV(C)]; };
        hidden_layer<PR, CB, KS_D0, DIN == kDinEncoded ? FP : kF32>(st, g, BiasAt{bias_s, 0}, gin, h0);
    }
    hidden6(std::integral_constant<int, 0>{}, BiasAt{bias_s, 256}, a.wscale + 1, std::true_type{});
    // Head of the depth network: B / 64 passes of 64 classes (32 * kRbPerPass).
    const int npass = a.B / (32 * kRbPerPass);
    constexpr int PASS_FRAGS = KS_H * kRbPerPass;
    // Passes are grouped so that a group spans exactly two chunks (a pass
    // spans CPP whole chunks, or PPC passes share one); the head is padded to
    // an even number of chunks, so the chunks of a missing pass that starts a
    // chunk are padding and are consumed in its place.
    static_assert(PASS_FRAGS >= kChunkFrags ? PASS_FRAGS % kChunkFrags == 0 : kChunkFrags % PASS_FRAGS == 0,
                  "passes and chunks nest");
    constexpr int CPP = PASS_FRAGS >= kChunkFrags ? PASS_FRAGS / kChunkFrags : 1;
    constexpr int PPC = PASS_FRAGS >= kChunkFrags ? 1 : kChunkFrags / PASS_FRAGS;
    static_assert(CPP <= 2, "pass grouping");
    constexpr int GP = CPP == 2 ? 1 : 2 * PPC;
    auto dump_scores = [&](int p, int R, int C, const f32x16& acc) {
        if (a.out_scores && part == 0 && valid[C]) {
            float* dst = a.out_scores + (size_t)rid[C] * a.B;
            const int rowb = 32 * kRbPerPass * p + 32 * R + 4 * g;
#pragma unroll
            for (int i = 0; i < 16; ++i) dst[rowb + 8 * (i / 4) + (i % 4)] = acc[i];
        }
    };
    // Per ray: sample depth t, width delta and class of sample k.
    int sel[CB][NCAP];
    float st_t[CB][NCAP], st_d[CB][NCAP];
    if constexpr (PLACE == kPlaceTopN) {
        TopList<NCAP> top[CB];
        sfor<CB>([&](auto C) { top[CV(C)].init(); });
        // Within a group, the scores of pass q wait in registers (the hidden
        // activations h1 are dead here) and enter the lists one per fragment
        // during the MFMAs of pass q + 1; the group's last pass inserts its
        // own after its MFMAs.
        constexpr int PF = KS_H * kRbPerPass;   // fragments per pass
        static_assert(PF >= 16 * kRbPerPass, "one insertion per fragment covers a pass's scores");
        for (int p0 = 0; p0 < npass; p0 += GP) {
            f32x16 held[kRbPerPass][CB];
            int held_p = 0;
            auto push_held = [&](auto F) {
                constexpr int f = CV(F);
                if constexpr (f < 16 * kRbPerPass) {
                    constexpr int R = f / 16, i = f % 16;
                    sfor<CB>([&](auto C) {
                        // The volatile asms hold the insertion at its step: the
                        // compiler would otherwise move it out of the MFMA
                        // stream, up to the chunk barrier or down past the pass.
                        float x = held[R][CV(C)][i];
                        asm volatile("" : "+v"(x));
                        top[CV(C)].push(x, 32 * kRbPerPass * held_p + 32 * R + 8 * (i / 4) + (i % 4));
#pragma unroll
                        for (int k = 0; k < NCAP; ++k) asm volatile("" : "+v"(top[CV(C)].v[k]));
                    });
                }
            };
            sfor<GP>([&](auto Q) {
                constexpr int q = CV(Q);
                const int p = p0 + q;
                if (p >= npass) {
                    constexpr int f0 = q * PASS_FRAGS;   // the pass's first fragment in the group
                    if constexpr (f0 % kChunkFrags == 0) {
                        sfor<CPP>([&](auto J) { st.template next<(f0 / kChunkFrags + CV(J)) & 1>(); });
                    }
                    if constexpr (q > 0) {
                        if (p == npass) sfor<16 * kRbPerPass>(push_held);   // the last pass's, held
                    }
                } else {
                    auto epi = [&](auto R, auto C, const f32x16& acc) {
                        if constexpr (q + 1 < GP) {
                            held[CV(R)][CV(C)] = acc;
                        } else {
                            const int rowb = 32 * kRbPerPass * p + 32 * CV(R);   // + 4 g: rebase below
#pragma unroll
                            for (int i = 0; i < 16; ++i) top[CV(C)].push(acc[i], rowb + 8 * (i / 4) + (i % 4));
                        }
                        dump_scores(p, CV(R), CV(C), acc);
                    };
                    if constexpr (q > 0) {
                        run_pass<FP, CB, KS_H, kRbPerPass, q * PASS_FRAGS>(
                            st, g, BiasAt{bias_s, kDepthHeadBias + 32 * kRbPerPass * p}, g0, epi, push_held);
                    } else {
                        run_pass<FP, CB, KS_H, kRbPerPass, q * PASS_FRAGS>(
                            st, g, BiasAt{bias_s, kDepthHeadBias + 32 * kRbPerPass * p}, g0, epi);
                    }
                    held_p = p;
                }
            });
        }
        sfor<CB>([&](auto C) {
            top[CV(C)].rebase(4 * g);
            top[CV(C)].merge_partner();
            top[CV(C)].ascending(a.N, sel[CV(C)]);
        });
    } else if constexpr (PLACE == kPlaceCdf) {
        // Inverse-CDF placement needs every class value of the ray; B <= 128
        // keeps them in registers (the hidden activations h1 are dead here).
        static_assert(PASS_FRAGS % kChunkFrags == 0, "a pass spans whole chunks");
        constexpr int NPM = 128 / (32 * kRbPerPass);
        float vals[CB][NPM][kRbPerPass][16];
        sfor<NPM>([&](auto PI) {
            constexpr int p = CV(PI);
            if (p < npass) {
                run_pass<FP, CB, KS_H, kRbPerPass, p * PASS_FRAGS>(
                    st, g, BiasAt{bias_s, kDepthHeadBias + 32 * kRbPerPass * p}, g0,
                    [&](auto R, auto C, const f32x16& acc) {
#pragma unroll
                        for (int i = 0; i < 16; ++i) vals[CV(C)][p][CV(R)][i] = sigmoid<FP == kF32>(acc[i]);
                        dump_scores(p, CV(R), CV(C), acc);
                    });
            } else {
                if constexpr (CPP == 1 && (p & 1)) st.template next<1>();   // padding chunk
                sfor<CB>([&](auto C) {
#pragma unroll
                    for (int R = 0; R < kRbPerPass; ++R)
#pragma unroll
                        for (int i = 0; i < 16; ++i) vals[CV(C)][p][R][i] = 0.0f;
                });
            }
        });
        sfor<CB>([&](auto C) {
            cdf_place<NPM, NCAP>(vals[CV(C)], g, a.N, a.B, a.cdf_u, a.near, a.dmax, a.log2_span1, st_t[CV(C)],
                                 st_d[CV(C)], sel[CV(C)]);
        });
    } else {
        // Inverse-CDF placement for B = 192 and 256, whose class values do
        // not fit in registers.  The steps are cdf_place's: 4-class block
        // sums, their prefix in class order, a target u located by that
        // prefix, then inside its block.
        //   sweep 1: the head's passes yield the block sums only; the ray's
        //            prefix goes to its row of the wave's LDS table, and each
        //            target's block b and its rest r = m - pre[b] come from a
        //            binary search of that row;
        //   sweep 2: the head runs again (the depth stream carries its
        //            chunks twice); each pass stages its class values in the
        //            table, and every target whose block lies in the pass
        //            reads that block's four values and is resolved.
        // Both lane groups of a ray compute the same targets.
        static_assert(CB == 1, "the LDS table holds one 32-ray column block per wave");
        static_assert(PASS_FRAGS % kChunkFrags == 0, "a pass spans whole chunks");
        constexpr int NPM = 256 / (32 * kRbPerPass);   // passes at B = 256
        constexpr int NLB = NPM * kRbPerPass * 4;      // lane-local blocks
        constexpr int NB = 2 * NLB;                    // blocks in class order
        constexpr int NT = 2 * NCAP - 1;               // targets: NCAP slice centres, NCAP - 1 inner slice ends
        static_assert(NB <= kCdfRayStride && NB == 64, "a ray's prefix fits its row; 4 bits of block per pass");
        const int tbase = wave * kCdfWaveFloats;
        const int rbase = tbase + col * kCdfRayStride;
        auto target_u = [&](int t) { return t < NCAP ? a.cdf_u[t] : a.cdf_u[kMaxSamples + t - NCAP]; };
        auto head_pass = [&](auto PI, auto&& epi) {
            constexpr int p = CV(PI);
            run_pass<FP, CB, KS_H, kRbPerPass, p * PASS_FRAGS, DONERF_CDFW_AHEAD>(
                st, g, BiasAt{bias_s, kDepthHeadBias + 32 * kRbPerPass * p}, g0, epi);
        };

        // sweep 1: block sums (absent passes of B = 192 add zeros)
        float bs[NLB];
        sfor<NPM>([&](auto PI) {
            constexpr int p = CV(PI);
            if (p < npass) {
                head_pass(PI, [&](auto R, auto C, const f32x16& acc) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const float v0 = sigmoid<FP == kF32>(acc[4 * q]), v1 = sigmoid<FP == kF32>(acc[4 * q + 1]);
                        const float v2 = sigmoid<FP == kF32>(acc[4 * q + 2]), v3 = sigmoid<FP == kF32>(acc[4 * q + 3]);
                        bs[(p * kRbPerPass + CV(R)) * 4 + q] = ((v0 + v1) + v2) + v3;
                    }
                    dump_scores(p, CV(R), CV(C), acc);
                });
            } else {
                if constexpr (CPP == 1 && (p & 1)) st.template next<1>();   // padding chunk
#pragma unroll
                for (int i = 0; i < kRbPerPass * 4; ++i) bs[p * kRbPerPass * 4 + i] = 0.0f;
            }
        });
        // prefix pre[b] (the blocks before b) in class order: block b lies
        // on lane group b & 1, lane-local block b >> 1; group g stores the
        // entries of parity g
        float total;
        {
            float pre = 0.0f;
#pragma unroll
            for (int b2 = 0; b2 < NB; b2 += 2) {
                const float own = bs[b2 >> 1];
                const float other = __shfl_xor(own, 32);
                const float e0 = g ? other : own;   // block b2 (group 0)
                const float e1 = g ? own : other;   // block b2 + 1 (group 1)
                const float pre1 = pre + e0;
                cdf_s[rbase + b2 + g] = g ? pre1 : pre;
                pre = pre1 + e1;
            }
            total = pre;
        }
        wave_lds_fence();
        // Block b of target t: the last with pre[b] <= m (pre[0] = 0), which
        // is cdf_place's count of block ends at or below m (m < total, so
        // b < B / 4).
        // Per target one byte holds 4 b, later 4 b + j = its class.
        uint32_t tk[(NT + 3) / 4];
        float tr[NT];
#pragma unroll
        for (int i = 0; i < (NT + 3) / 4; ++i) tk[i] = 0;
        sfor<NT>([&](auto T) {
            constexpr int t = CV(T);
            const float m = target_u(t) * total;
            int b = 0;
            float lo = 0.0f;
#pragma unroll
            for (int step = NB / 2; step >= 1; step >>= 1) {
                const float v = cdf_s[rbase + b + step];
                const bool take = v <= m;
                b = take ? b + step : b;
                lo = take ? v : lo;
            }
            tk[t / 4] |= (uint32_t)(4 * b) << (8 * (t % 4));
            tr[t] = m - lo;
            // four searches at a time: the scheduler would otherwise
            // interleave all of them and hold every step's compare mask
            if constexpr (t % 4 == 3) __builtin_amdgcn_sched_barrier(0);
        });

        // sweep 2: resolve each target in its block's pass; tr then holds
        // its coordinate s
        const float inv_b = 1.0f / (float)a.B;
        sfor<NPM>([&](auto PI) {
            constexpr int p = CV(PI);
            if (p < npass) {
                wave_lds_fence();   // the table's earlier reads come before these writes
                head_pass(PI, [&](auto R, auto C, const f32x16& acc) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        f32x4 v;
                        v[0] = sigmoid<FP == kF32>(acc[4 * q]);
                        v[1] = sigmoid<FP == kF32>(acc[4 * q + 1]);
                        v[2] = sigmoid<FP == kF32>(acc[4 * q + 2]);
                        v[3] = sigmoid<FP == kF32>(acc[4 * q + 3]);
                        *reinterpret_cast<f32x4*>(&cdf_s[tbase + 4 * ((CV(R) * 4 + q) * 64 + lane)]) = v;
                    }
                });
                wave_lds_fence();
                sfor<NT>([&](auto T) {
                    constexpr int t = CV(T);
                    const int kb = (int)(tk[t / 4] >> (8 * (t % 4))) & 255;
                    if ((kb >> 6) == p) {   // the block's pass (a resolved target keeps it)
                        // block b = 16 p + 8 R + 2 q + g': values of lane col + 32 g'
                        const int b = kb >> 2;
                        const int slot = (((b >> 3) & 1) * 4 + ((b >> 1) & 3)) * 64 + col + 32 * (b & 1);
                        const f32x4 w = *reinterpret_cast<const f32x4*>(&cdf_s[tbase + 4 * slot]);
                        const float r = tr[t];
                        const float c1 = w[0], c2 = c1 + w[1], c3 = c2 + w[2];
                        const int j = (r >= c1 ? 1 : 0) + (r >= c2 ? 1 : 0) + (r >= c3 ? 1 : 0);
                        const float base = j == 0 ? 0.0f : j == 1 ? c1 : j == 2 ? c2 : c3;
                        const float aj = j == 0 ? w[0] : j == 1 ? w[1] : j == 2 ? w[2] : w[3];
                        const float frac =
                            aj > 0.0f ? fminf(fmaxf((r - base) * __builtin_amdgcn_rcpf(aj), 0.0f), 1.0f) : 0.0f;
                        tr[t] = ((float)(4 * b + j) + frac) * inv_b;
                        tk[t / 4] += (uint32_t)j << (8 * (t % 4));
                    }
                });
            } else {
                if constexpr (CPP == 1 && (p & 1)) st.template next<1>();   // padding chunk
            }
        });
        // The ray's samples go to its row (depth, width at 2 k, 2 k + 1; class
        // at kCdfClass + k), where the shading loop reads them: held in
        // registers through that loop they would spill.
        wave_lds_fence();   // the staged values are read
        auto to_depth = [&](float s) { return a.near + exp2f(s * a.log2_span1) - 1.0f; };  // inverse of Eq. 3
        float lo_edge = a.near;
#pragma unroll
        for (int i = 0; i < NCAP; ++i) {
            if (i < a.N) {
                // (the last centre has no inner end after it: N <= NCAP)
                const float hi_edge = i + 1 < a.N ? to_depth(tr[NCAP + (i + 1 < NCAP ? i : 0)]) : a.dmax;
                cdf_s[rbase + 2 * i + g] = g ? hi_edge - lo_edge : to_depth(tr[i]);
                cdf_s[rbase + kCdfClass + i] = __int_as_float((int)(tk[i / 4] >> (8 * (i % 4))) & 255);
                lo_edge = hi_edge;
            }
        }
        wave_lds_fence();
    }
    // sample k of column block cb: depth, width
    auto sample_td = [&](int cb, int k, float& t, float& d) {
        if constexpr (PLACE == kPlaceTopN) {
            // Always a class index for finite scores; clamped so that no
            // sentinel can address outside the class table.
            const int bin = min(pick<true>(sel[cb], k), a.B - 1);
            t = bins_s[bin];
            d = bins_s[a.B + bin];
        } else if constexpr (PLACE == kPlaceCdf) {
            t = pick_f(st_t[cb], NCAP, k);
            d = pick_f(st_d[cb], NCAP, k);
        } else {
            const int row = wave * kCdfWaveFloats + col * kCdfRayStride;
            t = cdf_s[row + 2 * k];
            d = cdf_s[row + 2 * k + 1];
        }
    };

    // ---- shading network per sample, composited front to back
    const int s_bias = 7 * 256;
    float T[CB], Cr[CB], Cg[CB], Cb[CB], Dp[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) T[cb] = 1.0f, Cr[cb] = Cg[cb] = Cb[cb] = Dp[cb] = 0.0f;

    for (int k = k_begin; k < k_end; ++k) {
        u32x4 sin_[KS_S0][CB];
        float tk[CB], dk[CB];
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
            sample_td(cb, k, tk[cb], dk[cb]);
            float x[3], w[3];
#pragma unroll
            for (int c = 0; c < 3; ++c) x[c] = ray[cb].o[c] + tk[cb] * ray[cb].r[c];
            warp(a, x, w);
            float f[kSSlots];
            fourier<5, FP == kF32>(w, g, f);
            f[30] = g ? w[2] : w[0];
            f[31] = g ? 0.0f : w[1];
#pragma unroll
            for (int ks = 0; ks < KS_S0; ++ks) sin_[ks][cb] = P::pack(f + E * ks);
        }
        // Slot parity within a sample: its chunks add up to an even number,
        // so every sample starts in slot 0.
        constexpr int S0C = layer_chunks(PR, kSFirst, 128);
        constexpr int HEADC = layer_chunks(PR, kSHead, 128);
        constexpr int HIDC = 6 * layer_chunks(PR, kHiddenL, 128);
        static_assert((S0C + HIDC + HEADC) % 2 == 0, "a sample's chunks keep the slot parity");
        {
            auto gs = [&](auto K, auto C) { return sin_[CV(K)][CV(C)]; };
            hidden_layer<PR, CB, KS_S0, FP, 0, layer_even_padded(kSFirst)>(st, g, BiasAt{bias_s, s_bias}, gs, h0);
        }
        hidden6(std::integral_constant<int, S0C & 1>{}, BiasAt{bias_s, s_bias + 256}, a.wscale + 9,
                std::integral_constant<bool, !hid16(PR)>{});
        // compositing of one sample from its head outputs (r, g, b, sigma)
        auto composite = [&](auto C, float hr, float hg, float hb, float hs) {
            constexpr int cb = CV(C);
            const float cr = sigmoid<FP == kF32>(hr);
            const float cg = sigmoid<FP == kF32>(hg);
            const float cbl = sigmoid<FP == kF32>(hb);
            const float sigma = fmaxf(hs, 0.0f);
            const float tau = sigma * dk[cb];
            const float alpha = one_minus_exp_neg<FP == kF32>(tau);
            const float wgt = T[cb] * alpha;
            Cr[cb] += wgt * cr;
            Cg[cb] += wgt * cg;
            Cb[cb] += wgt * cbl;
            Dp[cb] += wgt * tk[cb];
            T[cb] *= exp_neg<FP == kF32>(tau);
        };
        if constexpr (hid16(PR)) {
            head16<kChunkFrags * ((S0C + HIDC) & 1)>(st, lane >> 4, BiasAt{bias_s, s_bias + 7 * 256}, h0, skip,
                                                     [&](const f32x4& o) {
                                                         composite(std::integral_constant<int, 0>{}, o[0], o[1], o[2], o[3]);
                                                     });
        } else {
            auto gh = [&](auto K, auto C) {
                if constexpr (CV(K) < KS_H) return h0[CV(K)][CV(C)];
                else return skip[CV(K) - KS_H][CV(C)];
            };
            run_pass<FP, CB, KS_H + KS_SK, 1, kChunkFrags * ((S0C + HIDC) & 1)>(
                st, g, BiasAt{bias_s, s_bias + 7 * 256}, gh, [&](auto R, auto C, const f32x16& acc) {
                    // lanes of group 0 hold rows 0..3 = (r, g, b, sigma) in registers 0..3
                    composite(C, acc[0], acc[1], acc[2], acc[3]);
                });
        }
    }
    st.finish();  // no copy into LDS may outlive the workgroup

    // ---- outputs (lane group 0 holds the composited values)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
        if (g == 0 && valid[cb]) {
            if (nsplit > 1) {
                const uint32_t local = tile_local * (32 * CB * NW) + wave * (32 * CB) + 32 * cb + col;
                float* q = a.partial + ((size_t)local * nsplit + part) * 5;
                q[0] = Cr[cb];
                q[1] = Cg[cb];
                q[2] = Cb[cb];
                q[3] = Dp[cb];
                q[4] = T[cb];
            } else {
                float* o = a.out_rgb + (size_t)rid[cb] * 3;
                o[0] = Cr[cb];
                o[1] = Cg[cb];
                o[2] = Cb[cb];
                if (a.out_depth) a.out_depth[rid[cb]] = Dp[cb];
            }
            if (a.out_bins && part == 0) {
                for (int k = 0; k < a.N; ++k) {
                    if constexpr (PLACE == kPlaceCdfWide)
                        a.out_bins[(size_t)rid[cb] * a.N + k] =
                            __float_as_int(cdf_s[wave * kCdfWaveFloats + col * kCdfRayStride + kCdfClass + k]);
                    else
                        a.out_bins[(size_t)rid[cb] * a.N + k] = pick<PLACE == kPlaceTopN>(sel[cb], k);
                }
            }
            if (a.out_samples && part == 0) {
                for (int k = 0; k < a.N; ++k) {
                    float t, d;
                    sample_td(cb, k, t, d);
                    a.out_samples[((size_t)rid[cb] * a.N + k) * 2 + 0] = t;
                    a.out_samples[((size_t)rid[cb] * a.N + k) * 2 + 1] = d;
                }
            }
        }
    }
}

// One render variant; ncap selects the sample capacity.
template <int PR, int CB, int NW, int OCC, int PL, int DIN>
hipError_t launch_variant(int ncap, const RenderArgs& a, dim3 grid, hipStream_t stream) {
    if (ncap == 4)
        hipLaunchKernelGGL((render_kernel<PR, CB, NW, OCC, 4, PL, DIN>), grid, dim3(64 * NW), 0, stream, a);
    else if (ncap == 8)
        hipLaunchKernelGGL((render_kernel<PR, CB, NW, OCC, 8, PL, DIN>), grid, dim3(64 * NW), 0, stream, a);
    else
        hipLaunchKernelGGL((render_kernel<PR, CB, NW, OCC, 16, PL, DIN>), grid, dim3(64 * NW), 0, stream, a);
    return hipGetLastError();
}

// Both depth inputs of one precision and placement.
template <int PR, int CB, int NW, int OCC, int PL>
hipError_t launch_placement(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream) {
    return din == kDinPositions ? launch_variant<PR, CB, NW, OCC, PL, kDinPositions>(ncap, a, grid, stream)
                                : launch_variant<PR, CB, NW, OCC, PL, kDinEncoded>(ncap, a, grid, stream);
}

}  // namespace
}  // namespace donerf
