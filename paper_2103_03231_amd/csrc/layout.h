// layout.h - register and memory layouts shared by the host packer and the
// gfx950 kernels.  Host and device both include it; nothing here touches HIP.
//
// Networks run in the transposed form Y^T = W X^T: weights are the MFMA A
// operand (rows = output units), activations the B operand (columns = rays or
// samples).  One MFMA step covers 32 output rows:
//   bf16: v_mfma_f32_32x32x16_bf16, 32 rows x 16 K; lane l holds row l%32 and
//         K slots 8*(l/32) + e, e = 0..7 (16 bytes)
//   fp32: four v_mfma_f32_32x32x2_f32, 32 rows x 8 K; lane l holds row l%32,
//         sub-step e = 0..3 reads K slot 2*e + l/32 (16 bytes)
//   fp8:  v_mfma_scale_f32_32x32x64_f8f6f4 on E4M3, 32 rows x 64 K; lane l
//         holds row l%32 and 32 K elements (32 bytes).  A and B place K the
//         same way, so element e of lane group g of A multiplies element e of
//         lane group g of B, whatever K the hardware assigns to it.
// A step's A operand is stored as 1 KiB units of 64 lanes x 16 bytes (one
// unit for fp32 and bf16, two for fp8: bytes 0-15 then 16-31 of each lane),
// so one ds_read_b128 per lane and unit fetches it without bank conflicts.
//
// Chaining.  The fp32 accumulator of a 32x32 MFMA block holds, on lane l
// with g = l/32, register i = 0..15 for row 8*(i/4) + 4*g + i%4 of the block
// and column l%32.  After bias, ReLU and (bf16) rounding those registers are
// used in place as the next layer's B operand.  The next layer's weight
// columns are permuted accordingly (chained_row), which is a relabelling of
// the hidden units and leaves the network's function unchanged.
#pragma once

#if defined(__HIPCC__)
#define DN_HD __host__ __device__
#else
#define DN_HD
#endif

namespace donerf {

constexpr int kHidden = 256;
constexpr int kDIn = 90;      // encode(unified origin / d_max, 10) + encode(dir, 4)
constexpr int kSIn = 63;      // encode(warped sample, 10)
constexpr int kSkip = 27;     // encode(dir, 4) into the last shading layer
constexpr int kSOut = 4;      // r, g, b, sigma
constexpr int kFragBytes = 1024;
#ifndef DONERF_CHUNK_FRAGS
#define DONERF_CHUNK_FRAGS 32
#endif
constexpr int kChunkFrags = DONERF_CHUNK_FRAGS;  // fragments per streamed chunk
constexpr int kChunkBytes = kChunkFrags * kFragBytes;

constexpr int kMaxPosesPerLaunch = 32;
#ifndef DONERF_RB_PER_PASS
#define DONERF_RB_PER_PASS 2
#endif
constexpr int kRbPerPass = DONERF_RB_PER_PASS;  // 32-row blocks per accumulator pass

// Arithmetic of a layer's MFMA steps (bool true/false convert to bf16/fp32).
enum Precision { kF32 = 0, kBF16 = 1, kFP8 = 2 };

// K elements per lane per step, K per step, 1 KiB units per step, bytes per
// element.
DN_HD constexpr int elems(int p) { return p == kFP8 ? 32 : p == kBF16 ? 8 : 4; }
DN_HD constexpr int kper(int p) { return p == kFP8 ? 64 : p == kBF16 ? 16 : 8; }
DN_HD constexpr int units(int p) { return p == kFP8 ? 2 : 1; }
DN_HD constexpr int elem_bytes(int p) { return p == kFP8 ? 1 : p == kBF16 ? 2 : 4; }
// Number of K steps for a padded K.
DN_HD constexpr int ksteps(int p, int kpad) { return kpad / kper(p); }

// Hidden unit (logical row of the previous layer) that feeds K step ks,
// lane group g, element e when the previous layer's accumulators are chained.
// bf16 / fp32: a 32-row block feeds 2 / 4 K steps.  fp8: a K step takes the
// 16 registers of two consecutive blocks, elements 0-15 from the first.
DN_HD constexpr int chained_row(int p, int ks, int g, int e) {
    return p == kFP8 ? 32 * (2 * ks + e / 16) + 8 * ((e % 16) / 4) + 4 * g + e % 4
                     : 32 * (ks / (16 / elems(p))) +
                           8 * (((ks % (16 / elems(p))) * elems(p) + e) / 4) + 4 * g +
                           (((ks % (16 / elems(p))) * elems(p) + e) % 4);
}

// bf16 networks run their six hidden layers on v_mfma_f32_16x16x32_bf16:
// 16 rows x 32 K per step, lane l holding row (A) or column (B) l % 16 and
// K elements 8 (l / 16) + e of lane group G = l / 16; the accumulator holds
// column l % 16, rows 4 G + i in register i.  A wave's 32 rays are two
// 16-column tiles, and a pass of four 16-row tiles has eight independent
// accumulation chains in the registers of two 32x32 blocks.  K step u of
// tile t is register 2 u + t of the 32x32 B operand array, and one
// v_permlane16_swap of registers 2 u and 2 u + 1 (lane quadrant 1 with 0,
// 3 with 2) converts between the two layouts in either direction.
DN_HD constexpr bool hid16(int net) { return net == kBF16; }
// Hidden unit that feeds 16x16 K step u, lane group G, element e when the
// previous 16x16 layer's accumulators are chained: row tiles 2 u and 2 u + 1
// give elements 0-3 and 4-7.
DN_HD constexpr int chained16(int u, int G, int e) { return 16 * (2 * u + e / 4) + 4 * G + e % 4; }
// The first hidden layer's input: the 32x32 chained layout after the swap
// (group G holds 32x32 K step 2 u + G % 2, lane group G / 2).
DN_HD constexpr int chained16_from32(int u, int G, int e) { return chained_row(kBF16, 2 * u + G % 2, G / 2, e); }
// A head after the hidden layers reads 32x32 K step ks, lane group g, after
// the swap back: 16x16 step ks / 2, group 2 g + ks % 2.
DN_HD constexpr int chained32_from16(int ks, int g, int e) { return chained16(ks / 2, 2 * g + ks % 2, e); }

// Per-lane feature slots.  Each column's features are split between lane
// groups g = 0 and 1 (lanes l and l+32 serve the same ray); lane slot s of
// group g sits at K step s / elems, element s % elems.  The maps give the
// index of the feature in the weight blob's input order, or -1 for padding.
// Frequencies alternate between the groups (k = 2t + g) so that both groups
// run the same instruction stream.
//
// Depth network input (90 features, 96 slots, 48 per group):
//   s in [0,30)  : position sin/cos at frequency 2t+g, t = s/6
//   s in [30,42) : direction sin/cos at frequency 2t+g, t = (s-30)/6
//   s in [42,45) : identity, position (g = 0) or direction (g = 1)
//   s in [45,48) : zero
DN_HD constexpr int d_feature(int g, int s) {
    return s < 30 ? 3 + 6 * (2 * (s / 6) + g) + s % 6
         : s < 42 ? 63 + 3 + 6 * (2 * ((s - 30) / 6) + g) + (s - 30) % 6
         : s < 45 ? (g == 0 ? s - 42 : 63 + s - 42)
         : -1;
}
constexpr int kDSlots = 48;
constexpr int kDKPad = 96;

// Shading network input (63 features, 64 slots, 32 per group):
//   s in [0,30) : sin/cos at frequency 2t+g
//   s == 30     : x (g = 0) or z (g = 1);  s == 31 : y (g = 0) or zero
DN_HD constexpr int s_feature(int g, int s) {
    return s < 30 ? 3 + 6 * (2 * (s / 6) + g) + s % 6
         : s == 30 ? (g == 0 ? 0 : 2)
         : (g == 0 ? 1 : -1);
}
constexpr int kSSlots = 32;
constexpr int kSKPad = 64;

// Direction skip into the last shading layer (27 features, 32 slots):
//   s in [0,12) : sin/cos at frequency 2t+g;  s in [12,15): identity (g = 0)
DN_HD constexpr int skip_feature(int g, int s) {
    return s < 12 ? 3 + 6 * (2 * (s / 6) + g) + s % 6
         : s < 15 ? (g == 0 ? s - 12 : -1)
         : -1;
}
constexpr int kSkipSlots = 16;
constexpr int kSkipKPad = 32;

// Depth network input of the paper (Sec. 5.2): unified origin, direction and
// one position per class centre, unencoded, 6 + 3 B values.  Position k is
// ((o - c) + c_k r) / d_max, so the layer's weights fold (host.cpp) into a
// 9-column layer over [u' (3), r (3), u_c (3)], u' = (o' - c) / d_max,
// u_c = (o - c) / d_max, run as fp32 fragments (K padded to 16).  K slot
// 8 ks + 2 e + g of the fp32 layout holds folded column K (< 9) or zero.
constexpr int kPIn = 9;
constexpr int kPKPad = 16;
DN_HD constexpr int p_feature(int ks, int g, int e) {
    return 8 * ks + 2 * e + g < kPIn ? 8 * ks + 2 * e + g : -1;
}

// Sample placement and depth-network input of a render variant.  kPlaceCdf
// keeps a ray's B <= 128 class values in registers; kPlaceCdfWide (B = 192,
// 256) runs the depth head twice, so the depth stream of such a network
// carries the head's chunks twice.
enum Placement { kPlaceTopN = 0, kPlaceCdf = 1, kPlaceCdfWide = 2 };
enum DepthInput { kDinEncoded = 0, kDinPositions = 1 };

// Layer roles in the streamed weight sequence.  kDFirstPos is the folded
// first depth layer of the positions input.
enum LayerKind { kDFirst = 0, kHiddenL = 1, kDHead = 2, kSFirst = 3, kSHead = 4, kDFirstPos = 5 };

struct LayerGeom {
    int out_rows;   // logical output units
    int in_cols;    // logical inputs (blob layout)
    int kpad;       // padded K consumed by the kernel
    int rb;         // 32-row output blocks
    int rbp;        // row blocks per accumulator pass
};

DN_HD constexpr LayerGeom layer_geom(int kind, int n_bins) {
    return kind == kDFirst  ? LayerGeom{kHidden, kDIn, kDKPad, 8, kRbPerPass}
         : kind == kDFirstPos ? LayerGeom{kHidden, kPIn, kPKPad, 8, kRbPerPass}
         : kind == kHiddenL ? LayerGeom{kHidden, kHidden, kHidden, 8, kRbPerPass}
         : kind == kDHead   ? LayerGeom{n_bins, kHidden, kHidden, n_bins / 32, kRbPerPass}
         : kind == kSFirst  ? LayerGeom{kHidden, kSIn, kSKPad, 8, kRbPerPass}
         :                    LayerGeom{kSOut, kHidden + kSkip, kHidden + kSkipKPad, 1, 1};
}

// Arithmetic of a layer in a network of precision net: the folded positions
// layer is fp32 in every network; an fp8 network keeps its first layers and
// heads in bf16 and runs the hidden layers in fp8.
DN_HD constexpr int frag_prec(int net, int kind) {
    return kind == kDFirstPos ? kF32 : net != kFP8 ? net : kind == kHiddenL ? kFP8 : kBF16;
}

// 1 KiB units a layer streams (before padding to whole chunks).
DN_HD constexpr int layer_frags(int net, int kind, int n_bins) {
    return layer_geom(kind, n_bins).rb * ksteps(frag_prec(net, kind), layer_geom(kind, n_bins).kpad) *
           units(frag_prec(net, kind));
}
// Chunks a layer streams.  The depth network's layers are padded with zeros
// to an even number of chunks, so that each starts in slot 0 of the two-slot
// LDS stream and the slot of every chunk is known at compile time.  The
// shading network's first layer and head are not: a sample's chunks add up to
// an even number (bf16 1 + 24 + 1, fp8 1 + 12 + 1, fp32 2 + 48 + 2), so every
// sample still starts in slot 0 and its layers' slots stay compile-time
// constants, and the two padding chunks per sample it saves are two barriers
// and two copies (0.45 % of the bf16 and 1.1 % of the fp8 step).
DN_HD constexpr bool layer_even_padded(int kind) { return !(kind == kSFirst || kind == kSHead); }
DN_HD constexpr int layer_chunks(int net, int kind, int n_bins) {
    return layer_even_padded(kind)
               ? (layer_frags(net, kind, n_bins) + 2 * kChunkFrags - 1) / (2 * kChunkFrags) * 2
               : (layer_frags(net, kind, n_bins) + kChunkFrags - 1) / kChunkFrags;
}

// Bias table: every layer's bias padded to 32 * rb floats; the depth
// network's seven ReLU layers, the shading network's eight layers, then the
// depth head (the one length that depends on B).
DN_HD constexpr int bias_len(int kind, int n_bins) { return 32 * layer_geom(kind, n_bins).rb; }

}  // namespace donerf
