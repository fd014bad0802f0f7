// Data-layout geometry of the batched latent-rollout evaluator: matrix
// fragment orders of the packed weights, chunk sizes, workspace helpers and
// the host-side model description.  Plain C++ (usable without the HIP
// compiler: the host packing code and its CPU tests include it alone).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/wm.h"

#ifndef __HIPCC__
#define __host__
#define __device__
#endif

namespace wm {

// --------------------------------------------------------------------------
// Matrix-fragment layout of the 32x32 matrix-core products (gfx950).
//
// Both products used here, v_mfma_f32_32x32x16_bf16 (8 bf16 per lane) and
// v_mfma_f32_32x32x2_f32 (1 float per lane), share one accumulator layout:
// lane L, accumulator register r in [0,16) holds row acc_row(L/32, r) and
// column L%32 of the 32x32 result.  The A (resp. B) operand of lane L holds
// row (resp. column) L%32, and operand slot j of lane half L/32 multiplies the
// same k in A and in B, so any consistent assignment of contraction indices
// to (half, slot) pairs is valid.  The kernels exploit that freedom so that
// every intermediate stays in registers:
//
//  * The rollout computes the transposed products  G^T = W1 . X^T  and
//    dZ^T = W2 . G^T, so weights are always the A operand and candidates are
//    the 32 columns.  The latent z of a candidate is carried in accumulator
//    layout (block b of 32 features, register r -> feature 32b+acc_row(h,r)),
//    and is fed back as the B operand of the next step's first product
//    without leaving its lane: operand fragment f of block b takes
//    registers [f*SL, f*SL+SL).  The hidden activations G^T come out of the
//    first product in the same layout and feed the second product the same
//    way.  The weight matrices are packed with their contraction columns in
//    that order (pack_* in wm_api.hip), so no data moves between lanes.
//  * The embedding part of [z; e] and all cost-model inputs use the natural
//    order: slot j of half h of fragment q is feature KF*q + SL*h + j.
// --------------------------------------------------------------------------
__host__ __device__ constexpr inline int acc_row(int half, int r) {
  return 8 * (r >> 2) + 4 * half + (r & 3);
}

// Operand-fragment geometry of a precision.
//   KF: contraction length of one product; SL: operand elements per lane;
//   G:  fragments per 16-byte lane group (the unit of an LDS read);
//   ES: bytes per stored weight element.
template <int KF_, int SL_, int G_, int ES_>
struct FragGeom {
  static constexpr int KF = KF_, SL = SL_, G = G_, ES = ES_;
};
using GeomBF16 = FragGeom<16, 8, 1, 2>;
using GeomF32 = FragGeom<2, 1, 4, 4>;

// Feature index held by operand slot (half, j) of fragment kf of the
// transition input X = [z; e] (width D + E).
template <class Gm>
__host__ __device__ constexpr inline int x_feature(int D, int kf, int half, int j) {
  constexpr int per_block = 32 / Gm::KF;      // fragments per 32-feature block of z
  if (kf < D / Gm::KF) {
    const int b = kf / per_block, f = kf % per_block;
    return 32 * b + acc_row(half, f * Gm::SL + j);
  }
  const int q = kf - D / Gm::KF;
  return D + Gm::KF * q + Gm::SL * half + j;
}

// Hidden unit (within a 32-wide chunk) held by slot (half, j) of the
// fragment f of GELU outputs that feeds the second product.
template <class Gm>
__host__ __device__ constexpr inline int g_feature(int f, int half, int j) {
  return acc_row(half, f * Gm::SL + j);
}

// Natural order (embedding part, cost-model inputs).
template <class Gm>
__host__ __device__ constexpr inline int nat_feature(int kf, int half, int j) {
  return Gm::KF * kf + Gm::SL * half + j;
}

// Byte offset of operand element (fragment F, lane L, slot j) inside a block
// of packed fragments: fragments are grouped G at a time, each group is
// 64 lanes x 16 bytes, lane-major.
template <class Gm>
__host__ __device__ constexpr inline int frag_offset(int F, int lane, int j) {
  return (F / Gm::G) * 1024 + lane * 16 + ((F % Gm::G) * Gm::SL + j) * Gm::ES;
}

// Chunk geometry of the transition weights: chunk c covers hidden units
// [32c, 32c+32).  Its W1 part is [NK1 fragments over the (D+E) inputs][b1
// tail: 32 floats in accumulator order]; its W2 part is [D/32 blocks x 32/KF
// fragments].  The two parts are stored in two arrays and staged separately
// (the rollout kernel overlaps one chunk's second product with the next
// chunk's first product).
template <class Gm>
struct TransChunk {
  static constexpr int nk1(int D, int E) { return (D + E) / Gm::KF; }
  static constexpr int nk2(int D) { return (D / 32) * (32 / Gm::KF); }
  static constexpr int w1_bytes(int D, int E) { return nk1(D, E) / Gm::G * 1024 + 128; }
  static constexpr int w2_bytes(int D) { return nk2(D) / Gm::G * 1024; }
};

// Chunk geometry of the cost-model first layer: one chunk = 32 hidden units,
// [Wc1 fragments over (D+E+HW) inputs][tail: bc1 then wc2, 32 floats each, in
// accumulator order].
template <class Gm>
struct CostChunk {
  static constexpr int nfrags(int D, int E, int HW) { return (D + E + HW) / Gm::KF; }
  static constexpr int ngroups(int D, int E, int HW) { return nfrags(D, E, HW) / Gm::G; }
  static constexpr int bytes(int D, int E, int HW) { return ngroups(D, E, HW) * 1024 + 256; }
};

// Transposed transition weights for the backward pass of the rollout loss.
//   W2^T chunk c: A fragments of dG^T[chunk] = W2^T[chunk] . Delta^T, rows =
//     the chunk's 32 hidden units, contraction over the latent in the same
//     slot order as the z part of X (x_feature), so Delta in accumulator
//     layout feeds it like z feeds the first product: nk2t = D / KF
//     fragments.
//   W1^T chunk c: for every 32-row output block of the (d + e) inputs
//     (latent blocks first, then embedding blocks), fragments over the
//     chunk's hidden units in GELU-operand order (g_feature), so dA^T feeds
//     it like G feeds the second product: ((D + E) / 32) x (32 / KF)
//     fragments.  Output row i of block b is input feature 32b + i.
template <class Gm>
struct TransT {
  static constexpr int nk2t(int D) { return D / Gm::KF; }
  static constexpr int w2t_bytes(int D) { return nk2t(D) / Gm::G * 1024; }
  static constexpr int nk1t(int D, int E) { return ((D + E) / 32) * (32 / Gm::KF); }
  static constexpr int w1t_bytes(int D, int E) { return nk1t(D, E) / Gm::G * 1024; }
};

// Hyperplane-normal map Wh [d][e] of the paper-form transition, packed as
// A-operand fragments of the product V^T = Wh . E^T: block b (rows
// [32b, 32b+32) of Wh, i.e. features of the latent in accumulator layout)
// holds E/KF fragments over the embedding in natural order, so the B operand
// is the step's embedding fragment set and V lands in the latent's layout.
template <class Gm>
struct HyperGeom {
  static constexpr int groups_per_block(int E) { return E / Gm::KF / Gm::G; }
  static constexpr int bytes(int D, int E) { return (D / 32) * groups_per_block(E) * 1024; }
};
// Transposed normal map for the paper-form loss backward: de += Wh^T . dv,
// with A fragments per 32-row block of the embedding and contraction over the
// latent in the z operand's slot order (x_feature), so dv in accumulator
// layout is the B operand: (E / 32) x (D / KF) fragments.
template <class Gm>
struct HyperT {
  static constexpr int groups_per_block(int D) { return D / Gm::KF / Gm::G; }
  static constexpr int bytes(int D, int E) { return (E / 32) * groups_per_block(D) * 1024; }
};
// The rollout kernel keeps Wh in LDS when the double-buffered chunks leave
// room for it (and for the embedding table), otherwise streams it from L2.
constexpr int WH_LDS_LIMIT = 112 * 1024;
constexpr bool wh_in_lds(int w1_chunk_bytes, int w2_chunk_bytes, int wh_bytes) {
  return 2 * (w1_chunk_bytes + w2_chunk_bytes) + wh_bytes <= WH_LDS_LIMIT;
}

// --------------------------------------------------------------------------
// Narrow tiles (bf16, 16 candidates): v_mfma_f32_16x16x32_bf16.  Lane L of
// the accumulator holds column L%16 and rows 4(L/16) + r, r < 4; operand
// lane L holds row (A) or column (B) L%16 and 8 contraction slots of lane
// group L/16.  As with the 32-wide products, the contraction order is free:
//  * a z operand fragment kf (32 features) is made of the accumulators of
//    latent blocks 2kf and 2kf+1 (16 features each): slot j of group g is
//    feature 32kf + 16(j/4) + 4g + j%4, so z never leaves its lane;
//  * the GELU outputs of a 32-unit hidden chunk (two 16-row output blocks)
//    form one operand fragment of the second product in the same order;
//  * embedding fragments use the natural order 32q + 8g + j.
// Packed blob (pack_transition_narrow in wm_api.hip), 1 KiB groups of A
// operands, gpk groups per operand fragment (bf16: 1, one 16x16x32 product;
// fp32: 2, four 16x16x4 products each, slots 4hh .. 4hh + 3 in half hh):
//   W1: chunk c, k-fragment kf, row block rb (16 hidden units 32c + 16rb..):
//       group ((c * NK + kf) * 2 + rb) * gpk + hh, NK = (D + E) / 32;
//   W2: chunk c, latent block b (16 rows): group (c * (D / 16) + b) * gpk + hh,
//       after W1;
//   then b1 (H floats) and b2 (D floats), natural order;
//   paper form: then Wh, latent block b (16 rows), embedding fragment q:
//       group (b * (E / 32) + q) * gpk + hh, slot j = embedding feature 32q + 8g + j.
// --------------------------------------------------------------------------
__host__ __device__ constexpr inline int narrow_x_feature(int D, int kf, int g, int j) {
  return kf < D / 32 ? 32 * kf + 16 * (j >> 2) + 4 * g + (j & 3) : D + 32 * (kf - D / 32) + 8 * g + j;
}
__host__ __device__ constexpr inline int narrow_g_feature(int g, int j) {
  return 16 * (j >> 2) + 4 * g + (j & 3);
}
struct Narrow {
  static constexpr size_t w1_groups(int D, int E, int H, int gpk) { return (size_t)(H / 32) * ((D + E) / 32) * 2 * gpk; }
  static constexpr size_t w2_groups(int D, int H, int gpk) { return (size_t)(H / 32) * (D / 16) * gpk; }
  static constexpr size_t bytes(int D, int E, int H, int gpk) {
    return (w1_groups(D, E, H, gpk) + w2_groups(D, H, gpk)) * 1024 + (size_t)(H + D) * 4;
  }
  static constexpr size_t wh_bytes(int D, int E, int gpk) { return (size_t)(D / 16) * (E / 32) * gpk * 1024; }
  // Transposed blob (rollout-loss backward), same operand orders:
  //   W2^T: chunk c, latent k-fragment kf (z-operand order), row block rb (16
  //         hidden units 32c + 16rb..): group ((c * D/32 + kf) * 2 + rb) * gpk + hh;
  //   W1^T: chunk c, output block ob of the D + E inputs (rows 16ob..), over
  //         the chunk's 32 hidden units in GELU-operand order:
  //         group W2T + (c * (D+E)/16 + ob) * gpk + hh.
  static constexpr size_t w2t_groups(int D, int H, int gpk) { return (size_t)(H / 32) * (D / 32) * 2 * gpk; }
  static constexpr size_t w1t_groups(int D, int E, int H, int gpk) { return (size_t)(H / 32) * ((D + E) / 16) * gpk; }
  static constexpr size_t t_bytes(int D, int E, int H, int gpk) {
    return (w2t_groups(D, H, gpk) + w1t_groups(D, E, H, gpk)) * 1024;
  }
  // paper form: then Wh^T, embedding block eb (16 rows), latent fragment kf
  // (z-operand order): group (eb * D/32 + kf) * gpk + hh after W1^T.
  static constexpr size_t wht_bytes(int D, int E, int gpk) { return (size_t)(E / 16) * (D / 32) * gpk * 1024; }
  // Cost-model blob (scores fused into the narrow rollout): Wc1 chunk cc
  // (32 cost-hidden units), k-fragment kf over [z_T; phi; h] (z-operand
  // order, then natural), row block rb: group ((cc * NKC + kf) * 2 + rb) *
  // gpk + hh, NKC = (D + E + HW) / 32; then bc1 and wc2 (C floats each).
  static constexpr size_t c_bytes(int D, int E, int HW, int C, int gpk) {
    return (size_t)(C / 32) * ((D + E + HW) / 32) * 2 * gpk * 1024 + (size_t)C * 8;
  }
};

// Action parameters per step are padded to PMAX in the embedding table
// (zero weights), so the kernels loop over a fixed count.
constexpr int PMAX = 8;

// Row stride (floats) of the type-embedding rows in the rollout table: four
// floats of padding put rows of different action types in different LDS
// banks (lanes of a wavefront read rows of different types at once).
__host__ __device__ constexpr inline int temb_stride(int E) { return E + 4; }

// Bucketing: one workgroup sorts batches of up to BUCKET_SINGLE_MAX
// candidates; larger batches use three passes over chunks of candidates
// (per-chunk length histograms in the workspace, one scan, a scatter).
constexpr int BUCKET_SINGLE_MAX = 8192;
constexpr int BUCKET_CHUNK = 4096;
// Chunks of a multi-workgroup bucketing (0: the single-workgroup kernel);
// at most 256 chunks, so the scan stays small for any batch.
inline int bucket_chunk(int B) {
  const int c = (B + 255) / 256;
  return c > BUCKET_CHUNK ? c : BUCKET_CHUNK;
}
inline int bucket_groups(int B) {
  return B <= BUCKET_SINGLE_MAX ? 0 : (B + bucket_chunk(B) - 1) / bucket_chunk(B);
}

// Device error bits (workspace error word).
enum : int { ERRBIT_LEN = 1, ERRBIT_TYPE = 2, ERRBIT_PARAM = 4, ERRBIT_TOKEN = 8 };

struct SegTable {
  int32_t n;                              // S
  int32_t off[WM_MAX_SEGMENTS + 1];
};

// Device-resident model (one allocation, carved up).
struct DevModel {
  wm_dims dims;
  int prec;                 // wm_precision
  uint8_t* base;            // the allocation
  const uint8_t* trans_w1;  // H/32 transition chunks, W1 part
  const uint8_t* trans_w2;  // H/32 transition chunks, W2 part
  const uint8_t* cost;      // C/32 cost chunks
  const uint8_t* trans_wh;  // Wh fragments (WM_NORM_L2 only)
  const uint8_t* trans_w2t; // H/32 chunks of W2^T (rollout-loss backward)
  const uint8_t* trans_w1t; // H/32 chunks of W1^T (rollout-loss backward)
  const uint8_t* trans_wht; // Wh^T fragments (paper-form rollout-loss backward)
  const uint8_t* trans_n;   // narrow-tile transition blob (d and e multiples of 32), or null
  const uint8_t* trans_nt;  // its transposed blob (rollout-loss backward), or null
  const uint8_t* cost_n;    // narrow cost-model blob (hw_dim a multiple of 32), or null
  const float* roll_tab;    // type_emb [K][E + 4] (padded rows), param_w^T [PMAX][E] (zero rows past P), param_b [E], b2 (acc order) [D]
  const float* emb_nat;     // the first three parts of roll_tab
  const float* enc_w1t;     // We1^T [F][Fh] (bf16-rounded values in bf16 mode)
  const float* enc_b1;      // [Fh]
  const float* enc_w2t;     // We2^T [Fh][D]
  const float* enc_b2;      // [D]
  float bc2;
  int w1_chunk_bytes, w2_chunk_bytes, cost_chunk_bytes, roll_tab_bytes;
  int wh_bytes;             // 0 unless WM_NORM_L2
};

// Tree-ensemble ranker: complete breadth-first trees of depth `depth`;
// node (feature, float bits of threshold) pairs [n_trees][2^depth - 1],
// leaves [n_trees][2^depth].  Feature indices are checked at creation.
struct DevForest {
  int32_t n_trees, depth, n_features;
  float base;
  uint8_t* alloc;
  const void* nodes;        // int2 (feature, threshold bits) pairs
  const float* leaves;
};
constexpr int FOREST_MAX_DEPTH = 12;
constexpr int TREE_MAX_FEATURES = 4096;

// Width of the structured action-feature vector: kind counts, length,
// per-slot mean and max of log2(param).
__host__ __device__ constexpr inline int phi_struct_dim(int K, int P) { return K + 1 + 2 * P; }

inline int train_splits(long long rows_bound) {
  const long long s = (rows_bound + 511) / 512;     // small batches: more splits, shorter row loops
  return (int)(s < 1 ? 1 : (s > 32 ? 32 : s));
}
// Row blocks of the embedding-gradient kernel (about 256 rows each).
inline int emb_blocks(long long rows_bound) {
  const long long s = (rows_bound + 255) / 256;
  return (int)(s < 1 ? 1 : (s > 512 ? 512 : s));
}

}  // namespace wm
