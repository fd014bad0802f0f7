// Host-side data preparation (wm_pack.cpp): weight packing into the
// matrix-fragment orders of the kernels, workspace layouts, segment checks.
// Plain C++ (no HIP types), so it also builds alone for the CPU tests.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "wm_layout.h"

namespace wm {

// fp32 -> bf16 bits, round to nearest even (NaN stays NaN); its float value
uint16_t f32_to_bf16(float f);
float bf16_value(float f);

// Transition chunks (TransChunk): for hidden chunk c, a W1 part [W1
// fragments over [z; e]][b1 tail] and a W2 part [W2 fragments], in two arrays.
template <class Gm>
void pack_transition(const wm_dims& dm, const wm_weights& w, std::vector<uint8_t>& w1blk,
                     std::vector<uint8_t>& w2blk);
// Narrow-tile blobs (Narrow): transition (plus Wh in the paper form), cost
// model, and the transposed transition of the rollout-loss backward.
std::vector<uint8_t> pack_transition_narrow(const wm_dims& dm, const wm_weights& w);
std::vector<uint8_t> pack_cost_narrow(const wm_dims& dm, const wm_weights& w);
std::vector<uint8_t> pack_transposed_narrow(const wm_dims& dm, const wm_weights& w);
// Transposed transition chunks (TransT), transposed normal map (HyperT),
// cost chunks (CostChunk), hyperplane-normal map (HyperGeom).
template <class Gm>
void pack_transposed(const wm_dims& dm, const wm_weights& w, std::vector<uint8_t>& w2t,
                     std::vector<uint8_t>& w1t);
template <class Gm>
std::vector<uint8_t> pack_hyper_t(const wm_dims& dm, const wm_weights& w);
template <class Gm>
std::vector<uint8_t> pack_cost(const wm_dims& dm, const wm_weights& w);
template <class Gm>
std::vector<uint8_t> pack_hyper(const wm_dims& dm, const wm_weights& w);

size_t align256(size_t x);

// Evaluator workspace: byte offsets of its parts (each 256-byte aligned).
struct WsLayout {
  size_t err, perm, hist, z0, zT, phi, phi_s, scores, total;
};
WsLayout ws_layout(const DevModel& m, int B, int T_max, int S, int n_hw);

// Rollout-loss workspace.
struct LossLayout {
  size_t err, perm, hist, off, row_src, X, A, G, P, SD, DE, V, SC, DV, lrow, pw1, pw2, pb1, pb2,
      pemb, pwh, total;
  int splits, emb_blocks;
};
LossLayout loss_layout(const DevModel& m, int B, int T_max);

// Checks a host segment table (0 = off[0] <= ... <= off[S] = B, 1 <= S <=
// WM_MAX_SEGMENTS) and fills the kernel-argument copy and the smallest
// segment size; on failure returns WM_ERR_INVALID_ARGUMENT with the reason
// in *msg.
wm_status check_segments(const int32_t* seg_off, int32_t S, int32_t B, SegTable* tab,
                         int32_t* min_seg, std::string* msg);

}  // namespace wm
