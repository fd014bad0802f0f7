// Host-side data preparation of the batched latent-rollout evaluator:
// packing of the weights into matrix-fragment order (the layouts are
// described in wm_layout.h), workspace layouts and the segment-table check.
// Plain C++: built into the library and, on its own, into the CPU tests
// (with the address and undefined-behaviour sanitizers).
#include "wm_pack.h"

#include <algorithm>
#include <cstring>
#include <string>
#include <vector>

namespace wm {

// ---- bf16 (round to nearest even) ----------------------------------------
uint16_t f32_to_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
  const uint32_t r = u + 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(r >> 16);
}
float bf16_value(float f) {
  const uint32_t u = (uint32_t)f32_to_bf16(f) << 16;
  float o;
  std::memcpy(&o, &u, 4);
  return o;
}

// Store one weight element of a packed fragment block.
template <class Gm>
static void put(std::vector<uint8_t>& blk, size_t base, int F, int lane, int j, float v) {
  const size_t off = base + (size_t)frag_offset<Gm>(F, lane, j);
  if (Gm::ES == 2) {
    const uint16_t b = f32_to_bf16(v);
    std::memcpy(&blk[off], &b, 2);
  } else {
    std::memcpy(&blk[off], &v, 4);
  }
}

static void put_f32(std::vector<uint8_t>& blk, size_t off, float v) { std::memcpy(&blk[off], &v, 4); }

// Transition chunks: for hidden chunk c, a W1 part [W1 fragments][b1 tail]
// and a W2 part [W2 fragments], in two arrays.
template <class Gm>
void pack_transition(const wm_dims& dm, const wm_weights& w, std::vector<uint8_t>& w1blk,
                     std::vector<uint8_t>& w2blk) {
  const int D = dm.d, E = dm.embed_dim, H = dm.trans_hidden, IN = D + E;
  const int B1 = TransChunk<Gm>::w1_bytes(D, E), B2 = TransChunk<Gm>::w2_bytes(D);
  const int NK1 = TransChunk<Gm>::nk1(D, E), NF2 = 32 / Gm::KF;
  w1blk.assign((size_t)(H / 32) * B1, 0);
  w2blk.assign((size_t)(H / 32) * B2, 0);
  for (int c = 0; c < H / 32; ++c) {
    const size_t base1 = (size_t)c * B1, base2 = (size_t)c * B2;
    for (int kf = 0; kf < NK1; ++kf)
      for (int L = 0; L < 64; ++L)
        for (int j = 0; j < Gm::SL; ++j) {
          const int m = L & 31, h = L >> 5;
          const int feat = x_feature<Gm>(D, kf, h, j);
          put<Gm>(w1blk, base1, kf, L, j, w.w1[(size_t)(32 * c + m) * IN + feat]);
        }
    for (int h = 0; h < 2; ++h)
      for (int r = 0; r < 16; ++r)
        put_f32(w1blk, base1 + (size_t)(B1 - 128) + (size_t)(h * 16 + r) * 4, w.b1[32 * c + acc_row(h, r)]);
    for (int db = 0; db < D / 32; ++db)
      for (int f = 0; f < NF2; ++f)
        for (int L = 0; L < 64; ++L)
          for (int j = 0; j < Gm::SL; ++j) {
            const int m = L & 31, h = L >> 5;
            const int hid = 32 * c + g_feature<Gm>(f, h, j);
            put<Gm>(w2blk, base2, db * NF2 + f, L, j, w.w2[(size_t)(32 * db + m) * H + hid]);
          }
  }
}

// Narrow-tile transition blob (layout at Narrow in wm_internal.h): bf16
// (gpk = 1, 8 bf16 per lane and group) or fp32 (gpk = 2, 4 floats per lane
// and group, slots 4hh .. 4hh + 3).
std::vector<uint8_t> pack_transition_narrow(const wm_dims& dm, const wm_weights& w) {
  const int D = dm.d, E = dm.embed_dim, H = dm.trans_hidden, IN = D + E, NK = IN / 32;
  const bool bf = dm.precision == WM_BF16, l2 = dm.norm == WM_NORM_L2;
  const int gpk = bf ? 1 : 2, per = 8 / gpk;                 // slots per lane and group
  std::vector<uint8_t> blk(Narrow::bytes(D, E, H, gpk) + (l2 ? Narrow::wh_bytes(D, E, gpk) : 0), 0);
  // slot j of the operand fragment starting at group frag_group0 (groups
  // counted from byte `base`): group half j / per, position j % per
  auto put_at = [&](size_t base, size_t frag_group0, int lane, int j, float v) {
    const size_t off = base + (frag_group0 + (size_t)(j / per)) * 1024 + (size_t)lane * 16;
    if (bf) {
      const uint16_t b = f32_to_bf16(v);
      std::memcpy(&blk[off + (size_t)(j % per) * 2], &b, 2);
    } else {
      std::memcpy(&blk[off + (size_t)(j % per) * 4], &v, 4);
    }
  };
  auto put = [&](size_t frag_group0, int lane, int j, float v) { put_at(0, frag_group0, lane, j, v); };
  for (int c = 0; c < H / 32; ++c)
    for (int kf = 0; kf < NK; ++kf)
      for (int rb = 0; rb < 2; ++rb)
        for (int L = 0; L < 64; ++L)
          for (int j = 0; j < 8; ++j) {
            const int hid = 32 * c + 16 * rb + (L & 15);
            put((((size_t)c * NK + kf) * 2 + rb) * gpk, L, j,
                w.w1[(size_t)hid * IN + narrow_x_feature(D, kf, L >> 4, j)]);
          }
  const size_t g2 = Narrow::w1_groups(D, E, H, gpk);
  for (int c = 0; c < H / 32; ++c)
    for (int b = 0; b < D / 16; ++b)
      for (int L = 0; L < 64; ++L)
        for (int j = 0; j < 8; ++j) {
          const int row = 16 * b + (L & 15), hid = 32 * c + narrow_g_feature(L >> 4, j);
          put(g2 + ((size_t)c * (D / 16) + b) * gpk, L, j, w.w2[(size_t)row * H + hid]);
        }
  const size_t tail = (g2 + Narrow::w2_groups(D, H, gpk)) * 1024;
  std::memcpy(&blk[tail], w.b1, (size_t)H * 4);
  std::memcpy(&blk[tail + (size_t)H * 4], w.b2, (size_t)D * 4);
  if (l2) {
    const size_t base = Narrow::bytes(D, E, H, gpk);          // 16-byte aligned
    for (int b = 0; b < D / 16; ++b)
      for (int q = 0; q < E / 32; ++q)
        for (int L = 0; L < 64; ++L)
          for (int j = 0; j < 8; ++j)
            put_at(base, ((size_t)b * (E / 32) + q) * gpk, L, j,
                w.wh[(size_t)(16 * b + (L & 15)) * E + 32 * q + 8 * (L >> 4) + j]);
  }
  return blk;
}

// Narrow cost-model blob (Narrow::c_bytes): Wc1 with the operand orders of
// the narrow rollout ([z_T] as z fragments, [phi; h] natural), bc1, wc2.
std::vector<uint8_t> pack_cost_narrow(const wm_dims& dm, const wm_weights& w) {
  const int D = dm.d, E = dm.embed_dim, HW = dm.hw_dim, C = dm.cost_hidden, IN = D + E + HW;
  const int NKC = IN / 32;
  const bool bf = dm.precision == WM_BF16;
  const int gpk = bf ? 1 : 2, per = 8 / gpk;
  std::vector<uint8_t> blk(Narrow::c_bytes(D, E, HW, C, gpk), 0);
  auto put = [&](size_t frag_group0, int lane, int j, float v) {
    const size_t off = (frag_group0 + (size_t)(j / per)) * 1024 + (size_t)lane * 16;
    if (bf) {
      const uint16_t b = f32_to_bf16(v);
      std::memcpy(&blk[off + (size_t)(j % per) * 2], &b, 2);
    } else {
      std::memcpy(&blk[off + (size_t)(j % per) * 4], &v, 4);
    }
  };
  for (int cc = 0; cc < C / 32; ++cc)
    for (int kf = 0; kf < NKC; ++kf)
      for (int rb = 0; rb < 2; ++rb)
        for (int L = 0; L < 64; ++L)
          for (int j = 0; j < 8; ++j) {
            const int row = 32 * cc + 16 * rb + (L & 15);
            put((((size_t)cc * NKC + kf) * 2 + rb) * gpk, L, j,
                w.wc1[(size_t)row * IN + narrow_x_feature(D, kf, L >> 4, j)]);
          }
  const size_t tail = (size_t)(C / 32) * NKC * 2 * gpk * 1024;
  std::memcpy(&blk[tail], w.bc1, (size_t)C * 4);
  std::memcpy(&blk[tail + (size_t)C * 4], w.wc2, (size_t)C * 4);
  return blk;
}

// Transposed narrow-tile blob for the rollout-loss backward (Narrow::t_bytes).
std::vector<uint8_t> pack_transposed_narrow(const wm_dims& dm, const wm_weights& w) {
  const int D = dm.d, E = dm.embed_dim, H = dm.trans_hidden, IN = D + E;
  const bool bf = dm.precision == WM_BF16, l2 = dm.norm == WM_NORM_L2;
  const int gpk = bf ? 1 : 2, per = 8 / gpk;
  std::vector<uint8_t> blk(Narrow::t_bytes(D, E, H, gpk) + (l2 ? Narrow::wht_bytes(D, E, gpk) : 0), 0);
  auto put = [&](size_t frag_group0, int lane, int j, float v) {
    const size_t off = (frag_group0 + (size_t)(j / per)) * 1024 + (size_t)lane * 16;
    if (bf) {
      const uint16_t b = f32_to_bf16(v);
      std::memcpy(&blk[off + (size_t)(j % per) * 2], &b, 2);
    } else {
      std::memcpy(&blk[off + (size_t)(j % per) * 4], &v, 4);
    }
  };
  for (int c = 0; c < H / 32; ++c)
    for (int kf = 0; kf < D / 32; ++kf)
      for (int rb = 0; rb < 2; ++rb)
        for (int L = 0; L < 64; ++L)
          for (int j = 0; j < 8; ++j) {
            const int hid = 32 * c + 16 * rb + (L & 15);
            const int lat = narrow_x_feature(D, kf, L >> 4, j);
            put((((size_t)c * (D / 32) + kf) * 2 + rb) * gpk, L, j, w.w2[(size_t)lat * H + hid]);
          }
  const size_t g1 = Narrow::w2t_groups(D, H, gpk);
  for (int c = 0; c < H / 32; ++c)
    for (int ob = 0; ob < IN / 16; ++ob)
      for (int L = 0; L < 64; ++L)
        for (int j = 0; j < 8; ++j) {
          const int feat = 16 * ob + (L & 15), hid = 32 * c + narrow_g_feature(L >> 4, j);
          put(g1 + ((size_t)c * (IN / 16) + ob) * gpk, L, j, w.w1[(size_t)hid * IN + feat]);
        }
  if (l2) {
    const size_t gh = g1 + Narrow::w1t_groups(D, E, H, gpk);
    for (int eb = 0; eb < E / 16; ++eb)
      for (int kf = 0; kf < D / 32; ++kf)
        for (int L = 0; L < 64; ++L)
          for (int j = 0; j < 8; ++j) {
            const int emb = 16 * eb + (L & 15), lat = narrow_x_feature(D, kf, L >> 4, j);
            put(gh + ((size_t)eb * (D / 32) + kf) * gpk, L, j, w.wh[(size_t)lat * E + emb]);
          }
  }
  return blk;
}

// Transposed transition chunks for the rollout-loss backward (see TransT).
template <class Gm>
void pack_transposed(const wm_dims& dm, const wm_weights& w, std::vector<uint8_t>& w2t,
                     std::vector<uint8_t>& w1t) {
  const int D = dm.d, E = dm.embed_dim, H = dm.trans_hidden, IN = D + E;
  const int B2 = TransT<Gm>::w2t_bytes(D), B1 = TransT<Gm>::w1t_bytes(D, E);
  const int NZ = TransT<Gm>::nk2t(D), NF2 = 32 / Gm::KF;
  w2t.assign((size_t)(H / 32) * B2, 0);
  w1t.assign((size_t)(H / 32) * B1, 0);
  for (int c = 0; c < H / 32; ++c) {
    for (int kf = 0; kf < NZ; ++kf)
      for (int L = 0; L < 64; ++L)
        for (int j = 0; j < Gm::SL; ++j) {
          const int m = L & 31, h = L >> 5;
          const int feat = x_feature<Gm>(D, kf, h, j);
          put<Gm>(w2t, (size_t)c * B2, kf, L, j, w.w2[(size_t)feat * H + 32 * c + m]);
        }
    for (int ob = 0; ob < IN / 32; ++ob)
      for (int f = 0; f < NF2; ++f)
        for (int L = 0; L < 64; ++L)
          for (int j = 0; j < Gm::SL; ++j) {
            const int m = L & 31, h = L >> 5;
            const int hid = 32 * c + g_feature<Gm>(f, h, j);
            put<Gm>(w1t, (size_t)c * B1, ob * NF2 + f, L, j, w.w1[(size_t)hid * IN + 32 * ob + m]);
          }
  }
}

// Transposed normal map: embedding block ob, fragment kf over the latent (z
// operand order) -> rows 32 ob + L%32 of Wh^T, i.e. Wh[feature][32 ob + m].
template <class Gm>
std::vector<uint8_t> pack_hyper_t(const wm_dims& dm, const wm_weights& w) {
  const int D = dm.d, E = dm.embed_dim, NZ = D / Gm::KF;
  std::vector<uint8_t> blk((size_t)HyperT<Gm>::bytes(D, E), 0);
  for (int ob = 0; ob < E / 32; ++ob)
    for (int kf = 0; kf < NZ; ++kf)
      for (int L = 0; L < 64; ++L)
        for (int j = 0; j < Gm::SL; ++j) {
          const int m = L & 31, h = L >> 5;
          const int feat = x_feature<Gm>(D, kf, h, j);
          put<Gm>(blk, 0, ob * NZ + kf, L, j, w.wh[(size_t)feat * E + 32 * ob + m]);
        }
  return blk;
}

// Cost chunks: for cost hidden chunk c, [Wc1 fragments][bc1 tail][wc2 tail].
template <class Gm>
std::vector<uint8_t> pack_cost(const wm_dims& dm, const wm_weights& w) {
  const int D = dm.d, E = dm.embed_dim, HW = dm.hw_dim, C = dm.cost_hidden, IN = D + E + HW;
  const int CB = CostChunk<Gm>::bytes(D, E, HW), NF = CostChunk<Gm>::nfrags(D, E, HW);
  const int NG = CostChunk<Gm>::ngroups(D, E, HW);
  std::vector<uint8_t> blk((size_t)(C / 32) * CB, 0);
  for (int c = 0; c < C / 32; ++c) {
    const size_t base = (size_t)c * CB;
    for (int kf = 0; kf < NF; ++kf)
      for (int L = 0; L < 64; ++L)
        for (int j = 0; j < Gm::SL; ++j) {
          const int m = L & 31, h = L >> 5;
          put<Gm>(blk, base, kf, L, j, w.wc1[(size_t)(32 * c + m) * IN + nat_feature<Gm>(kf, h, j)]);
        }
    for (int h = 0; h < 2; ++h)
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * c + acc_row(h, r);
        put_f32(blk, base + (size_t)NG * 1024 + (size_t)(h * 16 + r) * 4, w.bc1[row]);
        put_f32(blk, base + (size_t)NG * 1024 + 128 + (size_t)(h * 16 + r) * 4, w.wc2[row]);
      }
  }
  return blk;
}

// Hyperplane-normal map: block b, fragment q over the embedding (natural
// order) -> rows 32b + L%32 of Wh.
template <class Gm>
std::vector<uint8_t> pack_hyper(const wm_dims& dm, const wm_weights& w) {
  const int D = dm.d, E = dm.embed_dim, NE = E / Gm::KF;
  std::vector<uint8_t> blk((size_t)HyperGeom<Gm>::bytes(D, E), 0);
  for (int b = 0; b < D / 32; ++b)
    for (int q = 0; q < NE; ++q)
      for (int L = 0; L < 64; ++L)
        for (int j = 0; j < Gm::SL; ++j) {
          const int m = L & 31, h = L >> 5;
          put<Gm>(blk, 0, b * NE + q, L, j, w.wh[(size_t)(32 * b + m) * E + nat_feature<Gm>(q, h, j)]);
        }
  return blk;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }


WsLayout ws_layout(const DevModel& m, int B, int T_max, int S, int n_hw) {
  WsLayout L;
  size_t o = 0;
  L.err = o; o += 256;
  L.perm = o; o = align256(o + (size_t)B * 2 * sizeof(int32_t));   // (candidate, subgraph) pairs
  L.hist = o; o = align256(o + (size_t)bucket_groups(B) * (size_t)(T_max + 1) * 4);
  L.z0 = o; o = align256(o + (size_t)S * m.dims.d * 4);
  L.zT = o; o = align256(o + (size_t)B * m.dims.d * 4);
  L.phi = o; o = align256(o + (size_t)B * m.dims.embed_dim * 4);
  L.phi_s = o; o = align256(o + (size_t)B * phi_struct_dim(m.dims.n_kinds, m.dims.n_params) * 4);
  L.scores = o; o = align256(o + (size_t)n_hw * B * 4);
  L.total = o;
  return L;
}

// Rollout-loss workspace: bucketing, step activations (rows i * T_max + t),
// per-candidate step losses, partial gradient sums.

LossLayout loss_layout(const DevModel& m, int B, int T_max) {
  const wm_dims& dm = m.dims;
  const size_t D = dm.d, E = dm.embed_dim, H = dm.trans_hidden;
  const size_t K = dm.n_kinds, P = dm.n_params;
  const long long rows = (long long)B * T_max;
  const size_t R = (size_t)rows;
  LossLayout L;
  L.splits = train_splits(rows);
  L.emb_blocks = emb_blocks(rows);
  const size_t S = (size_t)L.splits;
  size_t o = 0;
  L.err = o; o += 256;
  L.perm = o; o = align256(o + (size_t)B * 2 * sizeof(int32_t));   // (candidate, subgraph) pairs
  L.hist = o; o = align256(o + (size_t)bucket_groups(B) * (size_t)(T_max + 1) * 4);
  L.off = o; o = align256(o + ((size_t)B + 1) * 4);
  L.row_src = o; o = align256(o + R * 4);
  L.X = o; o = align256(o + R * (D + E) * 4);
  L.A = o; o = align256(o + R * H * 4);
  L.G = o; o = align256(o + R * H * 4);
  L.P = o; o = align256(o + R * D * 4);
  L.SD = o; o = align256(o + R * D * 4);
  L.DE = o; o = align256(o + R * E * 4);
  const bool l2 = dm.norm == WM_NORM_L2;
  L.V = o; o = align256(o + (l2 ? R * D * 4 : 0));
  L.SC = o; o = align256(o + (l2 ? R * 16 : 0));
  L.DV = o; o = align256(o + (l2 ? R * D * 4 : 0));
  L.lrow = o; o = align256(o + R * 4);
  L.pw1 = o; o = align256(o + S * H * (D + E) * 4);
  L.pw2 = o; o = align256(o + S * D * H * 4);
  L.pb1 = o; o = align256(o + S * H * 4);
  L.pb2 = o; o = align256(o + S * D * 4);
  L.pemb = o; o = align256(o + (size_t)L.emb_blocks * (K * E + E * P + E) * 4);
  L.pwh = o; o = align256(o + (l2 ? S * D * E * 4 : 0));
  L.total = o;
  return L;
}

// Host checks of a segment table; fills the kernel-argument copy.  On
// failure returns the status and puts the reason in *msg.
wm_status check_segments(const int32_t* seg_off, int32_t S, int32_t B, SegTable* tab,
                         int32_t* min_seg, std::string* msg) {
  auto bad = [&](const std::string& m) {
    *msg = m;
    return WM_ERR_INVALID_ARGUMENT;
  };
  if (!seg_off) return bad("seg_off is NULL");
  if (S < 1 || S > WM_MAX_SEGMENTS) return bad("S must be in [1, " + std::to_string(WM_MAX_SEGMENTS) + "]");
  if (seg_off[0] != 0 || seg_off[S] != B) return bad("seg_off must start at 0 and end at B");
  int32_t mn = B;
  for (int s = 0; s < S; ++s) {
    if (seg_off[s + 1] < seg_off[s]) return bad("seg_off is not non-decreasing");
    mn = std::min(mn, seg_off[s + 1] - seg_off[s]);
  }
  tab->n = S;
  for (int s = 0; s <= S; ++s) tab->off[s] = seg_off[s];
  *min_seg = mn;
  return WM_OK;
}


template void pack_transition<GeomBF16>(const wm_dims&, const wm_weights&, std::vector<uint8_t>&,
                                        std::vector<uint8_t>&);
template void pack_transition<GeomF32>(const wm_dims&, const wm_weights&, std::vector<uint8_t>&,
                                       std::vector<uint8_t>&);
template void pack_transposed<GeomBF16>(const wm_dims&, const wm_weights&, std::vector<uint8_t>&,
                                        std::vector<uint8_t>&);
template void pack_transposed<GeomF32>(const wm_dims&, const wm_weights&, std::vector<uint8_t>&,
                                       std::vector<uint8_t>&);
template std::vector<uint8_t> pack_hyper_t<GeomBF16>(const wm_dims&, const wm_weights&);
template std::vector<uint8_t> pack_hyper_t<GeomF32>(const wm_dims&, const wm_weights&);
template std::vector<uint8_t> pack_cost<GeomBF16>(const wm_dims&, const wm_weights&);
template std::vector<uint8_t> pack_cost<GeomF32>(const wm_dims&, const wm_weights&);
template std::vector<uint8_t> pack_hyper<GeomBF16>(const wm_dims&, const wm_weights&);
template std::vector<uint8_t> pack_hyper<GeomF32>(const wm_dims&, const wm_weights&);

}  // namespace wm
