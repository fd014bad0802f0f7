// CPU check of the host-side data preparation (paper_2606_09312_amd/csrc/
// wm_pack.cpp), built with the address and undefined-behaviour sanitizers by
// tests/test_host_sanitize.py.
//
// Independent of the packing code: the operand conventions of the matrix-core
// products are restated here from the hardware's definition, not taken from
// the library's layout helpers.
//  * v_mfma_f32_32x32x16_bf16: lane L supplies row (A) / column (B) L % 32 and
//    the eight contraction slots 8 (L / 32) .. + 7 of a 16-wide k-block;
//  * v_mfma_f32_32x32x2_f32: lane L supplies row / column L % 32 and the one
//    contraction slot L / 32 of a 2-wide k-block;
//  * the 32x32 result: lane L, register r holds row 8 (r / 4) + 4 (L / 32) +
//    r % 4 and column L % 32.
// The rollout keeps z and the GELU outputs in result layout and feeds them
// back as B operands without moving data between lanes; the packed weights
// must therefore reproduce W . x exactly when multiplied, through the
// operand conventions above, with B operands assembled from result layouts.
// That is what the product checks below compute.  Blobs of the other
// layouts are checked to hold exactly the source values (as a multiset).
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <string>
#include <vector>

#include "wm_pack.h"

using namespace wm;

static int g_fail = 0;
#define CHECK(c, ...)                                  \
  do {                                                 \
    if (!(c)) {                                        \
      if (g_fail < 20) {                               \
        std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
        std::fprintf(stderr, __VA_ARGS__);             \
        std::fprintf(stderr, "\n");                    \
      }                                                \
      ++g_fail;                                        \
    }                                                  \
  } while (0)

// result-layout row of register r in lane half h (32x32 products)
static int res_row(int h, int r) { return 8 * (r / 4) + 4 * h + r % 4; }

static float rne_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u = (u + 0x7fffu + ((u >> 16) & 1u)) & 0xffff0000u;
  float o;
  std::memcpy(&o, &u, 4);
  return o;
}

struct Shape {
  const char* name;
  wm_precision prec;
  int d, e, K, P, H, C, hw;
};

struct Weights {
  std::vector<float> type_emb, param_w, param_b, w1, b1, w2, b2, wc1, bc1, wc2, wh;
  wm_weights view{};
};

static Weights make_weights(const wm_dims& dm, uint32_t seed) {
  std::mt19937 rng(seed);
  std::normal_distribution<float> nd(0.0f, 1.0f);
  auto fill = [&](std::vector<float>& v, size_t n) {
    v.resize(n);
    for (auto& x : v) x = nd(rng);
  };
  Weights W;
  const int D = dm.d, E = dm.embed_dim, H = dm.trans_hidden, C = dm.cost_hidden, HW = dm.hw_dim;
  fill(W.type_emb, (size_t)dm.n_kinds * E);
  fill(W.param_w, (size_t)E * dm.n_params);
  fill(W.param_b, E);
  fill(W.w1, (size_t)H * (D + E));
  fill(W.b1, H);
  fill(W.w2, (size_t)D * H);
  fill(W.b2, D);
  fill(W.wc1, (size_t)C * (D + E + HW));
  fill(W.bc1, C);
  fill(W.wc2, C);
  fill(W.wh, (size_t)D * E);
  W.view.type_emb = W.type_emb.data();
  W.view.param_w = W.param_w.data();
  W.view.param_b = W.param_b.data();
  W.view.w1 = W.w1.data();
  W.view.b1 = W.b1.data();
  W.view.w2 = W.w2.data();
  W.view.b2 = W.b2.data();
  W.view.wc1 = W.wc1.data();
  W.view.bc1 = W.bc1.data();
  W.view.wc2 = W.wc2.data();
  W.view.bc2 = 0.25f;
  W.view.wh = W.wh.data();
  return W;
}

// Operand element (fragment F, lane L, slot j) of a packed block, for
// bf16 (8 slots per lane, one fragment per 1 KiB group) or fp32 (one slot
// per lane, four fragments per group, fragment F % 4 at byte 4 (F % 4)).
static float operand(const std::vector<uint8_t>& blk, size_t base, bool bf, int F, int L, int j) {
  size_t off;
  if (bf) {
    off = base + (size_t)F * 1024 + (size_t)L * 16 + (size_t)j * 2;
    CHECK(off + 2 <= blk.size(), "operand offset %zu beyond %zu", off, blk.size());
    if (off + 2 > blk.size()) return 0.0f;
    uint16_t b;
    std::memcpy(&b, &blk[off], 2);
    const uint32_t u = (uint32_t)b << 16;
    float o;
    std::memcpy(&o, &u, 4);
    return o;
  }
  off = base + (size_t)(F / 4) * 1024 + (size_t)L * 16 + (size_t)(F % 4) * 4;
  CHECK(off + 4 <= blk.size(), "operand offset %zu beyond %zu", off, blk.size());
  if (off + 4 > blk.size()) return 0.0f;
  float o;
  std::memcpy(&o, &blk[off], 4);
  return o;
}

// One 32x32 product over nk fragments: out[m][n] = sum over fragments,
// halves and slots of A(F, lane (h, m), j) * B(F, lane (h, n), j).
template <class FA, class FB>
static void product(int nk, int slots, FA a, FB b, double (&out)[32][32]) {
  for (int m = 0; m < 32; ++m)
    for (int n = 0; n < 32; ++n) out[m][n] = 0.0;
  for (int F = 0; F < nk; ++F)
    for (int h = 0; h < 2; ++h)
      for (int j = 0; j < slots; ++j) {
        double bv[32];
        for (int n = 0; n < 32; ++n) bv[n] = b(F, h, n, j);
        for (int m = 0; m < 32; ++m) {
          const double av = a(F, 32 * h + m, j);
          if (av == 0.0) continue;
          for (int n = 0; n < 32; ++n) out[m][n] += av * bv[n];
        }
      }
}

static bool close(double x, double y, double scale) { return std::fabs(x - y) <= 1e-9 * scale + 1e-12; }

// Transition chunks: the first product over [z; e] and the second over the
// GELU outputs, both against W1 . x and W2 . g computed directly.
static void check_transition(const Shape& sh, const wm_dims& dm, const Weights& W) {
  const bool bf = dm.precision == WM_BF16;
  const int D = dm.d, E = dm.embed_dim, H = dm.trans_hidden, IN = D + E;
  const int KF = bf ? 16 : 2, SL = bf ? 8 : 1;
  std::vector<uint8_t> w1, w2;
  if (bf) pack_transition<GeomBF16>(dm, W.view, w1, w2);
  else pack_transition<GeomF32>(dm, W.view, w1, w2);
  const size_t B1 = (size_t)(IN / KF) * (bf ? 1024 : 256) + 128;   // fragments + b1 tail
  const size_t B2 = (size_t)(D / 32) * (32 / KF) * (bf ? 1024 : 256);
  CHECK(w1.size() == (size_t)(H / 32) * B1, "%s: W1 part size %zu", sh.name, w1.size());
  CHECK(w2.size() == (size_t)(H / 32) * B2, "%s: W2 part size %zu", sh.name, w2.size());
  if (g_fail) return;
  // candidates' inputs, exactly representable in bf16
  std::mt19937 rng(7);
  std::uniform_int_distribution<int> ui(-64, 64);
  std::vector<double> x((size_t)32 * IN), g((size_t)32 * H);
  for (auto& v : x) v = ui(rng) / 32.0;
  for (auto& v : g) v = ui(rng) / 32.0;
  const int chunks[3] = {0, H / 64, H / 32 - 1};
  for (int c : chunks) {
    const size_t base1 = (size_t)c * B1, base2 = (size_t)c * B2;
    // B operand of the first product: z fragments from the result layout of
    // the latent (block kf / (32 / KF), registers (kf % (32 / KF)) * SL + j),
    // embedding fragments in natural order
    const int per_block = 32 / KF, NZ = D / KF;
    auto bop = [&](int F, int h, int n, int j) -> double {
      if (F < NZ) {
        const int b = F / per_block, r = (F % per_block) * SL + j;
        return x[(size_t)n * IN + 32 * b + res_row(h, r)];
      }
      return x[(size_t)n * IN + D + KF * (F - NZ) + SL * h + j];
    };
    auto aop = [&](int F, int L, int j) -> double { return operand(w1, base1, bf, F, L, j); };
    double out[32][32];
    product(IN / KF, SL, aop, bop, out);
    for (int m = 0; m < 32; ++m)
      for (int n = 0; n < 32; ++n) {
        double ref = 0.0, sc = 0.0;
        for (int k = 0; k < IN; ++k) {
          const float wv = W.w1[(size_t)(32 * c + m) * IN + k];
          const double t = (double)(bf ? rne_bf16(wv) : wv) * x[(size_t)n * IN + k];
          ref += t;
          sc += std::fabs(t);
        }
        CHECK(close(out[m][n], ref, sc), "%s: first product chunk %d (%d, %d): %g vs %g", sh.name, c, m, n,
              out[m][n], ref);
      }
    // b1 tail: 32 floats in result order
    for (int h = 0; h < 2; ++h)
      for (int r = 0; r < 16; ++r) {
        float v;
        std::memcpy(&v, &w1[base1 + B1 - 128 + (size_t)(h * 16 + r) * 4], 4);
        CHECK(v == W.b1[32 * c + res_row(h, r)], "%s: b1 tail chunk %d", sh.name, c);
      }
    // second product: latent block db, GELU operand fragments from the
    // result layout of the chunk's first product (registers f * SL + j)
    for (int db = 0; db < D / 32; db += std::max(1, D / 32 - 1)) {
      auto bg = [&](int F, int h, int n, int j) -> double {
        return g[(size_t)n * H + 32 * c + res_row(h, F * SL + j)];
      };
      auto ag = [&](int F, int L, int j) -> double {
        return operand(w2, base2, bf, db * per_block + F, L, j);
      };
      product(per_block, SL, ag, bg, out);
      for (int m = 0; m < 32; ++m)
        for (int n = 0; n < 32; ++n) {
          double ref = 0.0, sc = 0.0;
          for (int k = 0; k < 32; ++k) {
            const float wv = W.w2[(size_t)(32 * db + m) * H + 32 * c + k];
            const double t = (double)(bf ? rne_bf16(wv) : wv) * g[(size_t)n * H + 32 * c + k];
            ref += t;
            sc += std::fabs(t);
          }
          CHECK(close(out[m][n], ref, sc), "%s: second product chunk %d block %d", sh.name, c, db);
        }
    }
  }
}

// Cost chunks: Wc1 over [z_T; phi; h] in natural order, bc1 and wc2 tails.
static void check_cost(const Shape& sh, const wm_dims& dm, const Weights& W) {
  const bool bf = dm.precision == WM_BF16;
  const int D = dm.d, E = dm.embed_dim, HW = dm.hw_dim, C = dm.cost_hidden, IN = D + E + HW;
  const int KF = bf ? 16 : 2, SL = bf ? 8 : 1;
  std::vector<uint8_t> blk = bf ? pack_cost<GeomBF16>(dm, W.view) : pack_cost<GeomF32>(dm, W.view);
  const size_t NG = (size_t)(IN / KF) / (bf ? 1 : 4);
  const size_t CB = NG * 1024 + 256;
  CHECK(blk.size() == (size_t)(C / 32) * CB, "%s: cost blob size %zu", sh.name, blk.size());
  if (g_fail) return;
  std::mt19937 rng(9);
  std::uniform_int_distribution<int> ui(-64, 64);
  std::vector<double> x((size_t)32 * IN);
  for (auto& v : x) v = ui(rng) / 32.0;
  for (int c : {0, C / 32 - 1}) {
    const size_t base = (size_t)c * CB;
    auto bop = [&](int F, int h, int n, int j) -> double { return x[(size_t)n * IN + KF * F + SL * h + j]; };
    auto aop = [&](int F, int L, int j) -> double { return operand(blk, base, bf, F, L, j); };
    double out[32][32];
    product(IN / KF, SL, aop, bop, out);
    for (int m = 0; m < 32; ++m)
      for (int n = 0; n < 32; ++n) {
        double ref = 0.0, sc = 0.0;
        for (int k = 0; k < IN; ++k) {
          const float wv = W.wc1[(size_t)(32 * c + m) * IN + k];
          const double t = (double)(bf ? rne_bf16(wv) : wv) * x[(size_t)n * IN + k];
          ref += t;
          sc += std::fabs(t);
        }
        CHECK(close(out[m][n], ref, sc), "%s: cost product chunk %d", sh.name, c);
      }
    for (int h = 0; h < 2; ++h)
      for (int r = 0; r < 16; ++r) {
        float b, w;
        std::memcpy(&b, &blk[base + NG * 1024 + (size_t)(h * 16 + r) * 4], 4);
        std::memcpy(&w, &blk[base + NG * 1024 + 128 + (size_t)(h * 16 + r) * 4], 4);
        CHECK(b == W.bc1[32 * c + res_row(h, r)] && w == W.wc2[32 * c + res_row(h, r)], "%s: cost tails", sh.name);
      }
  }
}

// Hyperplane-normal map: V^T = Wh . E^T per 32-row latent block, embedding
// operand in natural order.
static void check_hyper(const Shape& sh, const wm_dims& dm, const Weights& W) {
  const bool bf = dm.precision == WM_BF16;
  const int D = dm.d, E = dm.embed_dim, KF = bf ? 16 : 2, SL = bf ? 8 : 1;
  std::vector<uint8_t> blk = bf ? pack_hyper<GeomBF16>(dm, W.view) : pack_hyper<GeomF32>(dm, W.view);
  const int NE = E / KF;
  const size_t per_block = (size_t)NE / (bf ? 1 : 4) * 1024;
  CHECK(blk.size() == (size_t)(D / 32) * per_block, "%s: normal map size %zu", sh.name, blk.size());
  if (g_fail) return;
  std::mt19937 rng(11);
  std::uniform_int_distribution<int> ui(-64, 64);
  std::vector<double> e((size_t)32 * E);
  for (auto& v : e) v = ui(rng) / 32.0;
  for (int b : {0, D / 32 - 1}) {
    auto bop = [&](int F, int h, int n, int j) -> double { return e[(size_t)n * E + KF * F + SL * h + j]; };
    auto aop = [&](int F, int L, int j) -> double { return operand(blk, 0, bf, b * NE + F, L, j); };
    double out[32][32];
    product(NE, SL, aop, bop, out);
    for (int m = 0; m < 32; ++m)
      for (int n = 0; n < 32; ++n) {
        double ref = 0.0, sc = 0.0;
        for (int k = 0; k < E; ++k) {
          const float wv = W.wh[(size_t)(32 * b + m) * E + k];
          const double t = (double)(bf ? rne_bf16(wv) : wv) * e[(size_t)n * E + k];
          ref += t;
          sc += std::fabs(t);
        }
        CHECK(close(out[m][n], ref, sc), "%s: normal-map product block %d", sh.name, b);
      }
  }
}

// The values stored in [off, off + n) of a blob, as sorted bit patterns.
static std::vector<uint32_t> stored(const std::vector<uint8_t>& blk, size_t off, size_t n, bool bf) {
  std::vector<uint32_t> v(n);
  for (size_t i = 0; i < n; ++i) {
    if (bf) {
      uint16_t b;
      std::memcpy(&b, &blk[off + 2 * i], 2);
      v[i] = b;
    } else {
      std::memcpy(&v[i], &blk[off + 4 * i], 4);
    }
  }
  std::sort(v.begin(), v.end());
  return v;
}
static std::vector<uint32_t> source(const std::vector<const std::vector<float>*>& mats, bool bf) {
  std::vector<uint32_t> v;
  for (auto* m : mats)
    for (float f : *m) {
      if (bf) {
        v.push_back(f32_to_bf16(f));
      } else {
        uint32_t u;
        std::memcpy(&u, &f, 4);
        v.push_back(u);
      }
    }
  std::sort(v.begin(), v.end());
  return v;
}

// Narrow-tile and transposed blobs: every weight exactly once, tails exact.
static void check_permutations(const Shape& sh, const wm_dims& dm, const Weights& W) {
  const bool bf = dm.precision == WM_BF16, l2 = dm.norm == WM_NORM_L2;
  const int D = dm.d, E = dm.embed_dim, H = dm.trans_hidden, IN = D + E, ES = bf ? 2 : 4;
  if (D % 32 == 0 && E % 32 == 0) {
    const std::vector<uint8_t> tn = pack_transition_narrow(dm, W.view);
    const size_t nw1 = (size_t)H * IN, nw2 = (size_t)D * H;
    const size_t tail = (nw1 + nw2) * ES;
    CHECK(tn.size() == tail + (size_t)(H + D) * 4 + (l2 ? (size_t)D * E * ES : 0), "%s: narrow blob size", sh.name);
    if (!g_fail) {
      CHECK(stored(tn, 0, nw1, bf) == source({&W.w1}, bf), "%s: narrow W1 values", sh.name);
      CHECK(stored(tn, nw1 * ES, nw2, bf) == source({&W.w2}, bf), "%s: narrow W2 values", sh.name);
      CHECK(std::memcmp(&tn[tail], W.b1.data(), (size_t)H * 4) == 0, "%s: narrow b1", sh.name);
      CHECK(std::memcmp(&tn[tail + (size_t)H * 4], W.b2.data(), (size_t)D * 4) == 0, "%s: narrow b2", sh.name);
      if (l2)
        CHECK(stored(tn, tail + (size_t)(H + D) * 4, (size_t)D * E, bf) == source({&W.wh}, bf), "%s: narrow Wh",
              sh.name);
    }
    const std::vector<uint8_t> tt = pack_transposed_narrow(dm, W.view);
    CHECK(tt.size() == (nw1 + nw2 + (l2 ? (size_t)D * E : 0)) * ES, "%s: transposed narrow size", sh.name);
    if (!g_fail) {
      CHECK(stored(tt, 0, nw2, bf) == source({&W.w2}, bf), "%s: transposed narrow W2", sh.name);
      CHECK(stored(tt, nw2 * ES, nw1, bf) == source({&W.w1}, bf), "%s: transposed narrow W1", sh.name);
    }
    if (dm.hw_dim % 32 == 0 && dm.cost_hidden % 32 == 0) {
      const std::vector<uint8_t> cn = pack_cost_narrow(dm, W.view);
      const size_t nc = (size_t)dm.cost_hidden * (IN + dm.hw_dim);
      CHECK(cn.size() == nc * ES + (size_t)dm.cost_hidden * 8, "%s: narrow cost size", sh.name);
      if (!g_fail) CHECK(stored(cn, 0, nc, bf) == source({&W.wc1}, bf), "%s: narrow cost values", sh.name);
    }
  }
  if (IN % 32 == 0) {
    std::vector<uint8_t> w2t, w1t;
    if (bf) pack_transposed<GeomBF16>(dm, W.view, w2t, w1t);
    else pack_transposed<GeomF32>(dm, W.view, w2t, w1t);
    CHECK(w2t.size() == (size_t)D * H * ES && w1t.size() == (size_t)H * IN * ES, "%s: transposed sizes", sh.name);
    if (!g_fail) {
      CHECK(stored(w2t, 0, (size_t)D * H, bf) == source({&W.w2}, bf), "%s: transposed W2 values", sh.name);
      CHECK(stored(w1t, 0, (size_t)H * IN, bf) == source({&W.w1}, bf), "%s: transposed W1 values", sh.name);
    }
    if (l2 && E % 32 == 0) {
      const std::vector<uint8_t> ht = bf ? pack_hyper_t<GeomBF16>(dm, W.view) : pack_hyper_t<GeomF32>(dm, W.view);
      CHECK(ht.size() == (size_t)D * E * ES, "%s: transposed normal map size", sh.name);
      if (!g_fail) CHECK(stored(ht, 0, (size_t)D * E, bf) == source({&W.wh}, bf), "%s: transposed Wh", sh.name);
    }
  }
}

// Workspace layouts: 256-byte aligned parts in order, each large enough.
static void check_layouts(const Shape& sh, const wm_dims& dm) {
  DevModel m{};
  m.dims = dm;
  for (int B : {0, 1, 31, 4096, 8193, 65536})
    for (int S : {1, 32})
      for (int n_hw : {1, 2}) {
        const int T_max = 48;
        const WsLayout L = ws_layout(m, B, T_max, S, n_hw);
        const size_t off[] = {L.err, L.perm, L.hist, L.z0, L.zT, L.phi, L.phi_s, L.scores, L.total};
        const size_t need[] = {4, (size_t)B * 8, (size_t)bucket_groups(B) * (T_max + 1) * 4, (size_t)S * dm.d * 4,
                               (size_t)B * dm.d * 4, (size_t)B * dm.embed_dim * 4,
                               (size_t)B * (dm.n_kinds + 1 + 2 * dm.n_params) * 4, (size_t)n_hw * B * 4};
        for (int i = 0; i < 8; ++i) {
          CHECK(off[i] % 256 == 0, "%s: ws part %d misaligned", sh.name, i);
          CHECK(off[i + 1] >= off[i] + need[i], "%s: ws part %d too small (B=%d)", sh.name, i, B);
        }
      }
  for (int B : {1, 100, 8193}) {
    const int T_max = 64;
    const LossLayout L = loss_layout(m, B, T_max);
    const size_t R = (size_t)B * T_max, D = dm.d, E = dm.embed_dim, H = dm.trans_hidden;
    const size_t off[] = {L.err, L.perm, L.hist, L.off, L.row_src, L.X, L.A, L.G, L.P, L.SD, L.DE, L.V, L.SC,
                          L.DV, L.lrow, L.pw1, L.pw2, L.pb1, L.pb2, L.pemb, L.pwh, L.total};
    const bool l2 = dm.norm == WM_NORM_L2;
    const size_t S = L.splits;
    const size_t need[] = {4, (size_t)B * 8, (size_t)bucket_groups(B) * (T_max + 1) * 4, ((size_t)B + 1) * 4,
                           R * 4, R * (D + E) * 4, R * H * 4, R * H * 4, R * D * 4, R * D * 4, R * E * 4,
                           l2 ? R * D * 4 : 0, l2 ? R * 16 : 0, l2 ? R * D * 4 : 0, R * 4,
                           S * H * (D + E) * 4, S * D * H * 4, S * H * 4, S * D * 4,
                           (size_t)L.emb_blocks * (dm.n_kinds * E + E * dm.n_params + E) * 4,
                           l2 ? S * D * E * 4 : 0};
    for (int i = 0; i < 21; ++i) {
      CHECK(off[i] % 256 == 0, "%s: loss part %d misaligned", sh.name, i);
      CHECK(off[i + 1] >= off[i] + need[i], "%s: loss part %d too small (B=%d)", sh.name, i, B);
    }
  }
}

static void check_segments_table() {
  SegTable tab{};
  int32_t mn = -1;
  std::string msg;
  const int32_t ok3[] = {0, 5, 5, 12};
  CHECK(check_segments(ok3, 3, 12, &tab, &mn, &msg) == WM_OK && mn == 0 && tab.n == 3 && tab.off[3] == 12,
        "valid table rejected");
  const int32_t bad_end[] = {0, 5, 11};
  CHECK(check_segments(bad_end, 2, 12, &tab, &mn, &msg) == WM_ERR_INVALID_ARGUMENT && !msg.empty(), "end != B");
  const int32_t bad_start[] = {1, 12};
  CHECK(check_segments(bad_start, 1, 12, &tab, &mn, &msg) == WM_ERR_INVALID_ARGUMENT, "start != 0");
  const int32_t dec[] = {0, 7, 5, 12};
  CHECK(check_segments(dec, 3, 12, &tab, &mn, &msg) == WM_ERR_INVALID_ARGUMENT, "decreasing offsets");
  CHECK(check_segments(nullptr, 1, 0, &tab, &mn, &msg) == WM_ERR_INVALID_ARGUMENT, "null table");
  CHECK(check_segments(ok3, 0, 0, &tab, &mn, &msg) == WM_ERR_INVALID_ARGUMENT, "S = 0");
  std::vector<int32_t> big(WM_MAX_SEGMENTS + 2, 0);
  CHECK(check_segments(big.data(), WM_MAX_SEGMENTS + 1, 0, &tab, &mn, &msg) == WM_ERR_INVALID_ARGUMENT,
        "too many segments");
  std::vector<int32_t> full(WM_MAX_SEGMENTS + 1);
  for (int s = 0; s <= WM_MAX_SEGMENTS; ++s) full[s] = 3 * s;
  CHECK(check_segments(full.data(), WM_MAX_SEGMENTS, 3 * WM_MAX_SEGMENTS, &tab, &mn, &msg) == WM_OK && mn == 3 &&
            tab.off[WM_MAX_SEGMENTS] == 3 * WM_MAX_SEGMENTS,
        "largest table");
}

int main() {
  // the (precision, d, e) the kernels are built for, with the hidden widths of
  // the benchmark workloads
  const Shape shapes[] = {
      {"d64 fp32", WM_FP32, 64, 32, 12, 4, 128, 128, 16},
      {"d64 bf16", WM_BF16, 64, 32, 12, 4, 128, 128, 16},
      {"d256 fp32", WM_FP32, 256, 64, 16, 6, 512, 512, 32},
      {"d256 bf16", WM_BF16, 256, 64, 16, 6, 512, 512, 32},
      {"d256 bf16 H1024", WM_BF16, 256, 64, 16, 6, 1024, 512, 32},
      {"d512 bf16", WM_BF16, 512, 128, 16, 6, 2048, 1024, 32},
  };
  for (const Shape& sh : shapes)
    for (wm_norm norm : {WM_NORM_NONE, WM_NORM_L2}) {
      wm_dims dm{};
      dm.d = sh.d;
      dm.embed_dim = sh.e;
      dm.n_kinds = sh.K;
      dm.n_params = sh.P;
      dm.trans_hidden = sh.H;
      dm.cost_hidden = sh.C;
      dm.hw_dim = sh.hw;
      dm.precision = sh.prec;
      dm.norm = norm;
      const Weights W = make_weights(dm, 1234u + (uint32_t)sh.d);
      check_transition(sh, dm, W);
      check_cost(sh, dm, W);
      if (norm == WM_NORM_L2) check_hyper(sh, dm, W);
      check_permutations(sh, dm, W);
      check_layouts(sh, dm);
      std::printf("%s %s: %s\n", sh.name, norm == WM_NORM_L2 ? "l2" : "none", g_fail ? "FAIL" : "ok");
    }
  check_segments_table();
  // bf16 conversion: ties to even, NaN stays NaN
  CHECK(f32_to_bf16(1.0f + 1.0f / 256.0f) == 0x3f80, "tie to even (down)");
  CHECK(f32_to_bf16(1.0f + 3.0f / 256.0f) == 0x3f82, "tie to even (up)");
  CHECK((f32_to_bf16(std::nanf("")) & 0x7fff) > 0x7f80, "NaN");
  std::printf("%s (%d failures)\n", g_fail ? "FAILED" : "all ok", g_fail);
  return g_fail ? 1 : 0;
}
