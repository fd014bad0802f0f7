// C-ABI layer of the batched latent-rollout evaluator: model creation (weight
// repacking into matrix-fragment order), host-side argument validation,
// workspace carving, kernel orchestration, device error word, event timing.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "wm_internal.h"
#include "wm_pack.h"

using namespace wm;

struct wm_model {
  DevModel dm;
};

struct wm_forest {
  DevForest df;
};

namespace {

thread_local std::string g_last_error;

wm_status fail(wm_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

wm_status ok() {
  g_last_error.clear();
  return WM_OK;
}

#define WM_HIP_TRY(expr)                                                                 \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess) return fail(WM_ERR_DEVICE, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

// Segment-table check with the reason recorded as the last error.
wm_status check_segments(const int32_t* seg_off, int32_t S, int32_t B, SegTable* tab,
                         int32_t* min_seg) {
  std::string msg;
  const wm_status st = wm::check_segments(seg_off, S, B, tab, min_seg, &msg);
  return st == WM_OK ? st : fail(st, msg);
}

// ---- timing ----------------------------------------------------------------
constexpr int kTimingCap = 8192;
struct Timing {
  std::mutex mu;
  bool on = false;
  std::vector<hipEvent_t> start[TK_COUNT], stop[TK_COUNT];
  int count[TK_COUNT] = {};
} g_timing;

}  // namespace

namespace wm {
void timing_begin(int k, hipStream_t st) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  if (!g_timing.on || g_timing.count[k] >= kTimingCap) return;
  const int i = g_timing.count[k];
  if ((int)g_timing.start[k].size() <= i) {
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess) return;
    if (hipEventCreate(&b) != hipSuccess) { (void)hipEventDestroy(a); return; }
    g_timing.start[k].push_back(a);
    g_timing.stop[k].push_back(b);
  }
  (void)hipEventRecord(g_timing.start[k][i], st);
}
void timing_end(int k, hipStream_t st) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  if (!g_timing.on || g_timing.count[k] >= kTimingCap) return;
  const int i = g_timing.count[k];
  if ((int)g_timing.stop[k].size() <= i) return;
  (void)hipEventRecord(g_timing.stop[k][i], st);
  g_timing.count[k] = i + 1;
}
wm_status set_error(wm_status st, const std::string& msg) { return fail(st, msg); }
wm_status clear_error() { return ok(); }
}  // namespace wm

#define WM_TIMED(K, ST, CALL)                                              \
  do {                                                                     \
    timing_begin(K, ST);                                                   \
    hipError_t e_ = (CALL);                                                \
    timing_end(K, ST);                                                     \
    if (e_ != hipSuccess) return fail(WM_ERR_DEVICE, std::string("kernel launch: ") + hipGetErrorString(e_)); \
  } while (0)

// ---- allocation-free evaluation ----------------------------------------------
// Scratch of wm_evaluate_noalloc: one copy per GPU of the library's code
// object.  In host code `noalloc_scratch` only stands for the symbol; its
// device address, per device, comes from hipGetSymbolAddress.
static __device__ __align__(256) uint8_t noalloc_scratch[WM_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t* g_scratch[kMaxDevices] = {};

// The scratch's address on the current device (looked up once per device).
wm_status noalloc_scratch_ptr(uint8_t** out) {
  int dev = -1;
  WM_HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(WM_ERR_DEVICE, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    WM_HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(noalloc_scratch)));
    if (!p) return fail(WM_ERR_DEVICE, "hipGetSymbolAddress returned NULL for the scratch");
    g_scratch[dev] = static_cast<uint8_t*>(p);
  }
  *out = g_scratch[dev];
  return WM_OK;
}
}  // namespace

extern "C" {

const char* wm_last_error(void) { return g_last_error.c_str(); }

wm_status wm_model_create(const wm_dims* dims, const wm_weights* w, wm_model** out) {
  if (!dims || !w || !out) return fail(WM_ERR_INVALID_ARGUMENT, "null argument");
  *out = nullptr;
  const wm_dims& dm = *dims;
  if (dm.d <= 0 || dm.embed_dim <= 0 || dm.n_kinds <= 0 || dm.n_params <= 0 ||
      dm.trans_hidden <= 0 || dm.cost_hidden <= 0 || dm.hw_dim < 0 || dm.feat_dim < 0 ||
      (dm.feat_dim > 0 && dm.enc_hidden <= 0))
    return fail(WM_ERR_INVALID_ARGUMENT, "dims must be positive (hw_dim, feat_dim >= 0)");
  if (dm.precision != WM_FP32 && dm.precision != WM_BF16)
    return fail(WM_ERR_INVALID_ARGUMENT, "unknown precision");
  if (dm.norm != WM_NORM_NONE && dm.norm != WM_NORM_L2)
    return fail(WM_ERR_INVALID_ARGUMENT, "unknown norm");
  if (dm.norm == WM_NORM_L2 && !w->wh) return fail(WM_ERR_INVALID_ARGUMENT, "WM_NORM_L2 needs wh");
  if (!w->type_emb || !w->param_w || !w->param_b || !w->w1 || !w->b1 || !w->w2 || !w->b2 ||
      !w->wc1 || !w->bc1 || !w->wc2)
    return fail(WM_ERR_INVALID_ARGUMENT, "null weight pointer");
  if (dm.feat_dim > 0 && (!w->we1 || !w->be1 || !w->we2 || !w->be2))
    return fail(WM_ERR_INVALID_ARGUMENT, "null encoder weight pointer");
  if (!have_kernels(dm.precision, dm.d, dm.embed_dim))
    return fail(WM_ERR_UNSUPPORTED, "no kernels for this (precision, d, embed_dim)");
  if (dm.trans_hidden % 64 || dm.cost_hidden % 64 || dm.hw_dim % 16 || dm.hw_dim > 32 ||
      dm.n_kinds > 32 || dm.n_params > 8)
    return fail(WM_ERR_UNSUPPORTED,
                "need trans_hidden, cost_hidden % 64 == 0, hw_dim % 16 == 0 and <= 32, n_kinds <= 32, n_params <= 8");

  DevModel m{};
  m.dims = dm;
  m.prec = dm.precision;
  const int D = dm.d, E = dm.embed_dim, K = dm.n_kinds, P = dm.n_params, HW = dm.hw_dim;
  std::vector<uint8_t> tw1, tw2, cost, twh, tw2t, tw1t, twht, tn, tnt, cn;
  const bool l2 = dm.norm == WM_NORM_L2;
  if (m.prec == WM_BF16) {
    pack_transition<GeomBF16>(dm, *w, tw1, tw2);
    if ((D + E) % 32 == 0) pack_transposed<GeomBF16>(dm, *w, tw2t, tw1t);
    cost = pack_cost<GeomBF16>(dm, *w);
    if (l2) twh = pack_hyper<GeomBF16>(dm, *w);
    if (l2 && E % 32 == 0) twht = pack_hyper_t<GeomBF16>(dm, *w);
    m.w1_chunk_bytes = TransChunk<GeomBF16>::w1_bytes(D, E);
    m.w2_chunk_bytes = TransChunk<GeomBF16>::w2_bytes(D);
    m.cost_chunk_bytes = CostChunk<GeomBF16>::bytes(D, E, HW);
  } else {
    if ((D + E + HW) % 8 != 0) return fail(WM_ERR_UNSUPPORTED, "fp32 needs d + embed_dim + hw_dim % 8 == 0");
    pack_transition<GeomF32>(dm, *w, tw1, tw2);
    if ((D + E) % 32 == 0) pack_transposed<GeomF32>(dm, *w, tw2t, tw1t);
    cost = pack_cost<GeomF32>(dm, *w);
    if (l2) twh = pack_hyper<GeomF32>(dm, *w);
    if (l2 && E % 32 == 0) twht = pack_hyper_t<GeomF32>(dm, *w);
    m.w1_chunk_bytes = TransChunk<GeomF32>::w1_bytes(D, E);
    m.w2_chunk_bytes = TransChunk<GeomF32>::w2_bytes(D);
    m.cost_chunk_bytes = CostChunk<GeomF32>::bytes(D, E, HW);
  }
  if (D % 32 == 0 && E % 32 == 0) {
    tn = pack_transition_narrow(dm, *w);
    tnt = pack_transposed_narrow(dm, *w);
    if (HW % 32 == 0 && dm.cost_hidden % 32 == 0) cn = pack_cost_narrow(dm, *w);
  }
  // rollout table: type_emb [K][E + 4], param_w^T [PMAX][E], param_b [E], b2 (accumulator order)
  std::vector<float> tab;
  tab.reserve((size_t)K * temb_stride(E) + (size_t)PMAX * E + E + D + 4);
  for (int k = 0; k < K; ++k)
    for (int f = 0; f < temb_stride(E); ++f) tab.push_back(f < E ? w->type_emb[(size_t)k * E + f] : 0.0f);
  for (int p = 0; p < PMAX; ++p)
    for (int f = 0; f < E; ++f) tab.push_back(p < P ? w->param_w[(size_t)f * P + p] : 0.0f);
  for (int f = 0; f < E; ++f) tab.push_back(w->param_b[f]);
  for (int b = 0; b < D / 32; ++b)
    for (int h = 0; h < 2; ++h)
      for (int r = 0; r < 16; ++r) tab.push_back(w->b2[32 * b + acc_row(h, r)]);
  while (tab.size() % 4) tab.push_back(0.0f);
  m.roll_tab_bytes = (int)(tab.size() * 4);
  m.wh_bytes = (int)twh.size();
  if (rollout_lds_bytes(m) > 160 * 1024 || 2 * m.cost_chunk_bytes > 160 * 1024)
    return fail(WM_ERR_UNSUPPORTED, "weight chunks do not fit the 160 KiB LDS");

  // encoder (transposed; bf16-rounded values in bf16 mode)
  std::vector<float> enc;
  const int F = dm.feat_dim, Fh = dm.enc_hidden;
  size_t enc_w1t = 0, enc_b1 = 0, enc_w2t = 0, enc_b2 = 0;
  if (F > 0) {
    auto r = [&](float v) { return m.prec == WM_BF16 ? bf16_value(v) : v; };
    enc_w1t = enc.size();
    for (int f = 0; f < F; ++f)
      for (int o = 0; o < Fh; ++o) enc.push_back(r(w->we1[(size_t)o * F + f]));
    enc_b1 = enc.size();
    for (int o = 0; o < Fh; ++o) enc.push_back(w->be1[o]);
    enc_w2t = enc.size();
    for (int k = 0; k < Fh; ++k)
      for (int o = 0; o < D; ++o) enc.push_back(r(w->we2[(size_t)o * Fh + k]));
    enc_b2 = enc.size();
    for (int o = 0; o < D; ++o) enc.push_back(w->be2[o]);
  }

  size_t off = 0;
  const size_t o_tw1 = off; off = align256(off + tw1.size());
  const size_t o_tw2 = off; off = align256(off + tw2.size());
  const size_t o_cost = off; off = align256(off + cost.size());
  const size_t o_wh = off; off = align256(off + twh.size());
  const size_t o_w2t = off; off = align256(off + tw2t.size());
  const size_t o_w1t = off; off = align256(off + tw1t.size());
  const size_t o_wht = off; off = align256(off + twht.size());
  const size_t o_tn = off; off = align256(off + tn.size());
  const size_t o_tnt = off; off = align256(off + tnt.size());
  const size_t o_cn = off; off = align256(off + cn.size());
  const size_t o_tab = off; off = align256(off + tab.size() * 4);
  const size_t o_enc = off; off = align256(off + enc.size() * 4);
  void* dev = nullptr;
  if (hipMalloc(&dev, off) != hipSuccess) {
    (void)hipGetLastError();
    return fail(WM_ERR_OUT_OF_MEMORY, "hipMalloc of the model failed");
  }
  uint8_t* base = static_cast<uint8_t*>(dev);
  hipError_t e = hipMemcpy(base + o_tw1, tw1.data(), tw1.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(base + o_tw2, tw2.data(), tw2.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(base + o_cost, cost.data(), cost.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess && !twh.empty()) e = hipMemcpy(base + o_wh, twh.data(), twh.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess && !tw2t.empty()) e = hipMemcpy(base + o_w2t, tw2t.data(), tw2t.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess && !tw1t.empty()) e = hipMemcpy(base + o_w1t, tw1t.data(), tw1t.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess && !twht.empty()) e = hipMemcpy(base + o_wht, twht.data(), twht.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess && !tn.empty()) e = hipMemcpy(base + o_tn, tn.data(), tn.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess && !tnt.empty()) e = hipMemcpy(base + o_tnt, tnt.data(), tnt.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess && !cn.empty()) e = hipMemcpy(base + o_cn, cn.data(), cn.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(base + o_tab, tab.data(), tab.size() * 4, hipMemcpyHostToDevice);
  if (e == hipSuccess && !enc.empty()) e = hipMemcpy(base + o_enc, enc.data(), enc.size() * 4, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(dev);
    return fail(WM_ERR_DEVICE, std::string("hipMemcpy: ") + hipGetErrorString(e));
  }
  m.base = base;
  m.trans_w1 = base + o_tw1;
  m.trans_w2 = base + o_tw2;
  m.cost = base + o_cost;
  m.trans_wh = twh.empty() ? nullptr : base + o_wh;
  m.trans_w2t = tw2t.empty() ? nullptr : base + o_w2t;
  m.trans_w1t = tw1t.empty() ? nullptr : base + o_w1t;
  m.trans_wht = twht.empty() ? nullptr : base + o_wht;
  m.trans_n = tn.empty() ? nullptr : base + o_tn;
  m.trans_nt = tnt.empty() ? nullptr : base + o_tnt;
  m.cost_n = cn.empty() ? nullptr : base + o_cn;
  m.roll_tab = reinterpret_cast<const float*>(base + o_tab);
  m.emb_nat = m.roll_tab;
  const float* encp = reinterpret_cast<const float*>(base + o_enc);
  m.enc_w1t = encp + enc_w1t;
  m.enc_b1 = encp + enc_b1;
  m.enc_w2t = encp + enc_w2t;
  m.enc_b2 = encp + enc_b2;
  m.bc2 = w->bc2;
  wm_model* out_m = new (std::nothrow) wm_model;
  if (!out_m) {
    (void)hipFree(dev);
    return fail(WM_ERR_OUT_OF_MEMORY, "host allocation failed");
  }
  out_m->dm = m;
  *out = out_m;
  return ok();
}

void wm_model_destroy(wm_model* model) {
  if (!model) return;
  (void)hipFree(model->dm.base);
  delete model;
}

size_t wm_workspace_bytes(const wm_model* model, int32_t B, int32_t T_max, int32_t S, int32_t n_hw) {
  if (!model || B < 0 || T_max < 0 || T_max > WM_MAX_T || S < 1 || n_hw < 1) return 0;
  return ws_layout(model->dm, B, T_max, S, n_hw).total;
}

wm_status wm_encode_init(const wm_model* model, const float* feats, int32_t S, float* z0,
                         void* stream) {
  if (!model) return fail(WM_ERR_INVALID_ARGUMENT, "model is NULL");
  if (model->dm.dims.feat_dim <= 0) return fail(WM_ERR_INVALID_ARGUMENT, "model has no encoder");
  if (S < 0) return fail(WM_ERR_INVALID_ARGUMENT, "S < 0");
  if (S == 0) return ok();
  if (!feats || !z0) return fail(WM_ERR_INVALID_ARGUMENT, "feats/z0 is NULL");
  hipStream_t st = static_cast<hipStream_t>(stream);
  WM_TIMED(TK_ENCODE, st, launch_encode(model->dm, feats, S, z0, st));
  return ok();
}

static wm_status check_rollout_args(const wm_model* model, const float* z0, const int32_t* types,
                                    const int32_t* params, const int32_t* lens, int32_t B,
                                    int32_t T_max, const float* zT) {
  if (!model) return fail(WM_ERR_INVALID_ARGUMENT, "model is NULL");
  if (B < 0) return fail(WM_ERR_INVALID_ARGUMENT, "B < 0");
  if (T_max < 0 || T_max > WM_MAX_T)
    return fail(WM_ERR_INVALID_ARGUMENT, "T_max must be in [0, " + std::to_string(WM_MAX_T) + "]");
  if (B > 0 && (!z0 || !types || !params || !lens || !zT))
    return fail(WM_ERR_INVALID_ARGUMENT, "null input/output pointer");
  return WM_OK;
}

wm_status wm_rollout(const wm_model* model, const float* z0, const int32_t* seg_off, int32_t S,
                     const int32_t* types, const int32_t* params, const int32_t* lens, int32_t B,
                     int32_t T_max, float* zT, float* phi, void* ws, size_t ws_bytes,
                     void* stream) {
  wm_status s = check_rollout_args(model, z0, types, params, lens, B, T_max, zT);
  if (s != WM_OK) return s;
  SegTable seg;
  int32_t min_seg = 0;
  if ((s = check_segments(seg_off, S, B, &seg, &min_seg)) != WM_OK) return s;
  if (!ws) return fail(WM_ERR_INVALID_ARGUMENT, "workspace is NULL");
  const WsLayout L = ws_layout(model->dm, B, T_max, S, 1);
  if (ws_bytes < L.total) return fail(WM_ERR_INVALID_ARGUMENT, "workspace too small");
  if (B == 0) return ok();
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* w8 = static_cast<uint8_t*>(ws);
  int32_t* err = reinterpret_cast<int32_t*>(w8 + L.err);
  int2* perm = reinterpret_cast<int2*>(w8 + L.perm);
  WM_TIMED(TK_BUCKET, st, launch_bucket(lens, B, T_max, seg, perm, reinterpret_cast<int32_t*>(w8 + L.hist), err, st));
  bool phi_done = false;
  WM_TIMED(TK_ROLLOUT, st, launch_rollout(model->dm, z0, perm, types, params, lens, B, T_max, zT, phi,
                                          &phi_done, err, st));
  if (phi && !phi_done) WM_TIMED(TK_PHI, st, launch_phi(model->dm, types, params, lens, B, T_max, phi, st));
  return ok();
}

wm_status wm_score(const wm_model* model, const float* zT, const float* phi, int32_t B,
                   const float* hw, int32_t n_hw, float* scores, void* stream) {
  if (!model) return fail(WM_ERR_INVALID_ARGUMENT, "model is NULL");
  if (B < 0 || n_hw < 1) return fail(WM_ERR_INVALID_ARGUMENT, "need B >= 0 and n_hw >= 1");
  if (B == 0) return ok();
  if (!zT || !phi || !scores || (model->dm.dims.hw_dim > 0 && !hw))
    return fail(WM_ERR_INVALID_ARGUMENT, "null input/output pointer");
  hipStream_t st = static_cast<hipStream_t>(stream);
  WM_TIMED(TK_SCORE, st, launch_score(model->dm, zT, phi, B, hw, n_hw, scores, st));
  return ok();
}

static wm_status check_k(int32_t k, int32_t min_seg) {
  if (k < 1 || k > WM_MAX_K) return fail(WM_ERR_INVALID_ARGUMENT, "k must be in [1, " + std::to_string(WM_MAX_K) + "]");
  if (k > min_seg) return fail(WM_ERR_INVALID_ARGUMENT, "k exceeds the size of a segment");
  return WM_OK;
}

wm_status wm_topk(const float* scores, int32_t n_hw, int32_t B, const int32_t* seg_off, int32_t S,
                  int32_t k, int32_t* idx, float* val, void* stream) {
  if (B < 0 || n_hw < 1) return fail(WM_ERR_INVALID_ARGUMENT, "need B >= 0 and n_hw >= 1");
  SegTable seg;
  int32_t min_seg = 0;
  wm_status s = check_segments(seg_off, S, B, &seg, &min_seg);
  if (s != WM_OK) return s;
  if ((s = check_k(k, min_seg)) != WM_OK) return s;
  if (!scores || !idx) return fail(WM_ERR_INVALID_ARGUMENT, "null scores/idx");
  hipStream_t st = static_cast<hipStream_t>(stream);
  WM_TIMED(TK_TOPK, st, launch_topk(scores, n_hw, B, seg, k, idx, val, st));
  return ok();
}

wm_status wm_evaluate(const wm_model* model, const float* init, int32_t init_is_feats,
                      const int32_t* seg_off, int32_t S, const int32_t* types,
                      const int32_t* params, const int32_t* lens, int32_t B, int32_t T_max,
                      const float* hw, int32_t n_hw, int32_t k, float* scores, float* zT,
                      int32_t* idx, float* val, void* ws, size_t ws_bytes, void* stream) {
  if (!model) return fail(WM_ERR_INVALID_ARGUMENT, "model is NULL");
  if (init_is_feats && model->dm.dims.feat_dim <= 0)
    return fail(WM_ERR_INVALID_ARGUMENT, "init_is_feats needs a model with an encoder");
  // zT is checked below once a workspace fallback is known
  wm_status s = check_rollout_args(model, init, types, params, lens, B, T_max, reinterpret_cast<float*>(1));
  if (s != WM_OK) return s;
  if (n_hw < 1) return fail(WM_ERR_INVALID_ARGUMENT, "n_hw < 1");
  SegTable seg;
  int32_t min_seg = 0;
  if ((s = check_segments(seg_off, S, B, &seg, &min_seg)) != WM_OK) return s;
  if ((s = check_k(k, min_seg)) != WM_OK) return s;
  if (!idx) return fail(WM_ERR_INVALID_ARGUMENT, "idx is NULL");
  if (model->dm.dims.hw_dim > 0 && !hw) return fail(WM_ERR_INVALID_ARGUMENT, "hw is NULL");
  if (!ws) return fail(WM_ERR_INVALID_ARGUMENT, "workspace is NULL");
  const WsLayout L = ws_layout(model->dm, B, T_max, S, n_hw);
  if (ws_bytes < L.total) return fail(WM_ERR_INVALID_ARGUMENT, "workspace too small");

  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* w8 = static_cast<uint8_t*>(ws);
  int32_t* err = reinterpret_cast<int32_t*>(w8 + L.err);
  int2* perm = reinterpret_cast<int2*>(w8 + L.perm);
  float* z0 = const_cast<float*>(init);
  if (init_is_feats) {
    z0 = reinterpret_cast<float*>(w8 + L.z0);
    WM_TIMED(TK_ENCODE, st, launch_encode(model->dm, init, S, z0, st));
  }
  float* zTo = zT ? zT : reinterpret_cast<float*>(w8 + L.zT);
  float* phi = reinterpret_cast<float*>(w8 + L.phi);
  float* sc = scores ? scores : reinterpret_cast<float*>(w8 + L.scores);
  WM_TIMED(TK_BUCKET, st, launch_bucket(lens, B, T_max, seg, perm, reinterpret_cast<int32_t*>(w8 + L.hist), err, st));
  bool phi_done = false;
  ScoreFuse sf{hw, n_hw, sc, false};
  WM_TIMED(TK_ROLLOUT, st, launch_rollout(model->dm, z0, perm, types, params, lens, B, T_max, zTo, phi,
                                          &phi_done, err, st, &sf));
  if (!phi_done) WM_TIMED(TK_PHI, st, launch_phi(model->dm, types, params, lens, B, T_max, phi, st));
  if (!sf.done) WM_TIMED(TK_SCORE, st, launch_score(model->dm, zTo, phi, B, hw, n_hw, sc, st));
  WM_TIMED(TK_TOPK, st, launch_topk(sc, n_hw, B, seg, k, idx, val, st));
  return ok();
}

wm_status wm_evaluate_noalloc(const wm_model* model, const float* init, int32_t init_is_feats,
                              const int32_t* seg_off, int32_t S, const int32_t* types,
                              const int32_t* params, const int32_t* lens, int32_t B, int32_t T_max,
                              const float* hw, int32_t n_hw, int32_t k, float* scores, float* zT,
                              float* phi, int32_t* idx, float* val, int32_t* status, void* stream) {
  if (!model) return fail(WM_ERR_INVALID_ARGUMENT, "model is NULL");
  if (init_is_feats && model->dm.dims.feat_dim <= 0)
    return fail(WM_ERR_INVALID_ARGUMENT, "init_is_feats needs a model with an encoder");
  wm_status s = check_rollout_args(model, init, types, params, lens, B, T_max, zT);
  if (s != WM_OK) return s;
  if (n_hw < 1) return fail(WM_ERR_INVALID_ARGUMENT, "n_hw < 1");
  SegTable seg;
  int32_t min_seg = 0;
  if ((s = check_segments(seg_off, S, B, &seg, &min_seg)) != WM_OK) return s;
  if ((s = check_k(k, min_seg)) != WM_OK) return s;
  if (!idx) return fail(WM_ERR_INVALID_ARGUMENT, "idx is NULL");
  if (!scores || !phi) return fail(WM_ERR_INVALID_ARGUMENT, "scores and phi are required");
  if (!status) return fail(WM_ERR_INVALID_ARGUMENT, "status is NULL");
  if (model->dm.dims.hw_dim > 0 && !hw) return fail(WM_ERR_INVALID_ARGUMENT, "hw is NULL");
  // scratch layout: permutation, bucketing histograms, encoded initial latents
  const size_t o_perm = 0;
  const size_t o_hist = align256(o_perm + (size_t)B * sizeof(int2));
  const size_t o_z0 = align256(o_hist + (size_t)bucket_groups(B) * (size_t)(T_max + 1) * 4);
  const size_t need = o_z0 + (init_is_feats ? (size_t)S * model->dm.dims.d * 4 : 0);
  if (need > WM_NOALLOC_SCRATCH_BYTES)
    return fail(WM_ERR_INVALID_ARGUMENT, "the batch needs " + std::to_string(need) +
                                             " bytes of scratch, more than WM_NOALLOC_SCRATCH_BYTES");
  uint8_t* sp = nullptr;
  if ((s = noalloc_scratch_ptr(&sp)) != WM_OK) return s;

  hipStream_t st = static_cast<hipStream_t>(stream);
  int2* perm = reinterpret_cast<int2*>(sp + o_perm);
  WM_HIP_TRY(launch_clear_words(status, 64, st));
  float* z0 = const_cast<float*>(init);
  if (init_is_feats) {
    z0 = reinterpret_cast<float*>(sp + o_z0);
    WM_TIMED(TK_ENCODE, st, launch_encode(model->dm, init, S, z0, st));
  }
  WM_TIMED(TK_BUCKET, st, launch_bucket(lens, B, T_max, seg, perm, reinterpret_cast<int32_t*>(sp + o_hist),
                                        status, st));
  bool phi_done = false;
  ScoreFuse sf{hw, n_hw, scores, false};
  WM_TIMED(TK_ROLLOUT, st, launch_rollout(model->dm, z0, perm, types, params, lens, B, T_max, zT, phi,
                                          &phi_done, status, st, &sf));
  if (!phi_done) WM_TIMED(TK_PHI, st, launch_phi(model->dm, types, params, lens, B, T_max, phi, st));
  if (!sf.done) WM_TIMED(TK_SCORE, st, launch_score(model->dm, zT, phi, B, hw, n_hw, scores, st));
  WM_TIMED(TK_TOPK, st, launch_topk(scores, n_hw, B, seg, k, idx, val, st));
  return ok();
}

wm_status wm_forest_create(int32_t n_trees, int32_t depth, int32_t n_features, const int32_t* feat,
                           const float* thr, const float* leaf, float base, wm_forest** out) {
  if (!out) return fail(WM_ERR_INVALID_ARGUMENT, "out is NULL");
  *out = nullptr;
  if (!feat || !thr || !leaf) return fail(WM_ERR_INVALID_ARGUMENT, "null forest array");
  if (n_trees < 1 || depth < 1 || depth > FOREST_MAX_DEPTH || n_features < 1 || n_features > TREE_MAX_FEATURES)
    return fail(WM_ERR_INVALID_ARGUMENT, "need n_trees >= 1, 1 <= depth <= " + std::to_string(FOREST_MAX_DEPTH) +
                                          ", 1 <= n_features <= " + std::to_string(TREE_MAX_FEATURES));
  const size_t n_int = ((size_t)1 << depth) - 1;
  std::vector<int2> nodes((size_t)n_trees * n_int);
  for (size_t q = 0; q < nodes.size(); ++q) {
    if (feat[q] < 0 || feat[q] >= n_features)
      return fail(WM_ERR_INVALID_ARGUMENT, "feature index out of range at node " + std::to_string(q));
    int32_t bits;
    std::memcpy(&bits, &thr[q], 4);
    nodes[q] = make_int2(feat[q], bits);
  }
  const size_t nb = nodes.size() * sizeof(int2), lb = (size_t)n_trees * (n_int + 1) * 4;
  void* dev = nullptr;
  if (hipMalloc(&dev, align256(nb) + lb) != hipSuccess) {
    (void)hipGetLastError();
    return fail(WM_ERR_OUT_OF_MEMORY, "hipMalloc of the forest failed");
  }
  uint8_t* base8 = static_cast<uint8_t*>(dev);
  hipError_t e = hipMemcpy(base8, nodes.data(), nb, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(base8 + align256(nb), leaf, lb, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(dev);
    return fail(WM_ERR_DEVICE, std::string("hipMemcpy: ") + hipGetErrorString(e));
  }
  wm_forest* f = new (std::nothrow) wm_forest;
  if (!f) {
    (void)hipFree(dev);
    return fail(WM_ERR_OUT_OF_MEMORY, "host allocation failed");
  }
  f->df.n_trees = n_trees;
  f->df.depth = depth;
  f->df.n_features = n_features;
  f->df.base = base;
  f->df.alloc = base8;
  f->df.nodes = reinterpret_cast<const int2*>(base8);
  f->df.leaves = reinterpret_cast<const float*>(base8 + align256(nb));
  *out = f;
  return ok();
}

void wm_forest_destroy(wm_forest* forest) {
  if (!forest) return;
  (void)hipFree(forest->df.alloc);
  delete forest;
}

wm_status wm_phi_struct(const int32_t* types, const int32_t* params, const int32_t* lens, int32_t B,
                        int32_t T_max, int32_t n_kinds, int32_t n_params, float* phi_s, void* stream) {
  if (B < 0 || T_max < 0 || T_max > WM_MAX_T) return fail(WM_ERR_INVALID_ARGUMENT, "need B >= 0, 0 <= T_max <= WM_MAX_T");
  if (n_kinds < 1 || n_kinds > 32 || n_params < 1 || n_params > PMAX)
    return fail(WM_ERR_UNSUPPORTED, "need 1 <= n_kinds <= 32 and 1 <= n_params <= 8");
  if (B == 0) return ok();
  if (!types || !params || !lens || !phi_s) return fail(WM_ERR_INVALID_ARGUMENT, "null pointer");
  hipStream_t st = static_cast<hipStream_t>(stream);
  WM_TIMED(TK_PHI_STRUCT, st, launch_phi_struct(types, params, lens, B, T_max, n_kinds, n_params, phi_s, st));
  return ok();
}

wm_status wm_score_trees(const wm_forest* forest, const float* zT, int32_t d, const float* phi_s,
                         int32_t phi_dim, int32_t B, const float* hw, int32_t n_hw, int32_t hw_dim,
                         float* scores, void* stream) {
  if (!forest) return fail(WM_ERR_INVALID_ARGUMENT, "forest is NULL");
  if (B < 0 || n_hw < 1 || d < 0 || phi_dim < 0 || hw_dim < 0)
    return fail(WM_ERR_INVALID_ARGUMENT, "need B >= 0, n_hw >= 1, non-negative widths");
  if (d + phi_dim + hw_dim != forest->df.n_features)
    return fail(WM_ERR_INVALID_ARGUMENT, "d + phi_dim + hw_dim must equal the forest's n_features");
  if (B == 0) return ok();
  if (!zT || (phi_dim > 0 && !phi_s) || (hw_dim > 0 && !hw) || !scores)
    return fail(WM_ERR_INVALID_ARGUMENT, "null input/output pointer");
  hipStream_t st = static_cast<hipStream_t>(stream);
  WM_TIMED(TK_TREES, st, launch_score_trees(forest->df, zT, d, phi_s, phi_dim, B, hw, n_hw, hw_dim, scores, st));
  return ok();
}

wm_status wm_evaluate_trees(const wm_model* model, const wm_forest* forest, const float* init,
                            int32_t init_is_feats, const int32_t* seg_off, int32_t S,
                            const int32_t* types, const int32_t* params, const int32_t* lens,
                            int32_t B, int32_t T_max, const float* hw, int32_t n_hw, int32_t k,
                            float* scores, float* zT, int32_t* idx, float* val, void* ws,
                            size_t ws_bytes, void* stream) {
  if (!model || !forest) return fail(WM_ERR_INVALID_ARGUMENT, "model/forest is NULL");
  if (init_is_feats && model->dm.dims.feat_dim <= 0) return fail(WM_ERR_INVALID_ARGUMENT, "model has no encoder");
  wm_status s = check_rollout_args(model, init, types, params, lens, B, T_max, reinterpret_cast<float*>(1));
  if (s != WM_OK) return s;
  if (n_hw < 1) return fail(WM_ERR_INVALID_ARGUMENT, "n_hw < 1");
  const wm_dims& dm = model->dm.dims;
  const int phi_dim = phi_struct_dim(dm.n_kinds, dm.n_params);
  if (dm.d + phi_dim + dm.hw_dim != forest->df.n_features)
    return fail(WM_ERR_INVALID_ARGUMENT, "the forest's n_features must be d + (n_kinds + 1 + 2 n_params) + hw_dim");
  SegTable seg;
  int32_t min_seg = 0;
  if ((s = check_segments(seg_off, S, B, &seg, &min_seg)) != WM_OK) return s;
  if ((s = check_k(k, min_seg)) != WM_OK) return s;
  if (!idx) return fail(WM_ERR_INVALID_ARGUMENT, "idx is NULL");
  if (dm.hw_dim > 0 && !hw) return fail(WM_ERR_INVALID_ARGUMENT, "hw is NULL");
  if (!ws) return fail(WM_ERR_INVALID_ARGUMENT, "workspace is NULL");
  const WsLayout L = ws_layout(model->dm, B, T_max, S, n_hw);
  if (ws_bytes < L.total) return fail(WM_ERR_INVALID_ARGUMENT, "workspace too small");

  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* w8 = static_cast<uint8_t*>(ws);
  int32_t* err = reinterpret_cast<int32_t*>(w8 + L.err);
  int2* perm = reinterpret_cast<int2*>(w8 + L.perm);
  float* z0 = const_cast<float*>(init);
  if (init_is_feats) {
    z0 = reinterpret_cast<float*>(w8 + L.z0);
    WM_TIMED(TK_ENCODE, st, launch_encode(model->dm, init, S, z0, st));
  }
  float* zTo = zT ? zT : reinterpret_cast<float*>(w8 + L.zT);
  float* phs = reinterpret_cast<float*>(w8 + L.phi_s);
  float* sc = scores ? scores : reinterpret_cast<float*>(w8 + L.scores);
  WM_TIMED(TK_BUCKET, st, launch_bucket(lens, B, T_max, seg, perm, reinterpret_cast<int32_t*>(w8 + L.hist), err, st));
  bool phi_done = false;
  WM_TIMED(TK_ROLLOUT, st, launch_rollout(model->dm, z0, perm, types, params, lens, B, T_max, zTo, nullptr,
                                          &phi_done, err, st));
  WM_TIMED(TK_PHI_STRUCT, st, launch_phi_struct(types, params, lens, B, T_max, dm.n_kinds, dm.n_params, phs, st));
  WM_TIMED(TK_TREES, st, launch_score_trees(forest->df, zTo, dm.d, phs, phi_dim, B, hw, n_hw, dm.hw_dim, sc, st));
  WM_TIMED(TK_TOPK, st, launch_topk(sc, n_hw, B, seg, k, idx, val, st));
  return ok();
}

size_t wm_loss_workspace_bytes(const wm_model* model, int32_t B, int32_t T_max) {
  if (!model || B < 0 || T_max < 0 || T_max > WM_MAX_T) return 0;
  return loss_layout(model->dm, B, T_max).total;
}

wm_status wm_rollout_loss(const wm_model* model, const float* z0, const int32_t* seg_off, int32_t S,
                          const int32_t* types, const int32_t* params, const int32_t* lens,
                          int32_t B, int32_t T_max, const float* targets, const float* negatives,
                          int32_t n_neg, float lam, float gamma, float* loss, float* total,
                          const wm_grads* grads, void* ws, size_t ws_bytes, void* stream) {
  wm_status s = check_rollout_args(model, z0, types, params, lens, B, T_max, reinterpret_cast<float*>(1));
  if (s != WM_OK) return s;
  const DevModel& m = model->dm;
  const bool l2 = m.dims.norm == WM_NORM_L2;
  if (!have_train_kernels(m.prec, m.dims.d, m.dims.embed_dim) || !m.trans_w1t || !m.trans_w2t ||
      (l2 && !m.trans_wht))
    return fail(WM_ERR_UNSUPPORTED, "no rollout-loss kernels for this (precision, d, embed_dim)");
  if (n_neg < 1) return fail(WM_ERR_INVALID_ARGUMENT, "n_neg must be >= 1");
  if (!std::isfinite(lam) || !std::isfinite(gamma)) return fail(WM_ERR_INVALID_ARGUMENT, "lam and gamma must be finite");
  SegTable seg;
  int32_t min_seg = 0;
  if ((s = check_segments(seg_off, S, B, &seg, &min_seg)) != WM_OK) return s;
  if (!loss) return fail(WM_ERR_INVALID_ARGUMENT, "loss is NULL");
  if (B > 0 && T_max > 0 && (!targets || !negatives))
    return fail(WM_ERR_INVALID_ARGUMENT, "targets/negatives is NULL");
  if (grads && (!grads->w1 || !grads->b1 || !grads->w2 || !grads->b2 || !grads->type_emb ||
                !grads->param_w || !grads->param_b || (l2 && !grads->wh)))
    return fail(WM_ERR_INVALID_ARGUMENT, "null gradient pointer");
  if (!ws) return fail(WM_ERR_INVALID_ARGUMENT, "workspace is NULL");
  const LossLayout L = loss_layout(m, B, T_max);
  if (ws_bytes < L.total) return fail(WM_ERR_INVALID_ARGUMENT, "workspace too small");

  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* w8 = static_cast<uint8_t*>(ws);
  auto fptr = [&](size_t off) { return reinterpret_cast<float*>(w8 + off); };
  TrainIO io;
  io.z0 = z0; io.perm = reinterpret_cast<int2*>(w8 + L.perm); io.types = types; io.params = params;
  io.lens = lens; io.off = reinterpret_cast<int32_t*>(w8 + L.off);
  io.row_src = reinterpret_cast<int32_t*>(w8 + L.row_src);
  io.X = fptr(L.X); io.A = fptr(L.A); io.G = fptr(L.G); io.P = fptr(L.P);
  io.SD = fptr(L.SD); io.DE = fptr(L.DE); io.dz0 = grads ? grads->z0 : nullptr;
  io.V = l2 ? fptr(L.V) : nullptr; io.SC = l2 ? fptr(L.SC) : nullptr; io.DV = l2 ? fptr(L.DV) : nullptr;
  io.err = reinterpret_cast<int32_t*>(w8 + L.err); io.B = B; io.T_max = T_max;
  if (B > 0) {
    WM_TIMED(TK_BUCKET, st, launch_bucket(lens, B, T_max, seg, const_cast<int2*>(io.perm),
                                          reinterpret_cast<int32_t*>(w8 + L.hist), io.err, st));
    WM_TIMED(TK_BUCKET, st, launch_row_offsets(lens, B, T_max, io.off, st));
    WM_TIMED(TK_TRAIN_FWD, st, launch_train_fwd(m, io, st));
  } else {
    WM_TIMED(TK_BUCKET, st, launch_row_offsets(lens, 0, T_max, io.off, st));
  }
  WM_TIMED(TK_LOSS, st, launch_step_loss(io.P, targets, negatives, n_neg, lens, io.off, B, T_max,
                                          m.dims.d, lam, gamma, io.SD, fptr(L.lrow), loss, total, st));
  if (!grads) return ok();
  if (B > 0) WM_TIMED(TK_TRAIN_BWD, st, launch_train_bwd(m, io, st));
  GradParts gp;
  gp.w1 = fptr(L.pw1); gp.w2 = fptr(L.pw2); gp.b1 = fptr(L.pb1); gp.b2 = fptr(L.pb2);
  gp.emb = fptr(L.pemb); gp.wh = l2 ? fptr(L.pwh) : nullptr;
  gp.splits = L.splits; gp.emb_blocks = L.emb_blocks;
  WM_TIMED(TK_GRADS, st, launch_weight_grads(m, io, gp, grads->w1, grads->b1, grads->w2, grads->b2,
                                             grads->type_emb, grads->param_w, grads->param_b,
                                             l2 ? grads->wh : nullptr, st));
  return ok();
}

wm_status wm_device_status(void* ws, size_t ws_bytes, void* stream) {
  if (!ws || ws_bytes < 256) return fail(WM_ERR_INVALID_ARGUMENT, "workspace is NULL or too small");
  hipStream_t st = static_cast<hipStream_t>(stream);
  WM_HIP_TRY(hipStreamSynchronize(st));
  int32_t word = 0;
  WM_HIP_TRY(hipMemcpy(&word, ws, sizeof(word), hipMemcpyDeviceToHost));
  if (word == 0) return ok();
  WM_HIP_TRY(hipMemset(ws, 0, sizeof(word)));
  std::string msg = "input out of range:";
  if (word & ERRBIT_LEN) msg += " a length outside [0, T_max];";
  if (word & ERRBIT_TYPE) msg += " an action type outside [0, n_kinds);";
  if (word & ERRBIT_PARAM) msg += " an action parameter < 1;";
  if (word & ERRBIT_TOKEN) msg += " a token id outside [0, vocab);";
  return fail(WM_ERR_INPUT_RANGE, msg);
}

wm_status wm_timing_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  g_timing.on = on != 0;
  for (int k = 0; k < TK_COUNT; ++k) g_timing.count[k] = 0;
  return ok();
}

wm_status wm_timing_read(int32_t kernel, double* total_ms, int64_t* launches) {
  if (kernel < 0 || kernel >= TK_COUNT || !total_ms || !launches)
    return fail(WM_ERR_INVALID_ARGUMENT, "bad timing query");
  std::lock_guard<std::mutex> lk(g_timing.mu);
  double tot = 0.0;
  const int n = g_timing.count[kernel];
  for (int i = 0; i < n; ++i) {
    WM_HIP_TRY(hipEventSynchronize(g_timing.stop[kernel][i]));
    float ms = 0.0f;
    WM_HIP_TRY(hipEventElapsedTime(&ms, g_timing.start[kernel][i], g_timing.stop[kernel][i]));
    tot += ms;
  }
  *total_ms = tot;
  *launches = n;
  return ok();
}

}  // extern "C"
