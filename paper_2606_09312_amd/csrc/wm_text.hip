// Chunked transformer state encoder (Sec. 3.3): sliding-window chunks of
// each program's token sequence, a post-LayerNorm transformer backbone of the
// CodeBERT (RoBERTa) shape on every chunk, masked mean pooling per chunk, the
// mean over a program's chunks, and a linear projection head to the latent.
//
// All chunks of all programs are one batch of rows r = c * window + p (chunk
// c, position p; positions past a chunk's tokens are padding: never pooled,
// masked as attention keys).  Dense products run in one LDS-tiled
// matrix-core kernel (128 x 128 output tiles, 32-deep stages, operands
// rounded as product operands while they are staged); attention is the same
// kernel batched over (chunk, head) for the scores and for probabilities x
// values, with a row softmax in between.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <type_traits>
#include <vector>

#include "wm_internal.h"

using namespace wm;

struct wm_text_model {
  wm_text_dims dims;
  uint8_t* base;
  const float *tok_emb, *pos_emb, *ln0_g, *ln0_b;
  const float *wqkv, *bqkv, *wo, *bo, *ln1_g, *ln1_b, *w1, *b1, *w2, *b2, *ln2_g, *ln2_b;
  const float *wp, *bp;
  const __bf16 *wqkv16, *wo16, *w116, *w216;   // WM_BF16: the layer matrices as bf16
};

namespace wm {
namespace text {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float LN_EPS = 1e-5f;

// Matrix-core products of the two precisions (32 x 32 output, 16 or 2 deep).
struct BF {
  static constexpr int KF = 16, SL = 8;
  using Elem = __bf16;
  using Frag = bf16x8;
  static __device__ __forceinline__ f32x16 mfma(Frag a, Frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
struct FP {
  static constexpr int KF = 2, SL = 1;
  using Elem = float;
  using Frag = float;
  static __device__ __forceinline__ f32x16 mfma(Frag a, Frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x = fmaxf(x, __shfl_xor(x, m));
  return x;
}

// GELU(x) = x Phi(x) with erf from Abramowitz & Stegun 7.1.26 (|error| <=
// 1.5e-7), the same form as the evaluator's kernels.
__device__ __forceinline__ float gelu(float x) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f * 0.70710678118654752f, ax, 1.0f));
  float p = fmaf(1.061405429f, t, -1.453152027f);
  p = fmaf(p, t, 1.421413741f);
  p = fmaf(p, t, -0.284496736f);
  p = fmaf(p, t, 0.254829592f);
  const float ex = __builtin_amdgcn_exp2f((x * x) * (-0.5f * 1.4426950408889634f));
  const float erf_a = fmaf(-(p * t), ex, 1.0f);
  return 0.5f * fmaf(ax, erf_a, x);
}

// Programs and their chunks (host-built, passed by value).
struct TTable {
  int32_t S;
  int32_t chunk_off[WM_TEXT_MAX_PROGRAMS + 1];   // first chunk of each program
  int32_t tok_off[WM_TEXT_MAX_PROGRAMS + 1];     // first token of each program
};

__device__ __forceinline__ int program_of(const TTable& tt, int c) {
  int lo = 0, hi = tt.S - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (tt.chunk_off[mid] <= c) lo = mid; else hi = mid - 1;
  }
  return lo;
}
// First token and token count of chunk c.
__device__ __forceinline__ void chunk_span(const TTable& tt, int c, int window, int stride,
                                           int& first, int& len) {
  const int s = program_of(tt, c);
  first = tt.tok_off[s] + (c - tt.chunk_off[s]) * stride;
  len = min(window, tt.tok_off[s + 1] - first);
}

// ---------------------------------------------------------------------------
// h[r] = LN(tok_emb[id] + pos_emb[p]); padding rows are zero.  One wavefront
// per row, lanes over the features.
constexpr int LN_MAX_PER_LANE = 16;               // hidden <= 1024

__global__ __launch_bounds__(256) void embed_ln_kernel(const int32_t* __restrict__ tokens,
                                                       const TTable tt, int window, int stride,
                                                       const float* __restrict__ tok_emb,
                                                       const float* __restrict__ pos_emb,
                                                       const float* __restrict__ g,
                                                       const float* __restrict__ b, int H, int vocab,
                                                       int rows, float* __restrict__ h,
                                                       __bf16* __restrict__ hb, int32_t* err) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int c = r / window, p = r - c * window;
  int first, len;
  chunk_span(tt, c, window, stride, first, len);
  float* out = h + (size_t)r * H;
  if (p >= len) {
    for (int f = lane; f < H; f += 64) {
      out[f] = 0.0f;
      if (hb) hb[(size_t)r * H + f] = (__bf16)0.0f;
    }
    return;
  }
  int id = tokens[first + p];
  if (id < 0 || id >= vocab) {
    if (lane == 0) atomicOr(err, ERRBIT_TOKEN);
    id = 0;
  }
  float x[LN_MAX_PER_LANE];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < LN_MAX_PER_LANE; ++i) {
    const int f = lane + 64 * i;
    x[i] = f < H ? tok_emb[(size_t)id * H + f] + pos_emb[(size_t)p * H + f] : 0.0f;
    s += x[i];
  }
  const float mean = wave_sum(s) / (float)H;
  float v = 0.0f;
#pragma unroll
  for (int i = 0; i < LN_MAX_PER_LANE; ++i) {
    const int f = lane + 64 * i;
    if (f < H) v = fmaf(x[i] - mean, x[i] - mean, v);
  }
  const float rs = rsqrtf(wave_sum(v) / (float)H + LN_EPS);
#pragma unroll
  for (int i = 0; i < LN_MAX_PER_LANE; ++i) {
    const int f = lane + 64 * i;
    if (f < H) {
      const float o = (x[i] - mean) * rs * g[f] + b[f];
      out[f] = o;
      if (hb) hb[(size_t)r * H + f] = (__bf16)o;
    }
  }
}

// h[r] = LN(y[r]) (the residual sum is formed by the product's epilogue).
__global__ __launch_bounds__(256) void ln_kernel(const float* __restrict__ y,
                                                 const float* __restrict__ g,
                                                 const float* __restrict__ b, int H, int rows,
                                                 float* __restrict__ h, __bf16* __restrict__ hb) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const float* in = y + (size_t)r * H;
  float x[LN_MAX_PER_LANE];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < LN_MAX_PER_LANE; ++i) {
    const int f = lane + 64 * i;
    x[i] = f < H ? in[f] : 0.0f;
    s += x[i];
  }
  const float mean = wave_sum(s) / (float)H;
  float v = 0.0f;
#pragma unroll
  for (int i = 0; i < LN_MAX_PER_LANE; ++i) {
    const int f = lane + 64 * i;
    if (f < H) v = fmaf(x[i] - mean, x[i] - mean, v);
  }
  const float rs = rsqrtf(wave_sum(v) / (float)H + LN_EPS);
  float* out = h + (size_t)r * H;
#pragma unroll
  for (int i = 0; i < LN_MAX_PER_LANE; ++i) {
    const int f = lane + 64 * i;
    if (f < H) {
      const float o = (x[i] - mean) * rs * g[f] + b[f];
      out[f] = o;
      if (hb) hb[(size_t)r * H + f] = (__bf16)o;
    }
  }
}

// ---------------------------------------------------------------------------
// Batched product  C[b] = epi(alpha * A[b] . op(B[b])^T)  with
//   A[b](m, k) = A[offA(b) + m lda + k]
//   B[b](n, k) = B[offB(b) + n ldb + k]          (BT = false)
//              = B[offB(b) + k ldb + n]          (BT = true: stored k-major)
//   off(b) = (b / bdiv) s1 + (b % bdiv) s2
//   epi: + bias[n], then GELU, then + R[offC(b) + m ldr + n] (each optional)
// Workgroup = 4 wavefronts on a 128 x 128 output tile (2 x 2 matrix-core
// tiles each); 32-deep stages staged in LDS with rows of the contraction
// contiguous (one 16-byte LDS read per operand fragment); the next stage's
// loads are in flight during the current stage's products.
struct GemmArgs {
  const float* A;
  const float* B;
  float* C;
  const float* bias;
  const float* res;
  int M, N, K, lda, ldb, ldc, ldr, bdiv, tiles_n;
  long long sA1, sA2, sB1, sB2, sC1, sC2;
  float alpha;
  int gelu;
};
constexpr int GT = 128, GK = 32;

template <class PR, bool BT>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmArgs g) {
  using Elem = typename PR::Elem;
  using Frag = typename PR::Frag;
  constexpr bool BFM = std::is_same<PR, BF>::value;
  constexpr int KF = PR::KF, SL = PR::SL;
  constexpr int LDW = GK + (BFM ? 8 : 4);
  __shared__ __attribute__((aligned(16))) Elem As[GT * LDW];
  __shared__ __attribute__((aligned(16))) Elem Bs[GT * LDW];
  const int bidx = blockIdx.y;
  const long long offA = (long long)(bidx / g.bdiv) * g.sA1 + (long long)(bidx % g.bdiv) * g.sA2;
  const long long offB = (long long)(bidx / g.bdiv) * g.sB1 + (long long)(bidx % g.bdiv) * g.sB2;
  const long long offC = (long long)(bidx / g.bdiv) * g.sC1 + (long long)(bidx % g.bdiv) * g.sC2;
  const float* A = g.A + offA;
  const float* B = g.B + offB;
  const int m0 = (blockIdx.x / g.tiles_n) * GT, n0 = (blockIdx.x % g.tiles_n) * GT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // loaders: row-major operands by (row, 16-deep half), k-major B by (column, 16-deep half)
  const int lr = tid >> 1, lk = (tid & 1) * 16;
  const int bc = tid & (GT - 1), bk = (tid >> 7) * 16;
  float va[16], vb[16];
  auto load = [&](int k0) {
    const bool okA = m0 + lr < g.M;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 x = okA ? *reinterpret_cast<const f32x4*>(A + (size_t)(m0 + lr) * g.lda + k0 + lk + 4 * q)
                          : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int i = 0; i < 4; ++i) va[4 * q + i] = x[i];
    }
    if constexpr (!BT) {
      const bool okB = n0 + lr < g.N;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x4 x = okB ? *reinterpret_cast<const f32x4*>(B + (size_t)(n0 + lr) * g.ldb + k0 + lk + 4 * q)
                            : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int i = 0; i < 4; ++i) vb[4 * q + i] = x[i];
      }
    } else {
      const bool okB = n0 + bc < g.N;
#pragma unroll
      for (int j = 0; j < 16; ++j) vb[j] = okB ? B[(size_t)(k0 + bk + j) * g.ldb + n0 + bc] : 0.0f;
    }
  };
  auto store = [&]() {
    Elem* da = As + lr * LDW + lk;
    Elem* db = BT ? Bs + bc * LDW + bk : Bs + lr * LDW + lk;
    if constexpr (BFM) {
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        bf16x8 ea, eb;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          ea[j] = (__bf16)va[8 * h2 + j];
          eb[j] = (__bf16)vb[8 * h2 + j];
        }
        *reinterpret_cast<bf16x8*>(da + 8 * h2) = ea;
        *reinterpret_cast<bf16x8*>(db + 8 * h2) = eb;
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        *reinterpret_cast<f32x4*>(da + 4 * q) = f32x4{va[4 * q], va[4 * q + 1], va[4 * q + 2], va[4 * q + 3]};
        *reinterpret_cast<f32x4*>(db + 4 * q) = f32x4{vb[4 * q], vb[4 * q + 1], vb[4 * q + 2], vb[4 * q + 3]};
      }
    }
  };

  const int wm = wave & 1, wn = wave >> 1;
  const int cl = lane & 31, h = lane >> 5;
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  load(0);
  for (int k0 = 0; k0 < g.K; k0 += GK) {
    __syncthreads();
    store();
    __syncthreads();
    if (k0 + GK < g.K) load(k0 + GK);
#pragma unroll
    for (int ks = 0; ks < GK / KF; ++ks) {
      Frag fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const Elem* pa = As + (wm * 64 + i * 32 + cl) * LDW + ks * KF + h * SL;
        const Elem* pb = Bs + (wn * 64 + i * 32 + cl) * LDW + ks * KF + h * SL;
        fa[i] = *reinterpret_cast<const Frag*>(pa);
        fb[i] = *reinterpret_cast<const Frag*>(pb);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = PR::mfma(fa[i], fb[j], acc[i][j]);
    }
  }
  float* C = g.C + offC;
  const float* R = g.res ? g.res + offC : nullptr;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn * 64 + j * 32 + cl;
      if (n >= g.N) continue;
      const float bn = g.bias ? g.bias[n] : 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * 64 + i * 32 + acc_row(h, r);
        if (m >= g.M) continue;
        float v = fmaf(acc[i][j][r], g.alpha, bn);
        if (g.gelu) v = gelu(v);
        if (R) v += R[(size_t)m * g.ldr + n];
        C[(size_t)m * g.ldc + n] = v;
      }
    }
}

// bf16 dense product with operands stored as bf16 (the product-operand
// values themselves):  C = epi(A . W^T), A [M][K] and W [N][K] row-major,
// epilogue + bias[n], GELU, + residual R[m][n] (fp32), C fp32 or bf16.
// Workgroup = 8 wavefronts on a 256 x 128 tile (each 64 x 64, 2 x 2
// matrix-core tiles); 32-deep stages, 16-byte loads straight into LDS rows
// (contraction contiguous), the next stage's loads in flight meanwhile.
struct Gemm16Args {
  const __bf16* A;
  const __bf16* W;
  void* C;
  const float* bias;
  const float* res;
  int M, N, K, tiles_n, gelu;
};
constexpr int G16_BM = 256, G16_BN = 128, G16_LDW = GK + 8;

template <bool OUT16>
__global__ __launch_bounds__(512) void gemm16_kernel(const Gemm16Args g) {
  __shared__ __attribute__((aligned(16))) __bf16 As[G16_BM * G16_LDW];
  __shared__ __attribute__((aligned(16))) __bf16 Bs[G16_BN * G16_LDW];
  const int m0 = (blockIdx.x / g.tiles_n) * G16_BM, n0 = (blockIdx.x % g.tiles_n) * G16_BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // A: 2 units of 8 bf16 per thread, B: 1 unit
  bf16x8 ra[2], rb;
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int u = tid + 512 * i, row = u >> 2, q = u & 3;
      ra[i] = m0 + row < g.M ? *reinterpret_cast<const bf16x8*>(g.A + (size_t)(m0 + row) * g.K + k0 + 8 * q)
                             : bf16x8{};
    }
    const int row = tid >> 2, q = tid & 3;
    rb = n0 + row < g.N ? *reinterpret_cast<const bf16x8*>(g.W + (size_t)(n0 + row) * g.K + k0 + 8 * q)
                        : bf16x8{};
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int u = tid + 512 * i, row = u >> 2, q = u & 3;
      *reinterpret_cast<bf16x8*>(As + row * G16_LDW + 8 * q) = ra[i];
    }
    const int row = tid >> 2, q = tid & 3;
    *reinterpret_cast<bf16x8*>(Bs + row * G16_LDW + 8 * q) = rb;
  };
  const int wm = wave & 3, wn = wave >> 2;
  const int cl = lane & 31, h = lane >> 5;
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  load(0);
  for (int k0 = 0; k0 < g.K; k0 += GK) {
    __syncthreads();
    store();
    __syncthreads();
    if (k0 + GK < g.K) load(k0 + GK);
#pragma unroll
    for (int ks = 0; ks < GK / 16; ++ks) {
      bf16x8 fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        fa[i] = *reinterpret_cast<const bf16x8*>(As + (wm * 64 + i * 32 + cl) * G16_LDW + ks * 16 + h * 8);
        fb[i] = *reinterpret_cast<const bf16x8*>(Bs + (wn * 64 + i * 32 + cl) * G16_LDW + ks * 16 + h * 8);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = BF::mfma(fa[i], fb[j], acc[i][j]);
    }
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn * 64 + j * 32 + cl;
      if (n >= g.N) continue;
      const float bn = g.bias ? g.bias[n] : 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * 64 + i * 32 + acc_row(h, r);
        if (m >= g.M) continue;
        float v = acc[i][j][r] + bn;
        if (g.gelu) v = gelu(v);
        if (g.res) v += g.res[(size_t)m * g.N + n];
        if constexpr (OUT16) reinterpret_cast<__bf16*>(g.C)[(size_t)m * g.N + n] = (__bf16)v;
        else reinterpret_cast<float*>(g.C)[(size_t)m * g.N + n] = v;
      }
    }
}

// Row softmax of the attention scores, keys past the chunk's tokens masked.
// One wavefront per row (chunk c, head, query); in place.
constexpr int SM_MAX_PER_LANE = 16;               // window <= 1024
__global__ __launch_bounds__(256) void softmax_kernel(float* __restrict__ s, const TTable tt,
                                                      int window, int stride, int heads,
                                                      long long rows) {
  const int lane = threadIdx.x & 63;
  const long long r = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int c = (int)(r / ((long long)heads * window));
  int first, len;
  chunk_span(tt, c, window, stride, first, len);
  float* row = s + r * window;
  float x[SM_MAX_PER_LANE];
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < SM_MAX_PER_LANE; ++i) {
    const int k = lane + 64 * i;
    x[i] = (k < window && k < len) ? row[k] : -INFINITY;
    mx = fmaxf(mx, x[i]);
  }
  mx = wave_max(mx);
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < SM_MAX_PER_LANE; ++i) {
    x[i] = x[i] == -INFINITY ? 0.0f : __expf(x[i] - mx);
    sum += x[i];
  }
  const float inv = 1.0f / wave_sum(sum);
#pragma unroll
  for (int i = 0; i < SM_MAX_PER_LANE; ++i) {
    const int k = lane + 64 * i;
    if (k < window) row[k] = x[i] * inv;
  }
}

// Fused attention of one (chunk, head) per workgroup, bf16: wavefront w
// takes queries [32 w, 32 w + 32).  K and V of the chunk are staged in LDS
// once (K row-major, V transposed with its keys permuted into accumulator
// order); the scores are computed transposed, S^T = K . Q^T, so a query is a
// lane's column and its softmax statistics are per-lane sums completed across
// the lane pair (L, L^32).  Pass 1 forms the row maximum and sum online over
// 32-key blocks; pass 2 recomputes the scores, normalises them (the
// probabilities exactly as defined, rounded as product operands) and
// accumulates O^T = V^T . P with P straight from the accumulators (its key
// order is the one V was permuted into).
template <int DH>
__global__ __launch_bounds__(1024) void attention_kernel(const __bf16* __restrict__ qkv,
                                                         __bf16* __restrict__ ctx, const TTable tt,
                                                         int window, int stride, int heads, int H,
                                                         float scale) {
  constexpr int KS = DH / 16;                 // 16-deep steps over the head width
  constexpr int DB = DH / 32;                 // 32-row blocks of the head width
  constexpr int KW = DH + 8;                  // padded K row (bf16)
  extern __shared__ __attribute__((aligned(16))) __bf16 lds_att[];
  const int VW = window + 8;                  // padded V^T row (bf16)
  __bf16* Ks = lds_att;                       // [window][KW]
  __bf16* Vt = lds_att + (size_t)window * KW; // [DH][VW]
  const int c = blockIdx.x / heads, head = blockIdx.x % heads;
  int first, len;
  chunk_span(tt, c, window, stride, first, len);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nt = blockDim.x;
  const int cl = lane & 31, h = lane >> 5;
  const __bf16* base = qkv + (size_t)c * window * 3 * H + head * DH;
  const int nkb = (len + 31) / 32;

  // stage K (row-major) and V (transposed, keys in accumulator order per block)
  for (int u = tid; u < nkb * 32 * (DH / 8); u += nt) {
    const int key = u / (DH / 8), d8 = (u % (DH / 8)) * 8;
    bf16x8 kv = {}, vv = {};
    if (key < len) {
      kv = *reinterpret_cast<const bf16x8*>(base + (size_t)key * 3 * H + H + d8);
      vv = *reinterpret_cast<const bf16x8*>(base + (size_t)key * 3 * H + 2 * H + d8);
    }
    *reinterpret_cast<bf16x8*>(Ks + key * KW + d8) = kv;
    // key = 32 kb + acc_row(hh, 8 f + j)  ->  position 32 kb + 16 f + 8 hh + j
    const int kb = key >> 5, kr = key & 31;
    const int hh = (kr >> 2) & 1, rr = ((kr >> 3) << 2) | (kr & 3);
    const int pos = kb * 32 + (rr >> 3) * 16 + hh * 8 + (rr & 7);
#pragma unroll
    for (int i = 0; i < 8; ++i) Vt[(d8 + i) * VW + pos] = vv[i];
  }
  // this wavefront's queries as B operands: Q[q][16 kk + 8 h + j]
  const int q = wave * 32 + cl;
  bf16x8 qf[KS];
  {
    const __bf16* qrow = base + (size_t)min(q, window - 1) * 3 * H;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) qf[kk] = *reinterpret_cast<const bf16x8*>(qrow + 16 * kk + 8 * h);
  }
  __syncthreads();
  if (wave * 32 >= len) return;               // no valid query in this wavefront

  auto scores = [&](int kb) -> f32x16 {
    f32x16 sacc = {};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const bf16x8 kfrag = *reinterpret_cast<const bf16x8*>(Ks + (kb * 32 + cl) * KW + 16 * kk + 8 * h);
      sacc = BF::mfma(kfrag, qf[kk], sacc);
    }
    return sacc;
  };
  // pass 1: running maximum and sum of exp over the valid keys
  float mx = -INFINITY, sum = 0.0f;
  for (int kb = 0; kb < nkb; ++kb) {
    const f32x16 sacc = scores(kb);
    float bm = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (kb * 32 + acc_row(h, r) < len) bm = fmaxf(bm, sacc[r] * scale);
    const float nm = fmaxf(mx, bm);
    float bs = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (kb * 32 + acc_row(h, r) < len) bs += __expf(sacc[r] * scale - nm);
    sum = (mx == -INFINITY ? 0.0f : sum * __expf(mx - nm)) + bs;
    mx = nm;
  }
  {
    const float mo = __shfl_xor(mx, 32), so = __shfl_xor(sum, 32);
    const float m2 = fmaxf(mx, mo);
    sum = (mx == -INFINITY ? 0.0f : sum * __expf(mx - m2)) + (mo == -INFINITY ? 0.0f : so * __expf(mo - m2));
    mx = m2;
  }
  const float inv = 1.0f / sum;
  // pass 2: probabilities and O^T = V^T . P
  f32x16 oacc[DB];
#pragma unroll
  for (int b = 0; b < DB; ++b) oacc[b] = f32x16{};
  for (int kb = 0; kb < nkb; ++kb) {
    const f32x16 sacc = scores(kb);
    bf16x8 pf[2];
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int r = 8 * f + j;
        const float pv = kb * 32 + acc_row(h, r) < len ? __expf(sacc[r] * scale - mx) * inv : 0.0f;
        pf[f][j] = (__bf16)pv;
      }
#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
      for (int f = 0; f < 2; ++f) {
        const bf16x8 vfrag = *reinterpret_cast<const bf16x8*>(Vt + (b * 32 + cl) * VW + kb * 32 + 16 * f + 8 * h);
        oacc[b] = BF::mfma(vfrag, pf[f], oacc[b]);
      }
  }
  if (q < window) {             // the output as the next product's operand
    __bf16* orow = ctx + ((size_t)c * window + q) * H + head * DH;
#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) orow[32 * b + acc_row(h, r)] = (__bf16)oacc[b][r];
  }
}

// Mean of each chunk's rows over its tokens.  One workgroup per chunk.
// Masked mean over a chunk's tokens: one workgroup per chunk; thread t sums
// the feature quad t % (H/4) over the tokens p = t / (H/4) + k G (G token
// groups, 16-byte loads), then the G partial sums are added in group order.
constexpr int POOL_THREADS = 1024;
__global__ __launch_bounds__(POOL_THREADS) void pool_kernel(const float* __restrict__ h, const TTable tt,
                                                            int window, int stride, int H,
                                                            float* __restrict__ pooled) {
  typedef float f4 __attribute__((ext_vector_type(4)));
  __shared__ f4 part[POOL_THREADS];
  const int c = blockIdx.x, tid = threadIdx.x;
  int first, len;
  chunk_span(tt, c, window, stride, first, len);
  const float inv = 1.0f / (float)len;
  const int nq = H / 4, groups = POOL_THREADS / nq;        // H <= 1024: at least 4 groups
  const int q = tid % nq, grp = tid / nq;
  f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  if (grp < groups) {
    const f4* base = reinterpret_cast<const f4*>(h + (size_t)c * window * H) + q;
    for (int p = grp; p < len; p += groups) acc += base[(size_t)p * nq];
  }
  part[tid] = acc;
  __syncthreads();
  if (tid < nq) {
    f4 t = part[tid];
    for (int g2 = 1; g2 < groups; ++g2) t += part[g2 * nq + tid];
    *reinterpret_cast<f4*>(pooled + (size_t)c * H + 4 * tid) = t * inv;
  }
}

// Program vector (mean of its chunk vectors; zero for an empty program, as
// a product operand) and z = Wp v + bp.  One workgroup per program.
__global__ __launch_bounds__(256) void project_kernel(const float* __restrict__ pooled,
                                                      const TTable tt, int H, int d,
                                                      const float* __restrict__ wp,
                                                      const float* __restrict__ bp, int bf16,
                                                      float* __restrict__ z) {
  extern __shared__ float v[];
  const int s = blockIdx.x;
  const int c0 = tt.chunk_off[s], c1 = tt.chunk_off[s + 1];
  const float inv = c1 > c0 ? 1.0f / (float)(c1 - c0) : 0.0f;
  for (int f = threadIdx.x; f < H; f += blockDim.x) {
    float a = 0.0f;
    for (int c = c0; c < c1; ++c) a += pooled[(size_t)c * H + f];
    a *= inv;
    v[f] = bf16 ? (float)(__bf16)a : a;
  }
  __syncthreads();
  for (int o = threadIdx.x; o < d; o += blockDim.x) {
    float a = bp[o];
    for (int f = 0; f < H; ++f) a = fmaf(wp[(size_t)o * H + f], v[f], a);
    z[(size_t)s * d + o] = a;
  }
}

}  // namespace text
}  // namespace wm

using namespace wm::text;

namespace {

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

int n_chunks_of(int n_tokens, int window, int stride) {
  if (n_tokens <= 0) return 0;
  if (n_tokens <= window) return 1;
  return 1 + (n_tokens - window + stride - 1) / stride;
}

// bf16 with a fused-attention head width and window: operands stored as bf16
bool bf16_path(const wm_text_dims& d) {
  const int dh = d.hidden / d.heads;
  return d.precision == WM_BF16 && (dh == 32 || dh == 64) && d.window <= 512;
}

struct TextLayout {
  size_t err, h, qkv, sc, ctx, y, f, pooled, hb, qkvb, ctxb, fb, total;
};

TextLayout text_layout(const wm_text_dims& dm, int n_chunks) {
  const size_t rows = (size_t)n_chunks * dm.window, H = dm.hidden;
  const bool bf = bf16_path(dm);
  TextLayout L;
  size_t o = 0;
  L.err = o; o += 256;
  L.h = o; o = al256(o + rows * H * 4);
  L.qkv = o; o = al256(o + (bf ? 0 : rows * 3 * H * 4));
  L.sc = o; o = al256(o + (bf ? 0 : (size_t)n_chunks * dm.heads * dm.window * dm.window * 4));
  L.ctx = o; o = al256(o + (bf ? 0 : rows * H * 4));
  L.y = o; o = al256(o + rows * H * 4);
  L.f = o; o = al256(o + (bf ? 0 : rows * (size_t)dm.ffn * 4));
  L.pooled = o; o = al256(o + (size_t)n_chunks * H * 4);
  // bf16: the product operands (the fp32 qkv, scores, context and hidden
  // buffers above are then unused and sized zero)
  L.hb = o; o = al256(o + (bf ? rows * H * 2 : 0));
  L.qkvb = o; o = al256(o + (bf ? rows * 3 * H * 2 : 0));
  L.ctxb = o; o = al256(o + (bf ? rows * H * 2 : 0));
  L.fb = o; o = al256(o + (bf ? rows * (size_t)dm.ffn * 2 : 0));
  L.total = o;
  return L;
}

template <class PR>
hipError_t launch_gemm(const GemmArgs& g0, int batch, bool bt, hipStream_t st) {
  GemmArgs g = g0;
  g.tiles_n = (g.N + GT - 1) / GT;
  const dim3 grid(((g.M + GT - 1) / GT) * g.tiles_n, batch);
  if (bt) hipLaunchKernelGGL((gemm_kernel<PR, true>), grid, dim3(256), 0, st, g);
  else hipLaunchKernelGGL((gemm_kernel<PR, false>), grid, dim3(256), 0, st, g);
  return hipGetLastError();
}

GemmArgs dense(const float* A, int M, int K, const float* W, int N, float* C, const float* bias,
               const float* res, int gelu) {
  GemmArgs g{};
  g.A = A; g.B = W; g.C = C; g.bias = bias; g.res = res;
  g.M = M; g.N = N; g.K = K; g.lda = K; g.ldb = K; g.ldc = N; g.ldr = N; g.bdiv = 1;
  g.alpha = 1.0f; g.gelu = gelu;
  return g;
}

}  // namespace

extern "C" {

wm_status wm_text_model_create(const wm_text_dims* dims, const wm_text_weights* w, wm_text_model** out) {
  if (!dims || !w || !out) return set_error(WM_ERR_INVALID_ARGUMENT, "null argument");
  *out = nullptr;
  const wm_text_dims& d = *dims;
  if (d.vocab < 1 || d.hidden < 1 || d.heads < 1 || d.ffn < 1 || d.layers < 0 || d.window < 1 ||
      d.stride < 1 || d.stride > d.window || d.d < 1)
    return set_error(WM_ERR_INVALID_ARGUMENT, "dims must be positive with 1 <= stride <= window");
  if (d.precision != WM_FP32 && d.precision != WM_BF16)
    return set_error(WM_ERR_INVALID_ARGUMENT, "unknown precision");
  if (d.hidden % d.heads || (d.hidden / d.heads) % 32 || d.hidden % 32 || d.ffn % 32 || d.window % 32 ||
      d.hidden > 64 * LN_MAX_PER_LANE || d.window > 64 * SM_MAX_PER_LANE)
    return set_error(WM_ERR_UNSUPPORTED,
                     "need hidden, ffn, window and the head width multiples of 32, hidden <= 1024, window <= 1024");
  const float* req[] = {w->tok_emb, w->pos_emb, w->ln0_g, w->ln0_b, w->wp, w->bp};
  for (const float* p : req)
    if (!p) return set_error(WM_ERR_INVALID_ARGUMENT, "null weight pointer");
  if (d.layers > 0) {
    const float* lreq[] = {w->wqkv, w->bqkv, w->wo, w->bo, w->ln1_g, w->ln1_b, w->w1, w->b1, w->w2,
                           w->b2, w->ln2_g, w->ln2_b};
    for (const float* p : lreq)
      if (!p) return set_error(WM_ERR_INVALID_ARGUMENT, "null layer weight pointer");
  }
  const size_t H = d.hidden, F = d.ffn, L = d.layers;
  const bool bf = d.precision == WM_BF16;
  auto rnd = [&](float v) {
    if (!bf) return v;
    return (float)(__bf16)v;
  };
  struct Part { const float* src; size_t n; bool matrix; size_t off; };
  std::vector<Part> parts = {
      {w->tok_emb, (size_t)d.vocab * H, false, 0}, {w->pos_emb, (size_t)d.window * H, false, 0},
      {w->ln0_g, H, false, 0}, {w->ln0_b, H, false, 0},
      {w->wqkv, L * 3 * H * H, true, 0}, {w->bqkv, L * 3 * H, false, 0},
      {w->wo, L * H * H, true, 0}, {w->bo, L * H, false, 0},
      {w->ln1_g, L * H, false, 0}, {w->ln1_b, L * H, false, 0},
      {w->w1, L * F * H, true, 0}, {w->b1, L * F, false, 0},
      {w->w2, L * H * F, true, 0}, {w->b2, L * H, false, 0},
      {w->ln2_g, L * H, false, 0}, {w->ln2_b, L * H, false, 0},
      {w->wp, (size_t)d.d * H, true, 0}, {w->bp, (size_t)d.d, false, 0}};
  size_t total = 0;
  for (auto& p : parts) { p.off = total; total = al256(total + p.n * 4); }
  // bf16 copies of wqkv, wo, w1, w2 (parts 4, 6, 10, 12)
  const int mats[4] = {4, 6, 10, 12};
  size_t off16[4] = {0, 0, 0, 0};
  if (bf)
    for (int i = 0; i < 4; ++i) { off16[i] = total; total = al256(total + parts[mats[i]].n * 2); }
  void* dev = nullptr;
  if (hipMalloc(&dev, total) != hipSuccess) {
    (void)hipGetLastError();
    return set_error(WM_ERR_OUT_OF_MEMORY, "hipMalloc of the encoder failed");
  }
  uint8_t* base = static_cast<uint8_t*>(dev);
  std::vector<float> tmp;
  for (const auto& p : parts) {
    if (p.n == 0) continue;
    tmp.assign(p.src, p.src + p.n);
    if (p.matrix)
      for (auto& v : tmp) v = rnd(v);
    if (hipMemcpy(base + p.off, tmp.data(), p.n * 4, hipMemcpyHostToDevice) != hipSuccess) {
      (void)hipFree(dev);
      return set_error(WM_ERR_DEVICE, "hipMemcpy of the encoder weights failed");
    }
  }
  if (bf) {
    std::vector<__bf16> t16;
    for (int i = 0; i < 4; ++i) {
      const Part& p = parts[mats[i]];
      if (p.n == 0) continue;
      t16.resize(p.n);
      for (size_t j = 0; j < p.n; ++j) t16[j] = (__bf16)p.src[j];
      if (hipMemcpy(base + off16[i], t16.data(), p.n * 2, hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(dev);
        return set_error(WM_ERR_DEVICE, "hipMemcpy of the encoder weights failed");
      }
    }
  }
  wm_text_model* m = new (std::nothrow) wm_text_model;
  if (!m) {
    (void)hipFree(dev);
    return set_error(WM_ERR_OUT_OF_MEMORY, "host allocation failed");
  }
  m->dims = d;
  m->base = base;
  const float** dst[] = {&m->tok_emb, &m->pos_emb, &m->ln0_g, &m->ln0_b, &m->wqkv, &m->bqkv, &m->wo,
                         &m->bo, &m->ln1_g, &m->ln1_b, &m->w1, &m->b1, &m->w2, &m->b2, &m->ln2_g,
                         &m->ln2_b, &m->wp, &m->bp};
  for (size_t i = 0; i < parts.size(); ++i) *dst[i] = reinterpret_cast<const float*>(base + parts[i].off);
  const __bf16** dst16[] = {&m->wqkv16, &m->wo16, &m->w116, &m->w216};
  for (int i = 0; i < 4; ++i) *dst16[i] = bf ? reinterpret_cast<const __bf16*>(base + off16[i]) : nullptr;
  *out = m;
  return clear_error();
}

void wm_text_model_destroy(wm_text_model* m) {
  if (!m) return;
  (void)hipFree(m->base);
  delete m;
}

int32_t wm_text_chunks(const wm_text_model* m, const int32_t* tok_off, int32_t S) {
  if (!m || !tok_off || S < 1 || S > WM_TEXT_MAX_PROGRAMS || tok_off[0] != 0) return -1;
  long long n = 0;
  for (int s = 0; s < S; ++s) {
    if (tok_off[s + 1] < tok_off[s]) return -1;
    n += n_chunks_of(tok_off[s + 1] - tok_off[s], m->dims.window, m->dims.stride);
  }
  return n > (1LL << 30) / m->dims.window ? -1 : (int32_t)n;
}

size_t wm_text_workspace_bytes(const wm_text_model* m, int32_t n_chunks) {
  if (!m || n_chunks < 0) return 0;
  return text_layout(m->dims, n_chunks).total;
}

wm_status wm_encode_text(const wm_text_model* m, const int32_t* tokens, const int32_t* tok_off,
                         int32_t S, float* z0, void* ws, size_t ws_bytes, void* stream) {
  if (!m) return set_error(WM_ERR_INVALID_ARGUMENT, "model is NULL");
  if (!tok_off || S < 1 || S > WM_TEXT_MAX_PROGRAMS)
    return set_error(WM_ERR_INVALID_ARGUMENT, "need tok_off and 1 <= S <= " + std::to_string(WM_TEXT_MAX_PROGRAMS));
  const int32_t n_chunks = wm_text_chunks(m, tok_off, S);
  if (n_chunks < 0) return set_error(WM_ERR_INVALID_ARGUMENT, "tok_off must start at 0 and be non-decreasing");
  if (!z0 || (tok_off[S] > 0 && !tokens)) return set_error(WM_ERR_INVALID_ARGUMENT, "null tokens/z0");
  if (!ws) return set_error(WM_ERR_INVALID_ARGUMENT, "workspace is NULL");
  const wm_text_dims& d = m->dims;
  const TextLayout L = text_layout(d, n_chunks);
  if (ws_bytes < L.total) return set_error(WM_ERR_INVALID_ARGUMENT, "workspace too small");

  TTable tt;
  tt.S = S;
  tt.chunk_off[0] = 0;
  for (int s = 0; s < S; ++s) {
    tt.tok_off[s] = tok_off[s];
    tt.chunk_off[s + 1] = tt.chunk_off[s] + n_chunks_of(tok_off[s + 1] - tok_off[s], d.window, d.stride);
  }
  tt.tok_off[S] = tok_off[S];

  hipStream_t st = static_cast<hipStream_t>(stream);
  uint8_t* w8 = static_cast<uint8_t*>(ws);
  auto fp = [&](size_t o) { return reinterpret_cast<float*>(w8 + o); };
  int32_t* err = reinterpret_cast<int32_t*>(w8 + L.err);
  float *h = fp(L.h), *qkv = fp(L.qkv), *sc = fp(L.sc), *ctx = fp(L.ctx), *y = fp(L.y), *f = fp(L.f);
  float* pooled = fp(L.pooled);
  const int H = d.hidden, F = d.ffn, W = d.window, nh = d.heads, dh = H / nh;
  const int rows = n_chunks * W;
  const bool bf = d.precision == WM_BF16;
  // bf16 operand path: fused attention (head width 32 or 64, K and V of a
  // window in LDS) and products on bf16-stored operands
  const bool fused = bf16_path(d);
  auto gemm = [&](const GemmArgs& g, int batch, bool bt) {
    return bf ? launch_gemm<BF>(g, batch, bt, st) : launch_gemm<FP>(g, batch, bt, st);
  };
#define WM_TT(K, CALL)                                                                     \
  do {                                                                                     \
    timing_begin(K, st);                                                                   \
    hipError_t e_ = (CALL);                                                                \
    timing_end(K, st);                                                                     \
    if (e_ != hipSuccess) return set_error(WM_ERR_DEVICE, std::string("kernel launch: ") + hipGetErrorString(e_)); \
  } while (0)

  auto g16 = [&](const __bf16* A, int M, int K, const __bf16* Wm, int N, void* C, const float* bias,
                 const float* res, int gelu, bool out16) {
    Gemm16Args g;
    g.A = A; g.W = Wm; g.C = C; g.bias = bias; g.res = res; g.M = M; g.N = N; g.K = K; g.gelu = gelu;
    g.tiles_n = (N + G16_BN - 1) / G16_BN;
    const dim3 grid(((M + G16_BM - 1) / G16_BM) * g.tiles_n);
    if (out16) hipLaunchKernelGGL(gemm16_kernel<true>, grid, dim3(512), 0, st, g);
    else hipLaunchKernelGGL(gemm16_kernel<false>, grid, dim3(512), 0, st, g);
    return hipGetLastError();
  };
  auto ln = [&](const float* yin, const float* gm, const float* bt, __bf16* hbo) {
    hipLaunchKernelGGL(ln_kernel, dim3((rows + 3) / 4), dim3(256), 0, st, yin, gm, bt, H, rows, h, hbo);
    return hipGetLastError();
  };
  __bf16* hb = reinterpret_cast<__bf16*>(w8 + L.hb);
  __bf16* qkvb = reinterpret_cast<__bf16*>(w8 + L.qkvb);
  __bf16* ctxb = reinterpret_cast<__bf16*>(w8 + L.ctxb);
  __bf16* fb = reinterpret_cast<__bf16*>(w8 + L.fb);

  if (n_chunks > 0) {
    WM_TT(TK_TEXT_OTHER, [&]() { hipLaunchKernelGGL(embed_ln_kernel, dim3((rows + 3) / 4), dim3(256), 0, st, tokens,
                                             tt, W, d.stride, m->tok_emb, m->pos_emb, m->ln0_g, m->ln0_b,
                                             H, d.vocab, rows, h, fused ? hb : nullptr, err); return hipGetLastError(); }());
    for (int l = 0; l < d.layers; ++l) {
      const size_t lH = (size_t)l * H;
      if (fused) {
        // bf16: every product operand is stored as bf16
        WM_TT(TK_TEXT_GEMM, g16(hb, rows, H, m->wqkv16 + lH * 3 * H, 3 * H, qkvb, m->bqkv + 3 * lH,
                                nullptr, 0, true));
        const int lds = (W * (dh + 8) + dh * (W + 8)) * 2;
        auto kern = dh == 64 ? attention_kernel<64> : attention_kernel<32>;
        WM_TT(TK_TEXT_ATTN, [&]() {
          hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
          if (e != hipSuccess) { (void)hipGetLastError(); return e; }
          hipLaunchKernelGGL(kern, dim3(n_chunks * nh), dim3(64 * (W / 32)), lds, st, qkvb, ctxb, tt, W,
                             d.stride, nh, H, 1.0f / std::sqrt((float)dh));
          return hipGetLastError();
        }());
        WM_TT(TK_TEXT_GEMM, g16(ctxb, rows, H, m->wo16 + lH * H, H, y, m->bo + lH, h, 0, false));
        WM_TT(TK_TEXT_OTHER, ln(y, m->ln1_g + lH, m->ln1_b + lH, hb));
        WM_TT(TK_TEXT_GEMM, g16(hb, rows, H, m->w116 + (size_t)l * F * H, F, fb, m->b1 + (size_t)l * F,
                                nullptr, 1, true));
        WM_TT(TK_TEXT_GEMM, g16(fb, rows, F, m->w216 + (size_t)l * H * F, H, y, m->b2 + lH, h, 0, false));
        WM_TT(TK_TEXT_OTHER, ln(y, m->ln2_g + lH, m->ln2_b + lH, hb));
        continue;
      }
      // q, k, v
      WM_TT(TK_TEXT_GEMM, gemm(dense(h, rows, H, m->wqkv + lH * 3 * H, 3 * H, qkv, m->bqkv + 3 * lH,
                                     nullptr, 0), 1, false));
      // scores per (chunk, head): q k^T / sqrt(dh)
      GemmArgs s{};
      s.A = qkv; s.B = qkv + H; s.C = sc; s.M = W; s.N = W; s.K = dh;
      s.lda = 3 * H; s.ldb = 3 * H; s.ldc = W; s.bdiv = nh;
      s.sA1 = (long long)W * 3 * H; s.sA2 = dh; s.sB1 = s.sA1; s.sB2 = dh;
      s.sC1 = (long long)nh * W * W; s.sC2 = (long long)W * W;
      s.alpha = 1.0f / std::sqrt((float)dh);
      WM_TT(TK_TEXT_ATTN, gemm(s, n_chunks * nh, false));
      WM_TT(TK_TEXT_ATTN, [&]() { hipLaunchKernelGGL(softmax_kernel, dim3((unsigned)(((long long)n_chunks * nh * W + 3) / 4)),
                                              dim3(256), 0, st, sc, tt, W, d.stride, nh,
                                              (long long)n_chunks * nh * W); return hipGetLastError(); }());
      // context = P v per (chunk, head), into the head's columns
      GemmArgs pv{};
      pv.A = sc; pv.B = qkv + 2 * H; pv.C = ctx; pv.M = W; pv.N = dh; pv.K = W;
      pv.lda = W; pv.ldb = 3 * H; pv.ldc = H; pv.bdiv = nh;
      pv.sA1 = (long long)nh * W * W; pv.sA2 = (long long)W * W;
      pv.sB1 = (long long)W * 3 * H; pv.sB2 = dh;
      pv.sC1 = (long long)W * H; pv.sC2 = dh;
      pv.alpha = 1.0f;
      WM_TT(TK_TEXT_ATTN, gemm(pv, n_chunks * nh, true));
      // h = LN(h + ctx Wo^T + bo)
      WM_TT(TK_TEXT_GEMM, gemm(dense(ctx, rows, H, m->wo + lH * H, H, y, m->bo + lH, h, 0), 1, false));
      WM_TT(TK_TEXT_OTHER, ln(y, m->ln1_g + lH, m->ln1_b + lH, nullptr));
      // h = LN(h + GELU(h W1^T + b1) W2^T + b2)
      WM_TT(TK_TEXT_GEMM, gemm(dense(h, rows, H, m->w1 + (size_t)l * F * H, F, f, m->b1 + (size_t)l * F,
                                     nullptr, 1), 1, false));
      WM_TT(TK_TEXT_GEMM, gemm(dense(f, rows, F, m->w2 + (size_t)l * H * F, H, y, m->b2 + lH, h, 0), 1, false));
      WM_TT(TK_TEXT_OTHER, ln(y, m->ln2_g + lH, m->ln2_b + lH, nullptr));
    }
    WM_TT(TK_TEXT_OTHER, [&]() { hipLaunchKernelGGL(pool_kernel, dim3(n_chunks), dim3(POOL_THREADS), 0, st, h, tt, W,
                                             d.stride, H, pooled); return hipGetLastError(); }());
  }
  WM_TT(TK_TEXT_OTHER, [&]() { hipLaunchKernelGGL(project_kernel, dim3(S), dim3(256), H * (int)sizeof(float), st,
                                           pooled, tt, H, d.d, m->wp, m->bp, bf ? 1 : 0, z0); return hipGetLastError(); }());
#undef WM_TT
  return clear_error();
}

}  // extern "C"
