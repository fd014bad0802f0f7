// Device-side pieces shared by the kernel sources: operand types and
// precision traits of the matrix-core products, the GELU, LDS staging
// helpers and the argument block of the rollout kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wm_internal.h"

namespace wm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// Global-memory (address space 1) views.  A pointer that passes through an
// asm statement keeps its address space only if its type says so; a generic
// pointer would turn the loads into flat loads, which also count against the
// LDS counter, so every LDS wait would drain them.
typedef __attribute__((address_space(1))) const uint8_t gu8;
typedef __attribute__((address_space(1))) const u32x4 gu32x4;

// --------------------------------------------------------------------------
// Precision traits: operand fragment type, conversion, matrix-core product.

struct PBF16 : GeomBF16 {
  using Frag = bf16x8;
  static __device__ __forceinline__ f32x16 mfma(Frag a, Frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  // The same product with the accumulator held in VGPRs, for a chain whose
  // accumulator lives beside a latent that fills the AGPRs.  The compiler's
  // hazard checks do not see inline assembly: the caller provides NOPS wait
  // states before the product (its accumulator written by VALU just before)
  // and waits before the first VALU access to the result.
  template <int NOPS>
  static __device__ __forceinline__ void mfma_v(Frag a, Frag b, f32x16& c) {
    static_assert(NOPS >= 0 && NOPS <= 16, "one s_nop covers 1 to 16 wait states");
    if constexpr (NOPS > 0)
      asm volatile("s_nop %3\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0"
                   : "+v"(c) : "v"(a), "v"(b), "i"(NOPS - 1));
    else
      asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b));
  }
  // 8 floats -> 8 bf16 (round to nearest even)
  static __device__ __forceinline__ Frag cvt(const float* v) {
    Frag f;
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = (__bf16)v[j];
    return f;
  }
  // fragment `w` (0 <= w < G) of a 16-byte lane group
  static __device__ __forceinline__ Frag pick(u32x4 g, int) { return __builtin_bit_cast(Frag, g); }
  // all elements kept (mask = ~0) or zeroed (mask = 0)
  static __device__ __forceinline__ Frag mask(Frag f, uint32_t m) {
    u32x4 u = __builtin_bit_cast(u32x4, f);
    u &= m;
    return __builtin_bit_cast(Frag, u);
  }
  // two GELU outputs -> one packed register (bf16 pair), masked
  using Packed = uint32_t;
  static __device__ __forceinline__ Packed pack2(float a, float b, uint32_t m) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 v = {(__bf16)a, (__bf16)b};
    return __builtin_bit_cast(uint32_t, v) & m;
  }
  // operand fragment f (8 values = 4 packed pairs) of the second product
  static __device__ __forceinline__ Frag gfrag(const Packed (&gp)[8], int f) {
    const u32x4 u = {gp[4 * f], gp[4 * f + 1], gp[4 * f + 2], gp[4 * f + 3]};
    return __builtin_bit_cast(Frag, u);
  }
};

struct PF32 : GeomF32 {
  using Frag = float;
  static __device__ __forceinline__ f32x16 mfma(Frag a, Frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ Frag cvt(const float* v) { return v[0]; }
  // Copy the element out first: a bit_cast applied directly to a vector
  // element expression lowers to element 0 whatever the index.
  static __device__ __forceinline__ Frag pick(u32x4 g, int w) {
    const uint32_t u = g[w];
    return __uint_as_float(u);
  }
  static __device__ __forceinline__ Frag mask(Frag f, uint32_t m) {
    return __uint_as_float(__float_as_uint(f) & m);
  }
  // fp32 keeps both values of a pair unpacked
  struct Packed { float a, b; };
  static __device__ __forceinline__ Packed pack2(float a, float b, uint32_t m) {
    return {__uint_as_float(__float_as_uint(a) & m), __uint_as_float(__float_as_uint(b) & m)};
  }
  // operand fragment f (one value) of the second product
  static __device__ __forceinline__ Frag gfrag(const Packed (&gp)[8], int f) {
    return (f & 1) ? gp[f >> 1].b : gp[f >> 1].a;
  }
};

// GELU(x) = x * Phi(x) = (x + |x| * erf(|x| / sqrt 2)) / 2, with erf from
// Abramowitz & Stegun, Handbook of Mathematical Functions, formula 7.1.26:
//   erf(a) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-a^2),
//   t = 1 / (1 + p a), a >= 0, |error| <= 1.5e-7.
// The 1/sqrt 2 scaling is folded into the constants: one reciprocal, one
// exp2, ten multiply-adds, no branches; -> 0 and -> x in the tails, 0 at 0.
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

template <class PR>
__device__ __forceinline__ float op_value(float v) {   // the value a product operand takes
  if constexpr (PR::G == 1) return (float)(__bf16)v;
  else return v;
}

// 16 accumulator values of one 32-row block <-> a row in natural order
// (rows acc_row(h, 4q .. 4q+3) are consecutive: four 16-byte accesses).
__device__ __forceinline__ void store_acc(float* row, const f32x16& v, int h) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const f32x4 x = {v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
    *reinterpret_cast<f32x4*>(row + acc_row(h, 4 * q)) = x;
  }
}
__device__ __forceinline__ f32x16 load_acc(const float* row, int h) {
  f32x16 v;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const f32x4 x = *reinterpret_cast<const f32x4*>(row + acc_row(h, 4 * q));
#pragma unroll
    for (int i = 0; i < 4; ++i) v[4 * q + i] = x[i];
  }
  return v;
}

__device__ __forceinline__ u32x4 lds_group(const uint8_t* base, int group, int lane) {
  return *reinterpret_cast<const u32x4*>(base + group * 1024 + lane * 16);
}

// Copy `bytes` (multiple of 16) from global memory into LDS with the
// direct global->LDS path: every lane moves 16 bytes, a wavefront fills 1 KiB
// at LDS address base + lane*16.  Completion is tracked by vmcnt.
__device__ __forceinline__ void stage_to_lds(const uint8_t* __restrict__ src, uint8_t* dst,
                                             int bytes, int tid, int nthreads) {
  const int units = bytes >> 4;
  const int wave_base = tid & ~63;
  for (int u0 = 0; u0 < units; u0 += nthreads) {
    const int u = u0 + tid;
    if (u < units) {
      __builtin_amdgcn_global_load_lds(
          (const void*)(src + (size_t)u * 16),
          (__attribute__((address_space(3))) void*)(dst + (size_t)(u0 + wave_base) * 16), 16, 0, 0);
    }
  }
}

// Same copy with a compile-time size: straight-line code, one guarded tail.
template <int BYTES, int NT>
__device__ __forceinline__ void stage_fixed(const uint8_t* __restrict__ src, uint8_t* dst, int tid) {
  static_assert(BYTES % 16 == 0, "16-byte units");
  constexpr int UNITS = BYTES / 16, FULL = UNITS / NT;
  const int wave_base = tid & ~63;
#pragma unroll
  for (int i = 0; i < FULL; ++i) {
    __builtin_amdgcn_global_load_lds(
        (const void*)(src + (size_t)(i * NT + tid) * 16),
        (__attribute__((address_space(3))) void*)(dst + (size_t)(i * NT + wave_base) * 16), 16, 0, 0);
  }
  if constexpr (UNITS % NT != 0) {
    if (FULL * NT + tid < UNITS)
      __builtin_amdgcn_global_load_lds(
          (const void*)(src + (size_t)(FULL * NT + tid) * 16),
          (__attribute__((address_space(3))) void*)(dst + (size_t)(FULL * NT + wave_base) * 16), 16, 0, 0);
  }
}

__device__ __forceinline__ void wait_vm_then_barrier() {
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's global->LDS copies landed
  __syncthreads();
}

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// Subgraph of candidate i: the largest s with off[s] <= i.
__device__ __forceinline__ int segment_of(const SegTable& seg, int i) {
  int lo = 0, hi = seg.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (seg.off[mid] <= i) lo = mid; else hi = mid - 1;
  }
  return lo;
}


struct RollArgs {
  const uint8_t* w1;        // packed transition chunks, W1 part
  const uint8_t* w2;        // packed transition chunks, W2 part
  const uint8_t* wh;        // packed hyperplane-normal map (paper-form transition)
  const float* tab;         // rollout table (see DevModel::roll_tab)
  const float* z0;          // [S][D]
  const int2* perm;         // sorted (candidate, subgraph)
  const int32_t* types;     // [B][T_max]
  const int32_t* params;    // [B][T_max][P]
  const int32_t* lens;      // [B]
  float* zT;                // [B][D]
  float* phi;               // [B][E] mean step embedding, or null (the phi kernel computes it)
  int32_t* err;
  int B, T_max, P, K, H, tab_bytes;
  // training forward of the rollout loss (row-owned kernel only): the
  // activations of every valid step in compact rows off[i] + t
  float *X, *A, *G, *Pz;    // [R][D+E], [R][H], [R][H], [R][D]
  float *V, *SC;            // paper form: [R][D] Wh e, [R][4] v.z, v.v, |u|, 0
  const int32_t* off;
  int32_t* row_src;
  // scores fused into the narrow rollout: cost blob, hw [n_hw][HW], scores [n_hw][B]
  const uint8_t* costn;
  const float* hw;
  float* scores;
  float bc2;
  int n_hw, HW, C;
};

typedef __attribute__((address_space(3))) uint8_t lds_u8;
__device__ __forceinline__ lds_u8* to_lds(uint8_t* p) { return (lds_u8*)p; }

}  // namespace wm
