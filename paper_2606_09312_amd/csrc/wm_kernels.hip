// Hand-written gfx950 kernels of the batched latent-rollout evaluator.
//
//  bucket_kernel   counting sort of candidates by action-sequence length
//                  (longest first), length validation, subgraph lookup
//  rollout_kernel  the multi-step transition z <- z + W2 GELU(W1 [z; e] + b1) + b2
//                  (Eq. 1, Sec. 3.4), persistent over all steps of a tile of
//                  32 candidates per wavefront, latent kept in registers,
//                  weights streamed through LDS, matrix cores for both products
//  phi_kernel      mean action embedding (action features, Sec. 3.5)
//  score_kernel    cost model y = wc2 GELU(Wc1 [z_T; phi; h] + bc1) + bc2 (Eq. 3)
//  encode_kernel   initial latents from program features (Sec. 3.3, Eq. 4)
//  topk_kernel     per (hardware vector, subgraph) top-k by (-y, index)
//                  (Sec. 3.5): radix select + bitonic sort in LDS
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "wm_device.h"

namespace wm {

// ==========================================================================
// Bucketing: one workgroup sorts all candidates by length, longest first.
// perm[pos] = (candidate, subgraph).  Candidates are independent, so the order
// within one length bucket does not affect any result.

__global__ __launch_bounds__(1024) void bucket_kernel(const int32_t* __restrict__ lens, int B,
                                                       int T_max, const SegTable seg,
                                                       int2* __restrict__ perm,
                                                       int32_t* __restrict__ err) {
  extern __shared__ int bsm[];
  int* hist = bsm;
  int* cur = bsm + (T_max + 1);
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int i = tid; i <= T_max; i += nt) hist[i] = 0;
  __syncthreads();
  int bad = 0;
  for (int i = tid; i < B; i += nt) {
    int L = lens[i];
    if (L < 0 || L > T_max) { bad = 1; L = clampi(L, 0, T_max); }
    atomicAdd(&hist[L], 1);
  }
  if (bad) atomicOr(err, ERRBIT_LEN);
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int L = T_max; L >= 0; --L) { cur[L] = acc; acc += hist[L]; }
  }
  __syncthreads();
  for (int i = tid; i < B; i += nt) {
    const int L = clampi(lens[i], 0, T_max);
    const int pos = atomicAdd(&cur[L], 1);
    perm[pos] = make_int2(i, segment_of(seg, i));
  }
}

// Large batches: the same counting sort over chunks of candidates, one
// workgroup per chunk.  Pass 1 writes each chunk's length histogram to
// hist[chunk][L]; pass 2 (one workgroup) turns the histograms into each
// chunk's first output position per length (longest lengths first, chunks
// in order within a length); pass 3 scatters every chunk from those cursors.

__global__ __launch_bounds__(1024) void bucket_count_kernel(const int32_t* __restrict__ lens, int B,
                                                             int T_max, int chunk,
                                                             int32_t* __restrict__ hist,
                                                             int32_t* __restrict__ err) {
  extern __shared__ int bsm[];
  const int nb = T_max + 1, tid = threadIdx.x, nt = blockDim.x;
  for (int L = tid; L < nb; L += nt) bsm[L] = 0;
  __syncthreads();
  const int lo = blockIdx.x * chunk, hi = min(lo + chunk, B);
  int bad = 0;
  for (int i = lo + tid; i < hi; i += nt) {
    int L = lens[i];
    if (L < 0 || L > T_max) { bad = 1; L = clampi(L, 0, T_max); }
    atomicAdd(&bsm[L], 1);
  }
  if (bad) atomicOr(err, ERRBIT_LEN);
  __syncthreads();
  for (int L = tid; L < nb; L += nt) hist[(size_t)blockIdx.x * nb + L] = bsm[L];
}

// Exclusive scan of one value per thread over the workgroup (1024 threads).
__device__ __forceinline__ int block_exclusive_scan(int v, int* wsum) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int k = 0; k < nw; ++k) { const int t = wsum[k]; wsum[k] = acc; acc += t; }
  }
  __syncthreads();
  return wsum[w] + x - v;
}

__global__ __launch_bounds__(1024) void bucket_scan_kernel(int T_max, int groups,
                                                            int32_t* __restrict__ hist) {
  extern __shared__ int bsm[];
  int* base = bsm;                       // [nb]: first position of each length
  int* wsum = bsm + (T_max + 1);         // [16]
  const int nb = T_max + 1, tid = threadIdx.x, nt = blockDim.x;
  // thread tid owns positions [tid*per, tid*per + per) of the length order
  // T_max, T_max - 1, ..., 0 (longest first)
  const int per = (nb + nt - 1) / nt;
  int own = 0;
  for (int j = tid * per; j < min(nb, tid * per + per); ++j) {
    const int L = T_max - j;
    int tot = 0;
    for (int g = 0; g < groups; ++g) tot += hist[(size_t)g * nb + L];
    base[L] = tot;
    own += tot;
  }
  int run = block_exclusive_scan(own, wsum);
  for (int j = tid * per; j < min(nb, tid * per + per); ++j) {
    const int L = T_max - j;
    const int tot = base[L];
    base[L] = run;
    run += tot;
  }
  __syncthreads();
  // per-chunk cursors: chunks in order within each length
  for (int L = tid; L < nb; L += nt) {
    int c = base[L];
    for (int g = 0; g < groups; ++g) {
      const int v = hist[(size_t)g * nb + L];
      hist[(size_t)g * nb + L] = c;
      c += v;
    }
  }
}

__global__ __launch_bounds__(1024) void bucket_scatter_kernel(const int32_t* __restrict__ lens,
                                                               int B, int T_max, int chunk,
                                                               const SegTable seg,
                                                               const int32_t* __restrict__ hist,
                                                               int2* __restrict__ perm) {
  extern __shared__ int bsm[];
  const int nb = T_max + 1, tid = threadIdx.x, nt = blockDim.x;
  for (int L = tid; L < nb; L += nt) bsm[L] = hist[(size_t)blockIdx.x * nb + L];
  __syncthreads();
  const int lo = blockIdx.x * chunk, hi = min(lo + chunk, B);
  for (int i = lo + tid; i < hi; i += nt) {
    const int L = clampi(lens[i], 0, T_max);
    const int pos = atomicAdd(&bsm[L], 1);
    perm[pos] = make_int2(i, segment_of(seg, i));
  }
}

// ==========================================================================
// Rollout.
//
// Workgroup = WAVES wavefronts; wavefront w owns the 32 candidates at sorted
// positions [32*(WAVES*blockIdx.x + w), +32): lane L works on candidate
// column L%32 together with lane L^32.  All wavefronts of a workgroup walk the
// same sequence of 32-hidden-unit weight chunks, double-buffered in LDS, for
// T_wg steps (T_wg = longest sequence of the workgroup; sorted order keeps
// the tiles of a workgroup of similar length).  A candidate past its own
// length keeps z unchanged: its GELU outputs and b2 are zeroed, so the second
// product adds exact zeros.


// Copies of the next weight chunk (its W1 and/or W2 part) into LDS, issued
// a few at a time between the matrix-fragment groups of an iteration so the
// L2 -> LDS traffic runs continuously underneath the computation.

struct CopyPlan {
  uint32_t o1;        // byte offset of the W1 part in the W1 chunk array
  lds_u8* d1;
  bool e1;            // copy the W1 part
  uint32_t o2;        // byte offset of the W2 part in the W2 chunk array
  lds_u8* d2;
  bool e2;
};

// Copy sources as raw buffer resources over the packed chunk arrays: a copy
// is a buffer load straight to LDS with the chunk's byte offset in a scalar
// register and one lane offset (tid * 16) shared by all copies, so no 64-bit
// address is kept per copy.  The hardware bounds-checks every copy against
// the array size.
struct CopySrc {
  __amdgpu_buffer_rsrc_t r1, r2;
  uint32_t voff;      // tid * 16
  int wave_base;      // first thread of the wavefront (uniform)
};
typedef __attribute__((address_space(3))) void lds_void;

// `BYTES` (multiple of 16) from byte offset `off` of a buffer into LDS.
template <int BYTES, int NT>
__device__ __forceinline__ void stage_buf(__amdgpu_buffer_rsrc_t r, uint32_t off, uint8_t* dst,
                                          const CopySrc& cs, int tid) {
  static_assert(BYTES % 16 == 0, "16-byte units");
  constexpr int UNITS = BYTES / 16, FULL = UNITS / NT;
#pragma unroll
  for (int i = 0; i < FULL; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(dst + (size_t)(i * NT + cs.wave_base) * 16), 16,
                                             cs.voff, off + i * NT * 16, 0, 0);
  if constexpr (UNITS % NT != 0) {
    if (FULL * NT + tid < UNITS)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(dst + (size_t)(FULL * NT + cs.wave_base) * 16), 16,
                                               cs.voff, off + FULL * NT * 16, 0, 0);
  }
}


// Per-wavefront pieces of one transition step.  Chunk c covers hidden units
// [32c, 32c+32): the first product forms G^T[chunk] = b1 + W1[chunk] . X^T in
// accumulator layout, its GELU becomes the B operand of the second product,
// which accumulates dZ^T += W2[:, chunk] . G^T into the latent.
template <class PR, int D, int E>
struct Roll {
  using Frag = typename PR::Frag;
  static constexpr int KF = PR::KF, SL = PR::SL, G = PR::G;
  static constexpr int NZ = D / KF, NE = E / KF, NK1 = NZ + NE;
  static constexpr int NF2 = 32 / KF, NB = D / 32, NK2 = NB * NF2;
  static constexpr int W1B = TransChunk<PR>::w1_bytes(D, E);
  static constexpr int W2B = TransChunk<PR>::w2_bytes(D);
  static_assert(NK1 % G == 0 && NK2 % G == 0, "fragment groups");

  // One pipeline iteration as a single stream of "items" (one 16-byte-per-
  // lane fragment group read from LDS each): first the N1 groups of the first
  // product of the next chunk (from w1n), then the N2 groups of the second
  // product of the current chunk (from w2c).  Reads run P items ahead in a
  // register ring; the GELU of the current chunk's first product is computed
  // a few values per item while the next chunk's first product runs, and is
  // complete before the second product starts.  A scheduling fence after every
  // item keeps this order (left alone, the scheduler serialises read, wait and
  // matrix instruction at this register pressure).
  //   DO_G1: compute acc1n = b1 + W1[next chunk] . X^T
  //   DO_G2: GELU(acc1) -> second product into zacc
  // Copy unit u (16 bytes per lane) of a CopyPlan: units [0, U1) are the W1
  // part, [U1, U1 + U2) the W2 part.
  template <int NT>
  static constexpr int U1 = (W1B / 16 + NT - 1) / NT;
  template <int NT>
  static constexpr int U2 = (W2B / 16 + NT - 1) / NT;
  template <int NT>
  static __device__ __forceinline__ void copy_unit(const CopyPlan& cp, const CopySrc& cs, int u, int tid) {
    if (u < U1<NT>) {
      const int k = u * NT;
      if (cp.e1 && k + tid < W1B / 16)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(cs.r1, (lds_void*)(cp.d1 + (k + cs.wave_base) * 16), 16,
                                                 cs.voff, cp.o1 + k * 16, 0, 0);
    } else {
      const int k = (u - U1<NT>) * NT;
      if (cp.e2 && k + tid < W2B / 16)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(cs.r2, (lds_void*)(cp.d2 + (k + cs.wave_base) * 16), 16,
                                                 cs.voff, cp.o2 + k * 16, 0, 0);
    }
  }

  template <bool DO_G1, bool DO_G2, int NT, bool COPY>
  static __device__ __forceinline__ void iteration(const uint8_t* w1n, const uint8_t* w2c,
                                                   const Frag (&xz)[NZ], const Frag (&xe)[NE],
                                                   const f32x16& acc1, uint32_t mask,
                                                   f32x16& acc1n, f32x16 (&zacc)[NB],
                                                   int lane, int h, const CopyPlan& cp,
                                                   const CopySrc& cs, int tid) {
    constexpr int N1 = DO_G1 ? NK1 / G : 0;
    constexpr int N2 = DO_G2 ? NK2 / G : 0;
    // d = 512 (first product alone, its GELU after it): the accumulator in VGPRs
    constexpr bool VACC = DO_G1 && !DO_G2 && G == 1 && D >= 512;
    constexpr int NI = N1 + N2;
    constexpr int NU = COPY ? U1<NT> + U2<NT> : 0;     // copy units, spread over the items
    constexpr int P = 4;                                   // LDS reads in flight
    constexpr int PAIRS = 8;                               // GELU value pairs (16 values)
    if constexpr (DO_G1) {
      const float* b1t = reinterpret_cast<const float*>(w1n + (W1B - 128)) + 16 * h;
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(b1t + 4 * r4);
#pragma unroll
        for (int i = 0; i < 4; ++i) acc1n[4 * r4 + i] = v[i];
      }
    }
    // GELU outputs, packed two at a time as they are produced
    typename PR::Packed gp[PAIRS];
    if constexpr (DO_G2 && N1 == 0) {      // nothing to hide the GELU under
#pragma unroll
      for (int q = 0; q < PAIRS; ++q) gp[q] = PR::pack2(gelu(acc1[2 * q]), gelu(acc1[2 * q + 1]), mask);
    }
    u32x4 ring[P];
#pragma unroll
    for (int i = 0; i < P && i < NI; ++i)
      ring[i] = lds_group(i < N1 ? w1n : w2c, i < N1 ? i : i - N1, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const u32x4 grp = ring[i % P];
      if (i + P < NI) ring[i % P] = lds_group(i + P < N1 ? w1n : w2c, i + P < N1 ? i + P : i + P - N1, lane);
      if constexpr (NU > 0) {
#pragma unroll
        for (int u = 0; u < NU; ++u)
          if ((u * NI) / NU == i) copy_unit<NT>(cp, cs, u, tid);
      }
      if (i < N1) {
        if constexpr (VACC) {
          // accumulator in VGPRs (the latent fills the AGPRs): 5 wait states
          // after its VALU initialisation; the first VALU access follows
          // the iteration's closing wait
          const Frag b = i < NZ ? xz[i < NZ ? i : 0] : xe[i < NZ ? 0 : i - NZ];
          if (i == 0) PR::template mfma_v<5>(PR::pick(grp, 0), b, acc1n);
          else PR::template mfma_v<0>(PR::pick(grp, 0), b, acc1n);
        } else {
#pragma unroll
          for (int w = 0; w < G; ++w) {
            const int kf = i * G + w;
            acc1n = PR::mfma(PR::pick(grp, w), kf < NZ ? xz[kf < NZ ? kf : 0] : xe[kf < NZ ? 0 : kf - NZ], acc1n);
          }
        }
        if constexpr (DO_G2) {
          // value pairs spread evenly over the N1 items of the first product
#pragma unroll
          for (int q = 0; q < PAIRS; ++q)
            if ((q * N1) / PAIRS == i) gp[q] = PR::pack2(gelu(acc1[2 * q]), gelu(acc1[2 * q + 1]), mask);
        }
      } else {
#pragma unroll
        for (int w = 0; w < G; ++w) {
          const int F = (i - N1) * G + w;
          zacc[F / NF2] = PR::mfma(PR::pick(grp, w), PR::gfrag(gp, F % NF2), zacc[F / NF2]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // wait states between the last product into a VGPR accumulator and the
    // next VALU access to it (the accumulator is an operand, so no access is
    // scheduled above them)
    if constexpr (VACC && N2 == 0) asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(acc1n));
  }

  // SL consecutive floats of an LDS table row
  static __device__ __forceinline__ void row(const float* p, float (&v)[SL]) {
    if constexpr (SL % 4 == 0) {
#pragma unroll
      for (int q = 0; q < SL / 4; ++q) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(p + 4 * q);
#pragma unroll
        for (int i = 0; i < 4; ++i) v[4 * q + i] = x[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < SL; ++i) v[i] = p[i];
    }
  }
};

// Workgroup = WAVES wavefronts; wavefront w owns the 32 candidates at sorted
// positions [32*(WAVES*blockIdx.x + w), +32): lane L works on candidate
// column L%32 together with lane L^32.  All wavefronts of a workgroup walk the
// same sequence of weight chunks for T_wg steps (T_wg = longest sequence of the
// workgroup; sorted order keeps a workgroup's tiles of similar length).
//
// Software pipeline over chunks (W1 parts in w1a/w1b, W2 parts in w2a/w2b,
// four distinct LDS arrays): iteration c computes GELU of chunk c while the
// first product of chunk c+1 runs on the matrix cores, then the second
// product of chunk c; meanwhile the W2 part of chunk c+1 and the W1 part of
// chunk c+2 are copied into the buffers freed by the previous iteration.
// Paper-form transition (Sec. 3.4, TransH-style hyperplanes): before the
// residual update the latent loses its component along the unit normal of
// the action's hyperplane, v = Wh . e_t, and after it the latent is scaled to
// unit length.  Both are applied at the start of a step, on the previous
// step's output u:  z' = (u - alpha v) s  with  s = 1/|u|  (when the previous
// step was a real step of this candidate) and  alpha = (v.u)/(v.v)  (when
// this step is one), which equals normalising first and projecting onto the
// hyperplane of unit normal v/|v| afterwards.  V^T = Wh . E^T runs on the
// matrix cores with the step's embedding fragments as B operand, so v lands
// in the latent's accumulator layout; the dot products are per-lane partial
// sums completed across the lane pair (L, L^32) that holds one candidate.
template <class PR, int D, int E>
struct Hyper {
  using Frag = typename PR::Frag;
  static constexpr int NE = E / PR::KF, NB = D / 32, G = PR::G;
  static constexpr int GPB = HyperGeom<PR>::groups_per_block(E);   // fragment groups per block
  static constexpr int NG = NB * GPB;
  static constexpr int BYTES = HyperGeom<PR>::bytes(D, E);
  // keep V in registers between the two passes where the latent leaves room
  static constexpr bool HOLD = D <= 64 || (G == 1 && D <= 256);
  // d = 512: the latent fills the AGPRs; V's accumulator goes to VGPRs
  static constexpr bool VACC = G == 1 && D >= 512;
  // latent operand fragments: NF2 per 32-row block, SL values each per lane
  static constexpr int SL = PR::SL, NF2 = 32 / PR::KF, NZ = D / PR::KF;

  static __device__ __forceinline__ u32x4 group(const uint8_t* src, int g, int lane) {
    return *reinterpret_cast<const u32x4*>(src + g * 1024 + lane * 16);
  }
  // Per-lane base address for reads from global memory, made opaque to the
  // optimiser: otherwise the loop-invariant address of every fragment group
  // is hoisted out of the step loop and kept live (64 bits each), which
  // spills.  LDS addresses need no such care (16-bit immediate offsets).
  static __device__ __forceinline__ const uint8_t* lane_base(const uint8_t* src, int lane) {
    gu8* p = ((gu8*)(src)) + lane * 16;
    asm volatile("" : "+v"(p));
    return (const uint8_t*)p;
  }
  static __device__ __forceinline__ u32x4 gload(const uint8_t* p) {
    return *reinterpret_cast<gu32x4*>(((gu8*)(p)));
  }
  static __device__ __forceinline__ float pair_sum(float x) { return x + __shfl_xor(x, 32); }

  // One pass over V block by block (RD fragment-group reads in flight).
  //   PASS 0: partial dots v.z, v.v, z.z (and V kept when HOLD)
  //   PASS 1: z <- (z - al v) s
  template <int PASS, int RD, bool GLOBAL>
  static __device__ __forceinline__ void pass(const uint8_t* src, const Frag (&xe)[NE],
                                              f32x16 (&z)[NB], f32x16 (&vh)[HOLD ? NB : 1],
                                              float& vz, float& vv, float& zz, float al, float s,
                                              Frag (&xz)[NZ], int lane) {
    // global source: lane offset folded into an opaque base (lane argument 0)
    const uint8_t* base = GLOBAL ? lane_base(src, lane) : src;
    const int ln = GLOBAL ? 0 : lane;
    auto ld = [&](int g) -> u32x4 {
      if constexpr (GLOBAL) return gload(base + g * 1024);
      else return group(base, g, ln);
    };
    u32x4 ring[RD];
#pragma unroll
    for (int i = 0; i < RD && i < NG; ++i) ring[i] = ld(i);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      f32x16 vb = {};
#pragma unroll
      for (int k = 0; k < GPB; ++k) {
        const int g = b * GPB + k;
        const u32x4 grp = ring[g % RD];
        if (g + RD < NG) ring[g % RD] = ld(g + RD);
        if constexpr (VACC) {
          // accumulator in VGPRs (the latent fills the AGPRs): 5 wait
          // states after its zero initialisation
          if (k == 0) PR::template mfma_v<5>(PR::pick(grp, 0), xe[k], vb);
          else PR::template mfma_v<0>(PR::pick(grp, 0), xe[k], vb);
        } else {
#pragma unroll
          for (int w = 0; w < G; ++w) vb = PR::mfma(PR::pick(grp, w), xe[k * G + w], vb);
        }
        // keep the reads RD groups ahead, not hoisted all to the top
        __builtin_amdgcn_sched_barrier(0);
      }
      // wait states before the first VALU access to a VGPR accumulator (an
      // operand of the wait, so no access is scheduled above it)
      if constexpr (VACC) asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(vb));
      if constexpr (PASS == 0) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          vz = fmaf(vb[r], z[b][r], vz);
          vv = fmaf(vb[r], vb[r], vv);
          zz = fmaf(z[b][r], z[b][r], zz);
        }
        if constexpr (HOLD) vh[b] = vb;
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) z[b][r] = (z[b][r] - al * vb[r]) * s;
        frags_of(z[b], b, xz);
        asm volatile("" : "+a"(z[b]));    // the updated block back in the AGPRs here
      }
    }
  }

  // The step's operand fragments of latent block b (the state after the
  // projection), formed as each block is updated so that the latent is read
  // once.
  static __device__ __forceinline__ void frags_of(const f32x16& zb, int b, Frag (&xz)[NZ]) {
#pragma unroll
    for (int f = 0; f < NF2; ++f) {
      float v[SL];
#pragma unroll
      for (int j = 0; j < SL; ++j) v[j] = zb[f * SL + j];
      xz[b * NF2 + f] = PR::cvt(v);
      // formed here, not sunk to its first use (which would keep every
      // updated value alive, and spill)
      asm volatile("" : "+v"(xz[b * NF2 + f]));
    }
  }

  template <int RD, bool GLOBAL>
  // Also forms the step's latent operand fragments xz from the projected state.
  static __device__ __forceinline__ void step_in(f32x16 (&z)[NB], const Frag (&xe)[NE],
                                                 const uint8_t* src, bool project, bool renorm,
                                                 Frag (&xz)[NZ], int lane) {
    float vz = 0.0f, vv = 0.0f, zz = 0.0f;
    f32x16 vh[HOLD ? NB : 1];
    pass<0, RD, GLOBAL>(src, xe, z, vh, vz, vv, zz, 0.0f, 1.0f, xz, lane);
    vz = pair_sum(vz);
    vv = pair_sum(vv);
    zz = pair_sum(zz);
    const float s = (renorm && zz > 0.0f) ? rsqrtf(zz) : 1.0f;
    const float al = (project && vv > 0.0f) ? vz / vv : 0.0f;
    if constexpr (HOLD) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
#pragma unroll
        for (int r = 0; r < 16; ++r) z[b][r] = (z[b][r] - al * vh[b][r]) * s;
        frags_of(z[b], b, xz);
      }
    } else {
      // The latent lives in the AGPRs: this fence makes pass 1 read it there
      // again instead of keeping the copies pass 0 read for its dots (with
      // the fence after each update, 46 spilled VGPRs instead of 62).
#pragma unroll
      for (int b = 0; b < NB; ++b) asm volatile("" : "+a"(z[b]));
      pass<1, RD, GLOBAL>(src, xe, z, vh, vz, vv, zz, al, s, xz, lane);
    }
  }

  // z <- z / |z| (when `renorm` and z != 0)
  static __device__ __forceinline__ void unit(f32x16 (&z)[NB], bool renorm) {
    float zz = 0.0f;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) zz = fmaf(z[b][r], z[b][r], zz);
    zz = pair_sum(zz);
    const float s = (renorm && zz > 0.0f) ? rsqrtf(zz) : 1.0f;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) z[b][r] *= s;
  }
};

// Whether the persistent kernel also sums the action features: d <= 256 and
// its static chunk buffers, the table (at most 16 KiB) and the sums
// (WAVES * 32 rows of E + 1 floats) fit the 160 KiB of LDS.
template <class PR, int D, int E, int WAVES, bool NORM>
constexpr bool persistent_phi_ok() {
  constexpr int W1B = TransChunk<PR>::w1_bytes(D, E), W2B = TransChunk<PR>::w2_bytes(D);
  constexpr int WHB = HyperGeom<PR>::bytes(D, E);
  constexpr int stat = 2 * (W1B + W2B) + ((NORM && wh_in_lds(W1B, W2B, WHB)) ? WHB : 0);
  return D <= 256 && stat + 16 * 1024 + WAVES * 32 * (E + 1) * 4 <= 160 * 1024;
}

template <class PR, int D, int E, int WAVES, bool NORM>
__global__ __launch_bounds__(64 * WAVES, 1) void rollout_kernel(const RollArgs a) {
  using R = Roll<PR, D, E>;
  using Frag = typename PR::Frag;
  constexpr int KF = PR::KF, SL = PR::SL;
  // Overlap each chunk's GELU with the next chunk's first product (two
  // accumulators).  At d = 512 the latent fills the accumulator registers and
  // the second accumulator does not fit, so the chunks run one at a time.
  constexpr bool PIPE = D <= 256;
  constexpr int NZ = R::NZ, NE = R::NE, NF2 = R::NF2, NB = R::NB;
  constexpr int W1B = R::W1B, W2B = R::W2B;
  constexpr int NT = 64 * WAVES;

  __shared__ __attribute__((aligned(16))) uint8_t w1a[W1B];
  __shared__ __attribute__((aligned(16))) uint8_t w1b[W1B];
  __shared__ __attribute__((aligned(16))) uint8_t w2a[W2B];
  __shared__ __attribute__((aligned(16))) uint8_t w2b[W2B];
  using HY = Hyper<PR, D, E>;
  // the hyperplane-normal map stays in LDS when it fits beside the chunks
  constexpr bool WH_LDS = NORM && wh_in_lds(W1B, W2B, HY::BYTES);
  __shared__ __attribute__((aligned(16))) uint8_t whs[WH_LDS ? HY::BYTES : 16];
  extern __shared__ __attribute__((aligned(16))) float tab[];
  const float* t_emb = tab;                       // [K][E + 4]
  const float* t_pw = tab + a.K * temb_stride(E);              // [PMAX][E], zero rows past P
  const float* t_pb = t_pw + PMAX * E;            // [E]
  const float* t_b2 = t_pb + E;                   // [NB][2][16] accumulator order
  // action features (d <= 256; the launcher adds the area): running sums of
  // the step embeddings per candidate row, rows padded by one float
  constexpr bool PHI_OK = persistent_phi_ok<PR, D, E, WAVES, NORM>();
  const bool do_phi = PHI_OK && a.phi != nullptr;
  float* phib = tab + a.tab_bytes / 4;             // [WAVES * 32][E + 1]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  const int NC = a.H / 32;                        // even (checked on the host)

  // Tables and the first chunks.
  stage_to_lds(reinterpret_cast<const uint8_t*>(a.tab), reinterpret_cast<uint8_t*>(tab),
               a.tab_bytes, tid, NT);
  CopySrc cs;
  cs.r1 = __builtin_amdgcn_make_buffer_rsrc((void*)a.w1, (short)0, NC * W1B, 0x00020000);
  cs.r2 = __builtin_amdgcn_make_buffer_rsrc((void*)a.w2, (short)0, NC * W2B, 0x00020000);
  cs.voff = (uint32_t)tid * 16u;
  cs.wave_base = __builtin_amdgcn_readfirstlane(tid & ~63);
  stage_buf<W1B, NT>(cs.r1, 0u, w1a, cs, tid);
  stage_buf<W2B, NT>(cs.r2, 0u, w2a, cs, tid);
  if constexpr (PIPE) stage_buf<W1B, NT>(cs.r1, (uint32_t)W1B, w1b, cs, tid);
  if constexpr (WH_LDS) stage_fixed<HY::BYTES, NT>(a.wh, whs, tid);
  if (do_phi)
    for (int i = tid; i < WAVES * 32 * (E + 1); i += NT) phib[i] = 0.0f;

  const int pos = (blockIdx.x * WAVES + wave) * 32 + n;
  const bool valid = pos < a.B;
  const int2 pc = valid ? a.perm[pos] : make_int2(0, 0);
  const int cand = pc.x;
  const int len = valid ? clampi(a.lens[cand], 0, a.T_max) : 0;
  // Longest sequence in the workgroup: its first sorted position.
  const int T_wg = __builtin_amdgcn_readfirstlane(
      clampi(a.lens[a.perm[blockIdx.x * WAVES * 32].x], 0, a.T_max));

  // Latent in accumulator layout.
  f32x16 zacc[NB];
  {
    const float* zs = a.z0 + (size_t)pc.y * D;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(zs + 32 * b + acc_row(h, 4 * r4));
#pragma unroll
        for (int i = 0; i < 4; ++i) zacc[b][4 * r4 + i] = v[i];
      }
  }

  // Action of the current step (prefetched one step ahead; at d = 512, where
  // the latent fills the accumulator registers, loaded after the previous
  // step's chunks instead, so the prefetched values do not occupy registers
  // through the step).  Parameters past P read as 1 (log2 = 0) and meet
  // zero weights in the padded table.
  constexpr bool LATE_ACTION = D >= 512;
  int nx_type = 0;
  int nx_par[PMAX];
#pragma unroll
  for (int p = 0; p < PMAX; ++p) nx_par[p] = 1;
  if (0 < len) {
    nx_type = a.types[(size_t)cand * a.T_max];
#pragma unroll
    for (int p = 0; p < PMAX; ++p) if (p < a.P) nx_par[p] = a.params[(size_t)cand * a.T_max * a.P + p];
  }
  int errbits = 0;

  wait_vm_then_barrier();

  const int total = T_wg * NC;       // chunks processed by the workgroup
  for (int t = 0; t < T_wg; ++t) {
    const bool active = t < len;
    const float actf = active ? 1.0f : 0.0f;
    const uint32_t amask = active ? 0xFFFFFFFFu : 0u;
    // ---- action embedding e_t for features KF*q + SL*h + j (branch-free)
    const bool bad_type = active && (nx_type < 0 || nx_type >= a.K);
    const int ty = (active && !bad_type) ? nx_type : 0;
    bool bad_par = false;
    float u[PMAX];
#pragma unroll
    for (int p = 0; p < PMAX; ++p) {
      bad_par |= active && nx_par[p] < 1;
      u[p] = active ? log2f((float)nx_par[p]) : 0.0f;
    }
    errbits |= (bad_type ? ERRBIT_TYPE : 0) | (bad_par ? ERRBIT_PARAM : 0);
    if (!LATE_ACTION && t + 1 < len) {   // prefetch the next action
      const size_t row = (size_t)cand * a.T_max + t + 1;
      nx_type = a.types[row];
#pragma unroll
      for (int p = 0; p < PMAX; ++p) if (p < a.P) nx_par[p] = a.params[row * a.P + p];
    }
    Frag xe[NE];
#pragma unroll
    for (int q = 0; q < NE; ++q) {
      const int f0 = KF * q + SL * h;
      float ev[SL], tmp[SL];
      R::row(t_emb + ty * temb_stride(E) + f0, ev);
#pragma unroll
      for (int p = 0; p < PMAX; ++p) {
        R::row(t_pw + p * E + f0, tmp);
#pragma unroll
        for (int j = 0; j < SL; ++j) ev[j] = fmaf(tmp[j], u[p], ev[j]);
      }
      R::row(t_pb + f0, tmp);
#pragma unroll
      for (int j = 0; j < SL; ++j) ev[j] = (ev[j] + tmp[j]) * actf;
      xe[q] = PR::cvt(ev);
      if (do_phi) {
        float* ph = phib + (wave * 32 + n) * (E + 1) + f0;
#pragma unroll
        for (int j = 0; j < SL; ++j) ph[j] += ev[j];
      }
    }
    // ---- z operand fragments (state at the start of the step)
    Frag xz[NZ];
    if constexpr (NORM) {
      // unit length for the previous step's output, hyperplane projection
      // for this step; the operand fragments come from the projected state
      if constexpr (WH_LDS) HY::template step_in<4, false>(zacc, xe, whs, active, t > 0 && t <= len, xz, lane);
      else HY::template step_in<8, true>(zacc, xe, a.wh, active, t > 0 && t <= len, xz, lane);
    } else {
#pragma unroll
      for (int kf = 0; kf < NZ; ++kf) {
        float v[SL];
#pragma unroll
        for (int j = 0; j < SL; ++j) v[j] = zacc[kf / NF2][(kf % NF2) * SL + j];
        xz[kf] = PR::cvt(v);
      }
    }

    const int g0 = t * NC;
    // Chunk at position pos (0 <= pos < 2 NC, positions past NC belong to the
    // next step) of the workgroup's sequence: odd steps walk the chunks in
    // descending order, so a step starts with the chunks the previous one
    // used last.  Where the transition weights exceed an XCD's L2 (d = 512),
    // an ascending sweep every step would find each chunk evicted.
    auto chunk_of = [NC, t](int pos) -> uint32_t {
      const bool next = pos >= NC;
      const int c = next ? pos - NC : pos;
      return (uint32_t)((((t + (next ? 1 : 0)) & 1) != 0) ? NC - 1 - c : c);
    };
    const CopyPlan none = {0u, nullptr, false, 0u, nullptr, false};
    if constexpr (PIPE) {
      // first product of chunk 0 (its W1 part is in w1a); accumulators accA
      // and accB alternate between "GELU input" and "next first product"
      f32x16 accA, accB;
      R::template iteration<true, false, NT, false>(w1a, w2a, xz, xe, accB, amask, accA, zacc,
                                                    lane, h, none, cs, tid);
      __syncthreads();                 // all wavefronts are done with w1a
      for (int c = 0; c < NC; c += 2) {
        const int g = g0 + c;
        // -- chunk c: W2 part in w2a, next W1 part (chunk c+1) in w1b; the W2
        // part of chunk c+1 is copied into w2b and the W1 part of chunk c+2
        // into w1a (issued together up front: spreading them measured slower
        // for this schedule)
        if (g + 1 < total) stage_buf<W2B, NT>(cs.r2, chunk_of(c + 1) * (uint32_t)W2B, w2b, cs, tid);
        if (g + 2 < total) stage_buf<W1B, NT>(cs.r1, chunk_of(c + 2) * (uint32_t)W1B, w1a, cs, tid);
        __builtin_amdgcn_sched_barrier(0);
        R::template iteration<true, true, NT, false>(w1b, w2a, xz, xe, accA, amask, accB, zacc,
                                                     lane, h, none, cs, tid);
        wait_vm_then_barrier();
        // -- chunk c+1: W2 part in w2b, next W1 part (chunk c+2) in w1a.  At
        // c + 2 == NC this first product is discarded (w1a then holds the
        // next step's chunk 0 or stale data; the step prologue recomputes it
        // with the new X): one branch-free body keeps register use down.
        if (g + 2 < total) stage_buf<W2B, NT>(cs.r2, chunk_of(c + 2) * (uint32_t)W2B, w2a, cs, tid);
        if (g + 3 < total) stage_buf<W1B, NT>(cs.r1, chunk_of(c + 3) * (uint32_t)W1B, w1b, cs, tid);
        __builtin_amdgcn_sched_barrier(0);
        R::template iteration<true, true, NT, false>(w1a, w2b, xz, xe, accB, amask, accA, zacc,
                                                     lane, h, none, cs, tid);
        wait_vm_then_barrier();
      }
    } else {
      // one accumulator: first product, GELU, second product per chunk; chunk
      // c+1 (both parts) is copied into the other buffer pair meanwhile, the
      // copy instructions spread over the first product
      f32x16 acc;
      for (int c = 0; c < NC; c += 2) {
        const int g = g0 + c;
        const CopyPlan cp0 = {chunk_of(c + 1) * (uint32_t)W1B, to_lds(w1b), g + 1 < total,
                              chunk_of(c + 1) * (uint32_t)W2B, to_lds(w2b), g + 1 < total};
        R::template iteration<true, false, NT, true>(w1a, w2a, xz, xe, acc, amask, acc, zacc,
                                                     lane, h, cp0, cs, tid);
        R::template iteration<false, true, NT, false>(w1a, w2a, xz, xe, acc, amask, acc, zacc,
                                                      lane, h, none, cs, tid);
        wait_vm_then_barrier();
        const CopyPlan cp1 = {chunk_of(c + 2) * (uint32_t)W1B, to_lds(w1a), g + 2 < total,
                              chunk_of(c + 2) * (uint32_t)W2B, to_lds(w2a), g + 2 < total};
        R::template iteration<true, false, NT, true>(w1b, w2b, xz, xe, acc, amask, acc, zacc,
                                                     lane, h, cp1, cs, tid);
        R::template iteration<false, true, NT, false>(w1b, w2b, xz, xe, acc, amask, acc, zacc,
                                                      lane, h, none, cs, tid);
        wait_vm_then_barrier();
      }
    }
    if (LATE_ACTION && t + 1 < len) {    // the next action
      const size_t row = (size_t)cand * a.T_max + t + 1;
      nx_type = a.types[row];
#pragma unroll
      for (int p = 0; p < PMAX; ++p) if (p < a.P) nx_par[p] = a.params[row * a.P + p];
    }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) zacc[b][r] += t_b2[(b * 2 + h) * 16 + r] * actf;
  }
  // outputs of a workgroup's longest sequences still need their unit length
  if constexpr (NORM) HY::unit(zacc, T_wg > 0 && T_wg <= len);
  if (errbits) atomicOr(a.err, errbits);

  if (do_phi && valid) {         // phi = sum / len (0 when empty); the lane pair holds all features
    const float inv = len > 0 ? 1.0f / (float)len : 0.0f;
    const float* ph = phib + (wave * 32 + n) * (E + 1);
#pragma unroll
    for (int q = 0; q < NE; ++q)
#pragma unroll
      for (int j = 0; j < SL; ++j) {
        const int f = KF * q + SL * h + j;
        a.phi[(size_t)cand * E + f] = ph[f] * inv;
      }
  }
  if (valid) {
    float* zo = a.zT + (size_t)cand * D;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        f32x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = zacc[b][4 * r4 + i];
        *reinterpret_cast<f32x4*>(zo + 32 * b + acc_row(h, 4 * r4)) = v;
      }
  }
}

// ==========================================================================
// Small-batch rollout: when there are too few 32-candidate tiles to occupy
// the chip, one workgroup of SPLIT wavefronts works on one tile and splits the
// hidden units of every step among its wavefronts: wavefront w takes the
// chunks w, w + SPLIT, ...  Each wavefront streams its chunks' A fragments
// straight from L2 into a register ring (the wavefronts read different
// chunks, so staging in LDS would save nothing), accumulates a partial update
// dZ_w over the whole latent, and once per step the partial updates are
// summed through LDS: wavefront w owns latent blocks [w*NB/SPLIT, ...) in
// fp32, adds the sum and b2 to them, and publishes their bf16 (or fp32)
// operand fragments, which every wavefront reads back as X for the next step.
template <class PR, int D, int E>
struct SplitGeom {
  static constexpr int N1 = Roll<PR, D, E>::NK1 / PR::G;
  static constexpr int N2 = Roll<PR, D, E>::NK2 / PR::G;
  static constexpr int NI = N1 + N2;            // fragment groups per chunk
  // enough loads in flight to cover an L2 hit (~600 cycles): a bf16 group
  // feeds one 32-cycle product, an fp32 group four 64-cycle products
  static constexpr int ring_depth() {
    const int cap = PR::G == 1 ? 12 : 4;
    for (int r = cap; r > 1; --r)
      if (NI % r == 0) return r;
    return 1;
  }
  static constexpr int RD = ring_depth();       // loads in flight (divides NI)
};

//
// Paper-form transition: wavefront w also forms v = Wh . e for its own latent
// blocks (Wh fragments of those blocks stay in registers), and at the end of
// step t it folds the unit length of u_t and the projection of step t+1 into
// its blocks: the three dot products u.u, v.u, v.v are summed over the
// wavefronts through a small LDS area, in the same barrier interval as the
// partial-update reduction.
template <class PR, int D, int E, int SPLIT, bool NORM>
__global__ __launch_bounds__(64 * SPLIT, 1) void rollout_split_kernel(const RollArgs a) {
  using R = Roll<PR, D, E>;
  using SG = SplitGeom<PR, D, E>;
  using Frag = typename PR::Frag;
  constexpr int KF = PR::KF, SL = PR::SL, G = PR::G;
  constexpr int NZ = R::NZ, NE = R::NE, NF2 = R::NF2, NB = R::NB;
  constexpr int W1B = R::W1B, W2B = R::W2B;
  constexpr int NT = 64 * SPLIT;
  constexpr int NBQ = NB / SPLIT;               // latent blocks owned by a wavefront
  constexpr int N1 = SG::N1, NI = SG::NI, RD = SG::RD;
  constexpr int REGION = NB * 4 * 1024;         // one wavefront's partial update
  static_assert(NB % SPLIT == 0, "latent blocks split evenly");

  extern __shared__ __attribute__((aligned(16))) float tab[];
  const float* t_emb = tab;
  const float* t_pw = tab + a.K * temb_stride(E);
  const float* t_pb = t_pw + PMAX * E;
  const float* t_b2 = t_pb + E;
  uint8_t* red = reinterpret_cast<uint8_t*>(tab) + a.tab_bytes;   // SPLIT regions
  uint8_t* xbuf = red;                          // X fragments (reuses region space)
  float* dots = reinterpret_cast<float*>(red + (size_t)SPLIT * REGION);   // [SPLIT][3][32]
  using HY = Hyper<PR, D, E>;
  constexpr int GPB = HY::GPB;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  const int NC = a.H / 32;                      // >= SPLIT (checked on the host)

  stage_to_lds(reinterpret_cast<const uint8_t*>(a.tab), reinterpret_cast<uint8_t*>(tab),
               a.tab_bytes, tid, NT);

  const int pos = blockIdx.x * 32 + n;
  const bool valid = pos < a.B;
  const int2 pc = valid ? a.perm[pos] : make_int2(0, 0);
  const int cand = pc.x;
  const int len = valid ? clampi(a.lens[cand], 0, a.T_max) : 0;
  const int T_wg = __builtin_amdgcn_readfirstlane(
      clampi(a.lens[a.perm[blockIdx.x * 32].x], 0, a.T_max));

  // owned latent blocks (fp32) and the full X operand
  const float* zs = a.z0 + (size_t)pc.y * D;
  f32x16 zq[NBQ];
#pragma unroll
  for (int bq = 0; bq < NBQ; ++bq)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(zs + 32 * (w * NBQ + bq) + acc_row(h, 4 * r4));
#pragma unroll
      for (int i = 0; i < 4; ++i) zq[bq][4 * r4 + i] = v[i];
    }
  Frag xz[NZ];
#pragma unroll
  for (int kf = 0; kf < NZ; ++kf) {
    float v[SL];
#pragma unroll
    for (int j = 0; j < SL; ++j) v[j] = zs[x_feature<PR>(D, kf, h, j)];
    xz[kf] = PR::cvt(v);
  }

  const int32_t* ty_row = a.types + (size_t)cand * a.T_max;
  const int32_t* pa_row = a.params + (size_t)cand * a.T_max * a.P;
  int nx_type = 0;
  int nx_par[PMAX];
#pragma unroll
  for (int p = 0; p < PMAX; ++p) nx_par[p] = 1;
  if (0 < len) {
    nx_type = ty_row[0];
#pragma unroll
    for (int p = 0; p < PMAX; ++p) if (p < a.P) nx_par[p] = pa_row[p];
  }
  int errbits = 0;

  // Embedding fragments of step s (zero past the candidate's length); reads
  // the prefetched action of step s and prefetches step s + 1.
  auto embed_step = [&](int s, Frag (&xe)[NE]) {
    const bool act = s < len;
    const float af = act ? 1.0f : 0.0f;
    const bool bad_type = act && (nx_type < 0 || nx_type >= a.K);
    const int ty = (act && !bad_type) ? nx_type : 0;
    bool bad_par = false;
    float u[PMAX];
#pragma unroll
    for (int p = 0; p < PMAX; ++p) {
      bad_par |= act && nx_par[p] < 1;
      u[p] = act ? log2f((float)nx_par[p]) : 0.0f;
    }
    errbits |= (bad_type ? ERRBIT_TYPE : 0) | (bad_par ? ERRBIT_PARAM : 0);
    if (s + 1 < len) {
      nx_type = ty_row[s + 1];
#pragma unroll
      for (int p = 0; p < PMAX; ++p) if (p < a.P) nx_par[p] = pa_row[(size_t)(s + 1) * a.P + p];
    }
#pragma unroll
    for (int q = 0; q < NE; ++q) {
      const int f0 = KF * q + SL * h;
      float ev[SL], tmp[SL];
      R::row(t_emb + ty * temb_stride(E) + f0, ev);
#pragma unroll
      for (int p = 0; p < PMAX; ++p) {
        R::row(t_pw + p * E + f0, tmp);
#pragma unroll
        for (int j = 0; j < SL; ++j) ev[j] = fmaf(tmp[j], u[p], ev[j]);
      }
      R::row(t_pb + f0, tmp);
#pragma unroll
      for (int j = 0; j < SL; ++j) ev[j] = (ev[j] + tmp[j]) * af;
      xe[q] = PR::cvt(ev);
    }
  };

  // Paper form: Wh fragments of the owned blocks (constant over the launch).
  u32x4 whq[NORM ? NBQ * GPB : 1];
  if constexpr (NORM) {
#pragma unroll
    for (int i = 0; i < NBQ * GPB; ++i) whq[i] = HY::group(a.wh, w * NBQ * GPB + i, lane);
  }
  // Paper form, end of a step: zq <- (zq - alpha v) s over the owned blocks,
  // s = 1/|u| when the finished step was one of this candidate's, alpha =
  // (v.u)/(v.v) for the projection of step tn when that is one of its steps.
  auto boundary = [&](const Frag (&xe)[NE], bool renorm, bool project) {
    f32x16 vq[NBQ];
    float vz = 0.0f, vv = 0.0f, zz = 0.0f;
#pragma unroll
    for (int bq = 0; bq < NBQ; ++bq) {
      f32x16 vb = {};
#pragma unroll
      for (int k = 0; k < GPB; ++k)
#pragma unroll
        for (int ww = 0; ww < G; ++ww) vb = PR::mfma(PR::pick(whq[bq * GPB + k], ww), xe[k * G + ww], vb);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        vz = fmaf(vb[r], zq[bq][r], vz);
        vv = fmaf(vb[r], vb[r], vv);
        zz = fmaf(zq[bq][r], zq[bq][r], zz);
      }
      vq[bq] = vb;
    }
    vz = HY::pair_sum(vz);
    vv = HY::pair_sum(vv);
    zz = HY::pair_sum(zz);
    if (h == 0) {
      dots[(w * 3 + 0) * 32 + n] = vz;
      dots[(w * 3 + 1) * 32 + n] = vv;
      dots[(w * 3 + 2) * 32 + n] = zz;
    }
    __syncthreads();
    vz = 0.0f; vv = 0.0f; zz = 0.0f;
#pragma unroll
    for (int ww = 0; ww < SPLIT; ++ww) {
      vz += dots[(ww * 3 + 0) * 32 + n];
      vv += dots[(ww * 3 + 1) * 32 + n];
      zz += dots[(ww * 3 + 2) * 32 + n];
    }
    const float sc = (renorm && zz > 0.0f) ? rsqrtf(zz) : 1.0f;
    const float al = (project && vv > 0.0f) ? vz / vv : 0.0f;
#pragma unroll
    for (int bq = 0; bq < NBQ; ++bq)
#pragma unroll
      for (int r = 0; r < 16; ++r) zq[bq][r] = (zq[bq][r] - al * vq[bq][r]) * sc;
  };
  // publish the X fragments of the owned blocks, read back all of X
  auto exchange_x = [&]() {
#pragma unroll
    for (int bq = 0; bq < NBQ; ++bq)
#pragma unroll
      for (int f = 0; f < NF2; ++f) {
        const int kf = (w * NBQ + bq) * NF2 + f;
        float v[SL];
#pragma unroll
        for (int j = 0; j < SL; ++j) v[j] = zq[bq][f * SL + j];
        const Frag x = PR::cvt(v);
        *reinterpret_cast<Frag*>(xbuf + frag_offset<PR>(kf, lane, 0)) = x;
      }
    __syncthreads();
#pragma unroll
    for (int kf = 0; kf < NZ; ++kf) xz[kf] = *reinterpret_cast<const Frag*>(xbuf + frag_offset<PR>(kf, lane, 0));
    __syncthreads();                            // X read before the next step's partial updates
  };

  // A-fragment group i of chunk c (W1 part first, then W2 part)
  auto group_ptr = [&](int c, int i) -> const u32x4* {
    const uint8_t* base = i < N1 ? a.w1 + (size_t)c * W1B + (size_t)i * 1024
                                 : a.w2 + (size_t)c * W2B + (size_t)(i - N1) * 1024;
    return reinterpret_cast<const u32x4*>(base + lane * 16);
  };
  // register ring: slot i % RD holds group i of the current chunk; the last RD
  // groups of a chunk prefetch the first RD groups of the next one
  u32x4 ring[RD];
#pragma unroll
  for (int i = 0; i < RD; ++i) ring[i] = *group_ptr(w, i);

  wait_vm_then_barrier();

  Frag xe[NE];
  if constexpr (NORM) {
    // step 0: embedding, projection of z0 (no unit length: z0 is used as given)
    embed_step(0, xe);
    boundary(xe, false, 0 < len);
    exchange_x();
  }

  for (int t = 0; t < T_wg; ++t) {
    const bool active = t < len;
    const float actf = active ? 1.0f : 0.0f;
    const uint32_t amask = active ? 0xFFFFFFFFu : 0u;
    if constexpr (!NORM) embed_step(t, xe);

    f32x16 dz[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) dz[b] = f32x16{};
    for (int c = w; c < NC; c += SPLIT) {
      const int cn = (c + SPLIT < NC) ? c + SPLIT : w;     // next chunk of this wavefront
      const float* b1g = reinterpret_cast<const float*>(a.w1 + (size_t)c * W1B + (W1B - 128)) + 16 * h;
      f32x4 b1v[4];
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) b1v[r4] = *reinterpret_cast<const f32x4*>(b1g + 4 * r4);
      f32x16 acc = {};
      typename PR::Packed gp[8];
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const u32x4 grp = ring[i % RD];
        ring[i % RD] = (i + RD < NI) ? *group_ptr(c, i + RD) : *group_ptr(cn, i + RD - NI);
        if (i < N1) {
#pragma unroll
          for (int ww = 0; ww < G; ++ww) {
            const int kf = i * G + ww;
            acc = PR::mfma(PR::pick(grp, ww), kf < NZ ? xz[kf < NZ ? kf : 0] : xe[kf < NZ ? 0 : kf - NZ], acc);
          }
          if (i == N1 - 1) {
            // bias, GELU, mask -> operand of the second product
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4)
#pragma unroll
              for (int j = 0; j < 4; ++j) acc[4 * r4 + j] += b1v[r4][j];
#pragma unroll
            for (int q = 0; q < 8; ++q) gp[q] = PR::pack2(gelu(acc[2 * q]), gelu(acc[2 * q + 1]), amask);
          }
        } else {
#pragma unroll
          for (int ww = 0; ww < G; ++ww) {
            const int F = (i - N1) * G + ww;
            dz[F / NF2] = PR::mfma(PR::pick(grp, ww), PR::gfrag(gp, F % NF2), dz[F / NF2]);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    // ---- reduce the partial updates through LDS
    uint8_t* mine = red + (size_t)w * REGION;
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        f32x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = dz[b][4 * r4 + i];
        *reinterpret_cast<f32x4*>(mine + (b * 4 + r4) * 1024 + lane * 16) = v;
      }
    __syncthreads();
#pragma unroll
    for (int bq = 0; bq < NBQ; ++bq) {
      const int b = w * NBQ + bq;
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        f32x4 sum = *reinterpret_cast<const f32x4*>(red + (b * 4 + r4) * 1024 + lane * 16);
#pragma unroll
        for (int ww = 1; ww < SPLIT; ++ww)
          sum += *reinterpret_cast<const f32x4*>(red + (size_t)ww * REGION + (b * 4 + r4) * 1024 + lane * 16);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          zq[bq][4 * r4 + i] += sum[i] + t_b2[(b * 2 + h) * 16 + 4 * r4 + i] * actf;
      }
    }
    if constexpr (NORM) {
      // the barrier inside also turns the region space into the X buffer
      embed_step(t + 1, xe);
      boundary(xe, active, t + 1 < len);
    } else {
      __syncthreads();                          // region space becomes the X buffer
    }
    exchange_x();
  }
  if (errbits) atomicOr(a.err, errbits);
  if (valid) {
    float* zo = a.zT + (size_t)cand * D;
#pragma unroll
    for (int bq = 0; bq < NBQ; ++bq)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        f32x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = zq[bq][4 * r4 + i];
        *reinterpret_cast<f32x4*>(zo + 32 * (w * NBQ + bq) + acc_row(h, 4 * r4)) = v;
      }
  }
}

// ==========================================================================
// Row-owned rollout (d = 256, 32-candidate tiles): the training forward of
// the rollout loss above 8192 candidates (narrow tiles take every smaller
// batch, and every evaluator batch this kernel could take, so its evaluator
// form, TRAIN = false, is not dispatched).  One workgroup of W wavefronts per
// tile, two per SIMD in bf16.  Wavefront w computes the first
// product and GELU of the hidden chunks w, w + W, ... and writes the GELU
// outputs as operand fragments to LDS; after one barrier it forms the update
// of its own NB/W latent blocks over all NC chunks, reading every chunk's GELU
// fragments from LDS and the matching W2 rows from L2.  Nothing is reduced
// across wavefronts, there are two barriers per step, and the W2 rows a
// wavefront reads are only its own blocks', so each wavefront streams 1/W of
// the step's weights.  A step is one fully unrolled stream of 16-byte-per-lane
// weight groups (first-product groups of the wavefront's chunks, then its W2
// groups of every chunk) read RD ahead into a register ring that wraps into
// the next step (the weights are the same every step).
template <class PR, int D, int E, int NC, int W>
struct RowsGeom {
  using R = Roll<PR, D, E>;
  static constexpr int G = PR::G;
  static constexpr int NB = R::NB, NBW = NB / W;          // latent blocks per wavefront
  static constexpr int NCW = NC / W;                      // first-product chunks per wavefront
  static constexpr int N1 = R::NK1 / G;                   // W1 groups per chunk
  static constexpr int G2 = R::NF2 / G;                   // W2 groups per (chunk, block)
  static constexpr int N2 = NBW * G2;                     // W2 groups per chunk
  static constexpr int NA = NCW * N1, NI = NA + NC * N2;  // items per step
  static constexpr int GB = R::NF2 / G;                   // GELU fragment groups per chunk
  // groups in flight: the ring wraps into the next step, so item j must sit
  // in slot j % RD in every step, which needs RD to divide NI
  static constexpr int ring_depth() {
    const int cap = G == 1 ? 12 : 8;
    for (int r = cap; r > 1; --r)
      if (NI % r == 0) return r;
    return 1;
  }
  static constexpr int RD = ring_depth();
  static_assert(NB % W == 0 && NC % W == 0, "even split");
  // LDS: [table][GELU fragments: NC * GB KiB][X fragments: NZ / G KiB]
  //      [embedding fragments: NE / G KiB][dots]
  static constexpr int GELU_BYTES = NC * GB * 1024;
  static constexpr int X_BYTES = (R::NZ / G) * 1024;
  static constexpr int NEG = R::NE / G;                   // embedding fragment groups
  static constexpr int XE_BYTES = NEG * 1024;
};

template <class PR, int D, int E, int NC, int W, bool NORM, bool TRAIN = false>
__global__ __launch_bounds__(64 * W, 1) void rollout_rows_kernel(const RollArgs a) {
  using R = Roll<PR, D, E>;
  using RG = RowsGeom<PR, D, E, NC, W>;
  using Frag = typename PR::Frag;
  using HY = Hyper<PR, D, E>;
  constexpr int KF = PR::KF, SL = PR::SL, G = PR::G;
  constexpr int NZ = R::NZ, NE = R::NE, NF2 = R::NF2, NB = R::NB;
  constexpr int W1B = R::W1B, W2B = R::W2B;
  constexpr int NBW = RG::NBW, NCW = RG::NCW, N1 = RG::N1, G2 = RG::G2, N2 = RG::N2;
  constexpr int NA = RG::NA, NI = RG::NI, RD = RG::RD, GB = RG::GB;
  constexpr int NT = 64 * W;
  constexpr int GPB = HY::GPB;

  extern __shared__ __attribute__((aligned(16))) float tab[];
  const float* t_emb = tab;
  const float* t_pw = tab + a.K * temb_stride(E);
  const float* t_pb = t_pw + PMAX * E;
  const float* t_b2 = t_pb + E;
  uint8_t* gbuf = reinterpret_cast<uint8_t*>(tab) + a.tab_bytes;   // GELU fragments
  uint8_t* xbuf = gbuf + RG::GELU_BYTES;                            // X fragments
  uint8_t* xebuf = xbuf + RG::X_BYTES;                              // embedding fragments
  float* dots = reinterpret_cast<float*>(xebuf + RG::XE_BYTES);     // [W][3][32]
  // action features: the running sum of each owned embedding fragment, per
  // candidate row (rows padded by one float against bank conflicts)
  float* phib = dots + (NORM ? W * 3 * 32 : 0);                      // [32][E + 1]
  const bool do_phi = !TRAIN && a.phi != nullptr;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = lane & 31, h = lane >> 5;

  stage_to_lds(reinterpret_cast<const uint8_t*>(a.tab), reinterpret_cast<uint8_t*>(tab),
               a.tab_bytes, tid, NT);
  if (do_phi)
    for (int i = tid; i < 32 * (E + 1); i += NT) phib[i] = 0.0f;

  const int pos = blockIdx.x * 32 + n;
  const bool valid = pos < a.B;
  const int2 pc = valid ? a.perm[pos] : make_int2(0, 0);
  const int cand = pc.x;
  const int len = valid ? clampi(a.lens[cand], 0, a.T_max) : 0;
  const int T_wg = __builtin_amdgcn_readfirstlane(
      clampi(a.lens[a.perm[blockIdx.x * 32].x], 0, a.T_max));
  constexpr int IN = D + E;
  const size_t row0 = (TRAIN && valid) ? (size_t)a.off[cand] : 0;

  // owned latent blocks (fp32) and the full X operand
  const float* zs = a.z0 + (size_t)pc.y * D;
  f32x16 zq[NBW];
#pragma unroll
  for (int bq = 0; bq < NBW; ++bq)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(zs + 32 * (w * NBW + bq) + acc_row(h, 4 * r4));
#pragma unroll
      for (int i = 0; i < 4; ++i) zq[bq][4 * r4 + i] = v[i];
    }
  Frag xz[NZ];
#pragma unroll
  for (int kf = 0; kf < NZ; ++kf) {
    float v[SL];
#pragma unroll
    for (int j = 0; j < SL; ++j) v[j] = zs[x_feature<PR>(D, kf, h, j)];
    xz[kf] = PR::cvt(v);
  }

  const int32_t* ty_row = a.types + (size_t)cand * a.T_max;
  const int32_t* pa_row = a.params + (size_t)cand * a.T_max * a.P;
  int nx_type = 0;
  int nx_par[PMAX];
#pragma unroll
  for (int p = 0; p < PMAX; ++p) nx_par[p] = 1;
  if (0 < len) {
    nx_type = ty_row[0];
#pragma unroll
    for (int p = 0; p < PMAX; ++p) if (p < a.P) nx_par[p] = pa_row[p];
  }
  int errbits = 0;
  Frag xe[NE];

  // Action of step s: kind, log2 parameters, activity; error bits; prefetch
  // of step s + 1 (every wavefront: they all hold the tile's candidates).
  auto decode = [&](int s, int& ty, float (&u)[PMAX], float& af) {
    const bool act = s < len;
    af = act ? 1.0f : 0.0f;
    const bool bad_type = act && (nx_type < 0 || nx_type >= a.K);
    ty = (act && !bad_type) ? nx_type : 0;
    bool bad_par = false;
#pragma unroll
    for (int p = 0; p < PMAX; ++p) {
      bad_par |= act && nx_par[p] < 1;
      u[p] = act ? log2f((float)nx_par[p]) : 0.0f;
    }
    errbits |= (bad_type ? ERRBIT_TYPE : 0) | (bad_par ? ERRBIT_PARAM : 0);
    if (s + 1 < len) {
      nx_type = ty_row[s + 1];
#pragma unroll
      for (int p = 0; p < PMAX; ++p) if (p < a.P) nx_par[p] = pa_row[(size_t)(s + 1) * a.P + p];
    }
  };
  // embedding fragment q (features KF*q + SL*h + j)
  auto embed_vals = [&](int ty, const float (&u)[PMAX], float af, int q, float (&ev)[SL]) {
    const int f0 = KF * q + SL * h;
    float tmp[SL];
    R::row(t_emb + ty * temb_stride(E) + f0, ev);
#pragma unroll
    for (int p = 0; p < PMAX; ++p) {
      R::row(t_pw + p * E + f0, tmp);
#pragma unroll
      for (int j = 0; j < SL; ++j) ev[j] = fmaf(tmp[j], u[p], ev[j]);
    }
    R::row(t_pb + f0, tmp);
#pragma unroll
    for (int j = 0; j < SL; ++j) ev[j] = (ev[j] + tmp[j]) * af;
  };
  // running sum of fragment q's features (inactive steps add zero)
  auto phi_add = [&](int q, const float (&ev)[SL]) {
    float* ph = phib + n * (E + 1) + KF * q + SL * h;
#pragma unroll
    for (int j = 0; j < SL; ++j) ph[j] += ev[j];
  };
  // all fragments in this wavefront (paper form: the normal map needs them
  // before the step's exchange); the owner of each fragment group sums it
  auto embed_step = [&](int s, Frag (&xe)[NE]) {
    int ty;
    float u[PMAX], af;
    decode(s, ty, u, af);
#pragma unroll
    for (int q = 0; q < NE; ++q) {
      float ev[SL];
      embed_vals(ty, u, af, q, ev);
      xe[q] = PR::cvt(ev);
      if (do_phi && (q / G) % W == w) phi_add(q, ev);
      if constexpr (TRAIN) {
        if ((q / G) % W == w && s < len) {
          float* xo = a.X + (row0 + s) * IN + D + KF * q + SL * h;
#pragma unroll
          for (int j = 0; j < SL; ++j) xo[j] = op_value<PR>(ev[j]);
        }
      }
    }
  };
  // this wavefront's share of the fragment groups, into LDS (read back with X)
  auto embed_share = [&](int s) {
    int ty;
    float u[PMAX], af;
    decode(s, ty, u, af);
#pragma unroll
    for (int gq = 0; gq < RG::NEG; ++gq) {
      if (gq % W != w) continue;
#pragma unroll
      for (int k = 0; k < G; ++k) {
        const int q = gq * G + k;
        float ev[SL];
        embed_vals(ty, u, af, q, ev);
        *reinterpret_cast<Frag*>(xebuf + frag_offset<PR>(q, lane, 0)) = PR::cvt(ev);
        if (do_phi) phi_add(q, ev);
        if constexpr (TRAIN) {
          if (s < len) {
            float* xo = a.X + (row0 + s) * IN + D + KF * q + SL * h;
#pragma unroll
            for (int j = 0; j < SL; ++j) xo[j] = op_value<PR>(ev[j]);
          }
        }
      }
    }
  };

  // Paper form (see the split kernel): owned Wh fragments, dots through LDS.
  u32x4 whq[NORM ? NBW * GPB : 1];
  if constexpr (NORM) {
#pragma unroll
    for (int i = 0; i < NBW * GPB; ++i) whq[i] = HY::group(a.wh, w * NBW * GPB + i, lane);
  }
  // Training mode: the unit-length prediction of the finished step t and
  // |u| go to row t, the next step's v, v.z and v.v to row t + 1.
  auto boundary = [&](const Frag (&xe)[NE], bool renorm, bool project, int t) {
    f32x16 vq[NBW];
    float vz = 0.0f, vv = 0.0f, zz = 0.0f;
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq) {
      f32x16 vb = {};
#pragma unroll
      for (int k = 0; k < GPB; ++k)
#pragma unroll
        for (int ww = 0; ww < G; ++ww) vb = PR::mfma(PR::pick(whq[bq * GPB + k], ww), xe[k * G + ww], vb);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        vz = fmaf(vb[r], zq[bq][r], vz);
        vv = fmaf(vb[r], vb[r], vv);
        zz = fmaf(zq[bq][r], zq[bq][r], zz);
      }
      vq[bq] = vb;
    }
    vz = HY::pair_sum(vz);
    vv = HY::pair_sum(vv);
    zz = HY::pair_sum(zz);
    if (h == 0) {
      dots[(w * 3 + 0) * 32 + n] = vz;
      dots[(w * 3 + 1) * 32 + n] = vv;
      dots[(w * 3 + 2) * 32 + n] = zz;
    }
    __syncthreads();
    vz = 0.0f; vv = 0.0f; zz = 0.0f;
#pragma unroll
    for (int ww = 0; ww < W; ++ww) {
      vz += dots[(ww * 3 + 0) * 32 + n];
      vv += dots[(ww * 3 + 1) * 32 + n];
      zz += dots[(ww * 3 + 2) * 32 + n];
    }
    const float sc = (renorm && zz > 0.0f) ? rsqrtf(zz) : 1.0f;
    const float al = (project && vv > 0.0f) ? vz / vv : 0.0f;
    if constexpr (TRAIN) {
      if (renorm) {              // step t was active
        const size_t rt = row0 + t;
#pragma unroll
        for (int bq = 0; bq < NBW; ++bq) {
          f32x16 pv;
#pragma unroll
          for (int r = 0; r < 16; ++r) pv[r] = zq[bq][r] * sc;
          store_acc(a.Pz + rt * D + 32 * (w * NBW + bq), pv, h);
        }
        if (w == 0 && h == 0) a.SC[rt * 4 + 2] = sqrtf(zz);
      }
      if (project) {             // step t + 1 is active
        const size_t rs = row0 + (t + 1);
#pragma unroll
        for (int bq = 0; bq < NBW; ++bq) store_acc(a.V + rs * D + 32 * (w * NBW + bq), vq[bq], h);
        if (w == 0 && h == 0) {
          a.SC[rs * 4 + 0] = vz * sc;
          a.SC[rs * 4 + 1] = vv;
          a.SC[rs * 4 + 3] = 0.0f;
        }
      }
    }
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq)
#pragma unroll
      for (int r = 0; r < 16; ++r) zq[bq][r] = (zq[bq][r] - al * vq[bq][r]) * sc;
  };
  // publish the owned blocks' X fragments, read back all of X (own buffer:
  // the next overwrite comes after the next step's first barrier)
  auto exchange_x = [&]() {
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq)
#pragma unroll
      for (int f = 0; f < NF2; ++f) {
        const int kf = (w * NBW + bq) * NF2 + f;
        float v[SL];
#pragma unroll
        for (int j = 0; j < SL; ++j) v[j] = zq[bq][f * SL + j];
        const Frag x = PR::cvt(v);
        *reinterpret_cast<Frag*>(xbuf + frag_offset<PR>(kf, lane, 0)) = x;
      }
    __syncthreads();
#pragma unroll
    for (int kf = 0; kf < NZ; ++kf) xz[kf] = *reinterpret_cast<const Frag*>(xbuf + frag_offset<PR>(kf, lane, 0));
    if constexpr (!NORM) {
#pragma unroll
      for (int q = 0; q < NE; ++q) xe[q] = *reinterpret_cast<const Frag*>(xebuf + frag_offset<PR>(q, lane, 0));
    }
  };

  // Weight group of stream item i (i < NI), relative to the wavefront's two
  // base addresses; compile-time after unrolling.
  auto item_off = [](int i) -> size_t {
    if (i < NA) return (size_t)((i / N1) * W) * W1B + (size_t)(i % N1) * 1024;
    const int j = i - NA;
    return (size_t)(j / N2) * W2B + (size_t)(j % N2) * 1024;
  };
  gu8* baseA = ((gu8*)(a.w1)) + (size_t)w * W1B + lane * 16;
  gu8* baseB = ((gu8*)(a.w2)) + (size_t)(w * N2) * 1024 + lane * 16;
  auto item_ptr = [&](gu8* pA, gu8* pB, int i) -> gu32x4* {
    return reinterpret_cast<gu32x4*>((i < NA ? pA : pB) + item_off(i));
  };

  u32x4 ring[RD];
#pragma unroll
  for (int i = 0; i < RD; ++i) ring[i] = *item_ptr(baseA, baseB, i);

  wait_vm_then_barrier();

  if constexpr (NORM) {
    embed_step(0, xe);
    boundary(xe, false, 0 < len, -1);
  } else {
    embed_share(0);
  }
  exchange_x();

  for (int t = 0; t < T_wg; ++t) {
    const bool active = t < len;
    const float actf = active ? 1.0f : 0.0f;
    const uint32_t amask = active ? 0xFFFFFFFFu : 0u;
    // opaque per-step bases: the item addresses are rebuilt from them rather
    // than hoisted out of the step loop (one 64-bit address per item)
    gu8* pA = baseA;
    gu8* pB = baseB;
    asm volatile("" : "+v"(pA), "+v"(pB));
    const size_t row = row0 + t;
    if constexpr (TRAIN) {
      if (active) {            // X = [z; e]: the owned latent blocks (e: embed_share)
#pragma unroll
        for (int bq = 0; bq < NBW; ++bq) {
          f32x16 v;
#pragma unroll
          for (int r = 0; r < 16; ++r) v[r] = op_value<PR>(zq[bq][r]);
          store_acc(a.X + row * IN + 32 * (w * NBW + bq), v, h);
        }
        if (w == 0 && h == 0) a.row_src[row] = cand * a.T_max + t;
      }
    }

    f32x16 acc = {};
    f32x4 b1v[4];
    f32x16 dz[NBW];
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq) dz[bq] = f32x16{};
    typename PR::Packed gp[8];
    u32x4 gcur[GB], gnext[GB];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const u32x4 grp = ring[i % RD];
      ring[i % RD] = *item_ptr(pA, pB, (i + RD) % NI);   // wraps into the next step
      if (i < NA) {
        // ---- first product of chunk w + cw*W, group g
        const int cw = i / N1, g = i % N1;
        if (g == 0) {
          acc = f32x16{};
          const float* b1g = reinterpret_cast<const float*>(a.w1 + (size_t)(w + cw * W) * W1B + (W1B - 128)) + 16 * h;
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) b1v[r4] = *reinterpret_cast<const f32x4*>(b1g + 4 * r4);
        }
#pragma unroll
        for (int ww = 0; ww < G; ++ww) {
          const int kf = g * G + ww;
          acc = PR::mfma(PR::pick(grp, ww), kf < NZ ? xz[kf < NZ ? kf : 0] : xe[kf < NZ ? 0 : kf - NZ], acc);
        }
        if (g == N1 - 1) {
          // bias, GELU, mask -> operand fragments of chunk c in LDS
          const int c = w + cw * W;
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[4 * r4 + j] += b1v[r4][j];
          if constexpr (TRAIN) {
            f32x16 gv;
#pragma unroll
            for (int r = 0; r < 16; ++r) gv[r] = op_value<PR>(gelu(acc[r]));
#pragma unroll
            for (int q = 0; q < 8; ++q) gp[q] = PR::pack2(gv[2 * q], gv[2 * q + 1], amask);
            if (active) {
              store_acc(a.A + row * a.H + 32 * c, acc, h);
              store_acc(a.G + row * a.H + 32 * c, gv, h);
            }
          } else {
#pragma unroll
            for (int q = 0; q < 8; ++q) gp[q] = PR::pack2(gelu(acc[2 * q]), gelu(acc[2 * q + 1]), amask);
          }
#pragma unroll
          for (int f = 0; f < NF2; ++f)
            *reinterpret_cast<Frag*>(gbuf + frag_offset<PR>(c * NF2 + f, lane, 0)) = PR::gfrag(gp, f);
        }
        if (i == NA - 1) {
          __syncthreads();             // every chunk's GELU fragments are in LDS
#pragma unroll
          for (int gg = 0; gg < GB; ++gg) gcur[gg] = lds_group(gbuf, gg, lane);
#pragma unroll
          for (int gg = 0; gg < GB; ++gg) gnext[gg] = lds_group(gbuf, (NC > 1 ? GB : 0) + gg, lane);
        }
      } else {
        // ---- update of the owned blocks from chunk c, group k
        const int j = i - NA, c = j / N2, k = j % N2;
        const int bq = k / G2, gg2 = k % G2;
#pragma unroll
        for (int ww = 0; ww < G; ++ww) {
          const int f = gg2 * G + ww;             // GELU fragment of chunk c
          const u32x4 gf = gcur[(f * SL * PR::ES) / 16];
          Frag b;
          if constexpr (G == 1) b = PR::pick(gf, 0);
          else b = PR::pick(gf, f % G);
          dz[bq] = PR::mfma(PR::pick(grp, ww), b, dz[bq]);
        }
        if (k == N2 - 1) {
          // rotate the GELU fragments: chunk c+1 current, chunk c+2 prefetched
#pragma unroll
          for (int gg = 0; gg < GB; ++gg) gcur[gg] = gnext[gg];
          if (c + 2 < NC) {
#pragma unroll
            for (int gg = 0; gg < GB; ++gg) gnext[gg] = lds_group(gbuf, (c + 2) * GB + gg, lane);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // ---- owned blocks: z += dZ + b2
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq) {
      const int b = w * NBW + bq;
#pragma unroll
      for (int r = 0; r < 16; ++r) zq[bq][r] += dz[bq][r] + t_b2[(b * 2 + h) * 16 + r] * actf;
      if constexpr (TRAIN && !NORM) {
        if (active) store_acc(a.Pz + row * D + 32 * b, zq[bq], h);
      }
    }
    if constexpr (NORM) {
      embed_step(t + 1, xe);
      boundary(xe, active, t + 1 < len, t);
    } else {
      embed_share(t + 1);
    }
    exchange_x();
  }
  if (errbits) atomicOr(a.err, errbits);
  if (do_phi && valid) {         // phi = sum / len over the owned fragments (0 when empty)
    const float inv = len > 0 ? 1.0f / (float)len : 0.0f;
#pragma unroll
    for (int q = 0; q < NE; ++q) {
      if ((q / G) % W != w) continue;
      const float* ph = phib + n * (E + 1) + KF * q + SL * h;
#pragma unroll
      for (int j = 0; j < SL; ++j) a.phi[(size_t)cand * E + KF * q + SL * h + j] = ph[j] * inv;
    }
  }
  if (valid && !TRAIN) {
    float* zo = a.zT + (size_t)cand * D;
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        f32x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = zq[bq][4 * r4 + i];
        *reinterpret_cast<f32x4*>(zo + 32 * (w * NBW + bq) + acc_row(h, 4 * r4)) = v;
      }
  }
}

// ==========================================================================
// Narrow-tile rollout (d = 32 W): one workgroup of W wavefronts per tile of
// 16 candidates, on the 16x16 matrix-core products (layouts at Narrow in
// wm_internal.h).  For batches that give at most one tile per compute unit
// the kernel time is the longest tile's chain of steps, and a step of 16
// candidates is half the products and half the GELUs of a 32-candidate step
// with the same number of exchanges.
//  * wavefront w owns latent blocks 2w, 2w+1 (16 features each, 4 per lane),
//    which together are operand fragment w of z: it publishes that fragment
//    in LDS and, after a barrier, every wavefront reads all fragments of X;
//  * first product, for its chunks c = w, w + W, ...: two 16-row output
//    blocks per chunk over the NK fragments of X, bias, GELU, rounding, and
//    the chunk's GELU fragment into LDS;
//  * after a barrier, the update of its two latent blocks over every chunk.
// Weight groups stream from L2 through a register ring that wraps from
// step to step.  Wavefronts w < E/32 also embed the next step's action and
// sum the action features.
//
// An operand fragment is 8 values per lane (32 contraction slots over the 4
// lane groups).  bf16: one 16x16x32 product per fragment, one 1 KiB group of
// A operands.  fp32: four 16x16x4 products per 1 KiB group, two groups per
// fragment (slots 4hh .. 4hh + 3 in half hh); fragments in LDS as two 1 KiB
// halves.
typedef float f32x4n __attribute__((ext_vector_type(4)));
typedef float f32x8n __attribute__((ext_vector_type(8)));
constexpr int SCORE_MAX_HW = 32;        // hardware-vector width limit

struct NarrowBF16 {
  using XF = bf16x8;
  static constexpr int GPK = 1;                 // 1 KiB groups per fragment
  static __device__ __forceinline__ float op(float v) { return (float)(__bf16)v; }
  static __device__ __forceinline__ XF cvt(const float (&v)[8]) {
    XF f;
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = (__bf16)v[j];
    return f;
  }
  static __device__ __forceinline__ f32x4n mma(u32x4 grp, int, const XF& x, f32x4n acc) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, grp), x, acc, 0, 0, 0);
  }
  static __device__ __forceinline__ void store(uint8_t* buf, int frag, int lane, const XF& x) {
    *reinterpret_cast<XF*>(buf + frag * 1024 + lane * 16) = x;
  }
  static __device__ __forceinline__ XF load(const uint8_t* buf, int frag, int lane) {
    return *reinterpret_cast<const XF*>(buf + frag * 1024 + lane * 16);
  }
  // GELU outputs (masked) as an operand fragment
  static __device__ __forceinline__ XF gfrag(const float (&v)[8], uint32_t m) {
    u32x4 u = __builtin_bit_cast(u32x4, cvt(v));
    u &= m;
    return __builtin_bit_cast(XF, u);
  }
};

struct NarrowF32 {
  using XF = f32x8n;
  static constexpr int GPK = 2;
  static __device__ __forceinline__ float op(float v) { return v; }
  static __device__ __forceinline__ XF cvt(const float (&v)[8]) {
    XF f;
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = v[j];
    return f;
  }
  static __device__ __forceinline__ f32x4n mma(u32x4 grp, int hh, const XF& x, f32x4n acc) {
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const uint32_t a = grp[jj];
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a), x[4 * hh + jj], acc, 0, 0, 0);
    }
    return acc;
  }
  static __device__ __forceinline__ void store(uint8_t* buf, int frag, int lane, const XF& x) {
    const f32x4n lo = {x[0], x[1], x[2], x[3]}, hi = {x[4], x[5], x[6], x[7]};
    *reinterpret_cast<f32x4n*>(buf + (2 * frag) * 1024 + lane * 16) = lo;
    *reinterpret_cast<f32x4n*>(buf + (2 * frag + 1) * 1024 + lane * 16) = hi;
  }
  static __device__ __forceinline__ XF load(const uint8_t* buf, int frag, int lane) {
    const f32x4n lo = *reinterpret_cast<const f32x4n*>(buf + (2 * frag) * 1024 + lane * 16);
    const f32x4n hi = *reinterpret_cast<const f32x4n*>(buf + (2 * frag + 1) * 1024 + lane * 16);
    const XF x = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return x;
  }
  static __device__ __forceinline__ XF gfrag(const float (&v)[8], uint32_t m) {
    XF f;
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = __uint_as_float(__float_as_uint(v[j]) & m);
    return f;
  }
};

template <class NP, int D, int E, int NC, int W>
struct NarrowGeom {
  static constexpr int GPK = NP::GPK;
  static constexpr int NB = D / 16, NBW = NB / W;          // latent blocks, per wavefront
  static constexpr int NZ = D / 32, NE = E / 32, NK = NZ + NE;
  static constexpr int NCW = NC / W;                       // first-product chunks per wavefront
  static constexpr int NA = NCW * NK * 2 * GPK;            // first-product groups per step
  static constexpr int NI = NA + NC * NBW * GPK;           // groups per step
  static constexpr int W1G = NC * NK * 2 * GPK;            // W1 groups in the blob
  static constexpr int W2G = NC * NB * GPK;
  static constexpr int ring_depth() {
    for (int r = 12; r > 1; --r)
      if (NI % r == 0) return r;
    return 1;
  }
  static constexpr int RD = ring_depth();
  static_assert(NBW == 2 && NZ == W, "wavefront w owns z fragment w");
  static_assert(NC % W == 0 && NE <= W, "even split");
  static constexpr int G_BYTES = NC * GPK * 1024, X_BYTES = NK * GPK * 1024;
};

// TRAIN: the training forward of the rollout loss; stores, per valid step in
// compact row off[i] + t, the operands X = [z; e], the pre-activations A,
// the GELU outputs G and the prediction, as the 32-wide row-owned kernel
// does (paper form: the unit prediction, |u|, v and the dots v.z, v.v).
// SCORE: after the last step the workgroup also scores its candidates with
// the cost model (Eq. 3) for every hardware vector: wavefront w takes the
// cost-hidden chunks w, w + W, ...; the [z_T; phi] part of the first product
// is shared by the hardware vectors; partial scores are summed over the
// candidate's lane groups and then over the wavefronts in a fixed order.
constexpr int NARROW_SCORE_HW = 2;      // hardware vectors per fused launch
template <class NP, int D, int E, int NC, int W, bool NORM, bool TRAIN = false, bool SCORE = false>
__global__ __launch_bounds__(64 * W, 1) void rollout_narrow_kernel(const RollArgs a) {
  static_assert(!(TRAIN && SCORE), "scores belong to the evaluator");
  using NG = NarrowGeom<NP, D, E, NC, W>;
  using XF = typename NP::XF;
  constexpr int GPK = NG::GPK, NK = NG::NK, NZ = NG::NZ, NE = NG::NE, NB = NG::NB, NBW = NG::NBW;
  constexpr int NCW = NG::NCW, NA = NG::NA, NI = NG::NI, RD = NG::RD, NT = 64 * W;

  extern __shared__ __attribute__((aligned(16))) float tab[];
  const float* t_emb = tab;
  const float* t_pw = tab + a.K * temb_stride(E);
  const float* t_pb = t_pw + PMAX * E;
  uint8_t* gbuf = reinterpret_cast<uint8_t*>(tab) + a.tab_bytes;     // GELU fragments [NC]
  uint8_t* xbuf = gbuf + NG::G_BYTES;                                 // X fragments [NK]
  float* dots = reinterpret_cast<float*>(xbuf + NG::X_BYTES);         // paper form: [W][3][16]
  float* phib = dots + (NORM ? W * 3 * 16 : 0);                       // [16][E + 1]
  const bool do_phi = !TRAIN && a.phi != nullptr;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = lane & 15, g = lane >> 4;
  constexpr int IN = D + E;
  stage_to_lds(reinterpret_cast<const uint8_t*>(a.tab), reinterpret_cast<uint8_t*>(tab),
               a.tab_bytes, tid, NT);
  if (do_phi)
    for (int i = tid; i < 16 * (E + 1); i += NT) phib[i] = 0.0f;

  const int pos = blockIdx.x * 16 + n;
  const bool valid = pos < a.B;
  const int2 pc = valid ? a.perm[pos] : make_int2(0, 0);
  const int cand = pc.x;
  const int len = valid ? clampi(a.lens[cand], 0, a.T_max) : 0;
  const int T_wg = __builtin_amdgcn_readfirstlane(
      clampi(a.lens[a.perm[blockIdx.x * 16].x], 0, a.T_max));
  const size_t row0 = (TRAIN && valid) ? (size_t)a.off[cand] : 0;

  const float* b1n = reinterpret_cast<const float*>(a.w1 + (size_t)(NG::W1G + NG::W2G) * 1024);
  const float* b2n = b1n + NC * 32;
  // owned latent blocks 2w + bq, their b2, and the b1 of the own chunks
  const float* zs = a.z0 + (size_t)pc.y * D;
  f32x4n zq[NBW], b2v[NBW], b1v[NCW][2];
#pragma unroll
  for (int bq = 0; bq < NBW; ++bq) {
    zq[bq] = *reinterpret_cast<const f32x4n*>(zs + 16 * (w * NBW + bq) + 4 * g);
    b2v[bq] = *reinterpret_cast<const f32x4n*>(b2n + 16 * (w * NBW + bq) + 4 * g);
  }
#pragma unroll
  for (int cw = 0; cw < NCW; ++cw)
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
      b1v[cw][rb] = *reinterpret_cast<const f32x4n*>(b1n + 32 * (w + cw * W) + 16 * rb + 4 * g);

  const int32_t* ty_row = a.types + (size_t)cand * a.T_max;
  const int32_t* pa_row = a.params + (size_t)cand * a.T_max * a.P;
  int nx_type = 0;
  int nx_par[PMAX];
#pragma unroll
  for (int p = 0; p < PMAX; ++p) nx_par[p] = 1;
  if (0 < len) {
    nx_type = ty_row[0];
#pragma unroll
    for (int p = 0; p < PMAX; ++p) if (p < a.P) nx_par[p] = pa_row[p];
  }
  int errbits = 0;
  int s_cur = 0;                     // step of the embedding being built

  // Embedding of step s: the action's kind and log2 parameters (error bits,
  // prefetch of step s + 1), then fragment q (features 32q + 8g + j).
  auto decode = [&](int s, int& ty, float (&u)[PMAX], float& af) {
    const bool act = s < len;
    af = act ? 1.0f : 0.0f;
    const bool bad_type = act && (nx_type < 0 || nx_type >= a.K);
    ty = (act && !bad_type) ? nx_type : 0;
    bool bad_par = false;
#pragma unroll
    for (int p = 0; p < PMAX; ++p) {
      bad_par |= act && nx_par[p] < 1;
      u[p] = act ? log2f((float)nx_par[p]) : 0.0f;
    }
    errbits |= (bad_type ? ERRBIT_TYPE : 0) | (bad_par ? ERRBIT_PARAM : 0);
    if (s + 1 < len) {
      nx_type = ty_row[s + 1];
#pragma unroll
      for (int p = 0; p < PMAX; ++p) if (p < a.P) nx_par[p] = pa_row[(size_t)(s + 1) * a.P + p];
    }
  };
  // fragment q; the wavefront q also adds it to the phi sums
  auto embed_frag = [&](int q, int ty, const float (&u)[PMAX], float af) -> XF {
    const int f0 = 32 * q + 8 * g;
    float ev[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) ev[j] = t_emb[ty * temb_stride(E) + f0 + j];
#pragma unroll
    for (int p = 0; p < PMAX; ++p)
#pragma unroll
      for (int j = 0; j < 8; ++j) ev[j] = fmaf(t_pw[p * E + f0 + j], u[p], ev[j]);
#pragma unroll
    for (int j = 0; j < 8; ++j) ev[j] = (ev[j] + t_pb[f0 + j]) * af;
    if constexpr (TRAIN) {
      if (q == w && af != 0.0f) {     // the owner stores e of an active step
        float* xo = a.X + (row0 + s_cur) * IN + D + f0;
        const f32x4n lo = {NP::op(ev[0]), NP::op(ev[1]), NP::op(ev[2]), NP::op(ev[3])};
        const f32x4n hi = {NP::op(ev[4]), NP::op(ev[5]), NP::op(ev[6]), NP::op(ev[7])};
        *reinterpret_cast<f32x4n*>(xo) = lo;
        *reinterpret_cast<f32x4n*>(xo + 4) = hi;
      }
    }
    if (do_phi && q == w) {
      float* ph = phib + n * (E + 1) + f0;
#pragma unroll
      for (int j = 0; j < 8; ++j) ph[j] += ev[j];
    }
    return NP::cvt(ev);
  };
  // residual form: wavefront w < NE embeds fragment w into LDS
  auto embed_share = [&](int s) {
    if (w >= NE) return;
    s_cur = s;
    int ty;
    float u[PMAX], af;
    decode(s, ty, u, af);
    NP::store(xbuf, NZ + w, lane, embed_frag(w, ty, u, af));
  };
  // publish z fragment w (blocks 2w, 2w+1), read back all of X (paper
  // form: every wavefront holds the embedding fragments itself)
  XF xf[NK];
  XF xe[NORM ? NE : 1];
  auto exchange_x = [&]() {
    float v[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = zq[0][j];
      v[4 + j] = zq[1][j];
    }
    NP::store(xbuf, w, lane, NP::cvt(v));
    __syncthreads();
#pragma unroll
    for (int kf = 0; kf < NK; ++kf) {
      if (NORM && kf >= NZ) xf[kf] = xe[NORM ? kf - NZ : 0];
      else xf[kf] = NP::load(xbuf, kf, lane);
    }
  };
  // Paper form (Sec. 3.4): at a step boundary the finished step's u is
  // renormalised and, for an active next step, projected off the normal
  // v = Wh e of its embedding: z' = (u - (v.u / v.v) v) / |u|.  The owned
  // blocks' v come from the matrix cores (Wh groups in registers); the dots
  // are summed over the candidate's four lane groups, then over the
  // wavefronts through LDS.
  // bf16 holds the wavefront's Wh groups in registers; fp32 (twice the
  // groups, fewer free registers) reads them from L2 at each boundary
  constexpr bool WH_REG = GPK == 1;
  const uint8_t* whb = a.w1 + Narrow::bytes(D, E, NC * 32, GPK) + (size_t)w * NBW * NE * GPK * 1024 + lane * 16;
  u32x4 whq[NORM && WH_REG ? NBW * NE * GPK : 1];
  if constexpr (NORM && WH_REG) {
#pragma unroll
    for (int i = 0; i < NBW * NE * GPK; ++i) whq[i] = *reinterpret_cast<const u32x4*>(whb + (size_t)i * 1024);
  }
  auto wh_group = [&](int i) -> u32x4 {
    if constexpr (NORM && WH_REG) return whq[i];
    else return *reinterpret_cast<const gu32x4*>((gu8*)whb + (size_t)i * 1024);
  };
  auto embed_all = [&](int s) {
    s_cur = s;
    int ty;
    float u[PMAX], af;
    decode(s, ty, u, af);
#pragma unroll
    for (int q = 0; q < NE; ++q) xe[NORM ? q : 0] = embed_frag(q, ty, u, af);
  };
  // training: the unit prediction of the finished step t and |u| go to row
  // t, the next step's v, v.z and v.v to row t + 1
  auto boundary = [&](bool renorm, bool project, int t) {
    f32x4n vq[NBW];
    float vz = 0.0f, vv = 0.0f, zz = 0.0f;
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq) {
      f32x4n v = {};
#pragma unroll
      for (int q = 0; q < NE; ++q)
#pragma unroll
        for (int hh = 0; hh < GPK; ++hh)
          v = NP::mma(wh_group((bq * NE + q) * GPK + hh), hh, xe[NORM ? q : 0], v);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        vz = fmaf(v[r], zq[bq][r], vz);
        vv = fmaf(v[r], v[r], vv);
        zz = fmaf(zq[bq][r], zq[bq][r], zz);
      }
      vq[bq] = v;
    }
    vz += __shfl_xor(vz, 16); vz += __shfl_xor(vz, 32);
    vv += __shfl_xor(vv, 16); vv += __shfl_xor(vv, 32);
    zz += __shfl_xor(zz, 16); zz += __shfl_xor(zz, 32);
    if (g == 0) {
      dots[(w * 3 + 0) * 16 + n] = vz;
      dots[(w * 3 + 1) * 16 + n] = vv;
      dots[(w * 3 + 2) * 16 + n] = zz;
    }
    __syncthreads();
    vz = 0.0f; vv = 0.0f; zz = 0.0f;
#pragma unroll
    for (int ww = 0; ww < W; ++ww) {
      vz += dots[(ww * 3 + 0) * 16 + n];
      vv += dots[(ww * 3 + 1) * 16 + n];
      zz += dots[(ww * 3 + 2) * 16 + n];
    }
    const float sc = (renorm && zz > 0.0f) ? rsqrtf(zz) : 1.0f;
    const float al = (project && vv > 0.0f) ? vz / vv : 0.0f;
    if constexpr (TRAIN) {
      if (renorm) {                  // step t was active
        const size_t rt = row0 + t;
#pragma unroll
        for (int bq = 0; bq < NBW; ++bq) {
          const f32x4n pv = zq[bq] * sc;
          *reinterpret_cast<f32x4n*>(a.Pz + rt * D + 16 * (w * NBW + bq) + 4 * g) = pv;
        }
        if (w == 0 && g == 0) a.SC[rt * 4 + 2] = sqrtf(zz);
      }
      if (project) {                 // step t + 1 is active
        const size_t rs = row0 + (t + 1);
#pragma unroll
        for (int bq = 0; bq < NBW; ++bq)
          *reinterpret_cast<f32x4n*>(a.V + rs * D + 16 * (w * NBW + bq) + 4 * g) = vq[bq];
        if (w == 0 && g == 0) {
          a.SC[rs * 4 + 0] = vz * sc;
          a.SC[rs * 4 + 1] = vv;
          a.SC[rs * 4 + 3] = 0.0f;
        }
      }
    }
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq)
#pragma unroll
      for (int r = 0; r < 4; ++r) zq[bq][r] = (zq[bq][r] - al * vq[bq][r]) * sc;
  };

  // weight group of stream item i, relative to the wavefront's two bases
  auto item_off = [](int i) -> size_t {
    if (i < NA) {
      const int cw = i / (NK * 2 * GPK), r = i % (NK * 2 * GPK);
      return ((size_t)cw * W * NK * 2 * GPK + r) * 1024;
    }
    const int j = i - NA;       // (chunk, own block, half)
    const int c = j / (NBW * GPK), r = j % (NBW * GPK);
    return ((size_t)c * NB * GPK + r) * 1024;
  };
  gu8* baseA = ((gu8*)(a.w1)) + (size_t)(w * NK * 2 * GPK) * 1024 + lane * 16;
  gu8* baseB = ((gu8*)(a.w1)) + (size_t)(NG::W1G + w * NBW * GPK) * 1024 + lane * 16;
  auto item_ptr = [&](gu8* pA, gu8* pB, int i) -> gu32x4* {
    return reinterpret_cast<gu32x4*>((i < NA ? pA : pB) + item_off(i));
  };
  u32x4 ring[RD];
#pragma unroll
  for (int i = 0; i < RD; ++i) ring[i] = *item_ptr(baseA, baseB, i);

  wait_vm_then_barrier();
  if constexpr (NORM) {
    embed_all(0);
    boundary(false, 0 < len, -1);
  } else {
    embed_share(0);
  }
  exchange_x();

  for (int t = 0; t < T_wg; ++t) {
    const bool active = t < len;
    const float actf = active ? 1.0f : 0.0f;
    const uint32_t amask = active ? 0xFFFFFFFFu : 0u;
    gu8* pA = baseA;
    gu8* pB = baseB;
    asm volatile("" : "+v"(pA), "+v"(pB));
    const size_t row = row0 + t;
    if constexpr (TRAIN) {
      if (active) {                  // X = [z; e]: the owned latent blocks (e: embed_share)
#pragma unroll
        for (int bq = 0; bq < NBW; ++bq) {
          const f32x4n v = {NP::op(zq[bq][0]), NP::op(zq[bq][1]), NP::op(zq[bq][2]), NP::op(zq[bq][3])};
          *reinterpret_cast<f32x4n*>(a.X + row * IN + 16 * (w * NBW + bq) + 4 * g) = v;
        }
        if (w == 0 && g == 0) a.row_src[row] = cand * a.T_max + t;
      }
    }
    f32x4n acc[2], dz[NBW];
    acc[0] = f32x4n{}; acc[1] = f32x4n{};
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq) dz[bq] = f32x4n{};
    XF gcur = {}, gnext = {};
    // A chunk's bias-added pre-activations wait in pend while the next
    // chunk's products run; their GELUs are spread over that chunk's first
    // eight items (one per item), so the vector work of one chunk overlaps
    // the matrix work of the next.  The last chunk's GELUs run at once.
    constexpr int NPC = NK * 2 * GPK;                  // items per chunk
    constexpr bool DEFER = NPC >= 8;                   // eight items to spread them over
    float pend[8], gvp[8];
    auto finish_chunk = [&](int cwf, const float (&gv)[8]) {
      const int c = w + cwf * W;
      if constexpr (TRAIN) {
        if (active) {
#pragma unroll
          for (int rb2 = 0; rb2 < 2; ++rb2) {
            const f32x4n gq = {NP::op(gv[4 * rb2]), NP::op(gv[4 * rb2 + 1]), NP::op(gv[4 * rb2 + 2]),
                               NP::op(gv[4 * rb2 + 3])};
            *reinterpret_cast<f32x4n*>(a.G + row * a.H + 32 * c + 16 * rb2 + 4 * g) = gq;
          }
        }
      }
      NP::store(gbuf, c, lane, NP::gfrag(gv, amask));
    };
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const u32x4 grp = ring[i % RD];
      ring[i % RD] = *item_ptr(pA, pB, (i + RD) % NI);   // wraps into the next step
      if (i < NA) {
        const int cw = i / (NK * 2 * GPK), kf = (i / (2 * GPK)) % NK;
        const int rb = (i / GPK) % 2, hh = i % GPK;
        const int r_in = i % NPC;
        // the previous chunk's GELU number r_in
        if (DEFER && cw > 0 && r_in < 8) {
          gvp[r_in] = gelu(pend[r_in]);
          if (r_in == 7) finish_chunk(cw - 1, gvp);
        }
        acc[rb] = NP::mma(grp, hh, xf[kf], acc[rb]);
        if (kf == NK - 1 && rb == 1 && hh == GPK - 1) {
          float av8[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) av8[j] = acc[j >> 2][j & 3] + b1v[cw][j >> 2][j & 3];
          if constexpr (TRAIN) {
            if (active) {
              const int c = w + cw * W;
#pragma unroll
              for (int rb2 = 0; rb2 < 2; ++rb2) {
                const f32x4n av = {av8[4 * rb2], av8[4 * rb2 + 1], av8[4 * rb2 + 2], av8[4 * rb2 + 3]};
                *reinterpret_cast<f32x4n*>(a.A + row * a.H + 32 * c + 16 * rb2 + 4 * g) = av;
              }
            }
          }
          if (!DEFER || cw == NCW - 1) {   // last chunk: GELU, rounding, mask now
            float gv[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) gv[j] = gelu(av8[j]);
            finish_chunk(cw, gv);
          } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) pend[j] = av8[j];
          }
          acc[0] = f32x4n{};
          acc[1] = f32x4n{};
        }
        if (i == NA - 1) {
          __syncthreads();           // every chunk's GELU fragment is in LDS
          gcur = NP::load(gbuf, 0, lane);
          gnext = NP::load(gbuf, NC > 1 ? 1 : 0, lane);
        }
      } else {
        const int j = i - NA, c = j / (NBW * GPK), bq = (j / GPK) % NBW, hh = j % GPK;
        dz[bq] = NP::mma(grp, hh, gcur, dz[bq]);
        if (bq == NBW - 1 && hh == GPK - 1) {
          gcur = gnext;
          if (c + 2 < NC) gnext = NP::load(gbuf, c + 2, lane);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq) {
#pragma unroll
      for (int r = 0; r < 4; ++r) zq[bq][r] += dz[bq][r] + b2v[bq][r] * actf;
      if constexpr (TRAIN && !NORM) {
        if (active) *reinterpret_cast<f32x4n*>(a.Pz + row * D + 16 * (w * NBW + bq) + 4 * g) = zq[bq];
      }
    }
    if constexpr (NORM) {
      embed_all(t + 1);
      boundary(active, t + 1 < len, t);
    } else {
      embed_share(t + 1);
    }
    exchange_x();
  }
  if (errbits) atomicOr(a.err, errbits);
  if (do_phi && valid && w < NE) {   // phi = sum / len over the owned fragment (0 when empty)
    const float inv = len > 0 ? 1.0f / (float)len : 0.0f;
    const int f0 = 32 * w + 8 * g;
    const float* ph = phib + n * (E + 1) + f0;
#pragma unroll
    for (int j = 0; j < 8; ++j) a.phi[(size_t)cand * E + f0 + j] = ph[j] * inv;
  }
  if constexpr (SCORE) {
    // x = [z_T; phi; h]: z_T fragments from the last exchange, phi from the
    // sums (complete after that exchange's barrier), h per hardware vector
    constexpr int NHF = 1;                           // hw fragments (hw_dim <= 32)
    const int NH = a.HW / 32, NCC = a.C / 32, NKC = NZ + NE + NH;
    const float inv = len > 0 ? 1.0f / (float)len : 0.0f;
    XF pf[NE];
#pragma unroll
    for (int q = 0; q < NE; ++q) {
      float v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = phib[n * (E + 1) + 32 * q + 8 * g + j] * inv;
      pf[q] = NP::cvt(v);
    }
    XF hf[NARROW_SCORE_HW][NHF > 0 ? NHF : 1];
#pragma unroll
    for (int jj = 0; jj < NARROW_SCORE_HW; ++jj)
#pragma unroll
      for (int q = 0; q < (NHF > 0 ? NHF : 1); ++q) {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
          v[j] = (jj < a.n_hw && q < NH) ? a.hw[(size_t)jj * a.HW + 32 * q + 8 * g + j] : 0.0f;
        hf[jj][q] = NP::cvt(v);
      }
    const float* bc1n = reinterpret_cast<const float*>(a.costn + (size_t)NCC * NKC * 2 * GPK * 1024);
    const float* wc2n = bc1n + a.C;
    float part[NARROW_SCORE_HW] = {};
    for (int cc = w; cc < NCC; cc += W) {
      const uint8_t* cb = a.costn + (size_t)cc * NKC * 2 * GPK * 1024 + lane * 16;
      auto grp_at = [&](int kf, int rb, int hh) -> u32x4 {
        return *reinterpret_cast<const gu32x4*>((gu8*)cb + ((size_t)(kf * 2 + rb) * GPK + hh) * 1024);
      };
      f32x4n acc2[2] = {f32x4n{}, f32x4n{}};
#pragma unroll
      for (int kf = 0; kf < NZ + NE; ++kf)
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int hh = 0; hh < GPK; ++hh)
            acc2[rb] = NP::mma(grp_at(kf, rb, hh), hh, kf < NZ ? xf[kf < NZ ? kf : 0] : pf[kf < NZ ? 0 : kf - NZ], acc2[rb]);
      f32x4n b4[2], w4[2];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        b4[rb] = *reinterpret_cast<const f32x4n*>(bc1n + 32 * cc + 16 * rb + 4 * g);
        w4[rb] = *reinterpret_cast<const f32x4n*>(wc2n + 32 * cc + 16 * rb + 4 * g);
      }
#pragma unroll
      for (int jj = 0; jj < NARROW_SCORE_HW; ++jj) {
        if (jj < a.n_hw) {
          f32x4n aj[2] = {acc2[0], acc2[1]};
#pragma unroll
          for (int q = 0; q < (NHF > 0 ? NHF : 1); ++q)
            if (q < NH)
#pragma unroll
              for (int rb = 0; rb < 2; ++rb)
#pragma unroll
                for (int hh = 0; hh < GPK; ++hh) aj[rb] = NP::mma(grp_at(NZ + NE + q, rb, hh), hh, hf[jj][q], aj[rb]);
          float sum = 0.0f;
#pragma unroll
          for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int r = 0; r < 4; ++r) sum = fmaf(w4[rb][r], gelu(aj[rb][r] + b4[rb][r]), sum);
          part[jj] += sum;
        }
      }
    }
    // the candidate's four lane groups, then the wavefronts in order
    float* red = dots + (NORM ? W * 3 * 16 : 0) + 16 * (E + 1);          // [W][NARROW_SCORE_HW][16]
#pragma unroll
    for (int jj = 0; jj < NARROW_SCORE_HW; ++jj) {
      float v = part[jj];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (g == 0) red[(w * NARROW_SCORE_HW + jj) * 16 + n] = v;
    }
    __syncthreads();
    if (w == 0 && g == 0 && valid) {
#pragma unroll
      for (int jj = 0; jj < NARROW_SCORE_HW; ++jj) {
        if (jj < a.n_hw) {
          float y = 0.0f;
#pragma unroll
          for (int ww = 0; ww < W; ++ww) y += red[(ww * NARROW_SCORE_HW + jj) * 16 + n];
          a.scores[(size_t)jj * a.B + cand] = y + a.bc2;
        }
      }
    }
  }
  if (valid && !TRAIN) {
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq)
      *reinterpret_cast<f32x4n*>(a.zT + (size_t)cand * D + 16 * (w * NBW + bq) + 4 * g) = zq[bq];
  }
}

// ==========================================================================
// Action features: phi_i = (1/len_i) sum_t e_t.  The sum is regrouped by
// what varies per step:  sum_t e_t = sum_k n_k type_emb[k] + param_w .
// sum_t log2(params_t) + len_i param_b, with n_k the number of steps of
// kind k.  Kinds are clamped into range here (the rollout kernel reports
// them).

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

__device__ __forceinline__ float group16_sum(float x) {
  // butterfly over the 16 lanes of a group (xor 1, 2, 4, 8 stays inside it)
#pragma unroll
  for (int m = 8; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

// a4 where the rollout kernel does not sum phi itself: 16 lanes per candidate
// (four candidates per wavefront), lane s taking steps s, s + 16, ...; the
// kind counts and log2-parameter sums are reduced over the candidate's 16
// lanes, then lane s forms features s, s + 16, ... of the regrouped mean
// (0 for an empty sequence).
__global__ __launch_bounds__(256) void phi_kernel(const float* __restrict__ emb,
                                                   const int32_t* __restrict__ types,
                                                   const int32_t* __restrict__ params,
                                                   const int32_t* __restrict__ lens, int B,
                                                   int T_max, int E, int P, int K,
                                                   float* __restrict__ phi) {
  const int lane = threadIdx.x & 63, s = lane & 15;
  const int i = (blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * 4 + (lane >> 4);
  const bool valid = i < B;
  const float* t_emb = emb;
  const float* t_pw = emb + K * temb_stride(E);        // [PMAX][E], zero rows past P
  const float* t_pb = t_pw + PMAX * E;
  const int len = valid ? clampi(lens[i], 0, T_max) : 0;
  float cnt[32];                                       // n_k, K <= 32 (exact in float)
#pragma unroll
  for (int k = 0; k < 32; ++k) cnt[k] = 0.0f;
  float us[PMAX];                                      // sums of log2(params)
#pragma unroll
  for (int p = 0; p < PMAX; ++p) us[p] = 0.0f;
  const int32_t* ty_row = types + (size_t)(valid ? i : 0) * T_max;
  const int32_t* pa_row = params + (size_t)(valid ? i : 0) * T_max * P;
  for (int t = s; t < len; t += 16) {
    const int ty = clampi(ty_row[t], 0, K - 1);
#pragma unroll
    for (int k = 0; k < 32; ++k)
      if (k < K) cnt[k] += ty == k ? 1.0f : 0.0f;
#pragma unroll
    for (int p = 0; p < PMAX; ++p)
      if (p < P) us[p] += log2f((float)pa_row[(size_t)t * P + p]);
  }
  // every lane takes part in the reductions (invalid groups sum zeros)
#pragma unroll
  for (int k = 0; k < 32; ++k)
    if (k < K) cnt[k] = group16_sum(cnt[k]);
#pragma unroll
  for (int p = 0; p < PMAX; ++p) us[p] = p < P ? group16_sum(us[p]) : 0.0f;
  if (!valid) return;
  const float inv = len > 0 ? 1.0f / (float)len : 0.0f;
  for (int f = s; f < E; f += 16) {
    float acc = 0.0f;
#pragma unroll
    for (int k = 0; k < 32; ++k)
      if (k < K) acc = fmaf(cnt[k], t_emb[k * temb_stride(E) + f], acc);
#pragma unroll
    for (int p = 0; p < PMAX; ++p) acc = fmaf(us[p], t_pw[p * E + f], acc);
    phi[(size_t)i * E + f] = len > 0 ? fmaf(acc, inv, t_pb[f]) : 0.0f;
  }
}

// ==========================================================================
// Structured action features (the ranker's phi, Sec. 3.5): per candidate the
// number of steps of each kind, the length, and per parameter slot the mean
// and the maximum of log2(param) over the steps (all zero when the sequence
// is empty).  One wavefront per candidate, lanes over steps; kinds outside
// [0, K) are not counted.

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x = fmaxf(x, __shfl_xor(x, m));
  return x;
}

__global__ __launch_bounds__(256) void phi_struct_kernel(const int32_t* __restrict__ types,
                                                          const int32_t* __restrict__ params,
                                                          const int32_t* __restrict__ lens, int B,
                                                          int T_max, int K, int P,
                                                          float* __restrict__ phi_s) {
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (i >= B) return;                                  // whole wavefront leaves together
  const int len = clampi(lens[i], 0, T_max);
  const int32_t* ty_row = types + (size_t)i * T_max;
  const int32_t* pa_row = params + (size_t)i * T_max * P;
  int cnt[32];
#pragma unroll
  for (int k = 0; k < 32; ++k) cnt[k] = 0;
  float us[PMAX], um[PMAX];
#pragma unroll
  for (int p = 0; p < PMAX; ++p) { us[p] = 0.0f; um[p] = -INFINITY; }
  for (int t0 = 0; t0 < len; t0 += 64) {
    const int t = t0 + lane;
    const bool v = t < len;
    const int ty = v ? ty_row[t] : -1;
#pragma unroll
    for (int p = 0; p < PMAX; ++p)
      if (p < P && v) {
        const float u = log2f((float)pa_row[(size_t)t * P + p]);
        us[p] += u;
        um[p] = fmaxf(um[p], u);
      }
#pragma unroll
    for (int k = 0; k < 32; ++k)
      if (k < K) cnt[k] += __popcll(__ballot(ty == k));
  }
  float* o = phi_s + (size_t)i * phi_struct_dim(K, P);
  const float inv = len > 0 ? 1.0f / (float)len : 0.0f;
#pragma unroll
  for (int p = 0; p < PMAX; ++p) {
    if (p >= P) break;
    const float s = wave_sum(us[p]);
    const float m = wave_max(um[p]);
    if (lane == 0) {
      o[K + 1 + p] = len > 0 ? s * inv : 0.0f;
      o[K + 1 + P + p] = len > 0 ? m : 0.0f;
    }
  }
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < 32; ++k)
      if (k < K) o[k] = (float)cnt[k];
    o[K] = (float)len;
  }
}

// ==========================================================================
// Tree-ensemble ranker (the paper's G, Sec. 3.5): y = base + sum over trees
// of the leaf reached by x = [z_T ; phi_s ; h].  One workgroup per
// TREE_CPB candidates and one hardware vector: the candidates' x are staged
// in LDS, each thread walks trees tid, tid + 256, ... for all TREE_CPB
// candidates in lockstep (independent chains of dependent node loads; node
// i -> child 2i+1 when x[f] < c, else 2i+2, so a NaN goes right), and every
// candidate's leaf values are summed in a fixed order.

constexpr int TREE_THREADS = 256;
constexpr int TREE_CPB = 8;

__global__ __launch_bounds__(TREE_THREADS) void score_trees_kernel(
    const int2* __restrict__ nodes, const float* __restrict__ leaves, int NT, int depth, float base,
    const float* __restrict__ zT, int d, const float* __restrict__ phi_s, int phi_dim,
    const float* __restrict__ hw, int hw_dim, int B, float* __restrict__ scores) {
  extern __shared__ float tsm[];
  const int F = d + phi_dim + hw_dim;
  float* x = tsm;                                      // [TREE_CPB][F]
  float* red = tsm + TREE_CPB * F;                     // [TREE_THREADS / 64][TREE_CPB]
  const int i0 = blockIdx.x * TREE_CPB, j = blockIdx.y, tid = threadIdx.x;
  const int nc = min(TREE_CPB, B - i0);
  for (int q = tid; q < TREE_CPB * F; q += TREE_THREADS) {
    const int c = q / F, f = q - c * F;
    const int i = i0 + (c < nc ? c : 0);               // rows past the batch repeat the first
    float v;
    if (f < d) v = zT[(size_t)i * d + f];
    else if (f < d + phi_dim) v = phi_s[(size_t)i * phi_dim + (f - d)];
    else v = hw[(size_t)j * hw_dim + (f - d - phi_dim)];
    x[q] = v;
  }
  __syncthreads();
  const int n_int = (1 << depth) - 1;
  float acc[TREE_CPB];
#pragma unroll
  for (int c = 0; c < TREE_CPB; ++c) acc[c] = 0.0f;
  for (int t = tid; t < NT; t += TREE_THREADS) {
    const int2* tn = nodes + (size_t)t * n_int;
    int node[TREE_CPB];
#pragma unroll
    for (int c = 0; c < TREE_CPB; ++c) node[c] = 0;
    for (int l = 0; l < depth; ++l) {
#pragma unroll
      for (int c = 0; c < TREE_CPB; ++c) {
        const int2 nd = tn[node[c]];
        node[c] = 2 * node[c] + (x[c * F + nd.x] < __int_as_float(nd.y) ? 1 : 2);
      }
    }
    const float* tl = leaves + (size_t)t * (n_int + 1);
#pragma unroll
    for (int c = 0; c < TREE_CPB; ++c) acc[c] += tl[node[c] - n_int];
  }
#pragma unroll
  for (int c = 0; c < TREE_CPB; ++c) {
    const float v = wave_sum(acc[c]);
    if ((tid & 63) == 0) red[(tid >> 6) * TREE_CPB + c] = v;
  }
  __syncthreads();
  if (tid < nc) {
    float y = base;
#pragma unroll
    for (int w = 0; w < TREE_THREADS / 64; ++w) y += red[w * TREE_CPB + tid];
    scores[(size_t)j * B + i0 + tid] = y;
  }
}

// ==========================================================================
// Rollout loss and its gradients (the transition's training objective,
// Sec. 3.4).  Step activations live in compact rows r = off[i] + t of the
// workspace, off the exclusive prefix sum of the (clamped) lengths, so the
// valid steps of all candidates are rows [0, off[B]) with no padding;
// row_src[r] = i * T_max + t locates a row's action in the caller's tensors.
//
// train_fwd_kernel: one wavefront per 32-candidate tile (length-sorted),
// the residual-MLP step with the weight groups streamed from L2 into a
// register ring.  Per valid step it stores the product operands X = [z; e]
// (with the value the products see), the pre-activations A, the GELU outputs
// G (product-operand value) and the predicted state P = z_{t+1}.

struct TrainArgs {
  const uint8_t* w1;        // packed transition chunks (forward)
  const uint8_t* w2;
  const uint8_t* w2t;       // packed transposed chunks (backward)
  const uint8_t* w1t;
  const float* tab;         // rollout table
  const float* z0;          // [S][D]
  const int2* perm;
  const int32_t* types;
  const int32_t* params;
  const int32_t* lens;
  const int32_t* off;       // [B+1] row offsets
  int32_t* row_src;         // [R]  i * T_max + t of each row
  float* X;                 // [R][D+E]
  float* A;                 // [R][H]   pre-activations; the backward overwrites them with dA
  float* G;                 // [R][H]
  float* P;                 // [R][D]   predicted states
  float* SD;                // [R][D]   dL/dp seeds; the backward overwrites them with delta_{t+1}
  float* DE;                // [R][E]   gradient reaching the step's embedding
  const uint8_t* wh;        // paper form: packed normal map, and its transpose
  const uint8_t* wht;
  float* V;                 // [R][D]   Wh e
  float* SC;                // [R][4]   v.z, v.v, |u|, 0
  float* DV;                // [R][D]   dL/dv
  float* dz0;               // [B][D]   (may be null)
  int32_t* err;
  int B, T_max, P_, K, H, tab_bytes;
};

// d/dx [x Phi(x)] = Phi(x) + x phi(x), with erf from the same Abramowitz &
// Stegun 7.1.26 form as gelu() and phi(x) = exp(-x^2/2) / sqrt(2 pi).
__device__ __forceinline__ float gelu_grad(float x) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f * 0.70710678118654752f, ax, 1.0f));
  float p = fmaf(1.061405429f, t, -1.453152027f);
  p = fmaf(p, t, 1.421413741f);
  p = fmaf(p, t, -0.284496736f);
  p = fmaf(p, t, 0.254829592f);
  const float ex = __builtin_amdgcn_exp2f((x * x) * (-0.5f * 1.4426950408889634f));
  const float erf_a = fmaf(-(p * t), ex, 1.0f);
  return fmaf(0.5f, copysignf(erf_a, x), 0.5f) + x * ex * 0.3989422804014327f;
}

template <class PR, int D, int E>
struct TrainGeom {
  using R = Roll<PR, D, E>;
  static constexpr int G = PR::G;
  static constexpr int N1 = R::NK1 / G, N2 = R::NK2 / G, NIF = N1 + N2;    // forward groups per chunk
  static constexpr int NW2T = TransT<PR>::nk2t(D) / G;                    // backward: W2^T groups
  static constexpr int NW1T = TransT<PR>::nk1t(D, E) / G;                 // backward: W1^T groups
  static constexpr int NIB = NW2T + NW1T;
  static constexpr int NBE = E / 32;                                       // embedding output blocks
  // ring depth: a divisor of the groups per chunk, so the ring wraps from
  // one chunk (and step) into the next with every group in a fixed slot
  static constexpr int ring(int n) {
    const int cap = G == 1 ? 8 : 12;
    for (int r = cap; r > 1; --r)
      if (n % r == 0) return r;
    return 1;
  }
  static constexpr int RDF = ring(NIF), RDB = ring(NIB);
  static_assert(E % 32 == 0, "embedding blocks");
};

// Tile bookkeeping shared by the two step kernels.
struct TileInfo {
  int cand, seg, len, T_wg;
  bool valid;
};
__device__ __forceinline__ TileInfo tile_info(const TrainArgs& a, int tile, int n) {
  TileInfo ti;
  const int pos = tile * 32 + n;
  ti.valid = pos < a.B;
  const int2 pc = ti.valid ? a.perm[pos] : make_int2(0, 0);
  ti.cand = pc.x;
  ti.seg = pc.y;
  ti.len = ti.valid ? clampi(a.lens[pc.x], 0, a.T_max) : 0;
  // candidates are sorted longest first: the tile's first one sets its steps
  ti.T_wg = tile * 32 < a.B
                ? __builtin_amdgcn_readfirstlane(clampi(a.lens[a.perm[tile * 32].x], 0, a.T_max))
                : 0;
  return ti;
}

template <class PR, int D, int E, int WAVES, bool NORM>
__global__ __launch_bounds__(64 * WAVES, 1) void train_fwd_kernel(const TrainArgs a) {
  using R = Roll<PR, D, E>;
  using TG = TrainGeom<PR, D, E>;
  using Frag = typename PR::Frag;
  constexpr int KF = PR::KF, SL = PR::SL, G = PR::G;
  constexpr int NZ = R::NZ, NE = R::NE, NF2 = R::NF2, NB = R::NB;
  constexpr int W1B = R::W1B, W2B = R::W2B, N1 = TG::N1, NI = TG::NIF, RD = TG::RDF;
  constexpr int NT = 64 * WAVES, IN = D + E;

  extern __shared__ __attribute__((aligned(16))) float tab[];
  const float* t_emb = tab;
  const float* t_pw = tab + a.K * temb_stride(E);
  const float* t_pb = t_pw + PMAX * E;
  const float* t_b2 = t_pb + E;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  stage_to_lds(reinterpret_cast<const uint8_t*>(a.tab), reinterpret_cast<uint8_t*>(tab),
               a.tab_bytes, tid, NT);

  const TileInfo ti = tile_info(a, blockIdx.x * WAVES + wave, n);
  const int cand = ti.cand, len = ti.len, T_wg = ti.T_wg;
  const int NC = a.H / 32;
  const size_t row0 = ti.valid ? (size_t)a.off[cand] : 0;

  f32x16 zacc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) zacc[b] = load_acc(a.z0 + (size_t)ti.seg * D + 32 * b, h);
  const int32_t* ty_row = a.types + (size_t)cand * a.T_max;
  const int32_t* pa_row = a.params + (size_t)cand * a.T_max * a.P_;
  int errbits = 0;

  gu8* w1g = (gu8*)(a.w1) + lane * 16;
  gu8* w2g = (gu8*)(a.w2) + lane * 16;
  auto group_ptr = [&](int c, int i) -> gu32x4* {
    return reinterpret_cast<gu32x4*>(i < N1 ? w1g + (size_t)c * W1B + (size_t)i * 1024
                                            : w2g + (size_t)c * W2B + (size_t)(i - N1) * 1024);
  };
  u32x4 ring[RD];
#pragma unroll
  for (int i = 0; i < RD; ++i) ring[i] = *group_ptr(0, i);
  wait_vm_then_barrier();

  for (int t = 0; t < T_wg; ++t) {
    const bool active = t < len;
    const float actf = active ? 1.0f : 0.0f;
    const uint32_t amask = active ? 0xFFFFFFFFu : 0u;
    const size_t row = row0 + t;
    if (active && h == 0) a.row_src[row] = cand * a.T_max + t;
    // the step's action: kind and log2 parameters (zero embedding when done)
    int ty = 0;
    float u[PMAX];
#pragma unroll
    for (int p = 0; p < PMAX; ++p) u[p] = 0.0f;
    if (active) {
      const int tv = ty_row[t];
      if (tv < 0 || tv >= a.K) errbits |= ERRBIT_TYPE;
      else ty = tv;
#pragma unroll
      for (int p = 0; p < PMAX; ++p)
        if (p < a.P_) {
          const int pv = pa_row[(size_t)t * a.P_ + p];
          if (pv < 1) errbits |= ERRBIT_PARAM;
          u[p] = log2f((float)pv);
        }
    }
    float* xrow = a.X + row * IN;
    Frag xe[NE];
#pragma unroll
    for (int q = 0; q < NE; ++q) {
      const int f0 = KF * q + SL * h;
      float ev[SL], tmp[SL];
      R::row(t_emb + ty * temb_stride(E) + f0, ev);
#pragma unroll
      for (int p = 0; p < PMAX; ++p) {
        R::row(t_pw + p * E + f0, tmp);
#pragma unroll
        for (int j = 0; j < SL; ++j) ev[j] = fmaf(tmp[j], u[p], ev[j]);
      }
      R::row(t_pb + f0, tmp);
#pragma unroll
      for (int j = 0; j < SL; ++j) ev[j] = (ev[j] + tmp[j]) * actf;
      xe[q] = PR::cvt(ev);
      if (active) {
#pragma unroll
        for (int j = 0; j < SL; ++j) xrow[D + f0 + j] = op_value<PR>(ev[j]);
      }
    }
    // paper form: z' = z - (v.z / v.v) v with v = Wh e (two passes of V^T =
    // Wh . E^T on the matrix cores: the dots, then the projection)
    float s_vz = 0.0f, s_vv = 0.0f;
    if constexpr (NORM) {
      using HY = Hyper<PR, D, E>;
      constexpr int GPB = HY::GPB;
      gu8* whb = (gu8*)(a.wh) + lane * 16;
      auto vblock = [&](int b) -> f32x16 {
        f32x16 vb = {};
#pragma unroll
        for (int k = 0; k < GPB; ++k) {
          const u32x4 grp = *reinterpret_cast<gu32x4*>(whb + (size_t)(b * GPB + k) * 1024);
#pragma unroll
          for (int ww = 0; ww < G; ++ww) vb = PR::mfma(PR::pick(grp, ww), xe[k * G + ww], vb);
        }
        return vb;
      };
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const f32x16 vb = vblock(b);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s_vz = fmaf(vb[r], zacc[b][r], s_vz);
          s_vv = fmaf(vb[r], vb[r], s_vv);
        }
        if (active) store_acc(a.V + row * D + 32 * b, vb, h);
      }
      s_vz = HY::pair_sum(s_vz);
      s_vv = HY::pair_sum(s_vv);
      const float al = s_vv > 0.0f ? s_vz / s_vv : 0.0f;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const f32x16 vb = vblock(b);
#pragma unroll
        for (int r = 0; r < 16; ++r) zacc[b][r] -= al * vb[r];
      }
    }
    Frag xz[NZ];
#pragma unroll
    for (int kf = 0; kf < NZ; ++kf) {
      float v[SL];
#pragma unroll
      for (int j = 0; j < SL; ++j) v[j] = zacc[kf / NF2][(kf % NF2) * SL + j];
      xz[kf] = PR::cvt(v);
    }
    if (active) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        f32x16 v;
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = op_value<PR>(zacc[b][r]);
        store_acc(xrow + 32 * b, v, h);
      }
    }
    for (int c = 0; c < NC; ++c) {
      const int cn = c + 1 < NC ? c + 1 : 0;
      const float* b1g = reinterpret_cast<const float*>(a.w1 + (size_t)c * W1B + (W1B - 128)) + 16 * h;
      f32x16 acc;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(b1g + 4 * q);
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[4 * q + i] = v[i];
      }
      typename PR::Packed gp[8];
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const u32x4 grp = ring[i % RD];
        ring[i % RD] = (i + RD < NI) ? *group_ptr(c, i + RD) : *group_ptr(cn, i + RD - NI);
        if (i < N1) {
#pragma unroll
          for (int ww = 0; ww < G; ++ww) {
            const int kf = i * G + ww;
            acc = PR::mfma(PR::pick(grp, ww), kf < NZ ? xz[kf < NZ ? kf : 0] : xe[kf < NZ ? 0 : kf - NZ], acc);
          }
          if (i == N1 - 1) {
            f32x16 gv;
#pragma unroll
            for (int r = 0; r < 16; ++r) gv[r] = op_value<PR>(gelu(acc[r]));
#pragma unroll
            for (int q = 0; q < 8; ++q) gp[q] = PR::pack2(gv[2 * q], gv[2 * q + 1], amask);
            if (active) {
              store_acc(a.A + row * a.H + 32 * c, acc, h);
              store_acc(a.G + row * a.H + 32 * c, gv, h);
            }
          }
        } else {
#pragma unroll
          for (int ww = 0; ww < G; ++ww) {
            const int F = (i - N1) * G + ww;
            zacc[F / NF2] = PR::mfma(PR::pick(grp, ww), PR::gfrag(gp, F % NF2), zacc[F / NF2]);
          }
        }
      }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) zacc[b][r] += t_b2[(b * 2 + h) * 16 + r] * actf;
    if constexpr (NORM) {            // z_{t+1} = u / |u| (finished candidates stay as they are)
      float uu = 0.0f;
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) uu = fmaf(zacc[b][r], zacc[b][r], uu);
      uu = uu + __shfl_xor(uu, 32);
      const float nu = sqrtf(uu);
      const float sc = (active && nu > 0.0f) ? 1.0f / nu : 1.0f;
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) zacc[b][r] *= sc;
      if (active && h == 0) {
        const f32x4 sv = {s_vz, s_vv, nu, 0.0f};
        *reinterpret_cast<f32x4*>(a.SC + row * 4) = sv;
      }
    }
    if (active) {
#pragma unroll
      for (int b = 0; b < NB; ++b) store_acc(a.P + row * D + 32 * b, zacc[b], h);
    }
  }
  if (errbits) atomicOr(a.err, errbits);
}

// Per-step loss and its gradient with respect to the prediction: one
// wavefront per (candidate, step) slot; lane L holds features 4L..4L+3 (and
// +256, ...), so the prediction, the target and up to LOSS_NEG negatives
// are read in one pass of independent 16-byte loads.  The hardest negative
// is the nearest (first one on ties); a zero distance contributes a zero
// gradient.  targets / negatives are indexed by slot, P / SD / lrow by
// compact row.
constexpr int LOSS_NEG = 8;          // negatives per pass
__global__ __launch_bounds__(256) void loss_kernel(const float* __restrict__ P,
                                                   const float* __restrict__ targets,
                                                   const float* __restrict__ negatives, int NN,
                                                   const int32_t* __restrict__ lens,
                                                   const int32_t* __restrict__ off, int B,
                                                   int T_max, int D, float lam, float gamma,
                                                   float* __restrict__ SD, float* __restrict__ lrow) {
  const int lane = threadIdx.x & 63;
  const long long slot = (long long)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (slot >= (long long)B * T_max) return;            // whole wavefront leaves together
  const int i = (int)(slot / T_max), t = (int)(slot - (long long)i * T_max);
  if (t >= clampi(lens[i], 0, T_max)) return;
  const size_t row = (size_t)off[i] + t;
  const f32x4* p4 = reinterpret_cast<const f32x4*>(P + row * D);
  const f32x4* y4 = reinterpret_cast<const f32x4*>(targets + slot * D);
  const int D4 = D / 4;
  float m = 0.0f;
  for (int c = lane; c < D4; c += 64) {
    const f32x4 v = p4[c] - y4[c];
    m += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
  }
  const float match = wave_sum(m);
  const float dpos = sqrtf(match);
  float dmin = INFINITY;
  int hard = 0;
  for (int q0 = 0; q0 < NN; q0 += LOSS_NEG) {
    float sq[LOSS_NEG];
#pragma unroll
    for (int q = 0; q < LOSS_NEG; ++q) sq[q] = 0.0f;
    for (int c = lane; c < D4; c += 64) {
      const f32x4 pv = p4[c];
#pragma unroll
      for (int q = 0; q < LOSS_NEG; ++q) {
        if (q0 + q < NN) {
          const f32x4 v = pv - reinterpret_cast<const f32x4*>(negatives + (slot * NN + q0 + q) * D)[c];
          sq[q] += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
        }
      }
    }
#pragma unroll
    for (int q = 0; q < LOSS_NEG; ++q) {
      if (q0 + q < NN) {
        const float dq = sqrtf(wave_sum(sq[q]));
        if (dq < dmin) { dmin = dq; hard = q0 + q; }
      }
    }
  }
  const float hinge = dpos - dmin + gamma;
  const bool act = hinge > 0.0f;
  if (lane == 0) lrow[row] = lam * match + (1.0f - lam) * (act ? hinge : 0.0f);
  const float ip = dpos > 0.0f ? 1.0f / dpos : 0.0f;
  const float in = dmin > 0.0f ? 1.0f / dmin : 0.0f;
  const f32x4* n4 = reinterpret_cast<const f32x4*>(negatives + (slot * NN + hard) * D);
  f32x4* g4 = reinterpret_cast<f32x4*>(SD + row * D);
  const float wr = act ? (1.0f - lam) : 0.0f;
  for (int c = lane; c < D4; c += 64) {
    const f32x4 pv = p4[c], diff = pv - y4[c], dn = pv - n4[c];
    f32x4 g;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      g[k] = lam * 2.0f * diff[k];
      if (act) g[k] += wr * (diff[k] * ip - dn[k] * in);
    }
    g4[c] = g;
  }
}

// Per-candidate loss: the sum of its steps' losses in step order.
__global__ __launch_bounds__(256) void loss_sum_kernel(const float* __restrict__ lrow,
                                                       const int32_t* __restrict__ off, int B,
                                                       float* __restrict__ loss) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B) return;
  float s = 0.0f;
  for (int r = off[i]; r < off[i + 1]; ++r) s += lrow[r];
  loss[i] = s;
}

// Row offsets: off[i] = sum over j < i of clamp(lens[j], 0, T_max), i <= B.
// One workgroup; each thread sums a contiguous run, then a workgroup scan.
__global__ __launch_bounds__(1024) void row_offsets_kernel(const int32_t* __restrict__ lens, int B,
                                                           int T_max, int32_t* __restrict__ off) {
  __shared__ int wsum[16];
  const int per = (B + 1023) / 1024;
  const int i0 = threadIdx.x * per, i1 = min(B, i0 + per);
  int s = 0;
  for (int i = i0; i < i1; ++i) s += clampi(lens[i], 0, T_max);
  int run = block_exclusive_scan(s, wsum);
  for (int i = i0; i < i1; ++i) {
    off[i] = run;
    run += clampi(lens[i], 0, T_max);
  }
  if (threadIdx.x == 1023) off[B] = run;
}

// Sum of the per-candidate losses, one workgroup in a fixed order.
__global__ __launch_bounds__(1024) void loss_total_kernel(const float* __restrict__ loss, int B,
                                                          float* __restrict__ total) {
  __shared__ float part[16];
  float s = 0.0f;
  for (int i = threadIdx.x; i < B; i += 1024) s += loss[i];
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    float tot = 0.0f;
    for (int w = 0; w < 16; ++w) tot += part[w];
    *total = tot;
  }
}

// train_bwd_kernel: one wavefront per tile, steps from the last to the first.
// delta (accumulator layout) gains each step's seed and is stored as
// delta_{t+1} (for dW2, db2); as the B operand (product-operand value) it
// gives dG^T = W2^T . delta^T per hidden chunk; dA = dG * GELU'(A) (A is read
// back and overwritten with dA); then dX^T = W1^T . dA^T, whose latent blocks
// accumulate straight into delta (the residual path carries delta itself)
// and whose embedding blocks are stored as dE.  Finished candidates have no
// seed and a zero mask, so their delta passes through unchanged.
template <class PR, int D, int E, int WAVES, bool NORM>
__global__ __launch_bounds__(64 * WAVES, 1) void train_bwd_kernel(const TrainArgs a) {
  using R = Roll<PR, D, E>;
  using TG = TrainGeom<PR, D, E>;
  using Frag = typename PR::Frag;
  constexpr int SL = PR::SL, G = PR::G;
  constexpr int NZ = R::NZ, NF2 = R::NF2, NB = R::NB, NBE = TG::NBE;
  constexpr int NW2T = TG::NW2T, NI = TG::NIB, RD = TG::RDB;
  constexpr int W2TB = TransT<PR>::w2t_bytes(D), W1TB = TransT<PR>::w1t_bytes(D, E);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  const TileInfo ti = tile_info(a, blockIdx.x * WAVES + wave, n);
  const int cand = ti.cand, len = ti.len, T_wg = ti.T_wg;
  const int NC = a.H / 32;
  const size_t row0 = ti.valid ? (size_t)a.off[cand] : 0;

  gu8* w2g = (gu8*)(a.w2t) + lane * 16;
  gu8* w1g = (gu8*)(a.w1t) + lane * 16;
  auto group_ptr = [&](int c, int i) -> gu32x4* {
    return reinterpret_cast<gu32x4*>(i < NW2T ? w2g + (size_t)c * W2TB + (size_t)i * 1024
                                              : w1g + (size_t)c * W1TB + (size_t)(i - NW2T) * 1024);
  };
  u32x4 ring[RD];
#pragma unroll
  for (int i = 0; i < RD; ++i) ring[i] = *group_ptr(0, i);

  f32x16 dacc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) dacc[b] = f32x16{};
  for (int t = T_wg - 1; t >= 0; --t) {
    const bool active = t < len;
    const float actf = active ? 1.0f : 0.0f;
    const uint32_t amask = active ? 0xFFFFFFFFu : 0u;
    const size_t row = row0 + t;
    if (active) {
#pragma unroll
      for (int b = 0; b < NB; ++b) dacc[b] += load_acc(a.SD + row * D + 32 * b, h);
    }
    f32x4 sc = {0.0f, 0.0f, 0.0f, 0.0f};
    if constexpr (NORM) {
      // through z_{t+1} = u / |u|: du = (delta - (delta . z) z) / |u|
      if (active) sc = *reinterpret_cast<const f32x4*>(a.SC + row * 4);
      float dz = 0.0f;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const f32x16 zb = active ? load_acc(a.P + row * D + 32 * b, h) : f32x16{};
#pragma unroll
        for (int r = 0; r < 16; ++r) dz = fmaf(dacc[b][r], zb[r], dz);
      }
      dz = dz + __shfl_xor(dz, 32);
      const bool nrm = active && sc[2] > 0.0f;
      const float inu = nrm ? 1.0f / sc[2] : 1.0f;
      const float cz = nrm ? dz : 0.0f;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const f32x16 zb = nrm ? load_acc(a.P + row * D + 32 * b, h) : f32x16{};
#pragma unroll
        for (int r = 0; r < 16; ++r) dacc[b][r] = (dacc[b][r] - cz * zb[r]) * inu;
      }
    }
    if (active) {
#pragma unroll
      for (int b = 0; b < NB; ++b) store_acc(a.SD + row * D + 32 * b, dacc[b], h);   // du (delta_{t+1} in the residual form)
    }
    Frag dop[NZ];
#pragma unroll
    for (int kf = 0; kf < NZ; ++kf) {
      float v[SL];
#pragma unroll
      for (int j = 0; j < SL; ++j) v[j] = dacc[kf / NF2][(kf % NF2) * SL + j];
      dop[kf] = PR::cvt(v);
    }
    f32x16 deacc[NBE];
#pragma unroll
    for (int b = 0; b < NBE; ++b) deacc[b] = f32x16{};
    for (int c = 0; c < NC; ++c) {
      const int cn = c + 1 < NC ? c + 1 : 0;
      float* arow = a.A + row * a.H + 32 * c;
      const f32x16 av = active ? load_acc(arow, h) : f32x16{};
      f32x16 acc = {};
      typename PR::Packed dp[8];
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const u32x4 grp = ring[i % RD];
        ring[i % RD] = (i + RD < NI) ? *group_ptr(c, i + RD) : *group_ptr(cn, i + RD - NI);
        if (i < NW2T) {
#pragma unroll
          for (int ww = 0; ww < G; ++ww) acc = PR::mfma(PR::pick(grp, ww), dop[i * G + ww], acc);
          if (i == NW2T - 1) {
            f32x16 da;
#pragma unroll
            for (int r = 0; r < 16; ++r) da[r] = acc[r] * gelu_grad(av[r]) * actf;
            if (active) store_acc(arow, da, h);       // dA
#pragma unroll
            for (int q = 0; q < 8; ++q) dp[q] = PR::pack2(da[2 * q], da[2 * q + 1], amask);
          }
        } else {
#pragma unroll
          for (int ww = 0; ww < G; ++ww) {
            const int F = (i - NW2T) * G + ww;          // output block F / NF2, fragment F % NF2
            const int ob = F / NF2;
            if (ob < NB) dacc[ob] = PR::mfma(PR::pick(grp, ww), PR::gfrag(dp, F % NF2), dacc[ob]);
            else deacc[ob - NB] = PR::mfma(PR::pick(grp, ww), PR::gfrag(dp, F % NF2), deacc[ob - NB]);
          }
        }
      }
    }
    if constexpr (NORM) {
      // through z' = z - (w . z) w, w = v / |v|: dz = dz' - (w . dz') w,
      // dv = (dw - (w . dw) w) / |v| with dw = -((w . z) dz' + (w . dz') z),
      // where w . dw = -2 (w . z)(w . dz'); de += R(Wh)^T R(dv)
      const bool prj = active && sc[1] > 0.0f;
      const float inv = prj ? rsqrtf(sc[1]) : 0.0f;
      const float wz = sc[0] * inv;
      float wdz = 0.0f;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const f32x16 vb = prj ? load_acc(a.V + row * D + 32 * b, h) : f32x16{};
#pragma unroll
        for (int r = 0; r < 16; ++r) wdz = fmaf(vb[r], dacc[b][r], wdz);
      }
      wdz = (wdz + __shfl_xor(wdz, 32)) * inv;
      const float* zin = t > 0 ? a.P + (row - 1) * D : a.z0 + (size_t)ti.seg * D;
      gu8* whtb = (gu8*)(a.wht) + lane * 16;
      constexpr int NZG = NZ / G;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const f32x16 vb = prj ? load_acc(a.V + row * D + 32 * b, h) : f32x16{};
        const f32x16 zb = prj ? load_acc(zin + 32 * b, h) : f32x16{};
        f32x16 dv;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float wr = vb[r] * inv;
          dv[r] = (-(wz * dacc[b][r] + wdz * zb[r]) + 2.0f * wz * wdz * wr) * inv;
          dacc[b][r] -= wdz * wr;
        }
        if (active) store_acc(a.DV + row * D + 32 * b, dv, h);
#pragma unroll
        for (int f = 0; f < NF2; ++f) {
          float v[SL];
#pragma unroll
          for (int j = 0; j < SL; ++j) v[j] = dv[f * SL + j];
          const Frag dvf = PR::cvt(v);
          const int kf = b * NF2 + f;
#pragma unroll
          for (int ob = 0; ob < NBE; ++ob) {
            const u32x4 grp = *reinterpret_cast<gu32x4*>(whtb + (size_t)(ob * NZG + kf / G) * 1024);
            deacc[ob] = PR::mfma(PR::pick(grp, kf % G), dvf, deacc[ob]);
          }
        }
      }
    }
    if (active) {
#pragma unroll
      for (int b = 0; b < NBE; ++b) store_acc(a.DE + row * E + 32 * b, deacc[b], h);
    }
  }
  if (ti.valid && a.dz0) {
#pragma unroll
    for (int b = 0; b < NB; ++b) store_acc(a.dz0 + (size_t)cand * D + 32 * b, dacc[b], h);
  }
}

// Row range of one split of the compact rows [0, off[B]): equal shares,
// multiples of 32 rows.
__device__ __forceinline__ void split_rows(const int32_t* off, int B, int splits, int split,
                                           int& r0, int& r1) {
  const int Rv = off[B];
  const int rps = ((Rv + splits - 1) / splits + 31) & ~31;
  r0 = min(Rv, split * rps);
  r1 = min(Rv, r0 + rps);
}

// Row-owned backward (d = 256, one workgroup of W wavefronts per tile), the
// mirror of the row-owned forward.  Per step, from the last to the first:
//  * wavefront w owns latent blocks [w*NBW, (w+1)*NBW) of delta: it adds the
//    step's seed, stores delta_{t+1}, and publishes the blocks as operand
//    fragments in LDS; after a barrier every wavefront reads all of delta;
//  * phase 1, for its chunks c = w, w+W, ...: dG^T = W2^T[c] . delta^T,
//    dA = dG * GELU'(A) (stored), dA as fragments into LDS, and the
//    embedding outputs dE^T += W1^T[c][e blocks] . dA^T (a partial over its
//    chunks, summed across wavefronts through LDS in a fixed order);
//  * phase 2, for its own latent blocks over every chunk:
//    delta += W1^T[c][block] . dA^T[c] (dA fragments from LDS).
// Weight groups stream from L2 through a register ring that wraps from step
// to step.
template <class PR, int D, int E, int NC, int W>
struct BwdRowsGeom {
  using R = Roll<PR, D, E>;
  static constexpr int G = PR::G, NF2 = R::NF2, NB = R::NB, NBE = E / 32;
  static constexpr int NBW = NB / W, NCW = NC / W;
  static constexpr int GF = NF2 / G;                      // W1^T groups per (chunk, output block)
  static constexpr int N2T = TransT<PR>::nk2t(D) / G;     // W2^T groups per chunk
  static constexpr int NP1 = N2T + NBE * GF;              // phase-1 groups per chunk
  static constexpr int NA = NCW * NP1;                    // phase-1 items
  static constexpr int NI = NA + NC * NBW * GF;           // items per step
  static constexpr int ring_depth() {
    const int cap = G == 1 ? 8 : 12;
    for (int r = cap; r > 1; --r)
      if (NI % r == 0) return r;
    return 1;
  }
  static constexpr int RD = ring_depth();
  static_assert(NB % W == 0 && NC % W == 0 && NF2 % G == 0, "even split");
  // LDS: [table-free] [dA fragments: NC * GF KiB][delta fragments: NZ / G KiB]
  //      [dE partials: W * NBE * 4 KiB]
  static constexpr int DA_BYTES = NC * GF * 1024;
  static constexpr int DL_BYTES = (R::NZ / G) * 1024;
  static constexpr int DE_BYTES = W * NBE * 4096;
  static constexpr int LDS = DA_BYTES + DL_BYTES + DE_BYTES;
};

template <class PR, int D, int E, int NC, int W, bool NORM>
__global__ __launch_bounds__(64 * W, 1) void train_bwd_rows_kernel(const TrainArgs a) {
  using R = Roll<PR, D, E>;
  using BG = BwdRowsGeom<PR, D, E, NC, W>;
  using Frag = typename PR::Frag;
  constexpr int SL = PR::SL, G = PR::G;
  constexpr int NZ = R::NZ, NF2 = R::NF2, NB = R::NB, NBE = BG::NBE;
  constexpr int NBW = BG::NBW, NCW = BG::NCW, GF = BG::GF, N2T = BG::N2T, NP1 = BG::NP1;
  constexpr int NA = BG::NA, NI = BG::NI, RD = BG::RD;
  constexpr int W2TB = TransT<PR>::w2t_bytes(D), W1TB = TransT<PR>::w1t_bytes(D, E);

  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  uint8_t* dabuf = lds;                                   // dA fragments, chunk-major
  uint8_t* dlbuf = lds + BG::DA_BYTES;                    // delta fragments
  float* debuf = reinterpret_cast<float*>(lds + BG::DA_BYTES + BG::DL_BYTES);  // [W][NBE][2][16][32]
  float* dots = reinterpret_cast<float*>(lds + BG::LDS);  // paper form: [2][W][32]

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  const TileInfo ti = tile_info(a, blockIdx.x, n);
  const int cand = ti.cand, len = ti.len, T_wg = ti.T_wg;
  const size_t row0 = ti.valid ? (size_t)a.off[cand] : 0;

  // item i -> weight group (compile-time offsets after unrolling)
  auto item_ptr = [&](gu8* p2, gu8* p1, int i) -> gu32x4* {
    if (i < NA) {
      const int cw = i / NP1, k = i % NP1, c = w + cw * W;
      if (k < N2T) return reinterpret_cast<gu32x4*>(p2 + (size_t)c * W2TB + (size_t)k * 1024);
      const int q = (k - N2T) / GF, fg = (k - N2T) % GF;
      return reinterpret_cast<gu32x4*>(p1 + (size_t)c * W1TB + (size_t)((NB + q) * GF + fg) * 1024);
    }
    const int j = i - NA, c = j / (NBW * GF), bq = (j / GF) % NBW, fg = j % GF;
    return reinterpret_cast<gu32x4*>(p1 + (size_t)c * W1TB + (size_t)((w * NBW + bq) * GF + fg) * 1024);
  };
  gu8* base2 = ((gu8*)(a.w2t)) + lane * 16;
  gu8* base1 = ((gu8*)(a.w1t)) + lane * 16;
  u32x4 ring[RD];
#pragma unroll
  for (int i = 0; i < RD; ++i) ring[i] = *item_ptr(base2, base1, i);

  f32x16 dq[NBW];
#pragma unroll
  for (int bq = 0; bq < NBW; ++bq) dq[bq] = f32x16{};

  for (int t = T_wg - 1; t >= 0; --t) {
    const bool active = t < len;
    const float actf = active ? 1.0f : 0.0f;
    const uint32_t amask = active ? 0xFFFFFFFFu : 0u;
    const size_t row = row0 + t;
    gu8* p2 = base2;
    gu8* p1 = base1;
    asm volatile("" : "+v"(p2), "+v"(p1));
    // ---- owned delta blocks: seed, delta_{t+1} (paper form: du through the
    // normalisation, du = (delta - (delta . z) z) / |u| with z the unit
    // prediction), operand fragments in LDS
    f32x4 sc = {0.0f, 0.0f, 0.0f, 0.0f};
    if (active) {
#pragma unroll
      for (int bq = 0; bq < NBW; ++bq) dq[bq] += load_acc(a.SD + row * D + 32 * (w * NBW + bq), h);
    }
    if constexpr (NORM) {
      if (active) sc = *reinterpret_cast<const f32x4*>(a.SC + row * 4);
      f32x16 pb[NBW];
      float dz = 0.0f;
#pragma unroll
      for (int bq = 0; bq < NBW; ++bq) {
        pb[bq] = active ? load_acc(a.P + row * D + 32 * (w * NBW + bq), h) : f32x16{};
#pragma unroll
        for (int r = 0; r < 16; ++r) dz = fmaf(dq[bq][r], pb[bq][r], dz);
      }
      dz = dz + __shfl_xor(dz, 32);
      if (h == 0) dots[w * 32 + n] = dz;
      __syncthreads();
      dz = 0.0f;
#pragma unroll
      for (int ww = 0; ww < W; ++ww) dz += dots[ww * 32 + n];
      const bool nrm = active && sc[2] > 0.0f;
      const float inu = nrm ? 1.0f / sc[2] : 1.0f;
      const float cz = nrm ? dz : 0.0f;
#pragma unroll
      for (int bq = 0; bq < NBW; ++bq)
#pragma unroll
        for (int r = 0; r < 16; ++r) dq[bq][r] = (dq[bq][r] - cz * pb[bq][r]) * inu;
    }
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq) {
      const int b = w * NBW + bq;
      if (active) store_acc(a.SD + row * D + 32 * b, dq[bq], h);
#pragma unroll
      for (int f = 0; f < NF2; ++f) {
        float v[SL];
#pragma unroll
        for (int j = 0; j < SL; ++j) v[j] = dq[bq][f * SL + j];
        *reinterpret_cast<Frag*>(dlbuf + frag_offset<PR>(b * NF2 + f, lane, 0)) = PR::cvt(v);
      }
    }
    // pre-activations of the own chunks (read early, used after W2^T)
    f32x16 av[NCW];
#pragma unroll
    for (int cw = 0; cw < NCW; ++cw)
      av[cw] = active ? load_acc(a.A + row * a.H + 32 * (w + cw * W), h) : f32x16{};
    __syncthreads();
    Frag dop[NZ];
#pragma unroll
    for (int kf = 0; kf < NZ; ++kf) dop[kf] = *reinterpret_cast<const Frag*>(dlbuf + frag_offset<PR>(kf, lane, 0));

    f32x16 acc = {};
    f32x16 deacc[NBE];
#pragma unroll
    for (int q = 0; q < NBE; ++q) deacc[q] = f32x16{};
    f32x16 emlp = {};              // paper form: this wavefront's dE block, MLP part
    typename PR::Packed dp[8];
    constexpr int GB = NF2 / G;
    u32x4 dcur[GB], dnext[GB];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const u32x4 grp = ring[i % RD];
      ring[i % RD] = *item_ptr(p2, p1, (i + RD) % NI);   // wraps into the next step
      if (i < NA) {
        const int cw = i / NP1, k = i % NP1, c = w + cw * W;
        if (k < N2T) {
          if (k == 0) acc = f32x16{};
#pragma unroll
          for (int ww = 0; ww < G; ++ww) acc = PR::mfma(PR::pick(grp, ww), dop[k * G + ww], acc);
          if (k == N2T - 1) {
            f32x16 da;
#pragma unroll
            for (int r = 0; r < 16; ++r) da[r] = acc[r] * gelu_grad(av[cw][r]) * actf;
            if (active) store_acc(a.A + row * a.H + 32 * c, da, h);
#pragma unroll
            for (int q = 0; q < 8; ++q) dp[q] = PR::pack2(da[2 * q], da[2 * q + 1], amask);
#pragma unroll
            for (int f = 0; f < NF2; ++f)
              *reinterpret_cast<Frag*>(dabuf + frag_offset<PR>(c * NF2 + f, lane, 0)) = PR::gfrag(dp, f);
          }
        } else {
          const int q = (k - N2T) / GF, fg = (k - N2T) % GF;
#pragma unroll
          for (int ww = 0; ww < G; ++ww)
            deacc[q] = PR::mfma(PR::pick(grp, ww), PR::gfrag(dp, fg * G + ww), deacc[q]);
        }
        if (i == NA - 1) {
          // embedding partials into LDS, then every chunk's dA is published
#pragma unroll
          for (int q = 0; q < NBE; ++q)
#pragma unroll
            for (int r = 0; r < 16; ++r) debuf[(((w * NBE + q) * 2 + h) * 16 + r) * 32 + n] = deacc[q][r];
          __syncthreads();
          if (w < NBE) {            // dE block w: the partials in wavefront order
            f32x16 e = {};
#pragma unroll
            for (int ww = 0; ww < W; ++ww)
#pragma unroll
              for (int r = 0; r < 16; ++r) e[r] += debuf[(((ww * NBE + w) * 2 + h) * 16 + r) * 32 + n];
            if constexpr (NORM) emlp = e;
            else if (active) store_acc(a.DE + row * E + 32 * w, e, h);
          }
#pragma unroll
          for (int gg = 0; gg < GB; ++gg) dcur[gg] = lds_group(dabuf, gg, lane);
#pragma unroll
          for (int gg = 0; gg < GB; ++gg) dnext[gg] = lds_group(dabuf, (NC > 1 ? GB : 0) + gg, lane);
        }
      } else {
        const int j = i - NA, c = j / (NBW * GF), bq = (j / GF) % NBW, fg = j % GF;
#pragma unroll
        for (int ww = 0; ww < G; ++ww) {
          const int f = fg * G + ww;
          const u32x4 gf = dcur[(f * SL * PR::ES) / 16];
          Frag b;
          if constexpr (G == 1) b = PR::pick(gf, 0);
          else b = PR::pick(gf, f % G);
          dq[bq] = PR::mfma(PR::pick(grp, ww), b, dq[bq]);
        }
        if (bq == NBW - 1 && fg == GF - 1) {
#pragma unroll
          for (int gg = 0; gg < GB; ++gg) dcur[gg] = dnext[gg];
          if (c + 2 < NC) {
#pragma unroll
            for (int gg = 0; gg < GB; ++gg) dnext[gg] = lds_group(dabuf, (c + 2) * GB + gg, lane);
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (NORM) {
      // through z' = z - (w . z) w, w = v / |v| (as in the one-wavefront
      // kernel): dz = dz' - (w . dz') w, dv = (dw - (w . dw) w) / |v|,
      // de += R(Wh)^T R(dv); the dot w . dz' and the dE partials of the
      // owned blocks are summed across wavefronts through LDS
      const bool prj = active && sc[1] > 0.0f;
      const float inv = prj ? rsqrtf(sc[1]) : 0.0f;
      const float wz = sc[0] * inv;
      f32x16 vb[NBW];
      float wdz = 0.0f;
#pragma unroll
      for (int bq = 0; bq < NBW; ++bq) {
        vb[bq] = prj ? load_acc(a.V + row * D + 32 * (w * NBW + bq), h) : f32x16{};
#pragma unroll
        for (int r = 0; r < 16; ++r) wdz = fmaf(vb[bq][r], dq[bq][r], wdz);
      }
      wdz = wdz + __shfl_xor(wdz, 32);
      if (h == 0) dots[(W + w) * 32 + n] = wdz;
      __syncthreads();
      wdz = 0.0f;
#pragma unroll
      for (int ww = 0; ww < W; ++ww) wdz += dots[(W + ww) * 32 + n];
      wdz *= inv;
      const float* zin = t > 0 ? a.P + (row - 1) * D : a.z0 + (size_t)ti.seg * D;
      gu8* whtb = (gu8*)(a.wht) + lane * 16;
      constexpr int NZG = NZ / G;
      f32x16 den[NBE];
#pragma unroll
      for (int q = 0; q < NBE; ++q) den[q] = f32x16{};
#pragma unroll
      for (int bq = 0; bq < NBW; ++bq) {
        const int b = w * NBW + bq;
        const f32x16 zb = prj ? load_acc(zin + 32 * b, h) : f32x16{};
        f32x16 dv;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float wr = vb[bq][r] * inv;
          dv[r] = (-(wz * dq[bq][r] + wdz * zb[r]) + 2.0f * wz * wdz * wr) * inv;
          dq[bq][r] -= wdz * wr;
        }
        if (active) store_acc(a.DV + row * D + 32 * b, dv, h);
#pragma unroll
        for (int f = 0; f < NF2; ++f) {
          float v[SL];
#pragma unroll
          for (int j = 0; j < SL; ++j) v[j] = dv[f * SL + j];
          const Frag dvf = PR::cvt(v);
          const int kf = b * NF2 + f;
#pragma unroll
          for (int q = 0; q < NBE; ++q) {
            const u32x4 grp = *reinterpret_cast<gu32x4*>(whtb + (size_t)(q * NZG + kf / G) * 1024);
            den[q] = PR::mfma(PR::pick(grp, kf % G), dvf, den[q]);
          }
        }
      }
      // the MLP partials were read before this step's dot barrier
#pragma unroll
      for (int q = 0; q < NBE; ++q)
#pragma unroll
        for (int r = 0; r < 16; ++r) debuf[(((w * NBE + q) * 2 + h) * 16 + r) * 32 + n] = den[q][r];
      __syncthreads();
      if (w < NBE) {
        f32x16 e = emlp;
#pragma unroll
        for (int ww = 0; ww < W; ++ww)
#pragma unroll
          for (int r = 0; r < 16; ++r) e[r] += debuf[(((ww * NBE + w) * 2 + h) * 16 + r) * 32 + n];
        if (active) store_acc(a.DE + row * E + 32 * w, e, h);
      }
    }
    __syncthreads();                // dA / dE buffers are read before the next step writes them
  }
  if (ti.valid && a.dz0) {
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq) store_acc(a.dz0 + (size_t)cand * D + 32 * (w * NBW + bq), dq[bq], h);
  }
}

// Narrow-tile backward of the rollout loss (residual form; one workgroup of
// W wavefronts per tile of 16 candidates), the mirror of the narrow forward
// with the products of the 32-candidate row-owned backward.  Per step, from
// the last to the first:
//  * wavefront w owns latent blocks 2w, 2w+1 of delta: it adds the step's
//    seed, stores delta_{t+1}, and publishes the blocks as operand fragment w
//    in LDS; after a barrier every wavefront reads all of delta;
//  * for its chunks c = w, w + W, ...: dG^T = W2^T[c] . delta^T (two 16-row
//    blocks), dA = dG * GELU'(A) (stored), dA as an operand fragment into
//    LDS, and its partial dE^T += W1^T[c][e blocks] . dA^T (summed across
//    wavefronts through LDS in a fixed order);
//  * after a barrier, for its own latent blocks over every chunk:
//    delta += W1^T[c][block] . dA^T[c].
// Weight groups stream from L2 through a register ring that wraps from step
// to step (transposed blob at Narrow::t_bytes).
template <class NP, int D, int E, int NC, int W>
struct NarrowBwdGeom {
  static constexpr int GPK = NP::GPK;
  static constexpr int NB = D / 16, NBW = NB / W, NZ = D / 32, NBE = E / 16, IB = (D + E) / 16;
  static constexpr int NCW = NC / W;
  static constexpr int N2T = NZ * 2 * GPK;                 // W2^T groups per chunk
  static constexpr int NP1 = N2T + NBE * GPK;              // first-phase groups per chunk
  static constexpr int NA = NCW * NP1;
  static constexpr int NI = NA + NC * NBW * GPK;
  static constexpr int W2TG = NC * NZ * 2 * GPK;           // W2^T groups in the blob
  static constexpr int ring_depth() {
    for (int r = 12; r > 1; --r)
      if (NI % r == 0) return r;
    return 1;
  }
  static constexpr int RD = ring_depth();
  static_assert(NBW == 2 && NZ == W && NC % W == 0 && NBE <= W, "narrow split");
  // LDS: [dA fragments: NC][delta fragments: NZ][dE partials: W x NBE x 64 lanes x 4]
  static constexpr int DA_BYTES = NC * GPK * 1024, DL_BYTES = NZ * GPK * 1024;
  static constexpr int DE_BYTES = W * NBE * 64 * 16;
  static constexpr int LDS = DA_BYTES + DL_BYTES + DE_BYTES;
  static constexpr int DOTS_BYTES = 2 * W * 16 * 4;        // paper form: two dot products
};

// NORM (paper form, as the one-wavefront kernel): du through the
// normalisation at the start of a step, and dz, dv through the projection
// after the MLP part, with the dots summed over the lane groups and then the
// wavefronts through LDS; the normal map's dE partials (Wh^T . dv over the
// owned fragment) join the MLP ones.
template <class NP, int D, int E, int NC, int W, bool NORM>
__global__ __launch_bounds__(64 * W, 1) void train_bwd_narrow_kernel(const TrainArgs a) {
  using BG = NarrowBwdGeom<NP, D, E, NC, W>;
  using XF = typename NP::XF;
  constexpr int GPK = BG::GPK, NZ = BG::NZ, NBE = BG::NBE, IB = BG::IB, NBW = BG::NBW, NB = BG::NB;
  constexpr int NCW = BG::NCW, N2T = BG::N2T, NP1 = BG::NP1, NA = BG::NA, NI = BG::NI, RD = BG::RD;
  (void)NB;

  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  uint8_t* dabuf = lds;                                             // dA fragments [NC]
  uint8_t* dlbuf = lds + BG::DA_BYTES;                              // delta fragments [NZ]
  float* debuf = reinterpret_cast<float*>(lds + BG::DA_BYTES + BG::DL_BYTES);  // [W][NBE][64][4]
  float* dots = reinterpret_cast<float*>(lds + BG::LDS);            // paper form: [2][W][16]

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = lane & 15, g = lane >> 4;
  const int pos = blockIdx.x * 16 + n;
  const bool valid = pos < a.B;
  const int2 pc = valid ? a.perm[pos] : make_int2(0, 0);
  const int cand = pc.x;
  const int len = valid ? clampi(a.lens[cand], 0, a.T_max) : 0;
  const int T_wg = __builtin_amdgcn_readfirstlane(
      clampi(a.lens[a.perm[blockIdx.x * 16].x], 0, a.T_max));
  const size_t row0 = valid ? (size_t)a.off[cand] : 0;

  // item i -> weight group (compile-time offsets from three bases)
  gu8* baseA2 = ((gu8*)(a.w2t)) + (size_t)(w * N2T) * 1024 + lane * 16;
  gu8* baseA1 = ((gu8*)(a.w2t)) + (size_t)(BG::W2TG + (w * IB + NZ * 2) * GPK) * 1024 + lane * 16;
  gu8* baseB = ((gu8*)(a.w2t)) + (size_t)(BG::W2TG + w * NBW * GPK) * 1024 + lane * 16;
  auto item_ptr = [&](gu8* p2, gu8* p1, gu8* pb, int i) -> gu32x4* {
    if (i < NA) {
      const int cw = i / NP1, k = i % NP1;
      if (k < N2T) return reinterpret_cast<gu32x4*>(p2 + ((size_t)cw * W * N2T + k) * 1024);
      return reinterpret_cast<gu32x4*>(p1 + ((size_t)cw * W * IB * GPK + (k - N2T)) * 1024);
    }
    const int j = i - NA, c = j / (NBW * GPK), r = j % (NBW * GPK);
    return reinterpret_cast<gu32x4*>(pb + ((size_t)c * IB * GPK + r) * 1024);
  };
  u32x4 ring[RD];
#pragma unroll
  for (int i = 0; i < RD; ++i) ring[i] = *item_ptr(baseA2, baseA1, baseB, i);

  f32x4n dq[NBW];
#pragma unroll
  for (int bq = 0; bq < NBW; ++bq) dq[bq] = f32x4n{};

  for (int t = T_wg - 1; t >= 0; --t) {
    const bool active = t < len;
    const float actf = active ? 1.0f : 0.0f;
    const uint32_t amask = active ? 0xFFFFFFFFu : 0u;
    const size_t row = row0 + t;
    gu8* p2 = baseA2;
    gu8* p1 = baseA1;
    gu8* pb = baseB;
    asm volatile("" : "+v"(p2), "+v"(p1), "+v"(pb));
    // ---- owned delta blocks: seed, delta_{t+1} (paper form: du through the
    // normalisation, du = (delta - (delta . z) z) / |u| with z the unit
    // prediction), operand fragment w in LDS
    f32x4n sc = {0.0f, 0.0f, 0.0f, 0.0f};
    if (active) {
#pragma unroll
      for (int bq = 0; bq < NBW; ++bq)
        dq[bq] += *reinterpret_cast<const f32x4n*>(a.SD + row * D + 16 * (w * NBW + bq) + 4 * g);
    }
    if constexpr (NORM) {
      if (active) sc = *reinterpret_cast<const f32x4n*>(a.SC + row * 4);
      f32x4n pb[NBW];
      float dz = 0.0f;
#pragma unroll
      for (int bq = 0; bq < NBW; ++bq) {
        pb[bq] = active ? *reinterpret_cast<const f32x4n*>(a.P + row * D + 16 * (w * NBW + bq) + 4 * g) : f32x4n{};
#pragma unroll
        for (int r = 0; r < 4; ++r) dz = fmaf(dq[bq][r], pb[bq][r], dz);
      }
      dz += __shfl_xor(dz, 16);
      dz += __shfl_xor(dz, 32);
      if (g == 0) dots[w * 16 + n] = dz;
      __syncthreads();
      dz = 0.0f;
#pragma unroll
      for (int ww = 0; ww < W; ++ww) dz += dots[ww * 16 + n];
      const bool nrm = active && sc[2] > 0.0f;
      const float inu = nrm ? 1.0f / sc[2] : 1.0f;
      const float cz = nrm ? dz : 0.0f;
#pragma unroll
      for (int bq = 0; bq < NBW; ++bq) dq[bq] = (dq[bq] - cz * pb[bq]) * inu;
    }
    float v8[8];
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq) {
      if (active) *reinterpret_cast<f32x4n*>(a.SD + row * D + 16 * (w * NBW + bq) + 4 * g) = dq[bq];
#pragma unroll
      for (int r = 0; r < 4; ++r) v8[4 * bq + r] = dq[bq][r];
    }
    NP::store(dlbuf, w, lane, NP::cvt(v8));
    // pre-activations of the own chunks (read early, used after W2^T)
    f32x4n av[NCW][2];
#pragma unroll
    for (int cw = 0; cw < NCW; ++cw)
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
        av[cw][rb] = active ? *reinterpret_cast<const f32x4n*>(a.A + row * a.H + 32 * (w + cw * W) + 16 * rb + 4 * g)
                            : f32x4n{};
    __syncthreads();
    XF dop[NZ];
#pragma unroll
    for (int kf = 0; kf < NZ; ++kf) dop[kf] = NP::load(dlbuf, kf, lane);

    f32x4n acc[2], deacc[NBE];
    acc[0] = f32x4n{}; acc[1] = f32x4n{};
#pragma unroll
    for (int q = 0; q < NBE; ++q) deacc[q] = f32x4n{};
    XF dfr = {}, dcur = {}, dnext = {};
    f32x4n emlp = {};              // paper form: this wavefront's dE block, MLP part
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const u32x4 grp = ring[i % RD];
      ring[i % RD] = *item_ptr(p2, p1, pb, (i + RD) % NI);   // wraps into the next step
      if (i < NA) {
        const int cw = i / NP1, k = i % NP1;
        if (k < N2T) {
          const int kf = k / (2 * GPK), rb = (k / GPK) % 2, hh = k % GPK;
          acc[rb] = NP::mma(grp, hh, dop[kf], acc[rb]);
          if (k == N2T - 1) {
            const int c = w + cw * W;
            float da[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) da[j] = acc[j >> 2][j & 3] * gelu_grad(av[cw][j >> 2][j & 3]) * actf;
            if (active) {
#pragma unroll
              for (int rb2 = 0; rb2 < 2; ++rb2) {
                const f32x4n d4 = {da[4 * rb2], da[4 * rb2 + 1], da[4 * rb2 + 2], da[4 * rb2 + 3]};
                *reinterpret_cast<f32x4n*>(a.A + row * a.H + 32 * c + 16 * rb2 + 4 * g) = d4;   // dA
              }
            }
            dfr = NP::gfrag(da, amask);
            NP::store(dabuf, c, lane, dfr);
            acc[0] = f32x4n{};
            acc[1] = f32x4n{};
          }
        } else {
          const int q = (k - N2T) / GPK, hh = (k - N2T) % GPK;
          deacc[q] = NP::mma(grp, hh, dfr, deacc[q]);
        }
        if (i == NA - 1) {
          // embedding partials into LDS, then every chunk's dA is published
#pragma unroll
          for (int q = 0; q < NBE; ++q)
            *reinterpret_cast<f32x4n*>(debuf + ((w * NBE + q) * 64 + lane) * 4) = deacc[q];
          __syncthreads();
          if (w < NBE) {            // dE block w: the partials in wavefront order
            f32x4n e4 = {};
#pragma unroll
            for (int ww = 0; ww < W; ++ww) e4 += *reinterpret_cast<const f32x4n*>(debuf + ((ww * NBE + w) * 64 + lane) * 4);
            if constexpr (NORM) emlp = e4;
            else if (active) *reinterpret_cast<f32x4n*>(a.DE + row * E + 16 * w + 4 * g) = e4;
          }
          dcur = NP::load(dabuf, 0, lane);
          dnext = NP::load(dabuf, NC > 1 ? 1 : 0, lane);
        }
      } else {
        const int j = i - NA, c = j / (NBW * GPK), bq = (j / GPK) % NBW, hh = j % GPK;
        dq[bq] = NP::mma(grp, hh, dcur, dq[bq]);
        if (bq == NBW - 1 && hh == GPK - 1) {
          dcur = dnext;
          if (c + 2 < NC) dnext = NP::load(dabuf, c + 2, lane);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (NORM) {
      // through z' = z - (w . z) w, w = v / |v|: dz = dz' - (w . dz') w,
      // dv = (dw - (w . dw) w) / |v| with w . dw = -2 (w . z)(w . dz'),
      // de += R(Wh)^T R(dv)
      const bool prj = active && sc[1] > 0.0f;
      const float inv = prj ? rsqrtf(sc[1]) : 0.0f;
      const float wz = sc[0] * inv;
      f32x4n vb[NBW];
      float wdz = 0.0f;
#pragma unroll
      for (int bq = 0; bq < NBW; ++bq) {
        vb[bq] = prj ? *reinterpret_cast<const f32x4n*>(a.V + row * D + 16 * (w * NBW + bq) + 4 * g) : f32x4n{};
#pragma unroll
        for (int r = 0; r < 4; ++r) wdz = fmaf(vb[bq][r], dq[bq][r], wdz);
      }
      wdz += __shfl_xor(wdz, 16);
      wdz += __shfl_xor(wdz, 32);
      if (g == 0) dots[(W + w) * 16 + n] = wdz;
      __syncthreads();
      wdz = 0.0f;
#pragma unroll
      for (int ww = 0; ww < W; ++ww) wdz += dots[(W + ww) * 16 + n];
      wdz *= inv;
      const float* zin = t > 0 ? a.P + (row - 1) * D : a.z0 + (size_t)pc.y * D;
      float dv8[8];
#pragma unroll
      for (int bq = 0; bq < NBW; ++bq) {
        const f32x4n zb = prj ? *reinterpret_cast<const f32x4n*>(zin + 16 * (w * NBW + bq) + 4 * g) : f32x4n{};
        f32x4n dv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float wr = vb[bq][r] * inv;
          dv[r] = (-(wz * dq[bq][r] + wdz * zb[r]) + 2.0f * wz * wdz * wr) * inv;
          dq[bq][r] -= wdz * wr;
          dv8[4 * bq + r] = dv[r];
        }
        if (active) *reinterpret_cast<f32x4n*>(a.DV + row * D + 16 * (w * NBW + bq) + 4 * g) = dv;
      }
      // normal-map part of dE over the owned latent fragment w
      const XF dvf = NP::cvt(dv8);
      gu8* whtb = ((gu8*)(a.wht)) + lane * 16;
      f32x4n den[NBE];
#pragma unroll
      for (int q = 0; q < NBE; ++q) {
        den[q] = f32x4n{};
#pragma unroll
        for (int hh = 0; hh < GPK; ++hh) {
          const u32x4 grp = *reinterpret_cast<gu32x4*>(whtb + ((size_t)(q * NZ + w) * GPK + hh) * 1024);
          den[q] = NP::mma(grp, hh, dvf, den[q]);
        }
      }
      // the MLP partials were read before this step's dot barrier
#pragma unroll
      for (int q = 0; q < NBE; ++q)
        *reinterpret_cast<f32x4n*>(debuf + ((w * NBE + q) * 64 + lane) * 4) = den[q];
      __syncthreads();
      if (w < NBE) {
        f32x4n e4 = emlp;
#pragma unroll
        for (int ww = 0; ww < W; ++ww) e4 += *reinterpret_cast<const f32x4n*>(debuf + ((ww * NBE + w) * 64 + lane) * 4);
        if (active) *reinterpret_cast<f32x4n*>(a.DE + row * E + 16 * w + 4 * g) = e4;
      }
    }
    __syncthreads();                // dA / dE / delta buffers are read before the next step writes them
  }
  if (valid && a.dz0) {
#pragma unroll
    for (int bq = 0; bq < NBW; ++bq)
      *reinterpret_cast<f32x4n*>(a.dz0 + (size_t)cand * D + 16 * (w * NBW + bq) + 4 * g) = dq[bq];
  }
}

// Weight gradients as split-K products over the compact rows, two problems
// per launch (dW2 = sum R(delta) (x) g, dW1 = sum R(dA) (x) x):
//   part[split][m][n] = sum over the split's rows r of op(A[r][m]) * op(B[r][n])
// with the column sums of A (unrounded: db2, db1) on the side.  Workgroup =
// 4 wavefronts on a 128 x 128 output tile, each wavefront 64 x 64 (2 x 2
// matrix-core tiles); 32 rows per stage: every thread loads 8 consecutive
// rows of one column (coalesced across the wavefront), rounds them as
// product operands and writes them to LDS transposed (column-major, rows
// contiguous), so each lane's operand fragment is one 16-byte LDS read.  The
// next stage's loads are in flight during the current stage's products.
struct WgradProblem {
  const float* A;           // [rows][lda], columns [0, M)
  const float* Bm;          // [rows][ldb], columns [0, N)
  float* part;              // [splits][M][N]
  float* colsum;            // [splits][M] (may be null)
  int M, N, lda, ldb, tiles_n, tiles;
};
struct WgradArgs {
  WgradProblem p0, p1, p2;  // p2.tiles may be 0
  const int32_t* off;
  int B, splits;
};
constexpr int WG_T = 128, WG_KC = 32;

template <class PR>
__global__ __launch_bounds__(256) void wgrad_kernel(const WgradArgs a) {
  constexpr int KF = PR::KF, SL = PR::SL;
  constexpr bool BF = PR::G == 1;
  using Elem = typename std::conditional<BF, __bf16, float>::type;
  constexpr int LDW = WG_KC + (BF ? 8 : 4);               // padded LDS row (elements)
  __shared__ __attribute__((aligned(16))) Elem As[WG_T * LDW];
  __shared__ __attribute__((aligned(16))) Elem Bs[WG_T * LDW];
  __shared__ float csum[WG_T];
  // Workgroups are dealt to the 8 XCDs in turn: every tile of split s runs
  // on XCD s mod 8, so the split's rows come from HBM once per XCD and the
  // other tiles' re-reads hit that XCD's L2.
  const int tiles_all = a.p0.tiles + a.p1.tiles + a.p2.tiles;
  const int xcd = blockIdx.x % 8, k8 = blockIdx.x / 8;
  const int tile_id = k8 % tiles_all;
  const int split = (k8 / tiles_all) * 8 + xcd;
  if (split >= a.splits) return;
  const int which = tile_id < a.p0.tiles ? 0 : (tile_id < a.p0.tiles + a.p1.tiles ? 1 : 2);
  const WgradProblem& pr = which == 0 ? a.p0 : (which == 1 ? a.p1 : a.p2);
  const float* A = pr.A;
  const float* Bm = pr.Bm;
  float* part = pr.part;
  float* colsum = pr.colsum;
  const int M = pr.M, N = pr.N, lda = pr.lda, ldb = pr.ldb;
  const int tiles_n = pr.tiles_n;
  const int tile = tile_id - (which == 0 ? 0 : (which == 1 ? a.p0.tiles : a.p0.tiles + a.p1.tiles));
  const int m0 = (tile / tiles_n) * WG_T, n0 = (tile % tiles_n) * WG_T;
  int r0, r1;
  split_rows(a.off, a.B, a.splits, split, r0, r1);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = tid & (WG_T - 1), rg = tid >> 7;          // loader: column, row group (0, 1)
  const bool okA = m0 + c < M, okB = n0 + c < N;
  float va[2][8], vb[2][8];
  float cs = 0.0f;
  auto load = [&](int rb) {
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int r = rb + (rg + 2 * q) * 8 + j;
        const bool rv = r < r1;
        va[q][j] = (rv && okA) ? A[(size_t)r * lda + m0 + c] : 0.0f;
        vb[q][j] = (rv && okB) ? Bm[(size_t)r * ldb + n0 + c] : 0.0f;
      }
  };
  auto store = [&]() {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
#pragma unroll
      for (int j = 0; j < 8; ++j) cs += va[q][j];
      Elem* da = As + c * LDW + (rg + 2 * q) * 8;
      Elem* db = Bs + c * LDW + (rg + 2 * q) * 8;
      if constexpr (BF) {
        bf16x8 ea, eb;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          ea[j] = (__bf16)va[q][j];
          eb[j] = (__bf16)vb[q][j];
        }
        *reinterpret_cast<bf16x8*>(da) = ea;
        *reinterpret_cast<bf16x8*>(db) = eb;
      } else {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const f32x4 xa = {va[q][4 * k], va[q][4 * k + 1], va[q][4 * k + 2], va[q][4 * k + 3]};
          const f32x4 xb = {vb[q][4 * k], vb[q][4 * k + 1], vb[q][4 * k + 2], vb[q][4 * k + 3]};
          *reinterpret_cast<f32x4*>(da + 4 * k) = xa;
          *reinterpret_cast<f32x4*>(db + 4 * k) = xb;
        }
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
  if (r0 < r1) load(r0);
  for (int rb = r0; rb < r1; rb += WG_KC) {
    __syncthreads();                      // the previous stage's reads are done
    store();
    __syncthreads();
    if (rb + WG_KC < r1) load(rb + WG_KC);
#pragma unroll
    for (int ks = 0; ks < WG_KC / KF; ++ks) {
      typename PR::Frag fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const Elem* pa = As + (wm * 64 + i * 32 + cl) * LDW + ks * KF + h * SL;
        const Elem* pb = Bs + (wn * 64 + i * 32 + cl) * LDW + ks * KF + h * SL;
        if constexpr (BF) {
          fa[i] = *reinterpret_cast<const typename PR::Frag*>(pa);
          fb[i] = *reinterpret_cast<const typename PR::Frag*>(pb);
        } else {
          fa[i] = *pa;
          fb[i] = *pb;
        }
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = PR::mfma(fa[i], fb[j], acc[i][j]);
    }
  }
  float* o = part + (size_t)split * M * N;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn * 64 + j * 32 + cl;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * 64 + i * 32 + acc_row(h, r);
        if (m < M && n < N) o[(size_t)m * N + n] = acc[i][j][r];
      }
    }
  // column sums of A: the two row groups, in order (first column tile only)
  if (n0 == 0 && colsum) {
    __syncthreads();
    if (rg == 1) csum[c] = cs;
    __syncthreads();
    if (rg == 0 && okA) colsum[(size_t)split * M + m0 + c] = cs + csum[c];
  }
}

// All the split sums of one gradient call in one launch: job j adds the
// splits of `part` (stride apart) for its n outputs in a fixed order (eight
// running sums, k mod 8, so the loads are independent, then a fixed tree);
// the threads cover the jobs' outputs back to back.
constexpr int SUM_JOBS = 8;
struct SumJobs {
  const float* part[SUM_JOBS];
  float* out[SUM_JOBS];
  long long stride[SUM_JOBS];
  long long start[SUM_JOBS + 1];    // prefix of the output counts
  int splits[SUM_JOBS];
  int count;
};
__global__ __launch_bounds__(256) void sum_jobs_kernel(const SumJobs jb) {
  const long long q = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= jb.start[jb.count]) return;
  int j = 0;
  while (j + 1 < jb.count && q >= jb.start[j + 1]) ++j;
  const long long i = q - jb.start[j];
  const float* part = jb.part[j];
  const long long stride = jb.stride[j];
  const int splits = jb.splits[j];
  float s[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  int k = 0;
  for (; k + 8 <= splits; k += 8) {
#pragma unroll
    for (int u = 0; u < 8; ++u) s[u] += part[(size_t)(k + u) * stride + i];
  }
  for (int u = 0; k + u < splits; ++u) s[u] += part[(size_t)(k + u) * stride + i];
  jb.out[j][i] = ((s[0] + s[1]) + (s[2] + s[3])) + ((s[4] + s[5]) + (s[6] + s[7]));
}

// Embedding gradients over one block of the compact rows:
// part[block] = [ d type_emb (K x E) | d param_w (E x P) | d param_b (E) ].
// Rows are taken 64 at a time: their action kinds and log2 parameters are
// staged in LDS (one thread per row), then thread (row group g, feature f)
// walks rows g, g + RG, ... of the batch with per-kind bins in LDS (each
// thread owns its feature's column); the row groups are added in order.
constexpr int EMB_THREADS = 256, EMB_ROWS = 64;
__global__ __launch_bounds__(EMB_THREADS) void emb_grad_kernel(const float* __restrict__ DE, int E,
                                                               const int32_t* __restrict__ row_src,
                                                               const int32_t* __restrict__ types,
                                                               const int32_t* __restrict__ params,
                                                               int K, int P,
                                                               const int32_t* __restrict__ off, int B,
                                                               int splits, float* __restrict__ part) {
  extern __shared__ float bins[];                          // [RG][K + P + 1][E]
  __shared__ int s_ty[EMB_ROWS];
  __shared__ float s_u[EMB_ROWS][PMAX];
  const int RG = EMB_THREADS / E;
  const int f = threadIdx.x % E, g = threadIdx.x / E;
  const int W = K * E + E * P + E;
  int r0, r1;
  split_rows(off, B, splits, blockIdx.x, r0, r1);
  float* mine = bins + (size_t)g * (K + P + 1) * E;
  for (int k = 0; k < K + P + 1; ++k) mine[k * E + f] = 0.0f;
  for (int rb = r0; rb < r1; rb += EMB_ROWS) {
    const int nr = min(EMB_ROWS, r1 - rb);
    __syncthreads();
    if ((int)threadIdx.x < nr) {
      const int src = row_src[rb + threadIdx.x];
      s_ty[threadIdx.x] = types[src];
      for (int p = 0; p < P; ++p) s_u[threadIdx.x][p] = log2f((float)params[(size_t)src * P + p]);
    }
    __syncthreads();
    for (int q = g; q < nr; q += RG) {
      const float v = DE[(size_t)(rb + q) * E + f];
      const int ty = s_ty[q];
      if (ty >= 0 && ty < K) mine[ty * E + f] += v;
      for (int p = 0; p < P; ++p) mine[(K + p) * E + f] = fmaf(v, s_u[q][p], mine[(K + p) * E + f]);
      mine[(K + P) * E + f] += v;
    }
  }
  __syncthreads();
  if (g != 0) return;
  float* o = part + (size_t)blockIdx.x * W;
  for (int k = 0; k < K + P + 1; ++k) {
    float s = 0.0f;
    for (int q = 0; q < RG; ++q) s += bins[((size_t)q * (K + P + 1) + k) * E + f];
    if (k < K) o[k * E + f] = s;                            // type_emb [K][E]
    else if (k < K + P) o[K * E + f * P + (k - K)] = s;     // param_w [E][P]
    else o[K * E + E * P + f] = s;                          // param_b [E]
  }
}

// ==========================================================================
// Cost model.  Wavefront = 32 candidates (original order), workgroup walks
// the 32-wide chunks of the cost hidden layer with Wc1 fragments staged in
// LDS.  The [z_T; phi] product is shared by all hardware vectors; each vector
// adds its own small product.  Up to 4 hardware vectors per launch.

constexpr int SCORE_HW_PER_LAUNCH = 2;  // hardware vectors per score launch

struct ScoreArgs {
  const uint8_t* cost;
  const float* zT;
  const float* phi;
  const float* hw;    // [n_hw][HW]
  float* scores;      // [n_hw][B]
  float bc2;
  int B, C, HW, j0, nj, chunk_bytes;
};

template <class PR, int D, int E>
struct ScoreStep {
  using Frag = typename PR::Frag;
  static constexpr int KF = PR::KF, SL = PR::SL, G = PR::G;
  static constexpr int NX = (D + E) / KF;
  static constexpr int MAXH = SCORE_MAX_HW / KF;

  static __device__ __forceinline__ void chunk(const uint8_t* cur, int CB, int NH, int nj,
                                               const Frag (&x)[NX],
                                               const Frag (&hf)[SCORE_HW_PER_LAUNCH][MAXH],
                                               float (&part)[SCORE_HW_PER_LAUNCH], int lane, int h) {
    f32x16 acc = {};
#pragma unroll
    for (int g = 0; g < NX / G; ++g) {
      const u32x4 grp = lds_group(cur, g, lane);
#pragma unroll
      for (int w = 0; w < G; ++w) acc = PR::mfma(PR::pick(grp, w), x[g * G + w], acc);
    }
    const float* tail = reinterpret_cast<const float*>(cur + (CB - 256));
    const float* bc1t = tail + 16 * h;
    const float* wc2t = tail + 32 + 16 * h;
#pragma unroll
    for (int jj = 0; jj < SCORE_HW_PER_LAUNCH; ++jj) {
      if (jj < nj) {
        f32x16 accj = acc;
#pragma unroll
        for (int q = 0; q < MAXH; ++q) {
          if (q < NH) {
            const int F = NX + q;
            accj = PR::mfma(PR::pick(lds_group(cur, F / G, lane), F % G), hf[jj][q], accj);
          }
        }
        float s = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) s = fmaf(wc2t[r], gelu(accj[r] + bc1t[r]), s);
        part[jj] += s;
      }
    }
  }
};

template <class PR, int D, int E, int WAVES>
__global__ __launch_bounds__(64 * WAVES, 1) void score_kernel(const ScoreArgs a) {
  using SS = ScoreStep<PR, D, E>;
  using Frag = typename PR::Frag;
  constexpr int KF = PR::KF, SL = PR::SL;
  constexpr int NX = SS::NX, MAXH = SS::MAXH;
  constexpr int NT = 64 * WAVES;
  constexpr int CBMAX = CostChunk<PR>::bytes(D, E, SCORE_MAX_HW);
  __shared__ __attribute__((aligned(16))) uint8_t bufA[CBMAX];
  __shared__ __attribute__((aligned(16))) uint8_t bufB[CBMAX];
  const int CB = a.chunk_bytes;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  const int NH = a.HW / KF;
  const int NC = a.C / 32;                        // even (checked on the host)

  stage_to_lds(a.cost, bufA, CB, tid, NT);

  const int cand = (blockIdx.x * WAVES + wave) * 32 + n;
  const bool valid = cand < a.B;
  const int ci = valid ? cand : 0;

  Frag x[NX];
#pragma unroll
  for (int kf = 0; kf < NX; ++kf) {
    float v[SL];
#pragma unroll
    for (int j = 0; j < SL; ++j) {
      const int f = nat_feature<PR>(kf, h, j);
      v[j] = f < D ? a.zT[(size_t)ci * D + f] : a.phi[(size_t)ci * E + (f - D)];
    }
    x[kf] = PR::cvt(v);
  }
  Frag hf[SCORE_HW_PER_LAUNCH][MAXH];
#pragma unroll
  for (int jj = 0; jj < SCORE_HW_PER_LAUNCH; ++jj)
#pragma unroll
    for (int q = 0; q < MAXH; ++q) {
      float v[SL];
#pragma unroll
      for (int j = 0; j < SL; ++j)
        v[j] = (jj < a.nj && q < NH) ? a.hw[(size_t)(a.j0 + jj) * a.HW + nat_feature<PR>(q, h, j)] : 0.0f;
      hf[jj][q] = PR::cvt(v);
    }
  float part[SCORE_HW_PER_LAUNCH];
#pragma unroll
  for (int jj = 0; jj < SCORE_HW_PER_LAUNCH; ++jj) part[jj] = 0.0f;

  wait_vm_then_barrier();
  for (int c = 0; c < NC; c += 2) {
    stage_to_lds(a.cost + (size_t)(c + 1) * CB, bufB, CB, tid, NT);
    __builtin_amdgcn_sched_barrier(0);
    SS::chunk(bufA, CB, NH, a.nj, x, hf, part, lane, h);
    wait_vm_then_barrier();
    if (c + 2 < NC) stage_to_lds(a.cost + (size_t)(c + 2) * CB, bufA, CB, tid, NT);
    __builtin_amdgcn_sched_barrier(0);
    SS::chunk(bufB, CB, NH, a.nj, x, hf, part, lane, h);
    wait_vm_then_barrier();
  }
#pragma unroll
  for (int jj = 0; jj < SCORE_HW_PER_LAUNCH; ++jj) {
    if (jj < a.nj) {
      const float y = part[jj] + __shfl_xor(part[jj], 32) + a.bc2;
      if (valid && h == 0) a.scores[(size_t)(a.j0 + jj) * a.B + cand] = y;
    }
  }
}

// Cost model for small batches: a workgroup of SPLIT wavefronts per 32
// candidates, wavefront w taking cost-hidden chunks w, w + SPLIT, ... with
// fragments read straight from L2; the partial scores are summed through LDS
// in a fixed order (deterministic).
template <class PR, int D, int E, int SPLIT>
__global__ __launch_bounds__(64 * SPLIT, 1) void score_split_kernel(const ScoreArgs a) {
  using Frag = typename PR::Frag;
  constexpr int KF = PR::KF, SL = PR::SL, G = PR::G;
  constexpr int NX = (D + E) / KF;
  constexpr int MAXH = SCORE_MAX_HW / KF;
  constexpr int HPL = SCORE_HW_PER_LAUNCH;
  __shared__ float red[SPLIT][HPL][64];
  const int CB = a.chunk_bytes;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  const int NH = a.HW / KF;
  const int NC = a.C / 32;
  const int cand = blockIdx.x * 32 + n;
  const bool valid = cand < a.B;
  const int ci = valid ? cand : 0;

  Frag x[NX];
#pragma unroll
  for (int kf = 0; kf < NX; ++kf) {
    float v[SL];
#pragma unroll
    for (int j = 0; j < SL; ++j) {
      const int f = nat_feature<PR>(kf, h, j);
      v[j] = f < D ? a.zT[(size_t)ci * D + f] : a.phi[(size_t)ci * E + (f - D)];
    }
    x[kf] = PR::cvt(v);
  }
  Frag hf[HPL][MAXH];
#pragma unroll
  for (int jj = 0; jj < HPL; ++jj)
#pragma unroll
    for (int q = 0; q < MAXH; ++q) {
      float v[SL];
#pragma unroll
      for (int j = 0; j < SL; ++j)
        v[j] = (jj < a.nj && q < NH) ? a.hw[(size_t)(a.j0 + jj) * a.HW + nat_feature<PR>(q, h, j)] : 0.0f;
      hf[jj][q] = PR::cvt(v);
    }
  float part[HPL];
#pragma unroll
  for (int jj = 0; jj < HPL; ++jj) part[jj] = 0.0f;

  for (int c = w; c < NC; c += SPLIT) {
    const uint8_t* cb = a.cost + (size_t)c * CB;
    f32x16 acc = {};
#pragma unroll
    for (int g = 0; g < NX / G; ++g) {
      const u32x4 grp = *reinterpret_cast<const u32x4*>(cb + g * 1024 + lane * 16);
#pragma unroll
      for (int ww = 0; ww < G; ++ww) acc = PR::mfma(PR::pick(grp, ww), x[g * G + ww], acc);
    }
    const float* tail = reinterpret_cast<const float*>(cb + (CB - 256));
    float bc1t[16], wc2t[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      bc1t[r] = tail[16 * h + r];
      wc2t[r] = tail[32 + 16 * h + r];
    }
#pragma unroll
    for (int jj = 0; jj < HPL; ++jj) {
      if (jj < a.nj) {
        f32x16 accj = acc;
#pragma unroll
        for (int q = 0; q < MAXH; ++q) {
          if (q < NH) {
            const int F = NX + q;
            const u32x4 grp = *reinterpret_cast<const u32x4*>(cb + (F / G) * 1024 + lane * 16);
            accj = PR::mfma(PR::pick(grp, F % G), hf[jj][q], accj);
          }
        }
        float sum = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) sum = fmaf(wc2t[r], gelu(accj[r] + bc1t[r]), sum);
        part[jj] += sum;
      }
    }
  }
#pragma unroll
  for (int jj = 0; jj < HPL; ++jj) red[w][jj][lane] = part[jj];
  __syncthreads();
  if (w == 0) {
#pragma unroll
    for (int jj = 0; jj < HPL; ++jj) {
      if (jj < a.nj) {
        float y = red[0][jj][lane];
#pragma unroll
        for (int ww = 1; ww < SPLIT; ++ww) y += red[ww][jj][lane];
        y += __shfl_xor(y, 32) + a.bc2;
        if (valid && h == 0) a.scores[(size_t)(a.j0 + jj) * a.B + cand] = y;
      }
    }
  }
}

// ==========================================================================
// Encoder: one workgroup of ENC_THREADS per subgraph.  In bf16 mode the input
// and the hidden layer are rounded to bf16 (the weights already are).  Each
// layer splits its contraction over G = ENC_THREADS / outputs thread groups
// (coalesced weight reads across the outputs), and the G partial sums are
// added in group order.
constexpr int ENC_THREADS = 1024;

// out[o] = sum_k wt[k * N + o] x[k], o < N, through the partial-sum buffer
__device__ __forceinline__ void enc_layer(const float* __restrict__ wt, const float* x, int K, int N,
                                          float* part, float* out) {
  const int tid = threadIdx.x;
  for (int o0 = 0; o0 < N; o0 += ENC_THREADS) {
    const int n = min(N - o0, ENC_THREADS);
    const int G = ENC_THREADS / n, o = o0 + tid % n, grp = tid / n;
    const int kc = (K + G - 1) / G, k0 = grp * kc, k1 = min(K, k0 + kc);
    // eight independent loads in flight per thread (the loop is latency-bound)
    float acc = 0.0f;
    if (grp < G) {
      int k = k0;
      for (; k + 8 <= k1; k += 8) {
        float wv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) wv[u] = wt[(size_t)(k + u) * N + o];
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = fmaf(wv[u], x[k + u], acc);
      }
      for (; k < k1; ++k) acc = fmaf(wt[(size_t)k * N + o], x[k], acc);
    }
    part[tid] = acc;
    __syncthreads();
    if (tid < n) {
      float t = part[tid];
      for (int g2 = 1; g2 < G; ++g2) t += part[g2 * n + tid];
      out[o0 + tid] = t;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(ENC_THREADS) void encode_kernel(const float* __restrict__ feats,
                                                             const float* __restrict__ w1t,
                                                             const float* __restrict__ b1,
                                                             const float* __restrict__ w2t,
                                                             const float* __restrict__ b2, int F,
                                                             int Fh, int D, int bf16,
                                                             float* __restrict__ z0) {
  extern __shared__ float esm[];
  float* xs = esm;             // [F]
  float* hs = esm + F;         // [Fh]
  float* os = hs + Fh;         // [D]
  float* part = os + D;        // [ENC_THREADS]
  const int s = blockIdx.x;
  for (int f = threadIdx.x; f < F; f += blockDim.x) {
    const float v = feats[(size_t)s * F + f];
    xs[f] = bf16 ? (float)(__bf16)v : v;
  }
  __syncthreads();
  enc_layer(w1t, xs, F, Fh, part, hs);
  for (int o = threadIdx.x; o < Fh; o += blockDim.x) {
    const float g = gelu(hs[o] + b1[o]);
    hs[o] = bf16 ? (float)(__bf16)g : g;
  }
  __syncthreads();
  enc_layer(w2t, hs, Fh, D, part, os);
  for (int o = threadIdx.x; o < D; o += blockDim.x) z0[(size_t)s * D + o] = os[o] + b2[o];
}

// ==========================================================================
// Top-k per (hardware vector j, subgraph s): one workgroup of 1024 threads.
//
// Scores map to order-preserving unsigned keys (NaN lowest, -0 == +0).  A
// most-significant-digit radix select finds the k-th largest key K*; a second
// radix select over the (complemented) local index finds how many candidates
// tied at K* to keep, lowest index first.  The k selected candidates are then
// bitonic-sorted in LDS by the 64-bit key (score key, ~index).

__device__ __forceinline__ uint32_t score_key(float v) {
  if (v != v) return 0u;                // NaN ranks last
  if (v == 0.0f) v = 0.0f;              // -0 == +0
  const uint32_t u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int TOPK_THREADS = 1024;
constexpr int TOPK_WAVES = TOPK_THREADS / 64;

// Largest-first radix select over the keys that for_each(f) passes to f
// (each thread its own elements): returns the `need`-th largest key (1-based)
// and, in *rank_in_eq, how many elements equal to it must be taken.
template <class ForEach>
__device__ uint32_t radix_select(int need, ForEach for_each, uint32_t* hist_w, int* shared_int,
                                 int* rank_in_eq) {
  const int tid = threadIdx.x, wave = tid >> 6;
  uint32_t prefix = 0, mask = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < TOPK_WAVES * 256; i += TOPK_THREADS) hist_w[i] = 0;
    __syncthreads();
    for_each([&](uint32_t kk) {
      if ((kk & mask) == prefix) atomicAdd(&hist_w[wave * 256 + ((kk >> shift) & 255)], 1u);
    });
    __syncthreads();
    // combine the per-wave histograms into the first
    for (int b = tid; b < 256; b += TOPK_THREADS) {
      uint32_t s = 0;
      for (int w = 0; w < TOPK_WAVES; ++w) s += hist_w[w * 256 + b];
      hist_w[b] = s;
    }
    __syncthreads();
    if (tid < 64) {
      // lane l holds bins 255-4l .. 252-4l; an inclusive scan over lanes
      // (highest bins first) finds the bin where the count reaches `need`
      const int l = tid;
      int c4[4], sum = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c4[q] = (int)hist_w[255 - 4 * l - q];
        sum += c4[q];
      }
      int incl = sum;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off);
        if (l >= off) incl += v;
      }
      const unsigned long long hit = __ballot(incl >= need);
      const int first = __ffsll((long long)hit) - 1;
      if (l == first) {
        int rem = need - (incl - sum), digit = 255 - 4 * l;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (c4[q] >= rem) { digit = 255 - 4 * l - q; break; }
          rem -= c4[q];
        }
        shared_int[0] = digit;
        shared_int[1] = rem;
      }
    }
    __syncthreads();
    const int digit = shared_int[0];
    need = shared_int[1];
    prefix |= (uint32_t)digit << shift;
    mask |= 255u << shift;
    __syncthreads();
  }
  *rank_in_eq = need;
  return prefix;
}

// KPT > 0: the segment has at most KPT * TOPK_THREADS candidates and each
// thread keeps its keys in registers across the passes; KPT = 0 reads the
// scores again in every pass.
template <int KPT>
__global__ __launch_bounds__(TOPK_THREADS) void topk_kernel(const float* __restrict__ scores,
                                                            int B, const SegTable seg, int k,
                                                            int P2, int32_t* __restrict__ idx,
                                                            float* __restrict__ val) {
  __shared__ uint32_t hist_w[TOPK_WAVES * 256];
  __shared__ unsigned long long sel[WM_MAX_K];
  __shared__ int sh[4];
  const int S = seg.n;
  const int j = blockIdx.x / S, s = blockIdx.x % S;
  const int lo = seg.off[s], hi = seg.off[s + 1], n = hi - lo;
  const float* y = scores + (size_t)j * B + lo;
  const int tid = threadIdx.x;

  uint32_t keys[KPT > 0 ? KPT : 1];
  if constexpr (KPT > 0) {
#pragma unroll
    for (int q = 0; q < KPT; ++q) {
      const int i = tid + q * TOPK_THREADS;
      keys[q] = i < n ? score_key(y[i]) : 0u;
    }
  }
  // f(key, local index) over this thread's candidates
  auto each_key = [&](auto f) {
    if constexpr (KPT > 0) {
#pragma unroll
      for (int q = 0; q < KPT; ++q) {
        const int i = tid + q * TOPK_THREADS;
        if (i < n) f(keys[q], i);
      }
    } else {
      for (int i = tid; i < n; i += TOPK_THREADS) f(score_key(y[i]), i);
    }
  };

  int need_eq = 0;
  const uint32_t kstar = radix_select(
      k, [&](auto f) { each_key([&](uint32_t kk, int) { f(kk); }); }, hist_w, sh, &need_eq);
  // count of keys equal to K*
  if (tid == 0) { sh[2] = 0; sh[3] = 0; }
  __syncthreads();
  int my_eq = 0;
  each_key([&](uint32_t kk, int) { my_eq += (kk == kstar); });
  if (my_eq) atomicAdd(&sh[2], my_eq);
  __syncthreads();
  const int n_eq = sh[2];
  // ties at K*: keep the need_eq lowest local indices (largest ~index)
  uint32_t istar = 0;
  if (need_eq < n_eq) {
    int dummy = 0;
    istar = radix_select(
        need_eq,
        [&](auto f) { each_key([&](uint32_t kk, int i) { if (kk == kstar) f(~(uint32_t)i); }); },
        hist_w, sh, &dummy);
  }
  const uint32_t ilimit = (need_eq < n_eq) ? ~istar : 0xFFFFFFFFu;  // keep local index <= ilimit
  if (tid == 0) sh[3] = 0;
  for (int i = tid; i < P2; i += TOPK_THREADS) sel[i] = 0ull;
  __syncthreads();
  each_key([&](uint32_t kk, int i) {
    if (kk > kstar || (kk == kstar && (uint32_t)i <= ilimit)) {
      const int slot = atomicAdd(&sh[3], 1);
      if (slot < k) sel[slot] = ((unsigned long long)kk << 32) | (unsigned long long)(~(uint32_t)i);
    }
  });
  __syncthreads();
  // bitonic sort, descending
  for (int size = 2; size <= P2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < P2; i += TOPK_THREADS) {
        const int partner = i ^ stride;
        if (partner > i) {
          const bool desc = (i & size) == 0;
          const unsigned long long a0 = sel[i], a1 = sel[partner];
          if (desc ? (a0 < a1) : (a0 > a1)) { sel[i] = a1; sel[partner] = a0; }
        }
      }
      __syncthreads();
    }
  }
  for (int r = tid; r < k; r += TOPK_THREADS) {
    // (exactly k keys are selected; the clamp only guards the read)
    const int li = clampi((int)(~(uint32_t)(sel[r] & 0xFFFFFFFFull)), 0, n - 1);
    const size_t o = ((size_t)j * S + s) * k + r;
    idx[o] = lo + li;
    if (val) val[o] = y[li];
  }
}

// ==========================================================================
// Launchers.

namespace {


template <class PR, int D, int E, int WAVES, bool NORM>
hipError_t launch_rollout_t(const DevModel& m, const RollArgs& a, int blocks, hipStream_t st) {
  // the chunk buffers are static; the table and the phi sums are dynamic
  constexpr bool PHI_OK = persistent_phi_ok<PR, D, E, WAVES, NORM>();
  const int lds = m.roll_tab_bytes + (PHI_OK && a.phi ? WAVES * 32 * (E + 1) * 4 : 0);
  auto kern = rollout_kernel<PR, D, E, WAVES, NORM>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();   // do not leave the error for the caller's next HIP call
    return e;
  }
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(64 * WAVES), lds, st, a);
  return hipGetLastError();
}

template <class PR, int D, int E, int WAVES>
hipError_t launch_score_t(const DevModel& m, const ScoreArgs& a, int blocks, hipStream_t st) {
  const int lds = 0;                  // static chunk buffers
  auto kern = score_kernel<PR, D, E, WAVES>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();   // do not leave the error for the caller's next HIP call
    return e;
  }
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(64 * WAVES), lds, st, a);
  return hipGetLastError();
}

// Wavefronts per workgroup: as many as keep at least one workgroup per
// compute unit (256), so small batches spread over more units.
constexpr int SPLIT_MAX_TILES = 256;   // = compute units

inline int pick_waves(int tiles) {
  if (tiles >= 4 * 256) return 4;
  if (tiles >= 2 * 256) return 2;
  return 1;
}

// Instantiated (precision, d, e).  fp32 keeps z and its operand copy in
// registers (d floats per lane pair), which caps it at d = 256.
#define WM_CASE(P, PRT, D, E, CALL) \
  if (prec == P && d == D && e == E) { using PR = PRT; CALL(PR, D, E); }

#define WM_FOR_ALL_DE(CALL)                 \
  WM_CASE(WM_FP32, PF32, 64, 32, CALL)      \
  WM_CASE(WM_FP32, PF32, 256, 64, CALL)     \
  WM_CASE(WM_BF16, PBF16, 64, 32, CALL)     \
  WM_CASE(WM_BF16, PBF16, 256, 64, CALL)    \
  WM_CASE(WM_BF16, PBF16, 512, 128, CALL)

}  // namespace

bool have_kernels(int prec, int d, int e) {
#define WM_HAVE(PR, D, E) return true;
  WM_FOR_ALL_DE(WM_HAVE)
#undef WM_HAVE
  return false;
}

int rollout_lds_bytes(const DevModel& m) {
  int b = 2 * (m.w1_chunk_bytes + m.w2_chunk_bytes) + m.roll_tab_bytes;
  if (m.wh_bytes && wh_in_lds(m.w1_chunk_bytes, m.w2_chunk_bytes, m.wh_bytes)) b += m.wh_bytes;
  return b;
}

__global__ __launch_bounds__(64) void clear_words_kernel(int32_t* __restrict__ p, int n) {
  for (int i = threadIdx.x; i < n; i += 64) p[i] = 0;
}

hipError_t launch_clear_words(int32_t* p, int n, hipStream_t st) {
  hipLaunchKernelGGL(clear_words_kernel, dim3(1), dim3(64), 0, st, p, n);
  return hipGetLastError();
}

hipError_t launch_bucket(const int32_t* lens, int32_t B, int32_t T_max, const SegTable& seg,
                         int2* perm, int32_t* hist, int32_t* err, hipStream_t st) {
  const int groups = bucket_groups(B);
  if (groups == 0) {
    const int lds = 2 * (T_max + 1) * (int)sizeof(int);
    hipLaunchKernelGGL(bucket_kernel, dim3(1), dim3(1024), lds, st, lens, B, T_max, seg, perm, err);
    return hipGetLastError();
  }
  const int chunk = bucket_chunk(B);
  const int lds = (T_max + 1) * (int)sizeof(int);
  hipLaunchKernelGGL(bucket_count_kernel, dim3(groups), dim3(1024), lds, st, lens, B, T_max, chunk,
                     hist, err);
  hipLaunchKernelGGL(bucket_scan_kernel, dim3(1), dim3(1024), lds + 16 * (int)sizeof(int), st, T_max,
                     groups, hist);
  hipLaunchKernelGGL(bucket_scatter_kernel, dim3(groups), dim3(1024), lds, st, lens, B, T_max, chunk,
                     seg, hist, perm);
  return hipGetLastError();
}

template <class PR, int D, int E, int SPLIT, bool NORM>
hipError_t launch_rollout_split_t(const DevModel& m, const RollArgs& a, int tiles, hipStream_t st) {
  // table, SPLIT partial-update regions, and (paper form) the dot-product area
  const int lds = m.roll_tab_bytes + SPLIT * (D / 32) * 4 * 1024 + (NORM ? SPLIT * 3 * 32 * 4 : 0);
  auto kern = rollout_split_kernel<PR, D, E, SPLIT, NORM>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e;
  }
  hipLaunchKernelGGL(kern, dim3(tiles), dim3(64 * SPLIT), lds, st, a);
  return hipGetLastError();
}

// One (precision, d, e, transition form) without narrow tiles: split kernel
// for at most one tile per compute unit, else the persistent kernel with 1, 2
// or 4 wavefronts per workgroup.
template <class PR, int D, int E, bool NORM>
hipError_t launch_rollout_de(const DevModel& m, const RollArgs& a, int tiles, int blocks,
                             int waves, bool split, bool* phi_done, hipStream_t st) {
  *phi_done = a.phi != nullptr;
  // fp32 at d = 256 does not fit the split kernel's registers; the split
  // kernel leaves the action features to the phi kernel
  if constexpr (D <= 256 && (PR::G == 1 || D <= 64)) {
    constexpr int SPLIT = (D / 32) >= 4 ? 4 : (D / 32);
    if (split && m.dims.trans_hidden / 32 >= SPLIT) {
      RollArgs b = a;
      b.phi = nullptr;
      *phi_done = false;
      return launch_rollout_split_t<PR, D, E, SPLIT, NORM>(m, b, tiles, st);
    }
  }
  // the persistent kernel sums the action features where they fit its LDS
  const bool pok = waves == 4   ? persistent_phi_ok<PR, D, E, 4, NORM>()
                   : waves == 2 ? persistent_phi_ok<PR, D, E, 2, NORM>()
                                : persistent_phi_ok<PR, D, E, 1, NORM>();
  if (!pok) {
    RollArgs b = a;
    b.phi = nullptr;
    *phi_done = false;
    if (waves == 4) return launch_rollout_t<PR, D, E, 4, NORM>(m, b, blocks, st);
    if (waves == 2) return launch_rollout_t<PR, D, E, 2, NORM>(m, b, blocks, st);
    return launch_rollout_t<PR, D, E, 1, NORM>(m, b, blocks, st);
  }
  if (waves == 4) return launch_rollout_t<PR, D, E, 4, NORM>(m, a, blocks, st);
  if (waves == 2) return launch_rollout_t<PR, D, E, 2, NORM>(m, a, blocks, st);
  return launch_rollout_t<PR, D, E, 1, NORM>(m, a, blocks, st);
}

// Narrow tiles (16 candidates) for batches of at most two such tiles per
// compute unit: d = 256, e = 64 (8 wavefronts; bf16 with hidden widths 512
// and 1024, fp32 with 512) and d = 64, e = 32 (2 wavefronts, hidden width
// 128), both transition forms.  Up to 512 tiles they beat one 32-candidate
// tile per compute unit: candidates are sorted longest first, so the
// second tiles a compute unit takes are the short ones.
constexpr int NARROW_MAX_TILES = 512;
template <class NP, int NC, bool NORM, bool TRAIN = false, bool SCORE = false, int D = 256, int E = 64,
          int W = 8>
hipError_t launch_rollout_narrow(const DevModel& m, RollArgs a, int tiles, hipStream_t st) {
  using NG = NarrowGeom<NP, D, E, NC, W>;
  a.w1 = m.trans_n;
  const int lds = m.roll_tab_bytes + NG::G_BYTES + NG::X_BYTES + (NORM ? W * 3 * 16 * 4 : 0) +
                  (a.phi && !TRAIN ? 16 * (E + 1) * 4 : 0) + (SCORE ? W * NARROW_SCORE_HW * 16 * 4 : 0);
  auto kern = rollout_narrow_kernel<NP, D, E, NC, W, NORM, TRAIN, SCORE>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e;
  }
  hipLaunchKernelGGL(kern, dim3(tiles), dim3(64 * W), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_rollout(const DevModel& m, const float* z0, const int2* perm,
                          const int32_t* types, const int32_t* params, const int32_t* lens,
                          int32_t B, int32_t T_max, float* zT, float* phi, bool* phi_done,
                          int32_t* err, hipStream_t st, ScoreFuse* sf) {
  RollArgs a{};
  a.w1 = m.trans_w1; a.w2 = m.trans_w2; a.wh = m.trans_wh; a.tab = m.roll_tab; a.z0 = z0; a.perm = perm; a.types = types;
  a.params = params; a.lens = lens; a.zT = zT; a.phi = phi; a.err = err; a.B = B; a.T_max = T_max;
  a.P = m.dims.n_params; a.K = m.dims.n_kinds; a.H = m.dims.trans_hidden;
  a.tab_bytes = m.roll_tab_bytes;
  const int tiles = (B + 31) / 32;
  const int waves = pick_waves(tiles);
  const int blocks = (tiles + waves - 1) / waves;
  const int prec = m.prec, d = m.dims.d, e = m.dims.embed_dim;
  // At most one tile per compute unit: split each tile's hidden units over
  // the compute unit's SIMDs instead (d <= 256: the partial updates fit LDS).
  const bool split = tiles <= SPLIT_MAX_TILES && d <= 256;
  const bool norm = m.dims.norm == WM_NORM_L2;
  *phi_done = false;
  const int ntiles = (B + 15) / 16;
  if (d == 256 && e == 64 && m.trans_n && B > 0 && ntiles <= NARROW_MAX_TILES) {
    const int NC = m.dims.trans_hidden / 32;
    // scores fused: phi sums present, the narrow cost blob, at most two
    // hardware vectors of at most 32 features
    const bool fuse = sf && phi && m.cost_n && sf->n_hw >= 1 && sf->n_hw <= NARROW_SCORE_HW &&
                      m.dims.hw_dim <= SCORE_MAX_HW;
    if (fuse) {
      a.costn = m.cost_n; a.hw = sf->hw; a.scores = sf->scores; a.bc2 = m.bc2;
      a.n_hw = sf->n_hw; a.HW = m.dims.hw_dim; a.C = m.dims.cost_hidden;
    }
    auto narrow = [&](auto np, auto nc_tag, auto norm_tag) -> hipError_t {
      using NPT = decltype(np);
      constexpr int NCT = decltype(nc_tag)::value;
      constexpr bool NT = decltype(norm_tag)::value;
      *phi_done = phi != nullptr;
      if (fuse) {
        sf->done = true;
        return launch_rollout_narrow<NPT, NCT, NT, false, true>(m, a, ntiles, st);
      }
      return launch_rollout_narrow<NPT, NCT, NT, false, false>(m, a, ntiles, st);
    };
    using I16 = std::integral_constant<int, 16>;
    using I32 = std::integral_constant<int, 32>;
    using BT = std::true_type;
    using BF = std::false_type;
    if (prec == WM_BF16 && NC == 16) return norm ? narrow(NarrowBF16{}, I16{}, BT{}) : narrow(NarrowBF16{}, I16{}, BF{});
    if (prec == WM_BF16 && NC == 32) return norm ? narrow(NarrowBF16{}, I32{}, BT{}) : narrow(NarrowBF16{}, I32{}, BF{});
    if (prec == WM_FP32 && NC == 16) return norm ? narrow(NarrowF32{}, I16{}, BT{}) : narrow(NarrowF32{}, I16{}, BF{});
  }
  if (d == 64 && e == 32 && m.trans_n && B > 0 && ntiles <= NARROW_MAX_TILES && m.dims.trans_hidden == 128) {
    *phi_done = phi != nullptr;
    if (prec == WM_BF16)
      return norm ? launch_rollout_narrow<NarrowBF16, 4, true, false, false, 64, 32, 2>(m, a, ntiles, st)
                  : launch_rollout_narrow<NarrowBF16, 4, false, false, false, 64, 32, 2>(m, a, ntiles, st);
    return norm ? launch_rollout_narrow<NarrowF32, 4, true, false, false, 64, 32, 2>(m, a, ntiles, st)
                : launch_rollout_narrow<NarrowF32, 4, false, false, false, 64, 32, 2>(m, a, ntiles, st);
  }
#define WM_ROLL(PR, D, E)                                                                          \
  return norm ? launch_rollout_de<PR, D, E, true>(m, a, tiles, blocks, waves, split, phi_done, st)  \
              : launch_rollout_de<PR, D, E, false>(m, a, tiles, blocks, waves, split, phi_done, st);
  WM_FOR_ALL_DE(WM_ROLL)
#undef WM_ROLL
  return hipErrorInvalidValue;
}

hipError_t launch_phi(const DevModel& m, const int32_t* types, const int32_t* params,
                      const int32_t* lens, int32_t B, int32_t T_max, float* phi, hipStream_t st) {
  const int E = m.dims.embed_dim;
  if (B == 0) return hipSuccess;
  const int blocks = (B + 15) / 16;               // four wavefronts of four candidates each
  hipLaunchKernelGGL(phi_kernel, dim3(blocks), dim3(256), 0, st, m.emb_nat, types, params, lens,
                     B, T_max, E, m.dims.n_params, m.dims.n_kinds, phi);
  return hipGetLastError();
}

hipError_t launch_phi_struct(const int32_t* types, const int32_t* params, const int32_t* lens,
                             int32_t B, int32_t T_max, int32_t K, int32_t P, float* phi_s,
                             hipStream_t st) {
  if (B == 0) return hipSuccess;
  if (K > 32 || P > PMAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(phi_struct_kernel, dim3((B + 3) / 4), dim3(256), 0, st, types, params, lens, B,
                     T_max, K, P, phi_s);
  return hipGetLastError();
}

hipError_t launch_score_trees(const DevForest& f, const float* zT, int32_t d, const float* phi_s,
                              int32_t phi_dim, int32_t B, const float* hw, int32_t n_hw,
                              int32_t hw_dim, float* scores, hipStream_t st) {
  if (B == 0) return hipSuccess;
  const int lds = (TREE_CPB * (d + phi_dim + hw_dim) + (TREE_THREADS / 64) * TREE_CPB) * (int)sizeof(float);
  hipError_t e = hipFuncSetAttribute((const void*)score_trees_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e;
  }
  hipLaunchKernelGGL(score_trees_kernel, dim3((B + TREE_CPB - 1) / TREE_CPB, n_hw), dim3(TREE_THREADS), lds, st, static_cast<const int2*>(f.nodes),
                     f.leaves, f.n_trees, f.depth, f.base, zT, d, phi_s, phi_dim, hw, hw_dim, B,
                     scores);
  return hipGetLastError();
}

hipError_t launch_score(const DevModel& m, const float* zT, const float* phi, int32_t B,
                        const float* hw, int32_t n_hw, float* scores, hipStream_t st) {
  const int tiles = (B + 31) / 32;
  const int waves = pick_waves(tiles);
  const int blocks = (tiles + waves - 1) / waves;
  const int prec = m.prec, d = m.dims.d, e = m.dims.embed_dim;
  for (int j0 = 0; j0 < n_hw; j0 += SCORE_HW_PER_LAUNCH) {
    ScoreArgs a;
    a.cost = m.cost; a.zT = zT; a.phi = phi; a.hw = hw; a.scores = scores; a.bc2 = m.bc2;
    a.B = B; a.C = m.dims.cost_hidden; a.HW = m.dims.hw_dim; a.j0 = j0;
    a.nj = (n_hw - j0) < SCORE_HW_PER_LAUNCH ? (n_hw - j0) : SCORE_HW_PER_LAUNCH;
    a.chunk_bytes = m.cost_chunk_bytes;
    hipError_t err = hipErrorInvalidValue;
#define WM_SCORE(PR, D, E)                                                       \
  {                                                                              \
    if (tiles <= SPLIT_MAX_TILES && a.C / 32 >= 4) {                             \
      hipLaunchKernelGGL((score_split_kernel<PR, D, E, 4>), dim3(tiles), dim3(256), 0, st, a); \
      err = hipGetLastError();                                                   \
    } else if (waves == 4) err = launch_score_t<PR, D, E, 4>(m, a, blocks, st);  \
    else if (waves == 2) err = launch_score_t<PR, D, E, 2>(m, a, blocks, st);    \
    else err = launch_score_t<PR, D, E, 1>(m, a, blocks, st);                    \
  }
    WM_FOR_ALL_DE(WM_SCORE)
#undef WM_SCORE
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

hipError_t launch_topk(const float* scores, int32_t n_hw, int32_t B, const SegTable& seg,
                       int32_t k, int32_t* idx, float* val, hipStream_t st) {
  int P2 = 1;
  while (P2 < k) P2 <<= 1;
  int nmax = 0;
  for (int s = 0; s < seg.n; ++s) nmax = seg.off[s + 1] - seg.off[s] > nmax ? seg.off[s + 1] - seg.off[s] : nmax;
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3(n_hw * seg.n), dim3(TOPK_THREADS), 0, st, scores, B, seg, k, P2, idx, val);
  };
  if (nmax <= 2 * TOPK_THREADS) go(topk_kernel<2>);
  else if (nmax <= 8 * TOPK_THREADS) go(topk_kernel<8>);
  else if (nmax <= 32 * TOPK_THREADS) go(topk_kernel<32>);
  else go(topk_kernel<0>);
  return hipGetLastError();
}

hipError_t launch_encode(const DevModel& m, const float* feats, int32_t S, float* z0,
                         hipStream_t st) {
  const int F = m.dims.feat_dim, Fh = m.dims.enc_hidden, D = m.dims.d;
  const int lds = (F + Fh + D + ENC_THREADS) * (int)sizeof(float);
  hipLaunchKernelGGL(encode_kernel, dim3(S), dim3(ENC_THREADS), lds, st, feats, m.enc_w1t, m.enc_b1,
                     m.enc_w2t, m.enc_b2, F, Fh, D, m.prec == WM_BF16 ? 1 : 0, z0);
  return hipGetLastError();
}

// ---- rollout loss ----------------------------------------------------------

namespace {

// Training kernels are instantiated for the dims whose step state fits the
// registers of one wavefront (d <= 256).
#define WM_FOR_TRAIN_DE(CALL)               \
  WM_CASE(WM_FP32, PF32, 64, 32, CALL)      \
  WM_CASE(WM_FP32, PF32, 256, 64, CALL)     \
  WM_CASE(WM_BF16, PBF16, 64, 32, CALL)     \
  WM_CASE(WM_BF16, PBF16, 256, 64, CALL)

TrainArgs train_args(const DevModel& m, const TrainIO& io) {
  TrainArgs a;
  a.w1 = m.trans_w1; a.w2 = m.trans_w2; a.w2t = m.trans_w2t; a.w1t = m.trans_w1t;
  a.tab = m.roll_tab; a.z0 = io.z0; a.perm = io.perm; a.types = io.types; a.params = io.params;
  a.lens = io.lens; a.off = io.off; a.row_src = io.row_src;
  a.X = io.X; a.A = io.A; a.G = io.G; a.P = io.P; a.SD = io.SD; a.DE = io.DE;
  a.wh = m.trans_wh; a.wht = m.trans_wht; a.V = io.V; a.SC = io.SC; a.DV = io.DV;
  a.dz0 = io.dz0; a.err = io.err; a.B = io.B; a.T_max = io.T_max;
  a.P_ = m.dims.n_params; a.K = m.dims.n_kinds; a.H = m.dims.trans_hidden;
  a.tab_bytes = m.roll_tab_bytes;
  return a;
}

template <class PR, int D, int E, int WAVES, bool NORM>
hipError_t launch_train_fwd_t(const DevModel& m, const TrainArgs& a, int blocks, hipStream_t st) {
  const int lds = m.roll_tab_bytes;
  auto kern = train_fwd_kernel<PR, D, E, WAVES, NORM>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e;
  }
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(64 * WAVES), lds, st, a);
  return hipGetLastError();
}

template <class PR, int NC, int W, bool NORM>
hipError_t launch_train_bwd_rows(const TrainArgs& a, int tiles, hipStream_t st) {
  using BG = BwdRowsGeom<PR, 256, 64, NC, W>;
  constexpr int lds = BG::LDS + (NORM ? 2 * W * 32 * 4 : 0);
  static_assert(lds <= 160 * 1024, "LDS");
  auto kern = train_bwd_rows_kernel<PR, 256, 64, NC, W, NORM>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e;
  }
  hipLaunchKernelGGL(kern, dim3(tiles), dim3(64 * W), lds, st, a);
  return hipGetLastError();
}

template <class PR, int D, int E, bool NORM>
hipError_t launch_train_bwd_t(const TrainArgs& a, int tiles, hipStream_t st) {
  const int waves = pick_waves(tiles);
  const int blocks = (tiles + waves - 1) / waves;
  if (waves == 4) hipLaunchKernelGGL((train_bwd_kernel<PR, D, E, 4, NORM>), dim3(blocks), dim3(256), 0, st, a);
  else if (waves == 2) hipLaunchKernelGGL((train_bwd_kernel<PR, D, E, 2, NORM>), dim3(blocks), dim3(128), 0, st, a);
  else hipLaunchKernelGGL((train_bwd_kernel<PR, D, E, 1, NORM>), dim3(blocks), dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace

bool have_train_kernels(int prec, int d, int e) {
#define WM_HAVE_T(PR, D, E) return true;
  WM_FOR_TRAIN_DE(WM_HAVE_T)
#undef WM_HAVE_T
  return false;
}

// Rollout arguments of the training forward (no z_T, no phi).
RollArgs train_roll_args(const DevModel& m, const TrainIO& io, bool norm) {
  RollArgs a{};
  a.w1 = m.trans_w1; a.w2 = m.trans_w2; a.wh = norm ? m.trans_wh : nullptr; a.tab = m.roll_tab; a.z0 = io.z0;
  a.perm = io.perm; a.types = io.types; a.params = io.params; a.lens = io.lens; a.zT = nullptr;
  a.err = io.err; a.B = io.B; a.T_max = io.T_max; a.P = m.dims.n_params; a.K = m.dims.n_kinds;
  a.H = m.dims.trans_hidden; a.tab_bytes = m.roll_tab_bytes;
  a.X = io.X; a.A = io.A; a.G = io.G; a.Pz = io.P; a.off = io.off; a.row_src = io.row_src;
  a.V = io.V; a.SC = io.SC;
  return a;
}

// Training forward in the row-owned form (one workgroup per tile; d = 256).
template <class PR, int NC, int W, bool NORM>
hipError_t launch_train_fwd_rows(const DevModel& m, const TrainIO& io, int tiles, hipStream_t st) {
  const RollArgs a = train_roll_args(m, io, NORM);
  using RG = RowsGeom<PR, 256, 64, NC, W>;
  const int lds = m.roll_tab_bytes + RG::GELU_BYTES + RG::X_BYTES + RG::XE_BYTES + (NORM ? W * 3 * 32 * 4 : 0);
  auto kern = rollout_rows_kernel<PR, 256, 64, NC, W, NORM, true>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e;
  }
  hipLaunchKernelGGL(kern, dim3(tiles), dim3(64 * W), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_train_fwd(const DevModel& m, const TrainIO& io, hipStream_t st) {
  if (io.B == 0) return hipSuccess;
  const TrainArgs a = train_args(m, io);
  const int tiles = (io.B + 31) / 32;
  const bool norm = m.dims.norm == WM_NORM_L2;
  // both transition forms, up to NARROW_MAX_TILES = 512 tiles of 16 candidates
  // (two per compute unit): narrow tiles
  const int ntiles = (io.B + 15) / 16;
  if (m.dims.d == 256 && m.dims.embed_dim == 64 && m.trans_n && m.trans_nt && ntiles <= NARROW_MAX_TILES) {
    const int NC = m.dims.trans_hidden / 32;
    const RollArgs r = train_roll_args(m, io, norm);
    if (norm) {
      if (m.prec == WM_BF16 && NC == 16) return launch_rollout_narrow<NarrowBF16, 16, true, true>(m, r, ntiles, st);
      if (m.prec == WM_BF16 && NC == 32) return launch_rollout_narrow<NarrowBF16, 32, true, true>(m, r, ntiles, st);
      if (m.prec == WM_FP32 && NC == 16) return launch_rollout_narrow<NarrowF32, 16, true, true>(m, r, ntiles, st);
    } else {
      if (m.prec == WM_BF16 && NC == 16) return launch_rollout_narrow<NarrowBF16, 16, false, true>(m, r, ntiles, st);
      if (m.prec == WM_BF16 && NC == 32) return launch_rollout_narrow<NarrowBF16, 32, false, true>(m, r, ntiles, st);
      if (m.prec == WM_FP32 && NC == 16) return launch_rollout_narrow<NarrowF32, 16, false, true>(m, r, ntiles, st);
    }
  }
  if (m.dims.d == 64 && m.dims.embed_dim == 32 && m.dims.trans_hidden == 128 && m.trans_n && m.trans_nt &&
      ntiles <= NARROW_MAX_TILES) {
    const RollArgs r = train_roll_args(m, io, norm);
    if (m.prec == WM_BF16)
      return norm ? launch_rollout_narrow<NarrowBF16, 4, true, true, false, 64, 32, 2>(m, r, ntiles, st)
                  : launch_rollout_narrow<NarrowBF16, 4, false, true, false, 64, 32, 2>(m, r, ntiles, st);
    return norm ? launch_rollout_narrow<NarrowF32, 4, true, true, false, 64, 32, 2>(m, r, ntiles, st)
                : launch_rollout_narrow<NarrowF32, 4, false, true, false, 64, 32, 2>(m, r, ntiles, st);
  }
  if (m.dims.d == 256 && m.dims.embed_dim == 64) {
    const int NC = m.dims.trans_hidden / 32;
#define WM_TFWD_ROWS(N)                                                                              \
    if (m.prec == WM_BF16 && NC == 16) return launch_train_fwd_rows<PBF16, 16, 8, N>(m, io, tiles, st); \
    if (m.prec == WM_BF16 && NC == 32) return launch_train_fwd_rows<PBF16, 32, 8, N>(m, io, tiles, st); \
    if (m.prec == WM_FP32 && NC == 16) return launch_train_fwd_rows<PF32, 16, 4, N>(m, io, tiles, st);
    if (norm) { WM_TFWD_ROWS(true) } else { WM_TFWD_ROWS(false) }
#undef WM_TFWD_ROWS
  }
  const int waves = pick_waves(tiles);
  const int blocks = (tiles + waves - 1) / waves;
  const int prec = m.prec, d = m.dims.d, e = m.dims.embed_dim;
#define WM_TFWD(PR, D, E)                                                                      \
  if (norm) return waves == 4 ? launch_train_fwd_t<PR, D, E, 4, true>(m, a, blocks, st)          \
                 : waves == 2 ? launch_train_fwd_t<PR, D, E, 2, true>(m, a, blocks, st)          \
                              : launch_train_fwd_t<PR, D, E, 1, true>(m, a, blocks, st);         \
  return waves == 4 ? launch_train_fwd_t<PR, D, E, 4, false>(m, a, blocks, st)                   \
       : waves == 2 ? launch_train_fwd_t<PR, D, E, 2, false>(m, a, blocks, st)                   \
                    : launch_train_fwd_t<PR, D, E, 1, false>(m, a, blocks, st);
  WM_FOR_TRAIN_DE(WM_TFWD)
#undef WM_TFWD
  return hipErrorInvalidValue;
}

template <class NP, int NC, bool NORM, int D = 256, int E = 64, int W = 8>
hipError_t launch_train_bwd_narrow(const DevModel& m, TrainArgs a, int tiles, hipStream_t st) {
  using BG = NarrowBwdGeom<NP, D, E, NC, W>;
  constexpr int lds = BG::LDS + (NORM ? BG::DOTS_BYTES : 0);
  static_assert(lds <= 160 * 1024, "LDS");
  a.w2t = m.trans_nt;
  // paper form: the transposed normal map follows W1^T in the blob
  a.wht = NORM ? m.trans_nt + Narrow::t_bytes(D, E, NC * 32, NP::GPK) : nullptr;
  auto kern = train_bwd_narrow_kernel<NP, D, E, NC, W, NORM>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e;
  }
  hipLaunchKernelGGL(kern, dim3(tiles), dim3(64 * W), lds, st, a);
  return hipGetLastError();
}

hipError_t launch_train_bwd(const DevModel& m, const TrainIO& io, hipStream_t st) {
  if (io.B == 0) return hipSuccess;
  const TrainArgs a = train_args(m, io);
  const int tiles = (io.B + 31) / 32;
  const bool norm = m.dims.norm == WM_NORM_L2;
  // both transition forms, up to NARROW_MAX_TILES = 512 tiles of 16 candidates
  // (two per compute unit): narrow tiles
  const int ntiles = (io.B + 15) / 16;
  if (m.dims.d == 256 && m.dims.embed_dim == 64 && m.trans_nt && ntiles <= NARROW_MAX_TILES) {
    const int NC = m.dims.trans_hidden / 32;
    if (norm) {
      if (m.prec == WM_BF16 && NC == 16) return launch_train_bwd_narrow<NarrowBF16, 16, true>(m, a, ntiles, st);
      if (m.prec == WM_BF16 && NC == 32) return launch_train_bwd_narrow<NarrowBF16, 32, true>(m, a, ntiles, st);
      if (m.prec == WM_FP32 && NC == 16) return launch_train_bwd_narrow<NarrowF32, 16, true>(m, a, ntiles, st);
    } else {
      if (m.prec == WM_BF16 && NC == 16) return launch_train_bwd_narrow<NarrowBF16, 16, false>(m, a, ntiles, st);
      if (m.prec == WM_BF16 && NC == 32) return launch_train_bwd_narrow<NarrowBF16, 32, false>(m, a, ntiles, st);
      if (m.prec == WM_FP32 && NC == 16) return launch_train_bwd_narrow<NarrowF32, 16, false>(m, a, ntiles, st);
    }
  }
  if (m.dims.d == 64 && m.dims.embed_dim == 32 && m.dims.trans_hidden == 128 && m.trans_nt &&
      ntiles <= NARROW_MAX_TILES) {
    if (m.prec == WM_BF16)
      return norm ? launch_train_bwd_narrow<NarrowBF16, 4, true, 64, 32, 2>(m, a, ntiles, st)
                  : launch_train_bwd_narrow<NarrowBF16, 4, false, 64, 32, 2>(m, a, ntiles, st);
    return norm ? launch_train_bwd_narrow<NarrowF32, 4, true, 64, 32, 2>(m, a, ntiles, st)
                : launch_train_bwd_narrow<NarrowF32, 4, false, 64, 32, 2>(m, a, ntiles, st);
  }
  if (m.dims.d == 256 && m.dims.embed_dim == 64) {
    const int NC = m.dims.trans_hidden / 32;
#define WM_TBWD_ROWS(N)                                                                         \
    if (m.prec == WM_BF16 && NC == 16) return launch_train_bwd_rows<PBF16, 16, 8, N>(a, tiles, st); \
    if (m.prec == WM_BF16 && NC == 32) return launch_train_bwd_rows<PBF16, 32, 8, N>(a, tiles, st); \
    if (m.prec == WM_FP32 && NC == 16) return launch_train_bwd_rows<PF32, 16, 4, N>(a, tiles, st);
    if (norm) { WM_TBWD_ROWS(true) } else { WM_TBWD_ROWS(false) }
#undef WM_TBWD_ROWS
  }
  const int prec = m.prec, d = m.dims.d, e = m.dims.embed_dim;
#define WM_TBWD(PR, D, E) \
  return norm ? launch_train_bwd_t<PR, D, E, true>(a, tiles, st) : launch_train_bwd_t<PR, D, E, false>(a, tiles, st);
  WM_FOR_TRAIN_DE(WM_TBWD)
#undef WM_TBWD
  return hipErrorInvalidValue;
}

hipError_t launch_row_offsets(const int32_t* lens, int B, int T_max, int32_t* off, hipStream_t st) {
  hipLaunchKernelGGL(row_offsets_kernel, dim3(1), dim3(1024), 0, st, lens, B, T_max, off);
  return hipGetLastError();
}

hipError_t launch_step_loss(const float* P, const float* targets, const float* negatives, int NN,
                            const int32_t* lens, const int32_t* off, int B, int T_max, int D,
                            float lam, float gamma, float* SD, float* lrow, float* loss,
                            float* total, hipStream_t st) {
  const long long slots = (long long)B * T_max;
  if (slots > 0)
    hipLaunchKernelGGL(loss_kernel, dim3((unsigned)((slots + 3) / 4)), dim3(256), 0, st, P, targets,
                       negatives, NN, lens, off, B, T_max, D, lam, gamma, SD, lrow);
  if (B > 0)
    hipLaunchKernelGGL(loss_sum_kernel, dim3((B + 255) / 256), dim3(256), 0, st, lrow, off, B, loss);
  if (total) hipLaunchKernelGGL(loss_total_kernel, dim3(1), dim3(1024), 0, st, loss, B, total);
  return hipGetLastError();
}

hipError_t launch_weight_grads(const DevModel& m, const TrainIO& io, const GradParts& g,
                               float* gw1, float* gb1, float* gw2, float* gb2, float* gtemb,
                               float* gpw, float* gpb, float* gwh, hipStream_t st) {
  const int D = m.dims.d, E = m.dims.embed_dim, H = m.dims.trans_hidden, IN = D + E;
  const int K = m.dims.n_kinds, P = m.dims.n_params, W = K * E + E * P + E;
  const int S = g.splits;
  WgradArgs a;
  auto prob = [](const float* A, int M, int lda, const float* Bm, int N, int ldb, float* part,
                 float* colsum) {
    WgradProblem p;
    p.A = A; p.Bm = Bm; p.part = part; p.colsum = colsum; p.M = M; p.N = N; p.lda = lda; p.ldb = ldb;
    p.tiles_n = (N + WG_T - 1) / WG_T;
    p.tiles = ((M + WG_T - 1) / WG_T) * p.tiles_n;
    return p;
  };
  a.p0 = prob(io.SD, D, D, io.G, H, H, g.w2, g.b2);         // dW2 [D][H], db2
  a.p1 = prob(io.A, H, H, io.X, IN, IN, g.w1, g.b1);        // dW1 [H][IN], db1
  a.p2 = gwh ? prob(io.DV, D, D, io.X + D, E, IN, g.wh, nullptr)   // dWh [D][E] = sum R(dv) R(e)^T
             : WgradProblem{};
  a.off = io.off; a.B = io.B; a.splits = S;
  const dim3 grid((a.p0.tiles + a.p1.tiles + a.p2.tiles) * ((S + 7) / 8) * 8);
  if (m.prec == WM_BF16) hipLaunchKernelGGL(wgrad_kernel<PBF16>, grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL(wgrad_kernel<PF32>, grid, dim3(256), 0, st, a);
  if (E > EMB_THREADS || EMB_THREADS % E) return hipErrorInvalidValue;
  const int lds = (EMB_THREADS / E) * (K + P + 1) * E * (int)sizeof(float);
  hipError_t e = hipFuncSetAttribute((const void*)emb_grad_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return e;
  }
  hipLaunchKernelGGL(emb_grad_kernel, dim3(g.emb_blocks), dim3(EMB_THREADS), lds, st, io.DE, E,
                     io.row_src, io.types, io.params, K, P, io.off, io.B, g.emb_blocks, g.emb);
  SumJobs jb{};
  auto job = [&](const float* part, int splits, long long stride, long long n, float* out) {
    const int j = jb.count++;
    jb.part[j] = part; jb.out[j] = out; jb.stride[j] = stride; jb.splits[j] = splits;
    jb.start[j + 1] = jb.start[j] + n;
  };
  job(g.w1, S, (long long)H * IN, (long long)H * IN, gw1);
  job(g.w2, S, (long long)D * H, (long long)D * H, gw2);
  if (gwh) job(g.wh, S, (long long)D * E, (long long)D * E, gwh);
  job(g.b1, S, H, H, gb1);
  job(g.b2, S, D, D, gb2);
  job(g.emb, g.emb_blocks, (long long)W, (long long)K * E, gtemb);
  job(g.emb + (size_t)K * E, g.emb_blocks, (long long)W, (long long)E * P, gpw);
  job(g.emb + (size_t)K * E + (size_t)E * P, g.emb_blocks, (long long)W, E, gpb);
  const long long total = jb.start[jb.count];
  hipLaunchKernelGGL(sum_jobs_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, jb);
  return hipGetLastError();
}

}  // namespace wm
