// Internal declarations shared by the C-ABI layer (wm_api.hip) and the
// kernels (wm_kernels.hip).  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "../../include/wm.h"
#include "wm_layout.h"

namespace wm {

// Launchers (wm_kernels.hip).  Return hipSuccess or the launch error.
// zero n int32 words (a kernel rather than hipMemsetAsync, so the call is
// safe under stream capture)
hipError_t launch_clear_words(int32_t* p, int n, hipStream_t st);
// hist: bucket_groups(B) * (T_max + 1) ints of workspace (unused when 0)
hipError_t launch_bucket(const int32_t* lens, int32_t B, int32_t T_max, const SegTable& seg,
                         int2* perm, int32_t* hist, int32_t* err, hipStream_t st);
// Scores requested with a rollout (wm_evaluate): the narrow kernel computes
// them itself when it runs and sets `done`; otherwise launch_score does.
struct ScoreFuse {
  const float* hw;
  int32_t n_hw;
  float* scores;
  bool done;
};
// phi (may be null): the kernel families that can also sum the action
// features write them and set *phi_done; otherwise launch_phi computes them.
hipError_t launch_rollout(const DevModel& m, const float* z0, const int2* perm,
                          const int32_t* types, const int32_t* params, const int32_t* lens,
                          int32_t B, int32_t T_max, float* zT, float* phi, bool* phi_done,
                          int32_t* err, hipStream_t st, ScoreFuse* sf = nullptr);
hipError_t launch_phi(const DevModel& m, const int32_t* types, const int32_t* params,
                      const int32_t* lens, int32_t B, int32_t T_max, float* phi, hipStream_t st);
hipError_t launch_score(const DevModel& m, const float* zT, const float* phi, int32_t B,
                        const float* hw, int32_t n_hw, float* scores, hipStream_t st);
hipError_t launch_topk(const float* scores, int32_t n_hw, int32_t B, const SegTable& seg,
                       int32_t k, int32_t* idx, float* val, hipStream_t st);
hipError_t launch_encode(const DevModel& m, const float* feats, int32_t S, float* z0,
                         hipStream_t st);

hipError_t launch_phi_struct(const int32_t* types, const int32_t* params, const int32_t* lens,
                             int32_t B, int32_t T_max, int32_t K, int32_t P, float* phi_s,
                             hipStream_t st);
hipError_t launch_score_trees(const DevForest& f, const float* zT, int32_t d, const float* phi_s,
                              int32_t phi_dim, int32_t B, const float* hw, int32_t n_hw,
                              int32_t hw_dim, float* scores, hipStream_t st);

// Rollout loss (training objective of the transition): device buffers of
// one call.  Step activations are compact rows r = off[i] + t (see the
// kernels for their contents); their arrays are sized for B * T_max rows.
struct TrainIO {
  const float* z0;          // [S][D]
  const int2* perm;         // length-sorted (candidate, subgraph)
  const int32_t* types;
  const int32_t* params;
  const int32_t* lens;
  int32_t* off;             // [B+1] row offsets (written by launch_row_offsets)
  int32_t* row_src;         // [rows] i * T_max + t of each row
  float *X, *A, *G, *P, *SD, *DE;
  float *V, *SC, *DV;       // paper form: Wh e [rows][D], (v.z, v.v, |u|, 0) [rows][4], dL/dv [rows][D]
  float* dz0;               // [B][D] or null
  int32_t* err;
  int B, T_max;
};
// Weight-gradient partial sums of `splits` equal shares of the rows, added
// in order afterwards.
struct GradParts {
  float *w1, *w2, *b1, *b2, *emb, *wh;
  int splits, emb_blocks;
};
bool have_train_kernels(int prec, int d, int e);
hipError_t launch_row_offsets(const int32_t* lens, int B, int T_max, int32_t* off, hipStream_t st);
hipError_t launch_train_fwd(const DevModel& m, const TrainIO& io, hipStream_t st);
hipError_t launch_step_loss(const float* P, const float* targets, const float* negatives, int NN,
                            const int32_t* lens, const int32_t* off, int B, int T_max, int D,
                            float lam, float gamma, float* SD, float* lrow, float* loss,
                            float* total, hipStream_t st);
hipError_t launch_train_bwd(const DevModel& m, const TrainIO& io, hipStream_t st);
hipError_t launch_weight_grads(const DevModel& m, const TrainIO& io, const GradParts& parts,
                               float* gw1, float* gb1, float* gw2, float* gb2, float* gtemb,
                               float* gpw, float* gpb, float* gwh, hipStream_t st);

// Whether a (precision, d, e) combination has rollout/score kernels.
bool have_kernels(int prec, int d, int e);
// LDS bytes the rollout kernel needs for a model (0 if unsupported).
int rollout_lds_bytes(const DevModel& m);

// Kernel-family timing hooks (wm_api.hip).
enum TimedKernel { TK_ROLLOUT = 0, TK_SCORE = 1, TK_TOPK = 2, TK_BUCKET = 3, TK_PHI = 4, TK_ENCODE = 5,
                   TK_PHI_STRUCT = 6, TK_TREES = 7, TK_TRAIN_FWD = 8, TK_LOSS = 9,
                   TK_TRAIN_BWD = 10, TK_GRADS = 11, TK_TEXT_GEMM = 12, TK_TEXT_ATTN = 13,
                   TK_TEXT_OTHER = 14, TK_COUNT = 15 };
void timing_begin(int kernel, hipStream_t st);
void timing_end(int kernel, hipStream_t st);

// Thread-local last-error message of the C ABI (wm_api.hip).
wm_status set_error(wm_status st, const std::string& msg);
wm_status clear_error();

}  // namespace wm
