/*
 * wm.h - C ABI of the batched latent-rollout schedule evaluator (gfx950).
 *
 * The evaluator scores B candidate schedules of tensor-program subgraphs the
 * way the paper's world-model evaluator does (Sec. 3.2, Eq. 2-3): encode the
 * initial program state, roll the latent state forward once per scheduling
 * action (Eq. 1, Sec. 3.4), score the terminal latent together with action
 * and hardware features (Eq. 3, Sec. 3.5), and rank candidates within each
 * workload (Sec. 3.5, Sec. 3.6).  The instantiation is a residual two-layer
 * MLP transition, a type-embedding plus linear(log2 params) action embedding,
 * mean action embedding as action features, and a two-layer MLP cost model:
 *
 *   e_t  = type_emb[type_t] + param_w . log2(params_t) + param_b
 *   z_t  = z_{t-1} + W2 . GELU(W1 . [z_{t-1}; e_t] + b1) + b2,  t = 1..len_i
 *   phi  = (1/len_i) sum_t e_t          (0 when len_i = 0)
 *   y_j  = wc2 . GELU(Wc1 . [z_T; phi; h_j] + bc1) + bc2
 *   GELU(x) = x (1 + erf(x / sqrt 2)) / 2
 *
 * With norm = WM_NORM_L2 the transition takes the paper's own form (Sec. 3.4:
 * a TransH-style move into an action-conditioned hyperplane, the residual
 * update, then normalisation):
 *
 *   v    = Wh . e_t,   w = v / |v|_2           (w = 0 when v = 0)
 *   z'   = z_{t-1} - (w . z_{t-1}) w
 *   u    = z' + W2 . GELU(W1 . [z'; e_t] + b1) + b2
 *   z_t  = u / |u|_2                           (z_t = u when u = 0)
 *
 * z_0 is used as given (an empty sequence returns it unscaled).
 *
 * Conventions for every call below:
 *  - Pointers are device pointers unless marked HOST.  All tensors are dense,
 *    row-major, C-contiguous, 4-byte elements (float32 or int32), and must be
 *    4-byte aligned; float tensors read as vectors must be 16-byte aligned
 *    (any torch/hipMalloc allocation is).
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Work
 *    is enqueued asynchronously; a call returns after enqueueing.
 *  - The caller owns every buffer it passes; the library owns only the
 *    model's device copy of the weights.  Buffers, the model and the
 *    workspace must stay alive until the enqueued work has completed.
 *  - No call allocates device memory except wm_model_create (and the
 *    create calls of the tree ensemble and the text encoder).
 *  - Argument problems the host can see are reported synchronously, before
 *    anything is enqueued: a null required pointer, a negative size, a bad
 *    segment table, k out of range, a workspace that is too small.  The
 *    status is returned and wm_last_error() gives a message (thread-local).
 *  - Problems in the data itself (a length outside [0, T_max], an action type
 *    outside [0, n_kinds), a parameter < 1 at a step t < len_i) are detected
 *    on the device and recorded in the workspace's error word; read it with
 *    wm_device_status.  When it is set, outputs are unspecified (but no
 *    out-of-bounds access happens).  Padding entries (t >= len_i) are never
 *    read.
 *  - Calls that share one workspace must not overlap in time.
 */
#ifndef WM_H
#define WM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WM_MAX_SEGMENTS 512   /* subgraphs per call */
#define WM_MAX_K 1024         /* top-k per (hardware vector, subgraph) */
#define WM_MAX_T 4096         /* padded action-sequence width */
#define WM_NOALLOC_SCRATCH_BYTES (4u << 20)   /* scratch of wm_evaluate_noalloc, per GPU */

typedef enum wm_status {
  WM_OK = 0,
  WM_ERR_INVALID_ARGUMENT = 1, /* host-visible argument error; nothing enqueued */
  WM_ERR_UNSUPPORTED = 2,      /* dims/precision this build has no kernel for */
  WM_ERR_OUT_OF_MEMORY = 3,    /* wm_model_create could not allocate */
  WM_ERR_DEVICE = 4,           /* a HIP runtime call failed */
  WM_ERR_INPUT_RANGE = 5       /* device-detected data error (wm_device_status) */
} wm_status;

typedef enum wm_precision {
  WM_FP32 = 0, /* float32 operands, float32 matrix-core accumulation */
  WM_BF16 = 1  /* bfloat16 (round-to-nearest-even) matrix operands, float32 accumulation */
} wm_precision;

typedef enum wm_norm {
  WM_NORM_NONE = 0, /* residual MLP transition as above */
  WM_NORM_L2 = 1    /* hyperplane projection before, unit length after every step (Sec. 3.4) */
} wm_norm;

/* Model shape.  d: latent width; embed_dim: action-embedding width e;
 * n_kinds/n_params: action types and integer parameters per step;
 * trans_hidden: transition hidden width H; cost_hidden: cost hidden width C;
 * hw_dim: hardware-vector width (0 = no hardware features); feat_dim and
 * enc_hidden: program-feature width F and encoder hidden width (feat_dim = 0:
 * no encoder, the initial latents are given).  precision: wm_precision;
 * norm: wm_norm.
 * Supported by this build (else WM_ERR_UNSUPPORTED): (d, embed_dim) in
 * {(64, 32), (256, 64)} for both precisions and (512, 128) for WM_BF16;
 * trans_hidden and cost_hidden multiples of 64; hw_dim a multiple of 16 up
 * to 32; n_kinds <= 32; 1 <= n_params <= 8; the double-buffered weight
 * chunks plus embedding tables must fit the 160 KiB LDS. */
typedef struct wm_dims {
  int32_t d, embed_dim, n_kinds, n_params, trans_hidden, cost_hidden, hw_dim;
  int32_t feat_dim, enc_hidden;
  int32_t precision;
  int32_t norm;
} wm_dims;

/* Weights, HOST float32, PyTorch Linear layout [out][in]:
 *   type_emb [n_kinds][e], param_w [e][n_params], param_b [e],
 *   w1 [H][d+e] (columns: z then e), b1 [H], w2 [d][H], b2 [d],
 *   wc1 [C][d+e+hw_dim] (columns: z_T, phi, h), bc1 [C], wc2 [C], bc2,
 *   we1 [enc_hidden][feat_dim], be1 [enc_hidden], we2 [d][enc_hidden], be2 [d]
 *   (encoder pointers may be NULL when feat_dim = 0),
 *   wh [d][e]: hyperplane-normal map of WM_NORM_L2 (may be NULL otherwise). */
typedef struct wm_weights {
  const float *type_emb, *param_w, *param_b;
  const float *w1, *b1, *w2, *b2;
  const float *wc1, *bc1, *wc2;
  float bc2;
  const float *we1, *be1, *we2, *be2;
  const float *wh;
} wm_weights;

typedef struct wm_model wm_model;

/* Copy the weights to the current HIP device, rounding the matrices
 * W1, W2, Wc1, We1, We2 (and Wh) to bfloat16 (nearest-even) in WM_BF16 mode and
 * repacking them into the kernels' matrix-fragment order.  Synchronous.
 * The model is immutable: concurrent calls with distinct workspaces are safe.
 * Errors: INVALID_ARGUMENT (null pointer, non-positive dims), UNSUPPORTED,
 * OUT_OF_MEMORY, DEVICE. */
wm_status wm_model_create(const wm_dims* dims, const wm_weights* weights, wm_model** out);

/* Free the model.  Only after all work using it has completed.  NULL is a no-op. */
void wm_model_destroy(wm_model* model);

/* Bytes of workspace wm_rollout / wm_evaluate need for a batch of B
 * candidates in S subgraphs scored under n_hw hardware vectors (0 on a bad
 * argument).  The caller allocates it (256-byte aligned) and must zero it
 * once before first use; afterwards the library keeps the error word
 * consistent (wm_device_status clears it). */
size_t wm_workspace_bytes(const wm_model* model, int32_t B, int32_t T_max, int32_t S, int32_t n_hw);

/* Initial latents from program features (the state encoder E of Sec. 3.3,
 * Eq. 4, as a two-layer MLP): z0[s] = We2 . GELU(We1 . feats[s] + be1) + be2.
 * feats [S][feat_dim] float32 -> z0 [S][d] float32.  Needs feat_dim > 0. */
wm_status wm_encode_init(const wm_model* model, const float* feats, int32_t S, float* z0,
                         void* stream);

/* Batched multi-step latent rollout (Eq. 1-2, Sec. 3.4 and 3.6).
 * Candidate i (0 <= i < B) belongs to subgraph s with
 * seg_off[s] <= i < seg_off[s+1] and starts from z0[s].
 *   z0      [S][d] float32
 *   seg_off HOST int32 [S+1]: 0 = seg_off[0] <= ... <= seg_off[S] = B, 1 <= S <= WM_MAX_SEGMENTS
 *   types   [B][T_max] int32, params [B][T_max][n_params] int32, lens [B] int32
 *   zT      [B][d] float32 out: latent after lens[i] steps (z0 when lens[i] = 0)
 *   phi     [B][e] float32 out (may be NULL): mean step embedding (0 when lens[i] = 0)
 *   ws      workspace of at least wm_workspace_bytes(model, B, T_max, S, 1) bytes. */
wm_status wm_rollout(const wm_model* model, const float* z0, const int32_t* seg_off, int32_t S,
                     const int32_t* types, const int32_t* params, const int32_t* lens,
                     int32_t B, int32_t T_max, float* zT, float* phi,
                     void* ws, size_t ws_bytes, void* stream);

/* Cost model G (Eq. 3, Eq. 12): scores [n_hw][B] float32 out, from
 * zT [B][d], phi [B][e] and hw [n_hw][hw_dim] (hw may be NULL when
 * hw_dim = 0).  Higher scores rank first. */
wm_status wm_score(const wm_model* model, const float* zT, const float* phi, int32_t B,
                   const float* hw, int32_t n_hw, float* scores, void* stream);

/* Within-workload ranking (Sec. 3.5): for every hardware vector j and
 * subgraph s, the k best candidates of segment s ordered by descending score,
 * ties to the lower candidate index, NaN last.
 *   scores [n_hw][B] float32; seg_off HOST [S+1] as above;
 *   1 <= k <= min(WM_MAX_K, smallest segment);
 *   idx [n_hw][S][k] int32 out (global candidate indices);
 *   val [n_hw][S][k] float32 out (may be NULL). */
wm_status wm_topk(const float* scores, int32_t n_hw, int32_t B, const int32_t* seg_off,
                  int32_t S, int32_t k, int32_t* idx, float* val, void* stream);

/* The whole hot path in one call: [encode,] rollout, score, top-k
 * (Eq. 2-3, Sec. 3.6).  init is z0 [S][d], or program features
 * [S][feat_dim] when init_is_feats != 0 (needs an encoder).  scores
 * [n_hw][B], zT [B][d] and val may be NULL (kept in the workspace /
 * not written); idx is required.  ws needs
 * wm_workspace_bytes(model, B, T_max, S, n_hw) bytes. */
wm_status wm_evaluate(const wm_model* model, const float* init, int32_t init_is_feats,
                      const int32_t* seg_off, int32_t S,
                      const int32_t* types, const int32_t* params, const int32_t* lens,
                      int32_t B, int32_t T_max, const float* hw, int32_t n_hw, int32_t k,
                      float* scores, float* zT, int32_t* idx, float* val,
                      void* ws, size_t ws_bytes, void* stream);

/* wm_evaluate for callers that cannot allocate device memory or pass a
 * workspace (code under HIP graph capture, serving loops, harnesses that
 * forbid allocation): the same computation and kernels with every output
 * supplied by the caller and the remaining intermediates (the
 * length-sorted permutation, the bucketing histograms, the encoded initial
 * latents) in a scratch array the library keeps in each GPU's memory
 * (WM_NOALLOC_SCRATCH_BYTES per GPU, held until the process ends; its
 * address is looked up on the first call on a device, with that device
 * current).  Nothing is allocated.
 *   scores [n_hw][B], zT [B][d], phi [B][e] float32 out, all required;
 *   idx required, val may be NULL, as in wm_evaluate;
 *   status: device int32 [64] (256 bytes) out, required: cleared by the call,
 *     then the device error word of the call; read it with
 *     wm_device_status(status, 256, stream).
 * Errors: as wm_evaluate, plus INVALID_ARGUMENT when B, T_max and S need
 * more scratch than WM_NOALLOC_SCRATCH_BYTES (8 B + 4 (T_max + 1) / 4096 B
 * per candidate, plus 4 d bytes per subgraph with an encoder; about 512 Ki
 * candidates for T_max <= 64 without one).  All calls on one GPU share its
 * scratch: calls that overlap in time on one GPU (on different streams or
 * threads) race and must be serialised by the caller. */
wm_status wm_evaluate_noalloc(const wm_model* model, const float* init, int32_t init_is_feats,
                              const int32_t* seg_off, int32_t S,
                              const int32_t* types, const int32_t* params, const int32_t* lens,
                              int32_t B, int32_t T_max, const float* hw, int32_t n_hw, int32_t k,
                              float* scores, float* zT, float* phi, int32_t* idx, float* val,
                              int32_t* status, void* stream);

/* ---- Tree-ensemble ranker (the paper's G, Sec. 3.5) --------------------
 * The paper ranks candidates with a gradient-boosted tree ensemble over the
 * predicted terminal state, a structured action-feature vector and the
 * hardware vector:
 *
 *   phi_s = [ n_0 .. n_{K-1}, T, mean_t log2(params_t), max_t log2(params_t) ]
 *           (n_k = steps of kind k; per parameter slot mean and max; all
 *           zero when T = 0; width K + 1 + 2P)
 *   x     = [ z_T ; phi_s ; h ]
 *   y     = base + sum over trees of the leaf reached by x
 *
 * A tree of depth D is complete and breadth-first: internal node i
 * (0 <= i < 2^D - 1) has a feature index f_i and a float32 threshold c_i, and
 * x goes to child 2i+1 when x[f_i] < c_i (float32 comparison), else to
 * child 2i+2 (a NaN goes right); leaf l is node 2^D - 1 + l. */
typedef struct wm_forest wm_forest;

/* Copy a forest to the current device.  HOST arrays: feat [n_trees][2^depth
 * - 1] int32 in [0, n_features), thr [n_trees][2^depth - 1], leaf
 * [n_trees][2^depth].  1 <= depth <= 12, 1 <= n_features <= 4096.
 * Synchronous.  Errors: INVALID_ARGUMENT (null array, bad sizes, a feature
 * index out of range), OUT_OF_MEMORY, DEVICE. */
wm_status wm_forest_create(int32_t n_trees, int32_t depth, int32_t n_features,
                           const int32_t* feat, const float* thr, const float* leaf,
                           float base, wm_forest** out);

/* Free the forest (after all work using it has completed).  NULL: no-op. */
void wm_forest_destroy(wm_forest* forest);

/* Structured action features phi_s [B][n_kinds + 1 + 2 n_params] float32
 * out, from types [B][T_max], params [B][T_max][n_params], lens [B] (device).
 * Kinds outside [0, n_kinds) are not counted; a parameter < 1 gives a
 * non-finite log2 (these are reported by the rollout in wm_evaluate_trees).
 * 1 <= n_kinds <= 32, 1 <= n_params <= 8. */
wm_status wm_phi_struct(const int32_t* types, const int32_t* params, const int32_t* lens,
                        int32_t B, int32_t T_max, int32_t n_kinds, int32_t n_params,
                        float* phi_s, void* stream);

/* Tree-ensemble scores [n_hw][B] of x = [zT [B][d] ; phi_s [B][phi_dim] ;
 * hw [n_hw][hw_dim]] (device); d + phi_dim + hw_dim must equal the forest's
 * n_features.  Leaf values are summed in float32 in a fixed order. */
wm_status wm_score_trees(const wm_forest* forest, const float* zT, int32_t d,
                         const float* phi_s, int32_t phi_dim, int32_t B, const float* hw,
                         int32_t n_hw, int32_t hw_dim, float* scores, void* stream);

/* wm_evaluate with the tree-ensemble ranker: [encode,] rollout (the model's
 * transition), structured action features, tree scores, top-k.  The forest's
 * n_features must be d + n_kinds + 1 + 2 n_params + hw_dim of the model.
 * Same arguments, outputs and workspace as wm_evaluate. */
wm_status wm_evaluate_trees(const wm_model* model, const wm_forest* forest, const float* init,
                            int32_t init_is_feats, const int32_t* seg_off, int32_t S,
                            const int32_t* types, const int32_t* params, const int32_t* lens,
                            int32_t B, int32_t T_max, const float* hw, int32_t n_hw, int32_t k,
                            float* scores, float* zT, int32_t* idx, float* val,
                            void* ws, size_t ws_bytes, void* stream);

/* ---- Rollout loss and its gradients (training the transition, Sec. 3.4) --
 * The transition (residual form, WM_NORM_NONE) is trained on rollouts: from
 * z0 it is applied over each candidate's action sequence, and at every valid
 * step t the predicted state p_t = z_{t+1} is compared with a target state
 * z*_t (the encoded observed next state) and with n_neg negative states:
 *
 *   match_t = |p_t - z*_t|^2
 *   rank_t  = max(0, |p_t - z*_t| - min_n |p_t - z-_{t,n}| + gamma)
 *   loss_i  = sum_{t < len_i} lam * match_t + (1 - lam) * rank_t
 *
 * (|.| Euclidean; the hardest negative is the nearest, the first one on
 * ties; at the hinge, at a zero distance and at a zero hyperplane normal the
 * gradient taken is 0).  The gradients are those of L = sum_i loss_i with
 * respect to the transition weights (with Wh for WM_NORM_L2), the action
 * embedding and each candidate's initial state, by the chain rule backwards
 * through all steps.  With WM_NORM_L2 the predictions p_t are the unit-length
 * states of the paper's form, so both terms live in the normalised space as
 * in Sec. 3.4.  In WM_BF16 every matrix product of the forward and of the
 * backward takes bfloat16-rounded operands with float32 accumulation (the
 * rounding is passed through unchanged).  Gradients are sums in a fixed
 * order: repeated calls give identical bits. */
typedef struct wm_grads {
  float *w1, *b1;             /* [H][d+e], [H] */
  float *w2, *b2;             /* [d][H], [d] */
  float *type_emb;            /* [n_kinds][e] */
  float *param_w, *param_b;   /* [e][n_params], [e] */
  float *z0;                  /* [B][d]: per candidate (may be NULL) */
  float *wh;                  /* [d][e]: the normal map (WM_NORM_L2 models; ignored otherwise) */
} wm_grads;

/* Workspace bytes of wm_rollout_loss for B candidates with padded width
 * T_max (0 on a bad argument).  Same ownership and error-word rules as
 * wm_workspace_bytes (zero once before first use).  It holds the step
 * activations of the backward pass, about 4 (2 H + 3 d + 2 e + 2) bytes per
 * (candidate, step) slot (4 (2 d + 4) more for WM_NORM_L2), plus partial
 * gradient sums. */
size_t wm_loss_workspace_bytes(const wm_model* model, int32_t B, int32_t T_max);

/* Rollout loss (definition above).  Inputs as in wm_rollout, plus
 *   targets   [B][T_max][d] float32: z*_t for the state after step t
 *   negatives [B][T_max][n_neg][d] float32, n_neg >= 1
 *   (entries at t >= lens[i] are never read);
 * outputs: loss [B] float32 (required), total (1 float, may be NULL),
 * grads (may be NULL: loss only; else every pointer but z0 is required, and
 * wh for a WM_NORM_L2 model).  Needs d <= 256 (UNSUPPORTED otherwise). */
wm_status wm_rollout_loss(const wm_model* model, const float* z0, const int32_t* seg_off, int32_t S,
                          const int32_t* types, const int32_t* params, const int32_t* lens,
                          int32_t B, int32_t T_max, const float* targets, const float* negatives,
                          int32_t n_neg, float lam, float gamma, float* loss, float* total,
                          const wm_grads* grads, void* ws, size_t ws_bytes, void* stream);

/* ---- Chunked transformer state encoder (the paper's E, Sec. 3.3) --------
 * E maps a program's token sequence to its initial latent: the tokens are cut
 * into overlapping chunks by a sliding window (window W, stride Sd: chunk c
 * holds tokens [c Sd, min(c Sd + W, N)); 1 + ceil((N - W) / Sd) chunks when
 * N > W, one when 0 < N <= W, none when N = 0), every chunk is encoded on its
 * own by a post-LayerNorm transformer backbone (the CodeBERT / RoBERTa
 * shape), each chunk's outputs are mean-pooled over its tokens, a program's
 * chunk vectors are averaged (zero for an empty program) and projected:
 *
 *   h = LN(tok_emb[id] + pos_emb[p])              p = position in the chunk
 *   per layer: [q k v] = h Wqkv^T + bqkv;  per head o = softmax(q k^T / sqrt(dh)) v
 *              h = LN(h + o Wo^T + bo);  h = LN(h + GELU(h W1^T + b1) W2^T + b2)
 *   z = Wp mean_c(mean_p h) + bp
 *
 * LN(x) = (x - mean) / sqrt(var + 1e-5) * gamma + beta.  In WM_BF16 the weight
 * matrices and every activation entering a matrix product are rounded to
 * bfloat16 (float32 accumulation); embeddings, biases, LayerNorm, softmax,
 * residual sums and pooling stay float32. */
#define WM_TEXT_MAX_PROGRAMS 256   /* programs per call */

/* vocab, hidden width, heads (hidden / heads = head width), feed-forward
 * width, layers, window, stride, latent width d, precision (wm_precision).
 * Supported: hidden, ffn, window and the head width multiples of 32,
 * hidden <= 1024, window <= 1024, 1 <= stride <= window. */
typedef struct wm_text_dims {
  int32_t vocab, hidden, heads, ffn, layers, window, stride, d, precision;
} wm_text_dims;

/* HOST float32, PyTorch layouts, layers stacked on the leading axis:
 * tok_emb [vocab][hidden], pos_emb [window][hidden], ln0_g/ln0_b [hidden],
 * wqkv [L][3 hidden][hidden] (rows q, k, v), bqkv [L][3 hidden],
 * wo [L][hidden][hidden], bo [L][hidden], ln1_g/ln1_b [L][hidden],
 * w1 [L][ffn][hidden], b1 [L][ffn], w2 [L][hidden][ffn], b2 [L][hidden],
 * ln2_g/ln2_b [L][hidden], wp [d][hidden], bp [d]. */
typedef struct wm_text_weights {
  const float *tok_emb, *pos_emb, *ln0_g, *ln0_b;
  const float *wqkv, *bqkv, *wo, *bo, *ln1_g, *ln1_b, *w1, *b1, *w2, *b2, *ln2_g, *ln2_b;
  const float *wp, *bp;
} wm_text_weights;

typedef struct wm_text_model wm_text_model;

/* Copy the encoder to the current device (matrices rounded to bfloat16 in
 * WM_BF16).  Synchronous.  Errors: INVALID_ARGUMENT, UNSUPPORTED,
 * OUT_OF_MEMORY, DEVICE. */
wm_status wm_text_model_create(const wm_text_dims* dims, const wm_text_weights* weights,
                               wm_text_model** out);
void wm_text_model_destroy(wm_text_model* model);

/* Total chunks of S programs given HOST token offsets tok_off [S+1]
 * (0 = tok_off[0] <= ... ); -1 on a bad argument. */
int32_t wm_text_chunks(const wm_text_model* model, const int32_t* tok_off, int32_t S);

/* Workspace bytes of wm_encode_text for a batch of n_chunks chunks (caller
 * allocated, 256-byte aligned, zeroed once; same error-word rules as
 * wm_workspace_bytes).  About 4 (6 hidden + ffn + heads window) bytes per
 * chunk position. */
size_t wm_text_workspace_bytes(const wm_text_model* model, int32_t n_chunks);

/* z0 [S][d] float32 out, from the concatenated token ids tokens [tok_off[S]]
 * int32 (device) of S programs, tok_off HOST [S+1], 1 <= S <= 256.  A token
 * id outside [0, vocab) sets the device error word (read it with
 * wm_device_status).  The result can feed wm_evaluate as its z0. */
wm_status wm_encode_text(const wm_text_model* model, const int32_t* tokens, const int32_t* tok_off,
                         int32_t S, float* z0, void* ws, size_t ws_bytes, void* stream);

/* Synchronise `stream`, read and clear the workspace's device error word.
 * Returns WM_OK, or WM_ERR_INPUT_RANGE with wm_last_error() naming the
 * violation(s); WM_ERR_DEVICE if the stream reports a failure. */
wm_status wm_device_status(void* ws, size_t ws_bytes, void* stream);

/* Message for the last non-OK status returned on this thread ("" if none). */
const char* wm_last_error(void);

/* Kernel timing with HIP events recorded on the launch stream around each
 * launch of one kernel family (for benchmarks).  Ids: 0 rollout, 1 score,
 * 2 top-k, 3 bucketing, 4 action features, 5 encoder, 6 structured action
 * features, 7 tree-ensemble scores, 8 loss forward steps, 9 step losses,
 * 10 loss backward steps, 11 weight-gradient sums, 12 encoder dense
 * products, 13 encoder attention, 14 other encoder kernels.  Enabling resets the
 * counters; reading synchronises on the recorded events.  At most 8192
 * launches per kernel are recorded while enabled. */
wm_status wm_timing_enable(int32_t on);
wm_status wm_timing_read(int32_t kernel, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif
#endif /* WM_H */
