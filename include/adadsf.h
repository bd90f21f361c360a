/*
 * adadsf.h - C ABI of the MI355X (gfx950) depth-sparse Transformer layer forward.
 *
 * The library computes AdaDSF's inference path ("Adaptive Depth Sparse
 * Framework: Similarity-Driven Resource Allocation for Pre-Trained LLMs"):
 *   - a per-layer cosine-similarity statistic between a layer's input and
 *     output hidden states (Section 3.3, Eq. 4);
 *   - retention ratios from those statistics (Section 3.3, Eqs. 5-8), and
 *     K = floor(r * T) kept tokens per sequence (Section 3.4);
 *   - a lightweight MLP router scoring every token and a per-sequence Top-K
 *     (Section 3.4);
 *   - the decoder block (Section 3.1, Eqs. 1-2) run on the kept tokens only,
 *     with the skipped tokens passing through the residual path (Section 3.4).
 *
 * Conventions shared by every call
 * --------------------------------
 * Ownership. The caller owns every buffer. The library never allocates or
 *   frees device memory. Scratch space is a caller-provided device
 *   `workspace` of at least the size the matching *_workspace_size call returns.
 * Streams. Device work is enqueued on the given hipStream_t (0 = the null
 *   stream) and the call returns without waiting. The only exception is
 *   dsf_sim_finalize, which waits for its copy.
 * Errors. Every call returns a dsf_status and dsf_last_error() returns a
 *   message for the calling thread. Arguments are checked on the host before
 *   anything is enqueued, so an argument error (DSF_EINVAL, DSF_EUNSUPPORTED,
 *   DSF_EWORKSPACE) launches nothing, writes no output and needs no GPU. Only
 *   a HIP failure in the middle of a launch sequence (DSF_EHIP) can leave part
 *   of the work enqueued.
 * Positions. Caller-supplied positions (idx arguments) must lie in [0, T);
 *   kernels clamp them into that range so that a bad value cannot address
 *   memory outside the hidden-state rows (the result is then unspecified).
 * Layouts. Row-major and contiguous. Hidden states are [B, T, d]. Kept
 *   positions are int32 [B, k], strictly ascending within each sequence.
 *   Weight matrices are [out, in] (the in dimension contiguous). Every device
 *   pointer that is read or written as a vector must be 16-byte aligned.
 * Types. dtype selects the element type of hidden states, weights and
 *   activations: DSF_F32 (float) or DSF_BF16 (bfloat16 bits in uint16).
 *   Router scores are float in both cases. Arithmetic is fp32 (bf16 MFMA with
 *   fp32 accumulation on the bf16 path). The similarity statistic is fp64.
 * Determinism. There are no floating-point atomics. Equal inputs on the same
 *   device give bitwise-equal outputs.
 */
#ifndef ADADSF_H
#define ADADSF_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DSF_VERSION 10000 /* major * 10000 + minor * 100 + patch */

typedef enum dsf_status {
  DSF_OK = 0,
  DSF_EINVAL = 1,        /* null pointer, bad shape, k outside [0, T], misaligned pointer */
  DSF_EUNSUPPORTED = 2,  /* dtype, head_dim, router width or d outside the supported set */
  DSF_EWORKSPACE = 3,    /* workspace smaller than required */
  DSF_EHIP = 4,          /* a HIP runtime call failed; the message holds hipGetErrorString */
  DSF_ENODEVICE = 5      /* no usable GPU */
} dsf_status;

enum { DSF_F32 = 0, DSF_BF16 = 1 };

/* Block templates (the model family's own pre-norm block).
 * NEOX_PARALLEL: y = x + Attn(LN1(x)) + MLP_gelu(LN2(x)); LayerNorm with bias,
 *   biases on every projection, rotary on the first rotary_dims of each head.
 * QWEN_SEQ: h = x + Attn(RMS1(x)); y = h + MLP_swiglu(RMS2(h)); RMSNorm, bias on
 *   the QKV projection only, grouped-query attention. */
enum { DSF_BLOCK_NEOX_PARALLEL = 0, DSF_BLOCK_QWEN_SEQ = 1 };

/* flags */
enum {
  DSF_FLAG_DENSE = 1, /* run the unmodified layer on every token (no router, no Top-K) */
  /* Score-gated update, the training-side router-score pathway of Section
   * 3.4: a kept row becomes x + sigmoid(score) * delta instead of x + delta,
   * so that the loss depends on the router scores differentiably (see
   * dsf_gate_score_grad). Skipped rows are unchanged. Not with DSF_FLAG_DENSE. */
  DSF_FLAG_GATE = 2
};

/* clip modes for dsf_retention_from_similarity */
enum { DSF_CLIP_NONE = 0, DSF_CLIP_PLAIN = 1, DSF_CLIP_BUDGET = 2 };
/* rounding for dsf_k_from_retention */
enum { DSF_ROUND_FLOOR = 0, DSF_ROUND_CEIL = 1 };

/* Shape of one decoder layer. Every layer of a stack shares it. */
typedef struct dsf_layer_desc {
  int32_t block;        /* DSF_BLOCK_* */
  int32_t d_model;      /* d, a multiple of 8 */
  int32_t n_heads;      /* Hq */
  int32_t n_kv_heads;   /* Hkv; Hq % Hkv == 0 (query head h reads kv head h / (Hq/Hkv)) */
  int32_t head_dim;     /* hd in {32, 64, 128} */
  int32_t d_ff;         /* f, a multiple of 64 */
  int32_t rotary_dims;  /* R: even, 0 < R <= hd; rotate-half pairs (i, i + R/2) */
  int32_t d_router;     /* router hidden width d_r in {16, 32, 48, 64} */
  float norm_eps;       /* LayerNorm / RMSNorm epsilon */
  float reserved;       /* must be 0 */
  double rope_theta;    /* RoPE base; angle of pair i at position p is p * theta^(-2i/R) */
} dsf_layer_desc;

/* Device pointers of one layer's weights, all in the layer dtype.
 * Nullable entries are marked; a null bias means zero. */
typedef struct dsf_layer_weights {
  const void* router_w1;  /* [d_r, d] */
  const void* router_b1;  /* [d_r], nullable */
  const void* router_w2;  /* [d_r] */
  float router_b2;        /* scalar output bias */
  float reserved;         /* must be 0 */
  const void* norm1_w;    /* [d] */
  const void* norm1_b;    /* [d], NEOX only (must be null for QWEN) */
  const void* norm2_w;    /* [d] */
  const void* norm2_b;    /* [d], NEOX only (must be null for QWEN) */
  const void* w_qkv;      /* [(Hq + 2 Hkv) hd, d], rows in Q | K | V block order */
  const void* b_qkv;      /* [(Hq + 2 Hkv) hd], nullable */
  const void* w_o;        /* [d, Hq hd] */
  const void* b_o;        /* [d], nullable (NEOX) */
  const void* w_up;       /* NEOX: [f, d]; QWEN: [2f, d], gate rows then up rows */
  const void* b_up;       /* [f], nullable (NEOX) */
  const void* w_down;     /* [d, f] */
  const void* b_down;     /* [d], nullable (NEOX) */
} dsf_layer_weights;

/* ---------------------------------------------------------------- library */

int dsf_version(void);
/* Message of the calling thread's last failed call ("" if none). Valid until
 * that thread's next call into the library. */
const char* dsf_last_error(void);

/* ------------------------------------------- similarity statistic (Eq. 4) */

/* Workspace bytes dsf_sim_stats needs for n_tokens rows. */
size_t dsf_sim_workspace_size(int64_t n_tokens);

/* Section 3.3, Eq. 4. For every token row a = x_in[t, :], c = x_out[t, :]
 * (t < n_tokens, rows of d elements):
 *   cos_t = <a, c> / max(|a| |c|, 1e-8)   (products and sums in fp64),
 * then accum[0] += sum_t cos_t and accum[1] += n_tokens (fp64 device memory,
 * which the caller zeroes once before a calibration pass). per_token_cos
 * (nullable, device float [n_tokens]) receives cos_t. The sum is formed in a
 * fixed order, so the result is deterministic. n_tokens == 0 is a no-op. */
int dsf_sim_stats(const void* x_in, const void* x_out, int dtype, int64_t n_tokens, int d,
                  float* per_token_cos, double* accum, void* workspace, size_t workspace_bytes,
                  hipStream_t stream);

/* s_host[l] = accum[l][0] / accum[l][1] for l < L (Eq. 4 averaged over the
 * calibration tokens). accum_dev is device double [L][2], s_host host double
 * [L]. Waits for the copy on `stream`. A layer with a zero count gives NaN. */
int dsf_sim_finalize(const double* accum_dev, int L, double* s_host, hipStream_t stream);

/* ------------------------------------- retention allocation (host, fp64) */

/* Section 3.3, Eqs. 5-8, on the host in fp64:
 *   w~_i = exp((s_i - max s) / tau), w_i = w~_i / sum w~;
 *   z_i = beta (mean(w) - w_i);  r'_i = 0.05 + 0.9 / (1 + exp(-z_i));
 *   r_i = t L r'_i / sum r'.
 * tau <= 0 selects the ablation without temperature: r_i = t for every layer.
 * clip_mode: DSF_CLIP_NONE returns Eq. 8 as is (r_i may exceed 1);
 * DSF_CLIP_PLAIN caps at 1; DSF_CLIP_BUDGET caps at 1 and hands the excess to
 * the uncapped layers in proportion to r'_i, repeating until none exceeds 1,
 * so that sum r_i = t L still holds. Requires L >= 1, 0 < t <= 1, beta > 0,
 * finite s. r_out is host double [L]. */
int dsf_retention_from_similarity(const double* s, int L, double t, double tau, double beta,
                                  int clip_mode, double* r_out);

/* Section 3.4: K = floor(r T), evaluated as floor(r T + 1e-6) so that fp64
 * representation error cannot drop a token (DSF_ROUND_FLOOR), or
 * ceil(r T - 1e-6) (DSF_ROUND_CEIL); clamped to [0, T]. Returns k >= 0, or -1
 * on a bad argument (r not finite, T < 0, unknown rounding). Host only. */
int dsf_k_from_retention(double r, int T, int rounding);

/* ------------------------------------------------ routing (Section 3.4) */

/* Router scores: score[t] = sum_j w2[j] * ReLU(sum_i W1[j, i] x[t, i] + b1[j]) + b2
 * for the n_tokens rows of x (raw residual-stream rows, [n_tokens, d]).
 * W1 [d_r, d], b1 [d_r] (nullable), w2 [d_r] in dtype; scores device float
 * [n_tokens]. */
int dsf_router_score(const void* x, int dtype, int64_t n_tokens, int d, int d_r,
                     const void* w1, const void* b1, const void* w2, float b2,
                     float* scores, hipStream_t stream);

/* Gradient of a loss L with respect to the router scores through the
 * score-gated update (DSF_FLAG_GATE, Section 3.4). A kept row is
 * y = x + sigmoid(s) delta, so dL/ds = sigmoid'(s) <dy, delta>, which equals
 * (1 - sigmoid(s)) <dy, y - x>; skipped rows do not depend on s.
 *   dscore[b, t] = (1 - sigmoid(scores[b, t])) * sum_c dy[b, t, c] (x_out - x_in)[b, t, c]
 *                  for t in idx[b, :], and 0 for every other position.
 * dy, x_in (the layer input), x_out (the gated layer output): device [B, T, d]
 * in dtype, 16-byte aligned; scores: device float [B, T] (the scores the
 * layer used); idx: device int32 [B, k] (the kept positions, distinct per
 * sequence; entries outside [0, T) are ignored); dscore: device float
 * [B, T], fully overwritten. Products and the sum are in fp32. */
int dsf_gate_score_grad(const void* dy, const void* x_in, const void* x_out, int dtype,
                        const float* scores, const int32_t* idx, int B, int T, int k, int d,
                        float* dscore, hipStream_t stream);

/* Workspace bytes of dsf_router_backward (0 on a bad argument). */
size_t dsf_router_backward_workspace_size(int64_t n_tokens, int d, int d_r);

/* Backward of the router MLP (Section 3.4) given dscore = dL/dscore per token:
 * with z = W1 x + b1,
 *   dz = dscore * w2 * [z > 0],  dW1 = sum_t dz_t x_t^T,  db1 = sum_t dz_t,
 *   dw2 = sum_t dscore_t ReLU(z_t),  db2 = sum_t dscore_t,  dx_t += W1^T dz_t.
 * z is recomputed with the arithmetic of dsf_router_score, so the ReLU
 * decisions are those of the forward call. x [n_tokens, d], W1 [d_r, d], b1
 * [d_r] (nullable), w2 [d_r] in dtype; dscore device float [n_tokens]. The
 * weight gradients are device float: dW1 [d_r, d], db1 [d_r] (nullable; 0 is
 * not written when b1 is absent), dw2 [d_r], db2 [1], all overwritten. dx
 * (nullable) is device [n_tokens, d] in dtype and ACCUMULATED into (the
 * router's share of the input gradient is added, in fp32, then rounded once).
 * Sums run in an order fixed by the shape: repeated calls give identical bits.
 * The workspace (dsf_router_backward_workspace_size bytes, 256-byte aligned)
 * needs no initialisation; calls that overlap in time need separate ones. */
int dsf_router_backward(const void* x, int dtype, int64_t n_tokens, int d, int d_r,
                        const void* w1, const void* b1, const void* w2, const float* dscore,
                        float* dw1, float* db1, float* dw2, float* db2, void* dx,
                        void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Top-K_i per sequence. For each of the B sequences of T float scores,
 * writes the k positions with the largest scores to idx[b, 0..k) in ascending
 * position order. A larger score is preferred; equal scores prefer the lower
 * position; -0.0 equals +0.0; NaN ranks below every number. The result is
 * unique. scores device float [B, T], idx device int32 [B, k]. */
int dsf_topk_select(const float* scores, int B, int T, int k, int32_t* idx, hipStream_t stream);

/* Masked selection as compaction: out[b, j, :] = x[b, idx[b, j], :].
 * x [B, T, d], out [B, k, d] in dtype; idx int32 [B, k] with values in [0, T). */
int dsf_gather_rows(const void* x, int dtype, int B, int T, int d, const int32_t* idx, int k,
                    void* out, hipStream_t stream);

/* Residual bypass: x[b, idx[b, j], :] += delta[b, j, :] in place, the add in
 * fp32 and rounded once to dtype (round to nearest even). Skipped rows are not
 * touched. idx must hold distinct positions per sequence. */
int dsf_scatter_residual(void* x, const void* delta, int dtype, int B, int T, int d,
                         const int32_t* idx, int k, hipStream_t stream);

/* ----------------------------------- attention over kept tokens (Eq. 1) */

/* Eq. 1 with a causal mask over n kept tokens per sequence:
 *   out[b, j, h*hd:(h+1)*hd] = sum_{j' <= j} softmax_j'(q_j . k_j' / sqrt(hd)) v_j'
 * q [B, Hq, n, hd], k and v [B, Hkv, n, hd], out [B, n, Hq*hd], all dtype.
 * Query head h reads kv head h / (Hq / Hkv). Rotary embedding, if any, must
 * already be applied to q and k. hd in {32, 64, 128}. bf16: flash-style
 * online softmax in fp32, probabilities rounded to bf16 for the product with
 * v; a workgroup takes 64 queries (one 16-query group per wavefront) for
 * short sequences and 128 (two groups) otherwise, with bitwise the same
 * result; the environment variable DSF_ATTN_GROUPS=1 or =2, read at every
 * call, forces one (testing). */
int dsf_attention_forward(const void* q, const void* k, const void* v, int dtype, int B, int Hq,
                          int Hkv, int n, int hd, void* out, hipStream_t stream);

/* ----------------------------------------- the sparse layer and the stack */

/* Workspace bytes that dsf_sparse_block_forward / dsf_stack_forward need for
 * batch B, sequence length T and at most k_max kept tokens per sequence
 * (k_max = T for DSF_FLAG_DENSE). with_similarity != 0 adds room to keep each
 * layer's input for the similarity statistic. For DSF_BF16 it includes a
 * fixed 64 MiB (+ 2 KiB) for the partial sums and flags of the stream-K
 * projection schedule, followed by 4 B bytes of per-sequence counters of the
 * routing launch (below). The contents need no initialisation; each call
 * resets what it uses, so two calls that overlap in time (on different
 * streams) need two workspaces. Returns 0 on a bad argument.
 *
 * Routing launch. With DSF_BF16, T a multiple of 64 (at most 4096) and no
 * idx_in, the router and the per-sequence Top-K run as one launch: the last
 * of a sequence's router workgroups to finish selects its Top-K. Scores and
 * indices are bitwise those of the two separate kernels; the environment
 * variable DSF_UNFUSED_ROUTING=1, read at every call, runs those instead.
 *
 * Second stream. For GPT-NeoX blocks the FFN up projection runs on a
 * library-owned stream beside QKV and attention on the caller's stream,
 * ordered by event waits (which a graph capture of the caller's stream
 * records too). There is one such stream per device and host thread,
 * created by the thread's first call and destroyed with its events when the
 * thread exits. DSF_SINGLE_STREAM=1, read at every call, keeps all work on
 * the caller's stream (results are bitwise the same).
 *
 * Projection schedule. Each bf16 projection GEMM takes 256 x 256 output
 * tiles when they still fill the chip for more than a round (at least 320
 * tiles; 640 for forward projections with a reduction shorter than 2048;
 * the GPT-NeoX QKV and up projections, which run side by side, take one size
 * for both), 128 x 128 tiles otherwise; the environment variable
 * DSF_GEMM_TILE=small or =large, read at every launch, forces one size. With
 * 256 x 256 tiles each workgroup runs one tile; for the forward projections
 * other than the SwiGLU gate|up (bf16, on the call's workspace), when the
 * tiles would end in a last round at most half as many as the resident
 * workgroups, those last tiles go to a second launch that cuts each along K
 * into 2-4 pieces, the last piece adding the others' partial sums in a
 * fixed order (deterministic; rounds differently from the unsplit grid).
 * DSF_GEMM_TAIL=0, read at every launch, turns that split off. With
 * 128 x 128 tiles each
 * GEMM runs one output tile per workgroup; or, with more tiles than resident
 * workgroups, a persistent grid
 * taking whole tiles (same arithmetic); or, when that would end in a short
 * last round of tiles on a long reduction, a stream-K grid (workgroups split
 * the k-iterations of the last tiles and add their partial sums in a fixed
 * order, which rounds differently). All are deterministic. The environment
 * variable DSF_GEMM_SCHEDULE=classic, =persistent or =streamk, read at every
 * launch, forces one of them (testing and tuning).
 *
 * Call status. The first 4 bytes of the workspace hold a status word that
 * each call of dsf_sparse_block_forward, dsf_stack_forward,
 * dsf_stack_prefill, dsf_align_stack_forward and dsf_sparse_block_backward
 * clears at its start and that
 * its kernels OR bits into; read it with dsf_workspace_status once the call's
 * work is enqueued. A call with nothing to do (B, T or k zero), which
 * launches nothing, leaves the word as it was. DSF_WS_STATUS_SK_TIMEOUT: a stream-K workgroup, or the last
 * piece of a split tile, that must add an earlier workgroup's partial sum waits for it with a bounded spin of
 * 2^22 polls of its flag (the partial is normally ready within microseconds,
 * because the hardware dispatches workgroups in order); if the wait gives
 * up, the tile is written without that partial, so the call's output is
 * wrong, and this bit is set. The environment variable DSF_SK_SPIN_LIMIT
 * (polls per wait, read at every launch) exists for testing this report. */
size_t dsf_workspace_size(const dsf_layer_desc* desc, int dtype, int B, int T, int k_max,
                          int with_similarity);

enum { DSF_WS_STATUS_SK_TIMEOUT = 1 };

/* Status word of the last layer/stack call that used this workspace (see
 * above). Enqueues a 4-byte device-to-host copy on stream and waits for the
 * stream, so every call enqueued before it has finished. *status receives the
 * word (0: no failure). Returns DSF_EINVAL for a null pointer, DSF_EHIP if the
 * copy or the wait fails. */
int dsf_workspace_status(const void* workspace, uint32_t* status, hipStream_t stream);

/* Section 3.4: one sparse layer, in place on x [B, T, d].
 *   1. scores = router(x) for every token (skipped with DSF_FLAG_DENSE);
 *   2. idx = Top-K(scores, k) per sequence, or idx_in if given (teacher forcing);
 *   3. the block of Eqs. 1-2 runs on the kept rows only, at their original
 *      positions (RoPE angle uses idx), with kept tokens attending causally to
 *      kept tokens;
 *   4. x[b, idx[b, j]] = x[b, idx[b, j]] + delta[b, j] (with DSF_FLAG_GATE
 *      + sigmoid(scores[b, idx[b, j]]) delta[b, j]); skipped rows unchanged.
 * k in [0, T]; k == 0 leaves x untouched and launches nothing. With
 * DSF_FLAG_DENSE, k must equal T and every token is processed at positions
 * 0..T-1 (the unmodified layer). scores_out (device float [B, T]) and idx_out
 * (device int32 [B, k]) are nullable copies of the routing decision; idx_in
 * (nullable, device int32 [B, k], strictly ascending per sequence) replaces
 * the router's choice. */
int dsf_sparse_block_forward(const dsf_layer_desc* desc, const dsf_layer_weights* weights,
                             int dtype, void* x, int B, int T, int k, int flags,
                             float* scores_out, int32_t* idx_out, const int32_t* idx_in,
                             void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The depth-sparse stack: x <- layer_l(x, k[l]) for l = 0..L-1 (Section 3.4),
 * with k a host int array [L] (fixed per layer, so the loop never waits on
 * the GPU). weights is a host array [L] of device-pointer sets. With
 * sim_accum (nullable, device double [L][2], zeroed by the caller) each
 * layer's input is kept and dsf_sim_stats(input, output) accumulates into
 * sim_accum[l]: run with DSF_FLAG_DENSE this is the calibration pass of Eq. 4. */
int dsf_stack_forward(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int L,
                      int dtype, const int* k, void* x, int B, int T, int flags,
                      double* sim_accum, void* workspace, size_t workspace_bytes,
                      hipStream_t stream);

/* ------------------------- backward of the routed layer (Section 3.4) */

/* Gradients of one layer's weights, device fp32 in the weights' layouts
 * ([out, in] matrices, vectors as they are). A null entry is not computed;
 * the entries of weights the block template lacks (Qwen: b_o, b_up, b_down,
 * norm1_b, norm2_b) are ignored. Every computed gradient is written, not
 * accumulated. */
typedef struct dsf_layer_grads {
  float* w_qkv;
  float* b_qkv;
  float* w_o;
  float* b_o;
  float* w_up;
  float* b_up;
  float* w_down;
  float* b_down;
  float* norm1_w;
  float* norm1_b;
  float* norm2_w;
  float* norm2_b;
} dsf_layer_grads;

/* Workspace bytes of dsf_sparse_block_backward (0 on a bad argument or for
 * dtype DSF_F32, which the backward does not provide). */
size_t dsf_backward_workspace_size(const dsf_layer_desc* desc, int dtype, int B, int T, int k);

/* Backward of one routed layer (the training side of Section 3.4): given the
 * layer's input x [B, T, d], its kept positions idx [B, k] (as the forward
 * chose them: ascending, distinct, in [0, T)) and the gradient dy [B, T, d]
 * of the loss at the layer's output, writes
 *   dx [B, T, d]: dy at skipped rows; at kept rows dy + the gradient through
 *                 the block's update (the residual path carries dy);
 *   grads: the gradients of the block's weights.
 * With DSF_FLAG_GATE the forward was the gated layer, kept rows
 * x + sigmoid(s) delta with s = scores [B, T] (the router's output), and the
 * update's gradient is sigmoid(s) dy; the router's own share (through s) is
 * dsf_gate_score_grad followed by dsf_router_backward, which adds into dx.
 * The block's activations on the kept rows are recomputed from x (with the
 * forward's kernels) rather than kept by the forward. bf16 only
 * (DSF_EUNSUPPORTED for DSF_F32); fp32 accumulation, deterministic. k == 0
 * copies dy into dx and leaves the gradients unwritten. The weight gradients
 * reduce over every kept token into few output tiles: when that would leave
 * most of the chip idle, their GEMMs take the stream-K grid (equal pieces of
 * the k-iterations per workgroup, partial sums added in a fixed order). The
 * workspace starts with the same status word as the forward's (cleared by
 * every call with B, T > 0; DSF_WS_STATUS_SK_TIMEOUT if a stream-K wait gave
 * up), read with dsf_workspace_status. Errors: DSF_EINVAL for null or
 * misaligned pointers and bad sizes, DSF_EWORKSPACE for a short workspace. */
int dsf_sparse_block_backward(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int dtype,
                              const void* x, const void* dy, int B, int T, int k, const int32_t* idx,
                              const float* scores, int flags, void* dx, const dsf_layer_grads* grads,
                              void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ---------------------- incremental decoding with kept-token KV caches */

/* The paper treats the prefill only. Per-sequence Top-K (Section 3.4) needs
 * the whole sequence, so at decode time a new token is kept by layer l iff its
 * router score, taken on its hidden state at that layer, is >= a threshold
 * thr[l][b]. Each layer holds a cache of its kept tokens' keys and values
 * (after RoPE at their original positions): a kept token appends its key and
 * value and attends causally over the cache; a skipped token passes the layer
 * unchanged. Every step of the layer is causal, so decoding token by token
 * with the keep decisions of a prefill's Top-K reproduces that prefill.
 *
 * Caches, per layer l: cache_k[l] and cache_v[l] (host arrays [L] of device
 * pointers) are [B, Hkv, cap, hd] in dtype, 16-byte aligned, owned by the
 * caller; cache_len (device int32 [L][B]) counts the valid slots of each
 * (layer, sequence) and is updated by the calls. Slots at or beyond
 * cache_len are never read. */

/* Workspace bytes of dsf_decode_step for batch B, positions < max_pos and
 * caches of cap slots (0 on a bad argument, or cap > 65536). No
 * initialisation needed; overlapping calls need separate workspaces. */
size_t dsf_decode_workspace_size(const dsf_layer_desc* desc, int dtype, int B, int max_pos, int cap);

/* One decode step of the L-layer stack. x (device [B, d] in dtype, in place)
 * holds each sequence's new token, at original position pos[b] (device int32
 * [B]; clamped to [0, max_pos)). For l = 0..L-1, on the device:
 *   1. s = router(x[b]); scores_out (nullable, device float [L][B]) gets s;
 *   2. keep = s >= thr[l][b] (thr device float [L][B]: -inf keeps, +inf skips,
 *      a NaN score is not kept); a token that would be kept while its cache is
 *      full (cache_len == cap) is skipped; keep_out (nullable, device int32
 *      [L][B]) gets 1 (kept), 0 (skipped) or 2 (skipped: cache full);
 *   3. kept tokens: QKV with RoPE at pos[b]; key and value stored at slot
 *      cache_len[l][b], which then grows by one; the query attends over slots
 *      0..cache_len[l][b]-1 (itself included); x[b] += the block's update.
 *      Skipped tokens: x[b] unchanged (bitwise).
 * All B rows run through the projections and the keep flags are applied in
 * the cache append and the residual update, so nothing waits for the host.
 * Head dims 32, 64, 128; cap at most 65536 slots (DSF_EUNSUPPORTED above).
 * Errors: DSF_EINVAL for null or misaligned pointers and bad sizes,
 * DSF_EWORKSPACE for a short workspace. */
int dsf_decode_step(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int L, int dtype,
                    void* x, int B, const int32_t* pos, int max_pos, const float* thr,
                    float* scores_out, int32_t* keep_out, void* const* cache_k, void* const* cache_v,
                    int32_t* cache_len, int cap, void* workspace, size_t workspace_bytes,
                    hipStream_t stream);

/* For callers that cannot allocate device memory: code being captured into a
 * HIP graph, tight serving loops, harnesses that forbid hipMalloc. The same
 * step as dsf_decode_step, with the same arguments and results, but without
 * a workspace argument: its scratch is a static device array of
 * dsf_decode_static_scratch_bytes() bytes (32 MiB) that the library holds on
 * each device it runs on until the process ends. The call allocates nothing
 * (no hipMalloc or hipFree). A step whose dsf_decode_workspace_size exceeds
 * the array returns DSF_EWORKSPACE and enqueues nothing. Every call on one
 * device shares that device's array and leaves its contents behind; the step
 * clears what must start at zero itself. Two calls that can overlap on one
 * device (different streams or host threads) race: serialise them, or give
 * one of them dsf_decode_step with its own workspace. */
size_t dsf_decode_static_scratch_bytes(void);
int dsf_decode_step_static(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int L,
                           int dtype, void* x, int B, const int32_t* pos, int max_pos,
                           const float* thr, float* scores_out, int32_t* keep_out,
                           void* const* cache_k, void* const* cache_v, int32_t* cache_len, int cap,
                           hipStream_t stream);

/* Prefill into decode caches: dsf_stack_forward over x [B, T, d] with k[l]
 * kept tokens per layer (no flags, no similarity) that also stores each
 * layer's kept keys and values (RoPE at their positions, in position order)
 * in slots 0..k[l]-1 of cache_k[l] / cache_v[l] and sets cache_len[l][b] =
 * k[l] (k[l] <= cap). thr_out (nullable, device float [L][B]) gets the lowest
 * router score among each sequence's kept tokens (+inf for k[l] = 0): the
 * threshold that keeps a new token when it would rank among the prompt's
 * selection. Workspace: dsf_workspace_size(desc, dtype, B, T, max k, 0). */
int dsf_stack_prefill(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int L,
                      int dtype, const int* k, void* x, int B, int T, void* const* cache_k,
                      void* const* cache_v, int32_t* cache_len, int cap, float* thr_out,
                      void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------- alignment objective (Section 3.5, Eqs. 9-11) */

/* Workspace bytes of dsf_align_hidden and dsf_kl_align for n_rows rows (0 on
 * a bad argument). No initialisation needed; overlapping calls need separate
 * workspaces. */
size_t dsf_align_workspace_size(int64_t n_rows);

/* Eq. 9 summand: for each of n_tokens rows of h_sparse and h_dense ([n_tokens,
 * d] in dtype, 16-byte aligned), with softmax over the row's d features,
 *   sq[t] = sum_c (softmax(h_sparse[t])_c - softmax(h_dense[t])_c)^2,
 * and accum[0] += sum_t sq[t] (device double, added to). The layer's loss is
 * L_hid = sqrt(accum[0]) (the 2-norm over the whole hidden-state tensor).
 * per_token_sq (nullable, device float [n_tokens]) receives sq. Exponentials
 * in fp32, normalisers and sums in fp64, in an order fixed by the shape.
 * d a multiple of 8, at most 8192 (bf16) / 4096 (fp32). */
int dsf_align_hidden(const void* h_sparse, const void* h_dense, int dtype, int64_t n_tokens, int d,
                     float* per_token_sq, double* accum, void* workspace, size_t workspace_bytes,
                     hipStream_t stream);

/* Eq. 10 per row: KL(P_dense || P_sparse) = sum_c P_dense(c) log(P_dense(c) / P_sparse(c))
 * with P = softmax over the n_classes logits of a row. logits_dense and
 * logits_sparse are [n_rows, n_classes] in dtype, 16-byte aligned, n_classes a
 * multiple of 8. per_row_kl (nullable, device float [n_rows]) receives each
 * row's KL; accum[0] += their sum (device double). One pass over the logits
 * with an online maximum; exponentials fp32, sums fp64, fixed order. */
int dsf_kl_align(const void* logits_dense, const void* logits_sparse, int dtype, int64_t n_rows,
                 int n_classes, float* per_row_kl, double* accum, void* workspace,
                 size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes of dsf_align_stack_forward (0 on a bad argument). */
size_t dsf_align_stack_workspace_size(const dsf_layer_desc* desc, int dtype, int B, int T);

/* Dense-teacher / sparse-student forward of Section 3.5. x_sparse and x_dense
 * ([B, T, d] in dtype) hold the same input on entry. For l = 0..L-1:
 *   x_dense <- dense layer l (every token), x_sparse <- sparse layer l with
 *   k[l] kept tokens (as dsf_stack_forward), then
 *   hid_accum[l] += sum over tokens of the Eq. 9 summand of (x_sparse, x_dense).
 * L_hid^(l) = sqrt(hid_accum[l]); Eq. 11 is L_align + mean_l L_hid^(l).
 * hid_accum: device double [L], added to. flags: 0 or DSF_FLAG_GATE (the
 * student's gated update); DSF_FLAG_DENSE is rejected. d_model at most 8192
 * (bf16) / 4096 (fp32). */
int dsf_align_stack_forward(const dsf_layer_desc* desc, const dsf_layer_weights* weights, int L,
                            int dtype, const int* k, void* x_sparse, void* x_dense, int B, int T,
                            int flags, double* hid_accum, void* workspace, size_t workspace_bytes,
                            hipStream_t stream);

/* ------------------------------------------------------- kernel timing */

/* Per-kernel timing with HIP events recorded around each launch on the
 * launch's own stream. Used by the benchmark to attribute time to kernels.
 * dsf_timing_enable(n, mask) arms up to n launch records for the kernel
 * classes whose bit (1 << DSF_KIND_*) is set in mask; n == 0 disarms and
 * frees the events. dsf_timing_read waits for the recorded events and
 * returns, for the kernel class `kind`, the number of launches and their
 * summed duration in milliseconds, then clears that class. */
enum {
  DSF_KIND_SIM = 0, DSF_KIND_ROUTER = 1, DSF_KIND_TOPK = 2, DSF_KIND_NORM = 3,
  DSF_KIND_GEMM_QKV = 4, DSF_KIND_ATTN = 5, DSF_KIND_GEMM_O = 6, DSF_KIND_GEMM_UP = 7,
  DSF_KIND_GEMM_DOWN = 8, DSF_KIND_GATHER = 9, DSF_KIND_SCATTER = 10, DSF_KIND_OTHER = 11,
  DSF_KIND_BACKWARD = 12, DSF_KIND_ALIGN = 13, DSF_KIND_COUNT = 14
};
int dsf_timing_enable(int max_records, uint32_t kind_mask);
int dsf_timing_read(int kind, int* launches, double* total_ms);

#ifdef __cplusplus
}
#endif

#endif /* ADADSF_H */
