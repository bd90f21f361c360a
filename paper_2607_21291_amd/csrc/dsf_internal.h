// Host-side declarations shared by the library's translation units: kernel
// launchers (each defined next to its kernels) and the timing hooks.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "adadsf.h"

namespace dsf {

// ---- per-launch timing (api.hip) ----
// A scope brackets one launch with a start and a stop event. A deferred
// scope records neither itself: the launcher inside it takes the events with
// timing_claim and hands them to hipExtLaunchKernelGGL, which timestamps the
// kernel's own dispatch (no launch overhead inside the interval); if no
// launcher claims them the record is dropped.
void timing_begin(int kind, hipStream_t s, bool deferred);
bool timing_claim(hipEvent_t* start, hipEvent_t* stop);
void timing_end(int kind, hipStream_t s);

struct TimedScope {
  int kind;
  hipStream_t s;
  TimedScope(int k, hipStream_t st, bool deferred = false) : kind(k), s(st) { timing_begin(kind, s, deferred); }
  ~TimedScope() { timing_end(kind, s); }
};

// Launch kern<<<grid, block, 0, s>>>(args...), through hipExtLaunchKernelGGL
// with the events of an enclosing deferred scope when it hands them over.
template <typename K, typename... A>
inline void launch_with_timing(K kern, dim3 grid, dim3 block, hipStream_t s, A... args) {
  hipEvent_t e0, e1;
  if (timing_claim(&e0, &e1)) hipExtLaunchKernelGGL(kern, grid, block, 0, s, e0, e1, 0, args...);
  else kern<<<grid, block, 0, s>>>(args...);
}

// ---- router forward and backward (kernels_router.hip) ----
// Decode-time routing of the scored tokens, folded into the router (thr null:
// scores only): keep[t] = scores[t] >= thr[t] && len[t] < cap, gate[t] =
// keep ? +inf : -inf, keep_out[t] (nullable) = 1 kept, 0 skipped, 2 skipped
// because the cache is full.
struct RouteArgs {
  const float* thr;
  const int32_t* len;
  int cap;
  int32_t* keep;
  float* gate;
  int32_t* keep_out;
};
hipError_t launch_router(int dtype, const void* x, int64_t n, int d, int d_r, const void* w1,
                         const void* b1, const void* w2, float b2, float* scores, hipStream_t s,
                         const RouteArgs* route = nullptr);
// Router scores of B sequences of T tokens and each sequence's Top-K in one
// launch (bf16; router_topk_fusable). count: B words, zero before the launch
// and left zero.
bool router_topk_fusable(int dtype, int T, int d_r);
hipError_t launch_router_topk(const void* x, int B, int T, int d, int d_r, const void* w1, const void* b1,
                              const void* w2, float b2, float* scores, int k, int32_t* idx, uint32_t* count,
                              hipStream_t s);
// dscore[B, T] = 0, then at kept positions (1 - sigmoid(s)) <dy, x_out - x_in>
hipError_t launch_gate_grad(int dtype, const void* dy, const void* x_in, const void* x_out, const float* scores,
                            const int32_t* idx, int B, int T, int k, int d, float* dscore, hipStream_t s);
struct RouterBwdArgs {
  int dtype;
  const void* x; int64_t n; int d; int d_r;
  const void* w1; const void* b1; const void* w2;
  const float* dscore;
  float* dw1; float* db1; float* dw2; float* db2;  // db1 nullable
  void* dx;                                        // nullable; accumulated into
  void* workspace;                                 // router_bwd_workspace_bytes(n, d, d_r)
};
size_t router_bwd_workspace_bytes(int64_t n, int d, int d_r);
hipError_t launch_router_backward(const RouterBwdArgs& a, hipStream_t s);

// ---- alignment objective, Section 3.5 (kernels_align.hip) ----
int align_grid(int64_t n_tokens);  // blocks of the Eq. 9 kernel (partials written)
int align_max_d(int dtype);        // widest hidden row the Eq. 9 kernel keeps in registers
// accum[0] += sum over tokens of sum_c (softmax(hs) - softmax(hd))^2; partial: align_grid(n) doubles
hipError_t launch_align_hidden(int dtype, const void* hs, const void* hd, int64_t n, int d, float* per_tok,
                               double* partial, double* accum, hipStream_t s);
// accum[0] += sum over rows of KL(softmax(ld) || softmax(ls)); partial: rows doubles
hipError_t launch_kl_align(int dtype, const void* ld, const void* ls, int64_t rows, int C, float* per_row,
                           double* partial, double* accum, hipStream_t s);

// ---- streaming kernels (kernels_misc.hip) ----
// table[p][i] = (cos, sin)(p * theta^(-2i/R)), p < T, i < R/2, computed in fp64.
hipError_t launch_rope_table(float* table, int T, int R, double theta, hipStream_t s);
int sim_grid(int64_t n_tokens);
hipError_t launch_sim_stats(int dtype, const void* a, const void* c, int64_t n, int d, float* per_tok,
                            double* partial, double* accum, hipStream_t s);
hipError_t launch_topk(const float* scores, int B, int T, int k, int32_t* idx, hipStream_t s);
hipError_t launch_gather(int dtype, const void* x, int B, int T, int d, const int32_t* idx, int k,
                         void* out, hipStream_t s);
hipError_t launch_scatter(int dtype, void* x, const void* delta, int B, int T, int d,
                          const int32_t* idx, int k, hipStream_t s);
hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t s);
// dst[0 .. n) = 0 with a kernel (no memset node, so the call can be captured)
hipError_t launch_zero_u32(uint32_t* dst, int64_t n, hipStream_t s);

// Row normalisation of gathered rows. Output row r = b * kk + j reads source
// row src[b * src_rows + (idx ? idx[r] : j)] (src_rows = T for hidden states)
// or, with src_rows == 0, the compact row src[r]. rms != 0 selects RMSNorm
// (bias pointers must be null); out2 (nullable) receives a second
// normalisation of the same rows with (w2, b2).
struct NormArgs {
  int dtype;
  const void* src;
  int src_rows;
  const int32_t* idx;
  int B, kk, d;
  float eps;
  int rms;
  const void* w1; const void* b1; void* out1;
  const void* w2; const void* b2; void* out2;
};
hipError_t launch_norm(const NormArgs& a, hipStream_t s);

// ---- GEMMs with fused epilogues (kernels_gemm.hip) ----
// C[M, N] = A[M, K] . B[N, K]^T in fp32, then one of the epilogues below.
// Rows m < M are compacted tokens: m = b * kk + j at position pos = idx ? idx[m] : j.
enum EpiKind {
  EPI_QKV_ROPE = 0,   // + bias, RoPE on q/k heads, write q/k/v as [B, H, kk, hd]
  EPI_BIAS_GELU = 1,  // out[m, n] = gelu(C + bias)
  EPI_SWIGLU = 2,     // B rows interleaved gate/up; out[m, n] = silu(gate) * up, N = f
  EPI_RESID_STORE = 3,    // out[m, n] = x[b, pos, n] + C (+ bias)
  EPI_RESID_SCATTER = 4,  // x[b, pos, n] = resid + C + bias + bias2, resid = x[b, pos] or res[m]
  EPI_RESID_SCATTER_GATE = 5,  // x[b, pos, n] += sigmoid(gate[b, pos]) * (resid + C + bias + bias2 - x[b, pos])
  // backward of the block (bf16 only; one output tile per workgroup):
  EPI_STORE = 6,       // out[m, n] = C (+ bias), bf16
  EPI_STORE_F32 = 7,   // out[m, n] = C, fp32 (weight gradients)
  EPI_GELU_BWD = 8,    // out[m, n] = C * gelu'(res[m, n]) (res: the up projection's pre-activation, ld = ldo)
  EPI_SWIGLU_BWD = 9,  // N = f; res = [gate | up] pre-activations [M, 2f] (ld = ldo = 2f):
                       // out[m, n] = C * up * silu'(gate), out[m, f + n] = C * silu(gate)
};

struct GemmArgs {
  int dtype;
  int M, N, K;
  // A: [M, K1] from a, then [M, K - K1] from a2 (K1 == K: single source)
  const void* a; int lda; const void* a2; int lda2; int K1;
  // B: [N, K1] from b, then [N, K - K1] from b2
  const void* b; int ldb; const void* b2; int ldb2;
  int epi;
  const void* bias; const void* bias2;
  // token mapping
  int B, kk, T; const int32_t* idx;
  // EPI_QKV_ROPE
  void* q; void* k; void* v; int Hq, Hkv, hd, R; const float* rope;
  // EPI_BIAS_GELU / EPI_SWIGLU / EPI_RESID_STORE output [M, ldo]
  void* out; int ldo;
  // EPI_RESID_*: hidden states x [B, T, d] (d = N); res (nullable) compact residual [M, N]
  void* x; const void* res;
  // EPI_RESID_SCATTER_GATE: router scores [B, T] (fp32)
  const float* gate;
  // EPI_SWIGLU: f (gate rows [0, f), up rows [f, 2f))
  int f;
  // Stream-K workspace (nullable: then every launch is one tile per workgroup):
  // part holds gemm_partial_bytes(), flags gemm_flag_count() words that were
  // zeroed before the first launch using them; epoch is nonzero and distinct
  // for every launch between two zeroings.
  float* part; uint32_t* flags; uint32_t epoch;
  // Status word of the call (nullable): a stream-K finisher whose bounded
  // wait for a partial sum gives up ORs DSF_WS_STATUS_SK_TIMEOUT into it.
  // spin_limit is set by the launcher: polls of a flag before giving up.
  uint32_t* status; int spin_limit;
  // Few-row workspace (nullable): with M <= 16 rows (decode steps) a bf16 GEMM
  // splits K over workgroups; spart holds gemm_skinny_partial_bytes() and
  // scount gemm_skinny_counters() words, zero before the first launch using
  // them (each launch leaves them zero).
  float* spart; uint32_t* scount;
  // set by the launcher: number of M tiles; workgroups per XCD of a persistent
  // grid (0: one tile per workgroup); 1 if its last round is split along K
  int ntm; int px; int split;
  // set by the launcher for one-tile-per-workgroup grids: tiles are taken in
  // bands of group_m tile rows, column by column (0: row-major); ntn is the
  // number of N tiles
  int group_m; int ntn;
  // set by the launcher for the split last round (gemm_bf16_tail_kernel):
  // tiles tail0 .. tail0 + tail_r - 1 of the tile order, each split into
  // tail_s pieces of its k-tiles
  int tail0, tail_r, tail_s;
  // tile size chosen by the caller for a pair of GEMMs that share the chip
  // (0: the launcher's own rule, 1: 128 x 128, 2: 256 x 256)
  int tile_hint;
};
// Timing of a GEMM launched as two kernels: closes the record the first
// launch claimed and opens another of the same kind for the second.
void timing_continue();
hipError_t launch_gemm(const GemmArgs& g, hipStream_t s);
// GemmArgs::tile_hint for two forward projections run side by side, from the
// leading one's M x N and reduction K (0: leave each launch its own rule).
int gemm_pair_tile_hint(int M, int N, int K);

// ---- backward of the routed layer (kernels_bwd.hip) ----
// out[c][r] = op(in[r][c]) (op 0 copy, 1 GELU, 2 SiLU(in[r][c]) * in[r][C + c]);
// out's leading dimension ldo >= R, columns R .. ldo - 1 written as zeros.
hipError_t launch_transpose(int op, const void* in, int R, int C, int ldi, void* out, int ldo, hipStream_t s);
// out[c] = sum_r a[r][c] (x null) or sum_r a[r][c] (x[r][c] - mean[r]) rstd[r]
// (mean nullable: 0), in a fixed order; partial: colsum_chunks(R) * C floats.
int colsum_chunks(int R);
hipError_t launch_colsum(const void* a, int R, int C, int lda, const void* x, const float* mean, const float* rstd,
                         float* partial, float* out, hipStream_t s);
// out[b kk + j] = (scores ? sigmoid(scores[b, idx]) : 1) * dy[b, idx[b kk + j]]
hipError_t launch_gather_scale(const void* dy, int B, int T, int d, const int32_t* idx, int kk, const float* scores,
                               void* out, hipStream_t s);
// LayerNorm (rms false) or RMSNorm adjoint of M rows: acc (fp32) = or += dx;
// sum_out = add + dx (both nullable); mean/rstd [M] of each row kept.
hipError_t launch_norm_bwd(bool rms, const void* x, const void* dyn, const void* w, int M, int d, float eps, float* acc,
                           bool accumulate, const void* add, void* sum_out, float* mean, float* rstd, hipStream_t s);
// dqkv [B kk, (Hq + 2 Hkv) hd] (bf16) from head-major fp32 dq, dk, dv; RoPE turned back.
hipError_t launch_rope_bwd(const float* dq, const float* dk, const float* dv, const float* table, const int32_t* idx,
                           int B, int kk, int T, int Hq, int Hkv, int hd, int R, void* out, hipStream_t s);
// dx[b, idx] = dy[b, idx] + acc (fp32 add, one rounding)
hipError_t launch_scatter_grad(const void* dy, const float* acc, int B, int T, int d, const int32_t* idx, int kk,
                               void* dx, hipStream_t s);
// causal attention backward; q, k, v head-major (RoPE applied), o and dout
// token-major [B n, Hq hd]; lse [B, Hq, n] from the forward (launch_attention);
// dvec [B, Hq, n] (written, then read); dq [B, Hq, n, hd], dk and dv
// [B, Hkv, n, hd] fp32.
hipError_t launch_attention_bwd(const void* q, const void* k, const void* v, const void* o, const void* dout, int B,
                                int Hq, int Hkv, int n, int hd, const float* lse, float* dvec, float* dq, float* dk,
                                float* dv, hipStream_t s);
size_t gemm_partial_bytes();
int gemm_flag_count();
size_t gemm_skinny_partial_bytes();
int gemm_skinny_counters();

// ---- attention over kept tokens (kernels_attn.hip) ----
// q [B, Hq, n, hd], k/v [B, Hkv, n, hd] -> out [B, n, Hq*hd], causal over the n tokens.
// lse (nullable, bf16 only): float [B, Hq, n], the log of each query's softmax
// normaliser in natural units of q.k / sqrt(hd) (the backward's input).
hipError_t launch_attention(int dtype, const void* q, const void* k, const void* v, int B, int Hq,
                            int Hkv, int n, int hd, void* out, hipStream_t s, float* lse = nullptr);

// ---- incremental decoding (kernels_decode.hip) ----
int decode_attn_chunks(int cap);
constexpr int kDecodeMaxCap = 256 * 256;  // cache slots the decode attention supports
// q [B, Hq, hd]; caches [B, Hkv, cap, hd] with cache_len[b] valid slots;
// part: B * Hq * decode_attn_chunks(cap) * (hd + 2) floats; count: B * Hq + B
// words, zero before the launch (the launch leaves them zero); out [B, Hq * hd].
// keep (nullable): a kept sequence's new rows knew / vnew [B, Hkv, hd] join
// the attention as slot cache_len[b], are copied into that slot, and
// cache_len[b] grows by one (the cache append of a decode step).
hipError_t launch_decode_attention(int dtype, const void* q, const void* ck, const void* cv, int32_t* cache_len,
                                   const void* knew, const void* vnew, const int32_t* keep, int B, int Hq, int Hkv,
                                   int hd, int cap, float* part, uint32_t* count, void* out, hipStream_t s);
hipError_t launch_kv_fill(int dtype, const void* ks, const void* vs, void* ck, void* cv, int32_t* cache_len, int B,
                          int Hkv, int hd, int k, int cap, hipStream_t s);
hipError_t launch_kept_min_score(const float* scores, const int32_t* idx, int B, int T, int k, float* thr,
                                 hipStream_t s);

}  // namespace dsf
