// The token router of Section 3.4 on gfx950: the score MLP
// s = w2 . ReLU(W1 x + b1) + b2 for every token, and the training-side
// router-score pathway: the gradient of a loss through the score-gated
// residual update x + sigmoid(s) * delta with respect to the kept tokens'
// scores, and the backward of the score MLP (weights, biases and input).
//
// Every reduction runs in an order fixed by the shape (per-chunk partial sums
// added in chunk order), so results are bitwise repeatable; there are no
// floating-point atomics.
#include "dsf_device.h"
#include "dsf_internal.h"
#include "topk_block.h"

namespace dsf {

// ------------------------------------------------------------- forward

// bf16 router on MFMA. A workgroup scores 64 tokens (4 blocks of 16) against
// all d_r hidden units (DR / 16 column blocks of v_mfma_f32_16x16x32_bf16).
// The reduction over d is split between kRouterWaves wavefronts: wave w takes
// the 32-wide column slices w, w + NW, ... of all four token blocks, so each
// W1 fragment it loads serves 64 tokens (W1 traffic is a quarter of x's at
// d_r = 32), and the short per-wave loop keeps many loads in flight per CU.
// Within a slice each lane streams 16 contiguous bytes of its row; the MFMA's
// k slots are filled in that order and W1 is read in the same order, so the
// contraction is unchanged. The partial hidden sums meet in LDS.
constexpr int kRouterWaves = 8;
#ifndef DSF_ROUTER_TOKENS
#define DSF_ROUTER_TOKENS 64
#endif
constexpr int kRouterTokens = DSF_ROUTER_TOKENS;  // tokens per workgroup, a multiple of 16
static_assert(kRouterTokens % 16 == 0 && kRouterTokens <= 128, "token blocks of 16");

template <int DR>
using RouterPart = float[kRouterWaves][kRouterTokens][DR + 1];

// part[w][t][j] = wave w's share of sum_c x[row0 + t, c] * W1[j, c]. Rows
// past n are computed from row n - 1 and must be dropped by the caller.
template <int DR>
__device__ __forceinline__ void router_hidden_partials(const uint16_t* __restrict__ x, int64_t n, int d,
                                                       const uint16_t* __restrict__ w1, int64_t row0,
                                                       RouterPart<DR>& part) {
  constexpr int NB = DR / 16, NW = kRouterWaves, MT = kRouterTokens / 16;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const uint16_t* xr[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    int64_t row = row0 + 16 * mt + r;
    if (row > n - 1) row = n - 1;
    xr[mt] = x + row * d;
  }
  f32x4 acc[MT][NB];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mt][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  const bf16x8 zero = {};
#pragma unroll 4
  for (int kc = 32 * w; kc < d; kc += 32 * NW) {
    // d is a multiple of 8, so each lane's 8-element piece is wholly inside or past the end
    const int k0 = kc + 8 * g;
    const bool ok = k0 < d;
    bf16x8 wb[NB], xa[MT];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
      wb[nb] = ok ? *reinterpret_cast<const bf16x8*>(w1 + (16 * nb + r) * int64_t(d) + k0) : zero;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) xa[mt] = ok ? *reinterpret_cast<const bf16x8*>(xr[mt] + k0) : zero;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        acc[mt][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[mt], wb[nb], acc[mt][nb], 0, 0, 0);
  }
  // lane holds wave w's partial hidden[token 16 mt + 4 g + i][unit 16 nb + r]
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) part[w][16 * mt + 4 * g + i][16 * nb + r] = acc[mt][nb][i];
}

// Hidden pre-activation of unit j: b1[j] plus the wave partials in wave
// order. The forward pass and the backward recomputation share this order,
// so both take the same ReLU decisions.
template <int DR>
__device__ __forceinline__ float router_hidden(const RouterPart<DR>& part, const uint16_t* b1, int t, int j) {
  float h = b1 ? bf2f(b1[j]) : 0.f;
#pragma unroll
  for (int ww = 0; ww < kRouterWaves; ++ww) h += part[ww][t][j];
  return h;
}

// Decode-time routing of token t with score v (RouteArgs).
__device__ __forceinline__ void route_token(const RouteArgs& ra, int64_t t, float v) {
  const bool want = v >= ra.thr[t];
  const bool room = ra.len[t] < ra.cap;
  const int k = want && room;
  ra.keep[t] = k;
  ra.gate[t] = k ? INFINITY : -INFINITY;
  if (ra.keep_out) ra.keep_out[t] = want ? (room ? 1 : 2) : 0;
}

template <int DR>
__global__ __launch_bounds__(64 * kRouterWaves) void router_bf16_kernel(const uint16_t* __restrict__ x, int64_t n, int d,
                                                                         const uint16_t* __restrict__ w1,
                                                                         const uint16_t* __restrict__ b1,
                                                                         const uint16_t* __restrict__ w2, float b2,
                                                                         float* __restrict__ scores, RouteArgs ra) {
  __shared__ RouterPart<DR> part;
  const int64_t row0 = int64_t(blockIdx.x) * kRouterTokens;
  router_hidden_partials<DR>(x, n, d, w1, row0, part);
  __syncthreads();
  // threads 0..4 TM - 1: token t / 4, units q DR/4 .. (q + 1) DR/4 - 1 with
  // q = t % 4; the partial sums of a token are then added in a fixed order
  if (threadIdx.x >= 4 * kRouterTokens) return;
  const int t = threadIdx.x >> 2, q = threadIdx.x & 3;
  float v = 0.f;
#pragma unroll
  for (int jj = 0; jj < DR / 4; ++jj) {
    const int j = q * (DR / 4) + jj;
    const float h = router_hidden<DR>(part, b1, t, j);
    v = fmaf(bf2f(w2[j]), h > 0.f ? h : 0.f, v);
  }
  v += __shfl_xor(v, 1);
  v += __shfl_xor(v, 2);
  if (q == 0 && row0 + t < n) {
    scores[row0 + t] = v + b2;
    if (ra.thr) route_token(ra, row0 + t, v + b2);
  }
}

// fp32 hidden pre-activation of unit j for one row, by one wavefront: lane
// strided products, then a wave sum, then the bias (forward and backward).
__device__ __forceinline__ float router_hidden_f32(const float* __restrict__ row, int d,
                                                   const float* __restrict__ w1, const float* __restrict__ b1,
                                                   int j, int lane) {
  const float* wr = w1 + int64_t(j) * d;
  float h = 0.f;
  for (int i = lane; i < d; i += 64) h = fmaf(row[i], wr[i], h);
  return wave_sum(h) + (b1 ? b1[j] : 0.f);
}

// fp32 router: one wavefront per token, one hidden unit at a time.
__global__ __launch_bounds__(256) void router_f32_kernel(const float* __restrict__ x, int64_t n, int d, int dr,
                                                         const float* __restrict__ w1, const float* __restrict__ b1,
                                                         const float* __restrict__ w2, float b2,
                                                         float* __restrict__ scores, RouteArgs ra) {
  const int lane = threadIdx.x & 63;
  const int64_t t = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (t >= n) return;
  const float* row = x + t * d;
  float score = 0.f;
  for (int j = 0; j < dr; ++j) {
    const float h = router_hidden_f32(row, d, w1, b1, j, lane);
    score = fmaf(w2[j], h > 0.f ? h : 0.f, score);
  }
  if (lane == 0) {
    scores[t] = score + b2;
    if (ra.thr) route_token(ra, t, score + b2);
  }
}

hipError_t launch_router(int dtype, const void* x, int64_t n, int d, int d_r, const void* w1,
                         const void* b1, const void* w2, float b2, float* scores, hipStream_t s,
                         const RouteArgs* route) {
  if (n == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_ROUTER, s, true);
  const RouteArgs ra = route ? *route : RouteArgs{};
  if (dtype == DSF_F32) {
    launch_with_timing(router_f32_kernel, dim3(unsigned((n + 3) / 4)), dim3(256), s, (const float*)x, n, d, d_r,
                       (const float*)w1, (const float*)b1, (const float*)w2, b2, scores, ra);
    return hipGetLastError();
  }
  unsigned grid = unsigned((n + kRouterTokens - 1) / kRouterTokens);
  auto X = (const uint16_t*)x;
  auto W1 = (const uint16_t*)w1;
  auto B1 = (const uint16_t*)b1;
  auto W2 = (const uint16_t*)w2;
  switch (d_r) {
    case 16: launch_with_timing(router_bf16_kernel<16>, dim3(grid), dim3(64 * kRouterWaves), s, X, n, d, W1, B1, W2, b2, scores, ra); break;
    case 32: launch_with_timing(router_bf16_kernel<32>, dim3(grid), dim3(64 * kRouterWaves), s, X, n, d, W1, B1, W2, b2, scores, ra); break;
    case 48: launch_with_timing(router_bf16_kernel<48>, dim3(grid), dim3(64 * kRouterWaves), s, X, n, d, W1, B1, W2, b2, scores, ra); break;
    case 64: launch_with_timing(router_bf16_kernel<64>, dim3(grid), dim3(64 * kRouterWaves), s, X, n, d, W1, B1, W2, b2, scores, ra); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Router and per-sequence Top-K in one launch. The workgroups score their 64
// tokens as router_bf16_kernel does (same partials, same order: the scores
// are bitwise those of the router alone), store them with device-coherent
// stores and count themselves on their sequence's counter; the last of a
// sequence's T / 64 workgroups to arrive resets the counter and runs the
// Top-K of that sequence (topk_block.h, the same selection as the Top-K
// kernel) on scores read back with device-coherent loads, in the LDS the
// router partials used. No workgroup waits for another. Requires
// T % kRouterTokens == 0 and T <= kTopkLdsKeys; count[B] is zero before the
// launch and is left zero.
constexpr int kRouterThreads = 64 * kRouterWaves;

template <int DR>
__global__ __launch_bounds__(kRouterThreads) void router_topk_bf16_kernel(
    const uint16_t* __restrict__ x, int64_t n, int d, const uint16_t* __restrict__ w1,
    const uint16_t* __restrict__ b1, const uint16_t* __restrict__ w2, float b2, float* __restrict__ scores, int T,
    int k, int32_t* __restrict__ idx, uint32_t* __restrict__ count) {
  union Shared {
    RouterPart<DR> part;
    TopkShared<kRouterThreads, true> topk;
  };
  __shared__ Shared sh;
  __shared__ int is_last;
  const int64_t row0 = int64_t(blockIdx.x) * kRouterTokens;
  router_hidden_partials<DR>(x, n, d, w1, row0, sh.part);
  __syncthreads();
  if (threadIdx.x < 4 * kRouterTokens) {
    const int t = threadIdx.x >> 2, q = threadIdx.x & 3;
    float v = 0.f;
#pragma unroll
    for (int jj = 0; jj < DR / 4; ++jj) {
      const int j = q * (DR / 4) + jj;
      const float h = router_hidden<DR>(sh.part, b1, t, j);
      v = fmaf(bf2f(w2[j]), h > 0.f ? h : 0.f, v);
    }
    v += __shfl_xor(v, 1);
    v += __shfl_xor(v, 2);
    if (q == 0 && row0 + t < n) __hip_atomic_store(scores + row0 + t, v + b2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // the device-coherent stores complete before the counter moves; every wave
  // is done with the partials before the LDS is reused
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  const int b = int(row0 / T);
  if (threadIdx.x == 0) {
    const uint32_t old = __hip_atomic_fetch_add(count + b, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    is_last = old == uint32_t(T / kRouterTokens - 1);
    if (is_last) __hip_atomic_store(count + b, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!is_last) return;
  const float* sc = scores + int64_t(b) * T;
  topk_block<kRouterThreads, true>(
      [&](int t) { return __hip_atomic_load(sc + t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }, T, k,
      idx + int64_t(b) * k, sh.topk);
}

bool router_topk_fusable(int dtype, int T, int d_r) {
  return dtype == DSF_BF16 && T % kRouterTokens == 0 && T <= kTopkLdsKeys &&
         (d_r == 16 || d_r == 32 || d_r == 48 || d_r == 64);
}

hipError_t launch_router_topk(const void* x, int B, int T, int d, int d_r, const void* w1, const void* b1,
                              const void* w2, float b2, float* scores, int k, int32_t* idx, uint32_t* count,
                              hipStream_t s) {
  if (B == 0 || T == 0) return hipSuccess;
  if (!router_topk_fusable(DSF_BF16, T, d_r) || k < 1 || k > T) return hipErrorInvalidValue;
  TimedScope ts(DSF_KIND_ROUTER, s, true);
  const int64_t n = int64_t(B) * T;
  const unsigned grid = unsigned(n / kRouterTokens);
  auto X = (const uint16_t*)x;
  auto W1 = (const uint16_t*)w1;
  auto B1 = (const uint16_t*)b1;
  auto W2 = (const uint16_t*)w2;
  switch (d_r) {
    case 16: launch_with_timing(router_topk_bf16_kernel<16>, dim3(grid), dim3(kRouterThreads), s, X, n, d, W1, B1, W2, b2, scores, T, k, idx, count); break;
    case 32: launch_with_timing(router_topk_bf16_kernel<32>, dim3(grid), dim3(kRouterThreads), s, X, n, d, W1, B1, W2, b2, scores, T, k, idx, count); break;
    case 48: launch_with_timing(router_topk_bf16_kernel<48>, dim3(grid), dim3(kRouterThreads), s, X, n, d, W1, B1, W2, b2, scores, T, k, idx, count); break;
    default: launch_with_timing(router_topk_bf16_kernel<64>, dim3(grid), dim3(kRouterThreads), s, X, n, d, W1, B1, W2, b2, scores, T, k, idx, count); break;
  }
  return hipGetLastError();
}

// ------------------------------------------- gate score gradient (Sec. 3.4)

// With y[b, p] = x[b, p] + sigmoid(s) delta at a kept position p, a loss L
// has dL/ds = sigmoid'(s) <dy, delta> = (1 - sigmoid(s)) <dy, y - x>, because
// y - x = sigmoid(s) delta; skipped positions do not depend on s. One
// wavefront per kept token; dscore was zeroed beforehand. Positions outside
// [0, T) are ignored.
template <typename T>
__global__ __launch_bounds__(256) void gate_grad_kernel(const T* __restrict__ dy, const T* __restrict__ x_in,
                                                        const T* __restrict__ x_out,
                                                        const float* __restrict__ scores,
                                                        const int32_t* __restrict__ idx, int B, int Tn, int k, int d,
                                                        float* __restrict__ dscore) {
  constexpr int V = Elem<T>::kVec;
  const int lane = threadIdx.x & 63;
  const int64_t e = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (e >= int64_t(B) * k) return;
  const int b = int(e / k);
  const int p = idx[e];
  if (p < 0 || p >= Tn) return;
  const int64_t row = int64_t(b) * Tn + p;
  const T* g = dy + row * d;
  const T* a = x_in + row * d;
  const T* o = x_out + row * d;
  float acc = 0.f;
  for (int c = lane * V; c < d; c += 64 * V) {
    float gv[V], av[V], ov[V];
    load_vec(g + c, gv);
    load_vec(a + c, av);
    load_vec(o + c, ov);
#pragma unroll
    for (int i = 0; i < V; ++i) acc = fmaf(gv[i], ov[i] - av[i], acc);
  }
  acc = wave_sum(acc);
  if (lane == 0) dscore[row] = acc / (1.f + expf(scores[row]));
}

// The same with L lanes per kept token (64 / L tokens per wavefront) when the
// row splits evenly into C <= 8 vectors per lane, so that no lane idles.
template <typename T, int L, int C>
__global__ __launch_bounds__(256) void gate_grad_group_kernel(const T* __restrict__ dy, const T* __restrict__ x_in,
                                                              const T* __restrict__ x_out,
                                                              const float* __restrict__ scores,
                                                              const int32_t* __restrict__ idx, int B, int Tn, int k,
                                                              int d, float* __restrict__ dscore) {
  constexpr int V = Elem<T>::kVec, RW = 64 / L;
  const int lane = threadIdx.x & 63, hl = lane % L;
  const int64_t e = (int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6)) * RW + lane / L;
  const int64_t ee = e < int64_t(B) * k ? e : int64_t(B) * k - 1;
  const int b = int(ee / k);
  const int p = idx[ee];
  const bool ok = e < int64_t(B) * k && p >= 0 && p < Tn;
  const int64_t row = int64_t(b) * Tn + (ok ? p : 0);
  float acc = 0.f;
  float gv[C][V], av[C][V], ov[C][V];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const int64_t off = row * d + (hl + L * c) * V;
    load_vec(dy + off, gv[c]);
    load_vec(x_in + off, av[c]);
    load_vec(x_out + off, ov[c]);
  }
#pragma unroll
  for (int c = 0; c < C; ++c)
#pragma unroll
    for (int i = 0; i < V; ++i) acc = fmaf(gv[c][i], ov[c][i] - av[c][i], acc);
#pragma unroll
  for (int o = L / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o, kWave);
  if (hl == 0 && ok) dscore[row] = acc / (1.f + expf(scores[row]));
}

template <typename T, int L>
static void launch_gate_group(const T* dy, const T* xi, const T* xo, const float* sc, const int32_t* idx, int B,
                              int Tn, int k, int d, float* ds, int c, hipStream_t s) {
  const unsigned grid = unsigned((int64_t(B) * k + 4 * (64 / L) - 1) / (4 * (64 / L)));
  switch (c) {
    case 1: gate_grad_group_kernel<T, L, 1><<<grid, 256, 0, s>>>(dy, xi, xo, sc, idx, B, Tn, k, d, ds); break;
    case 2: gate_grad_group_kernel<T, L, 2><<<grid, 256, 0, s>>>(dy, xi, xo, sc, idx, B, Tn, k, d, ds); break;
    case 3: gate_grad_group_kernel<T, L, 3><<<grid, 256, 0, s>>>(dy, xi, xo, sc, idx, B, Tn, k, d, ds); break;
    case 4: gate_grad_group_kernel<T, L, 4><<<grid, 256, 0, s>>>(dy, xi, xo, sc, idx, B, Tn, k, d, ds); break;
    case 5: gate_grad_group_kernel<T, L, 5><<<grid, 256, 0, s>>>(dy, xi, xo, sc, idx, B, Tn, k, d, ds); break;
    case 6: gate_grad_group_kernel<T, L, 6><<<grid, 256, 0, s>>>(dy, xi, xo, sc, idx, B, Tn, k, d, ds); break;
    case 7: gate_grad_group_kernel<T, L, 7><<<grid, 256, 0, s>>>(dy, xi, xo, sc, idx, B, Tn, k, d, ds); break;
    default: gate_grad_group_kernel<T, L, 8><<<grid, 256, 0, s>>>(dy, xi, xo, sc, idx, B, Tn, k, d, ds); break;
  }
}

// true if the rows were handled by a lane-group kernel
template <typename T>
static bool launch_gate_grouped(const T* dy, const T* xi, const T* xo, const float* sc, const int32_t* idx, int B,
                                int Tn, int k, int d, float* ds, hipStream_t s) {
  const int nvec = d / Elem<T>::kVec;
  if (nvec % 64 == 0 && nvec / 64 <= 8) launch_gate_group<T, 64>(dy, xi, xo, sc, idx, B, Tn, k, d, ds, nvec / 64, s);
  else if (nvec % 32 == 0 && nvec / 32 <= 8) launch_gate_group<T, 32>(dy, xi, xo, sc, idx, B, Tn, k, d, ds, nvec / 32, s);
  else if (nvec % 16 == 0 && nvec / 16 <= 8) launch_gate_group<T, 16>(dy, xi, xo, sc, idx, B, Tn, k, d, ds, nvec / 16, s);
  else return false;
  return true;
}

hipError_t launch_gate_grad(int dtype, const void* dy, const void* x_in, const void* x_out, const float* scores,
                            const int32_t* idx, int B, int Tn, int k, int d, float* dscore, hipStream_t s) {
  if (int64_t(B) * Tn == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_BACKWARD, s);
  hipError_t e = launch_zero_u32(reinterpret_cast<uint32_t*>(dscore), int64_t(B) * Tn, s);
  if (e != hipSuccess || k == 0) return e;
  const unsigned grid = unsigned((int64_t(B) * k + 3) / 4);
  if (dtype == DSF_BF16) {
    auto D = (const uint16_t*)dy; auto I = (const uint16_t*)x_in; auto O = (const uint16_t*)x_out;
    if (!launch_gate_grouped(D, I, O, scores, idx, B, Tn, k, d, dscore, s))
      gate_grad_kernel<uint16_t><<<grid, 256, 0, s>>>(D, I, O, scores, idx, B, Tn, k, d, dscore);
  } else {
    auto D = (const float*)dy; auto I = (const float*)x_in; auto O = (const float*)x_out;
    if (!launch_gate_grouped(D, I, O, scores, idx, B, Tn, k, d, dscore, s))
      gate_grad_kernel<float><<<grid, 256, 0, s>>>(D, I, O, scores, idx, B, Tn, k, d, dscore);
  }
  return hipGetLastError();
}

// ------------------------------------------ router backward (Sec. 3.4)

// With z = W1 x + b1 and s = w2 . ReLU(z) + b2, and ds = dL/ds per token:
//   dz = ds * w2 * [z > 0]          dW1 = sum_t dz_t x_t^T    db1 = sum_t dz_t
//   dw2 = sum_t ds_t ReLU(z_t)       db2 = sum_t ds_t          dx_t = W1^T dz_t
// Launches:
//   tokens: per 64-token chunk, recompute z (same arithmetic and order as the
//     forward, hence the same ReLU decisions), then dz, the chunk's sums of
//     dz, ds ReLU(z) and ds, and dx += W1^T dz;
//   weights: partial dW1 over (column slab, token range);
//   reduce: the partials in fixed order into dW1, db1, dw2, db2.
// bf16 runs both contractions on MFMA. MFMA takes its k dimension
// contiguous in each lane's operand, so the tokens kernel multiplies
// W1^T (transposed once per call, k = units) by dz, and the weights kernel
// multiplies dz^T (written by the tokens kernel, k = tokens) by x tiles
// transposed through LDS. dz enters both as a bf16 pair hi + lo (hi = dz
// rounded to bf16, lo = the remainder rounded to bf16), which keeps about
// 16 significant bits: the products keep fp32-level accuracy. fp32 runs the
// same steps on the vector ALUs.

constexpr int kBwdTerms = 2;  // per-chunk sums: dz (db1) and ds ReLU(z) (dw2), then ds (db2)
constexpr int kBwdMaxSplits = 64;

// Token ranges of the weights kernel (a function of n only, so the summation
// order, and with it the result, does not depend on the device).
int router_bwd_splits(int64_t n) {
  const int64_t s = n / 256;
  return int(s < 1 ? 1 : (s > kBwdMaxSplits ? kBwdMaxSplits : s));
}

// Workspace: dz (fp32 [n, DR], or bf16 hi and lo [DR, npad] with npad = n
// rounded up to 32) | chunk terms | dW1 partials | W1^T (bf16 [d, DR]).
struct BwdLayout {
  size_t dz, terms, pw1, w1t, total;
  int64_t chunks, npad;
  int splits;
};
static BwdLayout bwd_layout(int64_t n, int d, int d_r) {
  auto up = [](size_t b) { return (b + 255) / 256 * 256; };
  BwdLayout L{};
  L.chunks = (n + kRouterTokens - 1) / kRouterTokens;
  L.npad = (n + 31) / 32 * 32;
  L.splits = router_bwd_splits(n);
  L.dz = 0;
  L.terms = up(sizeof(float) * size_t(L.npad) * d_r);
  L.pw1 = L.terms + up(sizeof(float) * size_t(L.chunks) * (kBwdTerms * d_r + 1));
  L.w1t = L.pw1 + up(sizeof(float) * size_t(L.splits) * d_r * d);
  L.total = L.w1t + up(sizeof(uint16_t) * size_t(d) * d_r);
  return L;
}

size_t router_bwd_workspace_bytes(int64_t n, int d, int d_r) { return bwd_layout(n, d, d_r).total; }

// z, dz and the per-chunk terms of a 64-token chunk, shared by both dtypes:
// dzs[t][j] = dz, part[1][t][j] = ds ReLU(z), ssum[t] = ds (0 past n). The
// hidden sums are in part (bf16: wave partials; fp32: part[0] holds z).
template <typename T, int DR, int LDZ>
__device__ __forceinline__ void router_bwd_chunk(RouterPart<DR>& part, float (*dzs)[LDZ], float* ssum,
                                                 const T* __restrict__ b1, const T* __restrict__ w2,
                                                 const float* __restrict__ ds, int64_t n, int64_t row0,
                                                 float* __restrict__ terms) {
  constexpr int NT = 64 * kRouterWaves, TM = kRouterTokens;
  for (int e = threadIdx.x; e < TM * DR; e += NT) {
    const int t = e / DR, j = e - t * DR;
    float h;
    if constexpr (sizeof(T) == 2) h = router_hidden<DR>(part, b1, t, j);
    else h = part[0][t][j];
    const float sv = row0 + t < n ? ds[row0 + t] : 0.f;
    const bool on = h > 0.f;
    dzs[t][j] = on ? sv * Elem<T>::to_f(w2[j]) : 0.f;
    part[1][t][j] = on ? sv * h : 0.f;  // only this thread reads or writes entry (t, j)
    if (j == 0) ssum[t] = sv;
  }
  __syncthreads();
  if (threadIdx.x < kBwdTerms * DR + 1) {
    const int j = threadIdx.x;
    float a = 0.f;
    if (j < DR) {
      for (int t = 0; t < TM; ++t) a += dzs[t][j];
    } else if (j < 2 * DR) {
      for (int t = 0; t < TM; ++t) a += part[1][t][j - DR];
    } else {
      for (int t = 0; t < TM; ++t) a += ssum[t];
    }
    terms[int64_t(blockIdx.x) * (kBwdTerms * DR + 1) + j] = a;
  }
}

// ---- bf16 on MFMA

template <int DR>
__global__ __launch_bounds__(256) void router_w1t_kernel(const uint16_t* __restrict__ w1, int d,
                                                         uint16_t* __restrict__ w1t) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;  // = c * DR + j
  if (i >= int64_t(d) * DR) return;
  const int c = int(i / DR), j = int(i - int64_t(c) * DR);
  w1t[i] = w1[int64_t(j) * d + c];
}

// v ~ hi + lo: hi = v rounded to bf16, lo = the remainder (exact in fp32) rounded to bf16
__device__ __forceinline__ __bf16 bf16_hi(float v) { return (__bf16)v; }
__device__ __forceinline__ __bf16 bf16_lo(float v, __bf16 hi) { return (__bf16)(v - (float)hi); }

template <int DR>
__global__ __launch_bounds__(64 * kRouterWaves) void router_bwd_tokens_bf16_kernel(
    const uint16_t* __restrict__ x, int64_t n, int d, const uint16_t* __restrict__ w1,
    const uint16_t* __restrict__ w1t, const uint16_t* __restrict__ b1, const uint16_t* __restrict__ w2,
    const float* __restrict__ ds, uint16_t* __restrict__ dx, uint16_t* __restrict__ dzt_hi,
    uint16_t* __restrict__ dzt_lo, int64_t npad, float* __restrict__ terms) {
  constexpr int NT = 64 * kRouterWaves, TM = kRouterTokens, KS = (DR + 31) / 32;
  __shared__ RouterPart<DR> part;
  __shared__ float dzs[TM][DR + 1];
  __shared__ float ssum[TM];
  const int64_t row0 = int64_t(blockIdx.x) * TM;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  router_hidden_partials<DR>(x, n, d, w1, row0, part);
  __syncthreads();
  router_bwd_chunk<uint16_t, DR, DR + 1>(part, dzs, ssum, b1, w2, ds, n, row0, terms);
  // dz^T as bf16 hi and lo, [DR, npad], for the weights kernel
  for (int e = threadIdx.x; e < TM * DR; e += NT) {
    const int j = e / TM, t = e - j * TM;
    if (row0 + t < n) {
      const float v = dzs[t][j];
      const __bf16 hi = bf16_hi(v);
      dzt_hi[j * npad + row0 + t] = __builtin_bit_cast(uint16_t, hi);
      dzt_lo[j * npad + row0 + t] = __builtin_bit_cast(uint16_t, bf16_lo(v, hi));
    }
  }
  if (!dx) return;
  // dx^T tiles: D[c][t] = sum_j W1^T[c][j] dz[t][j], 16 columns x 16 tokens
  // per MFMA; the lane holding D[4g + i][r] adds it to dx[t = 16 tb + r]
  // [c = 16 cb + 4g + i], i = 0..3 (one 8-byte read-modify-write)
  constexpr int TB = TM / 16;
  bf16x8 bh[TB][KS], bl[TB][KS];
#pragma unroll
  for (int tb = 0; tb < TB; ++tb)
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int j = 32 * ks + 8 * g + i;
        const float v = j < DR ? dzs[16 * tb + r][j] : 0.f;
        const __bf16 hi = bf16_hi(v);
        bh[tb][ks][i] = hi;
        bl[tb][ks][i] = bf16_lo(v, hi);
      }
  const bf16x8 zero = {};
  const int ncb = (d + 15) / 16;
  // software pipelined over this wave's column blocks: the W1^T fragments
  // and old dx values of block cb + NW are requested before block cb is
  // multiplied and stored
  bf16x8 a[KS], an[KS];
  u32x2 old[TB], on[TB];
  auto fetch = [&](int cb, bf16x8 (&aa)[KS], u32x2 (&oo)[TB]) {
    const int c = 16 * cb + r, c4 = 16 * cb + 4 * g;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int j0 = 32 * ks + 8 * g;
      aa[ks] = (c < d && j0 < DR) ? *reinterpret_cast<const bf16x8*>(w1t + int64_t(c) * DR + j0) : zero;
    }
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      const int64_t t = row0 + 16 * tb + r;
      oo[tb] = (t < n && c4 < d) ? *reinterpret_cast<const u32x2*>(dx + t * d + c4) : u32x2{0u, 0u};
    }
  };
  if (w < ncb) fetch(w, a, old);
  for (int cb = w; cb < ncb; cb += kRouterWaves) {
    if (cb + kRouterWaves < ncb) fetch(cb + kRouterWaves, an, on);
    const int c4 = 16 * cb + 4 * g;
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks], bh[tb][ks], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ks], bl[tb][ks], acc, 0, 0, 0);
      }
      const int64_t t = row0 + 16 * tb + r;
      if (t < n && c4 < d) {
        const float v0 = bf2f(uint16_t(old[tb][0] & 0xffffu)) + acc[0];
        const float v1 = bf2f(uint16_t(old[tb][0] >> 16)) + acc[1];
        const float v2 = bf2f(uint16_t(old[tb][1] & 0xffffu)) + acc[2];
        const float v3 = bf2f(uint16_t(old[tb][1] >> 16)) + acc[3];
        *reinterpret_cast<u32x2*>(dx + t * d + c4) =
            u32x2{uint32_t(f2bf(v0)) | (uint32_t(f2bf(v1)) << 16), uint32_t(f2bf(v2)) | (uint32_t(f2bf(v3)) << 16)};
      }
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) a[ks] = an[ks];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) old[tb] = on[tb];
  }
}

// Partial dW1 of token range s over a 64-column slab: D[j][c] =
// sum_t dz^T[j][t] x[t][c], k = 32 tokens per step. Wave w takes columns
// 16 w .. 16 w + 15 of the slab and every unit block. The x tile [32 tokens,
// 64 columns] is loaded one step ahead into registers and transposed through
// LDS (double buffered); the dz^T operands come straight from the workspace.
template <int DR>
__global__ __launch_bounds__(256) void router_bwd_w1_bf16_kernel(const uint16_t* __restrict__ x, int64_t n, int d,
                                                                 const uint16_t* __restrict__ dzt_hi,
                                                                 const uint16_t* __restrict__ dzt_lo, int64_t npad,
                                                                 int splits, float* __restrict__ pw1) {
  constexpr int NJ = DR / 16, P = 68;  // LDS row pitch in bf16 (136 bytes: spreads the column reads over banks)
  __shared__ __align__(16) uint16_t xt[2][32 * P];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int c0 = blockIdx.x * 64;
  const int s = blockIdx.y;
  const int64_t nk = (n + 31) / 32;
  const int64_t k0 = nk * s / splits, k1 = nk * (s + 1) / splits;
  const int lr = threadIdx.x >> 3, lc = (threadIdx.x & 7) * 8;
  auto load_tile = [&](int64_t kt) -> u32x4 {
    const int64_t t = kt * 32 + lr;
    const int c = c0 + lc;
    return (t < n && c < d) ? *reinterpret_cast<const u32x4*>(x + t * d + c) : u32x4{0u, 0u, 0u, 0u};
  };
  f32x4 acc[NJ];
#pragma unroll
  for (int jb = 0; jb < NJ; ++jb) acc[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // dz^T operands of step kt: rows j = 16 jb + r, tokens 32 kt + 8 g .. + 7
  // (inside the padded row; the pad past n holds no dz and is masked)
  auto load_dz = [&](int64_t kt, bf16x8 (&ah)[NJ], bf16x8 (&al)[NJ]) {
    const int64_t t8 = kt * 32 + 8 * g;
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb) {
      const int64_t off = int64_t(16 * jb + r) * npad + t8;
      ah[jb] = *reinterpret_cast<const bf16x8*>(dzt_hi + off);
      al[jb] = *reinterpret_cast<const bf16x8*>(dzt_lo + off);
      if (t8 + 8 > n) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (t8 + i >= n) ah[jb][i] = al[jb][i] = (__bf16)0.f;
      }
    }
  };
  u32x4 nxt = k0 < k1 ? load_tile(k0) : u32x4{0u, 0u, 0u, 0u};
  bf16x8 ah[NJ], al[NJ], ahn[NJ], aln[NJ];
  if (k0 < k1) load_dz(k0, ah, al);
  for (int64_t kt = k0; kt < k1; ++kt) {
    uint16_t* buf = xt[(kt - k0) & 1];
    *reinterpret_cast<u32x2*>(buf + lr * P + lc) = u32x2{nxt[0], nxt[1]};
    *reinterpret_cast<u32x2*>(buf + lr * P + lc + 4) = u32x2{nxt[2], nxt[3]};
    __syncthreads();
    if (kt + 1 < k1) {
      nxt = load_tile(kt + 1);
      load_dz(kt + 1, ahn, aln);
    }
    bf16x8 bx;
#pragma unroll
    for (int i = 0; i < 8; ++i) bx[i] = __builtin_bit_cast(__bf16, buf[(8 * g + i) * P + 16 * w + r]);
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb) {
      acc[jb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[jb], bx, acc[jb], 0, 0, 0);
      acc[jb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[jb], bx, acc[jb], 0, 0, 0);
    }
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb) {
      ah[jb] = ahn[jb];
      al[jb] = aln[jb];
    }
  }
  // lane holds D[j = 16 jb + 4 g + i][c = c0 + 16 w + r]
  const int c = c0 + 16 * w + r;
  if (c >= d) return;
#pragma unroll
  for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
    for (int i = 0; i < 4; ++i) pw1[(int64_t(s) * DR + 16 * jb + 4 * g + i) * d + c] = acc[jb][i];
}

// ---- fp32 on the vector ALUs

template <int DR>
__global__ __launch_bounds__(64 * kRouterWaves) void router_bwd_tokens_f32_kernel(
    const float* __restrict__ x, int64_t n, int d, const float* __restrict__ w1, const float* __restrict__ b1,
    const float* __restrict__ w2, const float* __restrict__ ds, float* __restrict__ dx, float* __restrict__ dz,
    float* __restrict__ terms) {
  constexpr int NT = 64 * kRouterWaves, TM = kRouterTokens;
  __shared__ RouterPart<DR> part;
  __shared__ __align__(16) float dzs[TM][DR];
  __shared__ float ssum[TM];
  const int64_t row0 = int64_t(blockIdx.x) * TM;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  // one wavefront per token, as in the fp32 forward; z (bias included) goes to part[0]
  for (int t = w; t < TM; t += kRouterWaves) {
    const int64_t row = row0 + t < n ? row0 + t : n - 1;
    for (int j = 0; j < DR; ++j) {
      const float h = router_hidden_f32(x + row * d, d, w1, b1, j, lane);
      if (lane == 0) part[0][t][j] = h;
    }
  }
  __syncthreads();
  router_bwd_chunk<float, DR, DR>(part, dzs, ssum, b1, w2, ds, n, row0, terms);
  for (int e = threadIdx.x; e < TM * DR; e += NT) {
    const int t = e / DR;
    if (row0 + t < n) dz[row0 * DR + e] = dzs[t][e - t * DR];
  }
  if (!dx) return;
  // dx[t, c:c+2] += sum_j dz[t, j] W1[j, c:c+2], two columns per thread
  const int tmax = n - row0 < TM ? int(n - row0) : TM;
  for (int c = 2 * threadIdx.x; c < d; c += 2 * NT) {
    float wa[DR], wb[DR];
#pragma unroll
    for (int j = 0; j < DR; ++j) {
      wa[j] = w1[int64_t(j) * d + c];
      wb[j] = w1[int64_t(j) * d + c + 1];
    }
    for (int t = 0; t < tmax; ++t) {
      float a = 0.f, b = 0.f;
#pragma unroll
      for (int j = 0; j < DR; ++j) {
        a = fmaf(dzs[t][j], wa[j], a);
        b = fmaf(dzs[t][j], wb[j], b);
      }
      float2* p = reinterpret_cast<float2*>(dx + (row0 + t) * d + c);
      float2 v = *p;
      v.x += a;
      v.y += b;
      *p = v;
    }
  }
}

// pw1[s][j][c] = sum over token range s of dz[t, j] x[t, c]; wave w holds
// units w DR/4 .. (w+1) DR/4, each lane two adjacent columns of a 128-column
// slab. A token's dz values are the same for the whole wave (scalar loads).
template <int DR>
__global__ __launch_bounds__(256) void router_bwd_w1_f32_kernel(const float* __restrict__ x, int64_t n, int d,
                                                                const float* __restrict__ dz, int splits,
                                                                float* __restrict__ pw1) {
  constexpr int U = DR / 4;
  const int w = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;
  const int c = blockIdx.x * 128 + 2 * lane;
  const int s = blockIdx.y;
  const int64_t t0 = n * s / splits, t1 = n * (s + 1) / splits;
  if (c >= d) return;
  float a0[U], a1[U];
#pragma unroll
  for (int u = 0; u < U; ++u) a0[u] = a1[u] = 0.f;
  for (int64_t t = t0; t < t1; ++t) {
    const float2 xv = *reinterpret_cast<const float2*>(x + t * d + c);
    const float* zr = dz + t * DR + w * U;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      a0[u] = fmaf(zr[u], xv.x, a0[u]);
      a1[u] = fmaf(zr[u], xv.y, a1[u]);
    }
  }
  float* out = pw1 + (int64_t(s) * DR + w * U) * d + c;
#pragma unroll
  for (int u = 0; u < U; ++u) *reinterpret_cast<float2*>(out + int64_t(u) * d) = float2{a0[u], a1[u]};
}

// ---- fixed-order reductions (both dtypes)

// Blocks [0, nbw): 64 outputs of dW1 each; wave q adds splits q, q + 4, ...
// in ascending order and the four wave sums meet in LDS in wave order. Then
// one wavefront per chunk term j: lanes take chunks lane, lane + 64, ... in
// order, and the lanes meet in a fixed butterfly.
template <int DR>
__global__ __launch_bounds__(256) void router_bwd_reduce_kernel(const float* __restrict__ pw1, int splits, int d,
                                                                const float* __restrict__ terms, int64_t chunks,
                                                                float* __restrict__ dw1, float* __restrict__ db1,
                                                                float* __restrict__ dw2, float* __restrict__ db2) {
  __shared__ float red[4][64];
  const int64_t nw = int64_t(DR) * d;
  const int64_t nbw = (nw + 63) / 64;
  const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
  if (blockIdx.x < nbw) {
    const int64_t i = int64_t(blockIdx.x) * 64 + lane;
    float a = 0.f;
    if (i < nw) {
      float v[kBwdMaxSplits / 4];  // at most splits / 4 per wave, all requested before the adds
#pragma unroll
      for (int u = 0; u < kBwdMaxSplits / 4; ++u) {
        const int s = q + 4 * u;
        v[u] = s < splits ? pw1[int64_t(s) * nw + i] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kBwdMaxSplits / 4; ++u) a += v[u];
    }
    red[q][lane] = a;
    __syncthreads();
    if (q == 0 && i < nw) dw1[i] = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
    return;
  }
  const int j = int(blockIdx.x - nbw) * 4 + q;
  if (j >= kBwdTerms * DR + 1) return;
  float a = 0.f;
  for (int64_t ch = lane; ch < chunks; ch += 64) a += terms[ch * (kBwdTerms * DR + 1) + j];
  a = wave_sum(a);
  if (lane != 0) return;
  if (j < DR) {
    if (db1) db1[j] = a;
  } else if (j < 2 * DR) {
    dw2[j - DR] = a;
  } else {
    *db2 = a;
  }
}

template <int DR>
static void launch_router_bwd_t(const RouterBwdArgs& a, hipStream_t s) {
  const BwdLayout L = bwd_layout(a.n, a.d, DR);
  char* ws = static_cast<char*>(a.workspace);
  float* terms = reinterpret_cast<float*>(ws + L.terms);
  float* pw1 = reinterpret_cast<float*>(ws + L.pw1);
  const unsigned chunks = unsigned(L.chunks);
  if (a.dtype == DSF_BF16) {
    uint16_t* w1t = reinterpret_cast<uint16_t*>(ws + L.w1t);
    uint16_t* dzt_hi = reinterpret_cast<uint16_t*>(ws + L.dz);
    uint16_t* dzt_lo = dzt_hi + int64_t(DR) * L.npad;
    if (a.dx)
      router_w1t_kernel<DR><<<unsigned((int64_t(a.d) * DR + 255) / 256), 256, 0, s>>>((const uint16_t*)a.w1, a.d, w1t);
    router_bwd_tokens_bf16_kernel<DR><<<chunks, 64 * kRouterWaves, 0, s>>>(
        (const uint16_t*)a.x, a.n, a.d, (const uint16_t*)a.w1, w1t, (const uint16_t*)a.b1, (const uint16_t*)a.w2,
        a.dscore, (uint16_t*)a.dx, dzt_hi, dzt_lo, L.npad, terms);
    router_bwd_w1_bf16_kernel<DR><<<dim3(unsigned((a.d + 63) / 64), unsigned(L.splits)), 256, 0, s>>>(
        (const uint16_t*)a.x, a.n, a.d, dzt_hi, dzt_lo, L.npad, L.splits, pw1);
  } else {
    float* dz = reinterpret_cast<float*>(ws + L.dz);
    router_bwd_tokens_f32_kernel<DR><<<chunks, 64 * kRouterWaves, 0, s>>>(
        (const float*)a.x, a.n, a.d, (const float*)a.w1, (const float*)a.b1, (const float*)a.w2, a.dscore,
        (float*)a.dx, dz, terms);
    router_bwd_w1_f32_kernel<DR><<<dim3(unsigned((a.d + 127) / 128), unsigned(L.splits)), 256, 0, s>>>(
        (const float*)a.x, a.n, a.d, dz, L.splits, pw1);
  }
  const int64_t nbw = (int64_t(DR) * a.d + 63) / 64;
  const int64_t nbt = (kBwdTerms * DR + 1 + 3) / 4;
  router_bwd_reduce_kernel<DR><<<unsigned(nbw + nbt), 256, 0, s>>>(pw1, L.splits, a.d, terms, L.chunks, a.dw1,
                                                                    a.db1, a.dw2, a.db2);
}

hipError_t launch_router_backward(const RouterBwdArgs& a, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_BACKWARD, s);
  switch (a.d_r) {
    case 16: launch_router_bwd_t<16>(a, s); break;
    case 32: launch_router_bwd_t<32>(a, s); break;
    case 48: launch_router_bwd_t<48>(a, s); break;
    case 64: launch_router_bwd_t<64>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dsf
