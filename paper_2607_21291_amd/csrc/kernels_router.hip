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
constexpr int kRouterTokens = 64;

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

template <int DR>
__global__ __launch_bounds__(64 * kRouterWaves) void router_bf16_kernel(const uint16_t* __restrict__ x, int64_t n, int d,
                                                                         const uint16_t* __restrict__ w1,
                                                                         const uint16_t* __restrict__ b1,
                                                                         const uint16_t* __restrict__ w2, float b2,
                                                                         float* __restrict__ scores) {
  __shared__ RouterPart<DR> part;
  const int64_t row0 = int64_t(blockIdx.x) * kRouterTokens;
  router_hidden_partials<DR>(x, n, d, w1, row0, part);
  __syncthreads();
  // threads 0..255: token t / 4, units q DR/4 .. (q + 1) DR/4 - 1 with
  // q = t % 4; the partial sums of a token are then added in a fixed order
  if (threadIdx.x >= 256) return;
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
  if (q == 0 && row0 + t < n) scores[row0 + t] = v + b2;
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
                                                         float* __restrict__ scores) {
  const int lane = threadIdx.x & 63;
  const int64_t t = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (t >= n) return;
  const float* row = x + t * d;
  float score = 0.f;
  for (int j = 0; j < dr; ++j) {
    const float h = router_hidden_f32(row, d, w1, b1, j, lane);
    score = fmaf(w2[j], h > 0.f ? h : 0.f, score);
  }
  if (lane == 0) scores[t] = score + b2;
}

hipError_t launch_router(int dtype, const void* x, int64_t n, int d, int d_r, const void* w1,
                         const void* b1, const void* w2, float b2, float* scores, hipStream_t s) {
  if (n == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_ROUTER, s);
  if (dtype == DSF_F32) {
    router_f32_kernel<<<unsigned((n + 3) / 4), 256, 0, s>>>((const float*)x, n, d, d_r, (const float*)w1,
                                                            (const float*)b1, (const float*)w2, b2, scores);
    return hipGetLastError();
  }
  unsigned grid = unsigned((n + kRouterTokens - 1) / kRouterTokens);
  auto X = (const uint16_t*)x;
  auto W1 = (const uint16_t*)w1;
  auto B1 = (const uint16_t*)b1;
  auto W2 = (const uint16_t*)w2;
  switch (d_r) {
    case 16: router_bf16_kernel<16><<<grid, 64 * kRouterWaves, 0, s>>>(X, n, d, W1, B1, W2, b2, scores); break;
    case 32: router_bf16_kernel<32><<<grid, 64 * kRouterWaves, 0, s>>>(X, n, d, W1, B1, W2, b2, scores); break;
    case 48: router_bf16_kernel<48><<<grid, 64 * kRouterWaves, 0, s>>>(X, n, d, W1, B1, W2, b2, scores); break;
    case 64: router_bf16_kernel<64><<<grid, 64 * kRouterWaves, 0, s>>>(X, n, d, W1, B1, W2, b2, scores); break;
    default: return hipErrorInvalidValue;
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

hipError_t launch_gate_grad(int dtype, const void* dy, const void* x_in, const void* x_out, const float* scores,
                            const int32_t* idx, int B, int Tn, int k, int d, float* dscore, hipStream_t s) {
  if (int64_t(B) * Tn == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_BACKWARD, s);
  hipError_t e = launch_zero_u32(reinterpret_cast<uint32_t*>(dscore), int64_t(B) * Tn, s);
  if (e != hipSuccess || k == 0) return e;
  const unsigned grid = unsigned((int64_t(B) * k + 3) / 4);
  if (dtype == DSF_BF16)
    gate_grad_kernel<uint16_t><<<grid, 256, 0, s>>>((const uint16_t*)dy, (const uint16_t*)x_in,
                                                   (const uint16_t*)x_out, scores, idx, B, Tn, k, d, dscore);
  else
    gate_grad_kernel<float><<<grid, 256, 0, s>>>((const float*)dy, (const float*)x_in, (const float*)x_out, scores,
                                                idx, B, Tn, k, d, dscore);
  return hipGetLastError();
}

// ------------------------------------------ router backward (Sec. 3.4)

// With z = W1 x + b1 and s = w2 . ReLU(z) + b2, and ds = dL/ds per token:
//   dz = ds * w2 * [z > 0]          dW1 = sum_t dz_t x_t^T    db1 = sum_t dz_t
//   dw2 = sum_t ds_t ReLU(z_t)       db2 = sum_t ds_t          dx_t = W1^T dz_t
// Three launches:
//   tokens: per 64-token chunk, recompute z (same arithmetic and order as the
//     forward, hence the same ReLU decisions), write dz [n, DR], the chunk's
//     sums of dz, ds ReLU(z) and ds, and add W1^T dz into dx;
//   weights: dW1 partials over (128-column slab, token range);
//   reduce: the partials in fixed order into dW1, db1, dw2, db2.

constexpr int kBwdTerms = 2;  // per-chunk sums: dz (db1) and ds ReLU(z) (dw2), then ds (db2)

template <int DR>
constexpr int bwd_terms_per_chunk() { return kBwdTerms * DR + 1; }

int router_bwd_splits(int64_t n) {
  const int64_t s = n / 256;
  return int(s < 1 ? 1 : (s > 64 ? 64 : s));
}

size_t router_bwd_workspace_bytes(int64_t n, int d, int d_r) {
  auto up = [](size_t b) { return (b + 255) / 256 * 256; };
  const int64_t chunks = (n + kRouterTokens - 1) / kRouterTokens;
  return up(sizeof(float) * size_t(n) * d_r) + up(sizeof(float) * size_t(chunks) * (kBwdTerms * d_r + 1)) +
         up(sizeof(float) * size_t(router_bwd_splits(n)) * d_r * d);
}

template <typename T, int DR>
__global__ __launch_bounds__(64 * kRouterWaves) void router_bwd_tokens_kernel(
    const T* __restrict__ x, int64_t n, int d, const T* __restrict__ w1, const T* __restrict__ b1,
    const T* __restrict__ w2, const float* __restrict__ ds, T* __restrict__ dx, float* __restrict__ dz,
    float* __restrict__ terms) {
  constexpr int NT = 64 * kRouterWaves, TM = kRouterTokens;
  __shared__ RouterPart<DR> part;
  __shared__ __align__(16) float dzs[TM][DR];
  __shared__ float ssum[TM];
  const int64_t row0 = int64_t(blockIdx.x) * TM;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if constexpr (sizeof(T) == 2) {
    router_hidden_partials<DR>(x, n, d, w1, row0, part);
  } else {
    // one wavefront per token, as in the fp32 forward; the full sum (bias
    // included) goes to part[0]
    for (int t = w; t < TM; t += kRouterWaves) {
      const int64_t row = row0 + t < n ? row0 + t : n - 1;
      for (int j = 0; j < DR; ++j) {
        const float h = router_hidden_f32(x + row * d, d, w1, b1, j, lane);
        if (lane == 0) part[0][t][j] = h;
      }
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < TM * DR; e += NT) {
    const int t = e / DR, j = e - t * DR;
    float h;
    if constexpr (sizeof(T) == 2) h = router_hidden<DR>(part, b1, t, j);
    else h = part[0][t][j];
    const float sv = row0 + t < n ? ds[row0 + t] : 0.f;
    const bool on = h > 0.f;
    const float g = on ? sv * Elem<T>::to_f(w2[j]) : 0.f;
    dzs[t][j] = g;
    part[1][t][j] = on ? sv * h : 0.f;  // only this thread reads or writes entry (t, j)
    if (j == 0) ssum[t] = sv;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < TM * DR; e += NT) {
    const int t = e / DR;
    if (row0 + t < n) dz[row0 * DR + e] = dzs[t][e - t * DR];
  }
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
  if (!dx) return;
  // dx[t, c:c+2] += sum_j dz[t, j] W1[j, c:c+2], two columns per thread
  const int tmax = n - row0 < TM ? int(n - row0) : TM;
  for (int c = 2 * threadIdx.x; c < d; c += 2 * NT) {
    float wa[DR], wb[DR];
#pragma unroll
    for (int j = 0; j < DR; ++j) {
      wa[j] = Elem<T>::to_f(w1[int64_t(j) * d + c]);
      wb[j] = Elem<T>::to_f(w1[int64_t(j) * d + c + 1]);
    }
    for (int t = 0; t < tmax; ++t) {
      float a = 0.f, b = 0.f;
#pragma unroll
      for (int j = 0; j < DR; j += 4) {
        const float4 z4 = *reinterpret_cast<const float4*>(&dzs[t][j]);
        a = fmaf(z4.x, wa[j], a);
        b = fmaf(z4.x, wb[j], b);
        a = fmaf(z4.y, wa[j + 1], a);
        b = fmaf(z4.y, wb[j + 1], b);
        a = fmaf(z4.z, wa[j + 2], a);
        b = fmaf(z4.z, wb[j + 2], b);
        a = fmaf(z4.w, wa[j + 3], a);
        b = fmaf(z4.w, wb[j + 3], b);
      }
      T* p = dx + (row0 + t) * d + c;
      if constexpr (sizeof(T) == 2) {
        uint32_t v = *reinterpret_cast<const uint32_t*>(p);
        const float lo = bf2f(uint16_t(v & 0xffffu)) + a, hi = bf2f(uint16_t(v >> 16)) + b;
        *reinterpret_cast<uint32_t*>(p) = uint32_t(f2bf(lo)) | (uint32_t(f2bf(hi)) << 16);
      } else {
        float2 v = *reinterpret_cast<const float2*>(p);
        v.x += a;
        v.y += b;
        *reinterpret_cast<float2*>(p) = v;
      }
    }
  }
}

// dW1 partial of token range s: pw1[s][j][c] = sum_t dz[t, j] x[t, c]. A
// workgroup covers a 128-column slab: wave w holds units w DR/4 .. (w+1) DR/4,
// each lane two adjacent columns. The units' dz values of a token are the
// same for the whole wave and come through the scalar cache.
template <typename T, int DR>
__global__ __launch_bounds__(256) void router_bwd_w1_kernel(const T* __restrict__ x, int64_t n, int d,
                                                            const float* __restrict__ dz, int splits,
                                                            float* __restrict__ pw1) {
  constexpr int U = DR / 4, UNR = 8;
  const int w = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;
  const int c = blockIdx.x * 128 + 2 * lane;
  const int s = blockIdx.y;
  const int64_t t0 = n * s / splits, t1 = n * (s + 1) / splits;
  if (c >= d) return;
  float a0[U], a1[U];
#pragma unroll
  for (int u = 0; u < U; ++u) a0[u] = a1[u] = 0.f;
  int64_t t = t0;
  for (; t + UNR <= t1; t += UNR) {
    float xv[UNR][2];
#pragma unroll
    for (int q = 0; q < UNR; ++q) {
      const T* p = x + (t + q) * d + c;
      if constexpr (sizeof(T) == 2) {
        const uint32_t v = *reinterpret_cast<const uint32_t*>(p);
        xv[q][0] = bf2f(uint16_t(v & 0xffffu));
        xv[q][1] = bf2f(uint16_t(v >> 16));
      } else {
        const float2 v = *reinterpret_cast<const float2*>(p);
        xv[q][0] = v.x;
        xv[q][1] = v.y;
      }
    }
#pragma unroll
    for (int q = 0; q < UNR; ++q) {
      const float* zr = dz + (t + q) * DR + w * U;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        a0[u] = fmaf(zr[u], xv[q][0], a0[u]);
        a1[u] = fmaf(zr[u], xv[q][1], a1[u]);
      }
    }
  }
  for (; t < t1; ++t) {
    const T* p = x + t * d + c;
    const float x0 = Elem<T>::to_f(p[0]), x1 = Elem<T>::to_f(p[1]);
    const float* zr = dz + t * DR + w * U;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      a0[u] = fmaf(zr[u], x0, a0[u]);
      a1[u] = fmaf(zr[u], x1, a1[u]);
    }
  }
  float* out = pw1 + (int64_t(s) * DR + w * U) * d + c;
#pragma unroll
  for (int u = 0; u < U; ++u) *reinterpret_cast<float2*>(out + int64_t(u) * d) = float2{a0[u], a1[u]};
}

// Fixed-order sums of the partials: dW1 over token ranges, the per-chunk
// terms over chunks.
template <int DR>
__global__ __launch_bounds__(256) void router_bwd_reduce_kernel(const float* __restrict__ pw1, int splits, int d,
                                                                const float* __restrict__ terms, int64_t chunks,
                                                                float* __restrict__ dw1, float* __restrict__ db1,
                                                                float* __restrict__ dw2, float* __restrict__ db2) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int64_t nw = int64_t(DR) * d;
  if (i < nw) {
    float a = 0.f;
    for (int s = 0; s < splits; ++s) a += pw1[int64_t(s) * nw + i];
    dw1[i] = a;
    return;
  }
  const int j = int(i - nw);
  if (j >= kBwdTerms * DR + 1) return;
  float a = 0.f;
  for (int64_t ch = 0; ch < chunks; ++ch) a += terms[ch * (kBwdTerms * DR + 1) + j];
  if (j < DR) {
    if (db1) db1[j] = a;
  } else if (j < 2 * DR) {
    dw2[j - DR] = a;
  } else {
    *db2 = a;
  }
}

template <typename T, int DR>
static void launch_router_bwd_t(const RouterBwdArgs& a, hipStream_t s) {
  const int64_t chunks = (a.n + kRouterTokens - 1) / kRouterTokens;
  const int splits = router_bwd_splits(a.n);
  char* ws = static_cast<char*>(a.workspace);
  auto up = [](size_t b) { return (b + 255) / 256 * 256; };
  float* dz = reinterpret_cast<float*>(ws);
  float* terms = reinterpret_cast<float*>(ws + up(sizeof(float) * size_t(a.n) * DR));
  float* pw1 = reinterpret_cast<float*>(ws + up(sizeof(float) * size_t(a.n) * DR) +
                                        up(sizeof(float) * size_t(chunks) * (kBwdTerms * DR + 1)));
  router_bwd_tokens_kernel<T, DR><<<unsigned(chunks), 64 * kRouterWaves, 0, s>>>(
      (const T*)a.x, a.n, a.d, (const T*)a.w1, (const T*)a.b1, (const T*)a.w2, a.dscore, (T*)a.dx, dz, terms);
  router_bwd_w1_kernel<T, DR><<<dim3(unsigned((a.d + 127) / 128), unsigned(splits)), 256, 0, s>>>(
      (const T*)a.x, a.n, a.d, dz, splits, pw1);
  const int64_t outs = int64_t(DR) * a.d + kBwdTerms * DR + 1;
  router_bwd_reduce_kernel<DR><<<unsigned((outs + 255) / 256), 256, 0, s>>>(pw1, splits, a.d, terms, chunks, a.dw1,
                                                                            a.db1, a.dw2, a.db2);
}

hipError_t launch_router_backward(const RouterBwdArgs& a, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_BACKWARD, s);
  const bool bf = a.dtype == DSF_BF16;
  switch (a.d_r) {
    case 16: bf ? launch_router_bwd_t<uint16_t, 16>(a, s) : launch_router_bwd_t<float, 16>(a, s); break;
    case 32: bf ? launch_router_bwd_t<uint16_t, 32>(a, s) : launch_router_bwd_t<float, 32>(a, s); break;
    case 48: bf ? launch_router_bwd_t<uint16_t, 48>(a, s) : launch_router_bwd_t<float, 48>(a, s); break;
    case 64: bf ? launch_router_bwd_t<uint16_t, 64>(a, s) : launch_router_bwd_t<float, 64>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dsf
