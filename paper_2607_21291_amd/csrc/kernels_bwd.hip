// Backward of the routed layer (the training side of Section 3.4) on gfx950:
// the kernels of the block's adjoint on the kept rows that are not projection
// GEMMs (those run on the forward's GEMM kernels with backward epilogues).
//
//   - transposes of [rows, cols] bf16 matrices (weights, and activations
//     whose token dimension becomes the reduction of a weight gradient),
//     optionally applying the forward activation on the way (GELU of the up
//     projection, or SiLU(gate) * up);
//   - column sums in a fixed order (bias and norm-gain gradients);
//   - gather of the output gradient at the kept rows, scaled by the gate;
//   - LayerNorm / RMSNorm adjoints of one row per wavefront;
//   - the RoPE adjoint with the head-major -> token-major relayout of q/k/v;
//   - causal attention backward over the kept tokens in two passes, both on
//     v_mfma_f32_16x16x32_bf16 and both deterministic (no atomics): one pass
//     per query block for dQ (and the softmax statistics), one per key block
//     for dK and dV, which adds the query heads of a GQA group in order;
//   - the final scatter: dx = dy, plus the block's gradient at the kept rows.
#include <hip/hip_ext.h>

#include "attn_tiles.h"
#include "dsf_device.h"
#include "dsf_internal.h"

namespace dsf {

// ----------------------------------------------------------- transposes

// out[c][r] = op(in[r][c]) for r < R, c < C; out has leading dimension ldo
// >= R and its columns R .. ldo-1 are written as zeros (so that a token
// count padded to a multiple of 64 can be a GEMM reduction). op: 0 copy,
// 1 GELU, 2 SiLU(in[r][c]) * in[r][C + c] (SwiGLU of a [R, 2C] gate|up row).
template <int OP>
__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ in, int R, int C, int ldi,
                                                        uint16_t* __restrict__ out, int ldo) {
  __shared__ float tile[64][65];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int rr = ty; rr < 64; rr += 4) {
    const int r = r0 + rr, c = c0 + tx;
    float v = 0.f;
    if (r < R && c < C) {
      const int64_t o = int64_t(r) * ldi + c;
      v = bf2f(in[o]);
      if constexpr (OP == 1) v = gelu_bf16(v);
      if constexpr (OP == 2) v = silu_bf16(v) * bf2f(in[o + C]);
    }
    tile[rr][tx] = v;
  }
  __syncthreads();
  for (int cc = ty; cc < 64; cc += 4) {
    const int c = c0 + cc, r = r0 + tx;
    if (c < C && r < ldo) out[int64_t(c) * ldo + r] = f2bf(tile[tx][cc]);
  }
}

// The same with 16-byte accesses on both sides (C, ldi and ldo multiples of
// 8, 16-byte aligned bases): a thread loads 8 columns of an input row and
// stores 8 rows of an output row.
template <int OP>
__global__ __launch_bounds__(256) void transpose_vec_kernel(const uint16_t* __restrict__ in, int R, int C, int ldi,
                                                            uint16_t* __restrict__ out, int ldo) {
  __shared__ float tile[64][65];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
  const int t = threadIdx.x, v = t & 7, q = t >> 3;  // vector index, row (column) within a pass
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int rr = q + 32 * i, r = r0 + rr, c = c0 + 8 * v;
    float x[8];
    if (r < R && c < C) {
      const int64_t o = int64_t(r) * ldi + c;
      const u32x4 raw = *reinterpret_cast<const u32x4*>(in + o);
      u32x4 up{};
      if constexpr (OP == 2) up = *reinterpret_cast<const u32x4*>(in + o + C);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[2 * e] = __uint_as_float(raw[e] << 16);
        x[2 * e + 1] = __uint_as_float(raw[e] & 0xffff0000u);
        if constexpr (OP == 1) {
          x[2 * e] = gelu_bf16(x[2 * e]);
          x[2 * e + 1] = gelu_bf16(x[2 * e + 1]);
        }
        if constexpr (OP == 2) {
          x[2 * e] = silu_bf16(x[2 * e]) * __uint_as_float(up[e] << 16);
          x[2 * e + 1] = silu_bf16(x[2 * e + 1]) * __uint_as_float(up[e] & 0xffff0000u);
        }
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = 0.f;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) tile[rr][8 * v + e] = x[e];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int cc = q + 32 * i, c = c0 + cc, r = r0 + 8 * v;
    if (c < C && r < ldo) {
      u32x4 pk;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        pk[e] = uint32_t(f2bf(tile[8 * v + 2 * e][cc])) | (uint32_t(f2bf(tile[8 * v + 2 * e + 1][cc])) << 16);
      *reinterpret_cast<u32x4*>(out + int64_t(c) * ldo + r) = pk;
    }
  }
}

hipError_t launch_transpose(int op, const void* in, int R, int C, int ldi, void* out, int ldo, hipStream_t s) {
  if (R <= 0 || C <= 0) return hipSuccess;
  const dim3 grid((C + 63) / 64, (ldo + 63) / 64);
  const auto* i = (const uint16_t*)in;
  auto* o = (uint16_t*)out;
  const bool vec = C % 8 == 0 && ldi % 8 == 0 && ldo % 8 == 0 && reinterpret_cast<uintptr_t>(in) % 16 == 0 &&
                   reinterpret_cast<uintptr_t>(out) % 16 == 0;
  if (vec) {
    if (op == 0) transpose_vec_kernel<0><<<grid, 256, 0, s>>>(i, R, C, ldi, o, ldo);
    else if (op == 1) transpose_vec_kernel<1><<<grid, 256, 0, s>>>(i, R, C, ldi, o, ldo);
    else transpose_vec_kernel<2><<<grid, 256, 0, s>>>(i, R, C, ldi, o, ldo);
  } else {
    if (op == 0) transpose_kernel<0><<<grid, 256, 0, s>>>(i, R, C, ldi, o, ldo);
    else if (op == 1) transpose_kernel<1><<<grid, 256, 0, s>>>(i, R, C, ldi, o, ldo);
    else transpose_kernel<2><<<grid, 256, 0, s>>>(i, R, C, ldi, o, ldo);
  }
  return hipGetLastError();
}

// ----------------------------------------------------------- column sums

// partial[chunk][c] = sum over the kColRows rows of chunk of a[r][c]
// (xhat == null) or a[r][c] * (x[r][c] - mean[r]) * rstd[r]; then out[c] =
// sum over chunks in order. With 16-byte rows (C, lda multiples of 8, aligned
// bases) a workgroup is 32 column vectors of 8 columns by 8 row lanes: row
// lane j adds rows j, j + 8, ... of the chunk in order, then the 8 lane sums
// are added in lane order. Otherwise a thread adds one column's rows in
// order. Every order is fixed by the shape.
constexpr int kColRows = 256;
constexpr int kColLanes = 8;

__global__ __launch_bounds__(256) void colsum_partial_vec_kernel(const uint16_t* __restrict__ a, int R, int C,
                                                                 int lda, const uint16_t* __restrict__ x,
                                                                 const float* __restrict__ mean,
                                                                 const float* __restrict__ rstd,
                                                                 float* __restrict__ partial) {
  __shared__ float red[kColLanes][32 * 8 + 4];
  const int cv = threadIdx.x & 31, rl = threadIdx.x >> 5;
  const int c0 = (blockIdx.x * 32 + cv) * 8;
  const int r0 = blockIdx.y * kColRows, r1 = min(R, r0 + kColRows);
  float s[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) s[e] = 0.f;
  if (c0 < C) {
    constexpr int U = 4;  // rows of this lane loaded before they are added
    for (int rb = r0 + rl; rb < r1; rb += U * kColLanes) {
      u32x4 va[U], vx[U];
      float mu[U], rs[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = rb + u * kColLanes;
        if (r < r1) {
          va[u] = *reinterpret_cast<const u32x4*>(a + int64_t(r) * lda + c0);
          if (x) {
            vx[u] = *reinterpret_cast<const u32x4*>(x + int64_t(r) * lda + c0);
            mu[u] = mean ? mean[r] : 0.f;
            rs[u] = rstd[r];
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (rb + u * kColLanes < r1) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const uint32_t wa = va[u][e >> 1];
            float v = __uint_as_float((e & 1) ? (wa & 0xffff0000u) : (wa << 16));
            if (x) {
              const uint32_t wx = vx[u][e >> 1];
              v *= (__uint_as_float((e & 1) ? (wx & 0xffff0000u) : (wx << 16)) - mu[u]) * rs[u];
            }
            s[e] += v;
          }
        }
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[rl][cv * 8 + e] = s[e];
  __syncthreads();
  // thread t sums column t of the workgroup's 256 over the lanes in order
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c < C) {
    float t = 0.f;
#pragma unroll
    for (int l = 0; l < kColLanes; ++l) t += red[l][threadIdx.x];
    partial[int64_t(blockIdx.y) * C + c] = t;
  }
}

__global__ __launch_bounds__(256) void colsum_partial_kernel(const uint16_t* __restrict__ a, int R, int C, int lda,
                                                             const uint16_t* __restrict__ x,
                                                             const float* __restrict__ mean,
                                                             const float* __restrict__ rstd,
                                                             float* __restrict__ partial) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int r0 = blockIdx.y * kColRows, r1 = min(R, r0 + kColRows);
  if (c >= C) return;
  float s = 0.f;
  for (int r = r0; r < r1; ++r) {
    float v = bf2f(a[int64_t(r) * lda + c]);
    if (x) v *= (bf2f(x[int64_t(r) * lda + c]) - (mean ? mean[r] : 0.f)) * rstd[r];
    s += v;
  }
  partial[int64_t(blockIdx.y) * C + c] = s;
}

__global__ __launch_bounds__(256) void colsum_final_kernel(const float* __restrict__ partial, int chunks, int C,
                                                           float* __restrict__ out) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  float s = 0.f;
  constexpr int U = 8;  // partials loaded before they are added (in order)
  for (int k = 0; k < chunks; k += U) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (k + u < chunks) v[u] = partial[int64_t(k + u) * C + c];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (k + u < chunks) s += v[u];
  }
  out[c] = s;
}

int colsum_chunks(int R) { return (R + kColRows - 1) / kColRows; }

hipError_t launch_colsum(const void* a, int R, int C, int lda, const void* x, const float* mean, const float* rstd,
                         float* partial, float* out, hipStream_t s) {
  if (C <= 0) return hipSuccess;
  const int chunks = colsum_chunks(R);
  const bool vec = C % 8 == 0 && lda % 8 == 0 && reinterpret_cast<uintptr_t>(a) % 16 == 0 &&
                   (!x || reinterpret_cast<uintptr_t>(x) % 16 == 0);
  if (chunks > 0) {
    const uint16_t *ap = (const uint16_t*)a, *xp = (const uint16_t*)x;
    const dim3 grid((C + 255) / 256, chunks);
    if (vec) colsum_partial_vec_kernel<<<grid, 256, 0, s>>>(ap, R, C, lda, xp, mean, rstd, partial);
    else colsum_partial_kernel<<<grid, 256, 0, s>>>(ap, R, C, lda, xp, mean, rstd, partial);
  }
  colsum_final_kernel<<<(C + 255) / 256, 256, 0, s>>>(partial, chunks, C, out);
  return hipGetLastError();
}

// ------------------------------------------------- gather of the gradient

// out[m][:] = g_m * dy[b][idx[m]][:], m = b * kk + j, with g_m = sigmoid of
// the token's router score (gate) or 1. 16-byte vectors; d % 8 == 0.
__global__ __launch_bounds__(256) void gather_scale_kernel(const uint16_t* __restrict__ dy, int T, int d,
                                                           const int32_t* __restrict__ idx, int kk, int M,
                                                           const float* __restrict__ scores,
                                                           uint16_t* __restrict__ out) {
  const int nv = d / 8;
  const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= int64_t(M) * nv) return;
  const int m = int(e / nv), c = int(e - int64_t(m) * nv) * 8;
  const int b = m / kk;
  const int p = clamp_pos(idx[m], T);
  float v[8];
  load_vec(dy + (int64_t(b) * T + p) * d + c, v);
  if (scores) {
    const float g = 1.f / (1.f + expf(-scores[int64_t(b) * T + p]));
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] *= g;
  }
  store_vec(out + int64_t(m) * d + c, v);
}

hipError_t launch_gather_scale(const void* dy, int B, int T, int d, const int32_t* idx, int kk, const float* scores,
                               void* out, hipStream_t s) {
  const int64_t n = int64_t(B) * kk * (d / 8);
  if (n == 0) return hipSuccess;
  gather_scale_kernel<<<int((n + 255) / 256), 256, 0, s>>>((const uint16_t*)dy, T, d, idx, kk, B * kk, scores,
                                                           (uint16_t*)out);
  return hipGetLastError();
}

// ------------------------------------------------------ norm adjoints

// One wavefront per row m of x [M, d] (the norm's input) and dyn [M, d] (the
// gradient at the norm's output), gain w [d]:
//   LayerNorm: xhat = (x - mean) * rstd, g = dyn * w,
//              dx = rstd * (g - mean(g) - xhat * mean(g * xhat));
//   RMSNorm:   xhat = x * rstd, dx = rstd * (g - xhat * mean(g * xhat)).
// dx goes to acc (fp32 [M, d]): acc = dx, or acc += dx with accumulate. With
// add and sum_out (both bf16 [M, d]): sum_out = add + dx (Qwen's
// d(attention output) = d(delta) + d(h)). mean/rstd of each row are kept for
// the gain gradient (a column sum over rows).
template <bool RMS>
__global__ __launch_bounds__(256) void norm_bwd_kernel(const uint16_t* __restrict__ x,
                                                       const uint16_t* __restrict__ dyn,
                                                       const uint16_t* __restrict__ w, int M, int d, float eps,
                                                       float* __restrict__ acc, int accumulate,
                                                       const uint16_t* __restrict__ add, uint16_t* __restrict__ sum_out,
                                                       float* __restrict__ mean_out, float* __restrict__ rstd_out) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= M) return;
  const uint16_t* xr = x + int64_t(m) * d;
  const uint16_t* gr = dyn + int64_t(m) * d;
  float s1 = 0.f, s2 = 0.f;
  for (int c = lane * 8; c < d; c += 512) {
    float v[8];
    load_vec(xr + c, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      s1 += v[i];
      s2 += v[i] * v[i];
    }
  }
  s1 = wave_sum(s1);
  s2 = wave_sum(s2);
  const float mean = RMS ? 0.f : s1 / float(d);
  const float var = RMS ? s2 / float(d) : fmaxf(s2 / float(d) - mean * mean, 0.f);
  const float rstd = 1.f / sqrtf(var + eps);
  float sg = 0.f, sgx = 0.f;
  for (int c = lane * 8; c < d; c += 512) {
    float v[8], g[8], wv[8];
    load_vec(xr + c, v);
    load_vec(gr + c, g);
    load_vec(w + c, wv);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float gi = g[i] * wv[i];
      sg += gi;
      sgx += gi * (v[i] - mean) * rstd;
    }
  }
  sg = wave_sum(sg) / float(d);
  sgx = wave_sum(sgx) / float(d);
  for (int c = lane * 8; c < d; c += 512) {
    float v[8], g[8], wv[8], dx[8];
    load_vec(xr + c, v);
    load_vec(gr + c, g);
    load_vec(w + c, wv);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float xh = (v[i] - mean) * rstd;
      dx[i] = rstd * (g[i] * wv[i] - (RMS ? 0.f : sg) - xh * sgx);
    }
    float* ar = acc + int64_t(m) * d + c;
    if (accumulate) {
#pragma unroll
      for (int i = 0; i < 8; ++i) ar[i] += dx[i];
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) ar[i] = dx[i];
    }
    if (sum_out) {
      float a[8];
      load_vec(add + int64_t(m) * d + c, a);
#pragma unroll
      for (int i = 0; i < 8; ++i) a[i] += dx[i];
      store_vec(sum_out + int64_t(m) * d + c, a);
    }
  }
  if (lane == 0) {
    mean_out[m] = mean;
    rstd_out[m] = rstd;
  }
}

hipError_t launch_norm_bwd(bool rms, const void* x, const void* dyn, const void* w, int M, int d, float eps, float* acc,
                           bool accumulate, const void* add, void* sum_out, float* mean, float* rstd, hipStream_t s) {
  if (M == 0) return hipSuccess;
  const dim3 grid((M + 3) / 4);
  const auto *xx = (const uint16_t*)x, *g = (const uint16_t*)dyn, *ww = (const uint16_t*)w, *ad = (const uint16_t*)add;
  if (rms)
    norm_bwd_kernel<true><<<grid, 256, 0, s>>>(xx, g, ww, M, d, eps, acc, accumulate, ad, (uint16_t*)sum_out, mean,
                                               rstd);
  else
    norm_bwd_kernel<false><<<grid, 256, 0, s>>>(xx, g, ww, M, d, eps, acc, accumulate, ad, (uint16_t*)sum_out,
                                                mean, rstd);
  return hipGetLastError();
}

// --------------------------------------------- RoPE adjoint and relayout

// dqkv[m][col] (bf16, token-major [M, (Hq + 2 Hkv) hd]) from the head-major
// fp32 gradients at the rotated q and k (and at v). A rotated pair (i,
// i + R/2) at position p was turned by the angle a = p * theta^(-2i/R); its
// gradient turns back: d_i' = d_i cos a + d_{i+R/2} sin a,
// d_{i+R/2}' = d_{i+R/2} cos a - d_i sin a. table: [T][R/2][2] (cos, sin).
__global__ __launch_bounds__(256) void rope_bwd_kernel(const float* __restrict__ dq, const float* __restrict__ dk,
                                                       const float* __restrict__ dv, const float* __restrict__ table,
                                                       const int32_t* __restrict__ idx, int kk, int T, int Hq,
                                                       int Hkv, int hd, int R, int M, uint16_t* __restrict__ out) {
  const int cols = (Hq + 2 * Hkv) * hd;
  const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= int64_t(M) * cols) return;
  const int m = int(e / cols), col = int(e - int64_t(m) * cols);
  const int b = m / kk, j = m - b * kk;
  const int p = idx ? clamp_pos(idx[m], T) : j;
  const int qc = Hq * hd, kc = Hkv * hd;
  const float* src;
  int head, dim, heads;
  bool rot = true;
  if (col < qc) {
    src = dq; heads = Hq; head = col / hd; dim = col % hd;
  } else if (col < qc + kc) {
    src = dk; heads = Hkv; head = (col - qc) / hd; dim = (col - qc) % hd;
  } else {
    src = dv; heads = Hkv; head = (col - qc - kc) / hd; dim = (col - qc - kc) % hd; rot = false;
  }
  const float* row = src + ((int64_t(b) * heads + head) * kk + j) * hd;
  float v = row[dim];
  if (rot && dim < R) {
    const int half = R / 2;
    if (dim < half) {
      const float* cs = table + (int64_t(p) * half + dim) * 2;
      v = v * cs[0] + row[dim + half] * cs[1];
    } else {
      const float* cs = table + (int64_t(p) * half + dim - half) * 2;
      v = v * cs[0] - row[dim - half] * cs[1];
    }
  }
  out[e] = f2bf(v);
}

// The same, eight columns per thread (one 16-byte store): the eight dims of
// a chunk lie in one head and, with R a multiple of 16, in one half of the
// rotated dims, so their partners and their (cos, sin) pairs are contiguous.
// The index arithmetic is done once per chunk in 32 bits (the launcher checks
// that the chunks fit) and the head dim is a power of two. Each element's
// arithmetic is the one of rope_bwd_kernel.
__global__ __launch_bounds__(256) void rope_bwd_vec_kernel(const float* __restrict__ dq, const float* __restrict__ dk,
                                                           const float* __restrict__ dv,
                                                           const float* __restrict__ table,
                                                           const int32_t* __restrict__ idx, int kk, int T, int Hq,
                                                           int Hkv, int hshift, int R, uint32_t chunks,
                                                           uint16_t* __restrict__ out) {
  const int hd = 1 << hshift;
  const uint32_t cpr = uint32_t(Hq + 2 * Hkv) << (hshift - 3);  // 8-column chunks per row
  const uint32_t e = blockIdx.x * 256u + threadIdx.x;
  if (e >= chunks) return;
  const uint32_t m = e / cpr;
  const int col0 = int(e - m * cpr) * 8;
  const int b = int(m) / kk, j = int(m) - b * kk;
  const int p = idx ? clamp_pos(idx[m], T) : j;
  const int qc = Hq << hshift, kc = Hkv << hshift;
  const float* src;
  int c = col0, heads;
  bool rot = true;
  if (c < qc) {
    src = dq; heads = Hq;
  } else if (c < qc + kc) {
    src = dk; heads = Hkv; c -= qc;
  } else {
    src = dv; heads = Hkv; c -= qc + kc; rot = false;
  }
  const int head = c >> hshift, dim0 = c & (hd - 1);
  const float* row = src + ((int64_t(b) * heads + head) * kk + j) * hd;
  float v[8];
  *reinterpret_cast<float4*>(v) = *reinterpret_cast<const float4*>(row + dim0);
  *reinterpret_cast<float4*>(v + 4) = *reinterpret_cast<const float4*>(row + dim0 + 4);
  if (rot && dim0 < R) {
    const int half = R / 2;
    const bool lo = dim0 < half;
    const float* pr = row + (lo ? dim0 + half : dim0 - half);
    float pv[8];
    *reinterpret_cast<float4*>(pv) = *reinterpret_cast<const float4*>(pr);
    *reinterpret_cast<float4*>(pv + 4) = *reinterpret_cast<const float4*>(pr + 4);
    const float4* cs = reinterpret_cast<const float4*>(table + (int64_t(p) * half + (lo ? dim0 : dim0 - half)) * 2);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 t = cs[q];
      v[2 * q] = lo ? v[2 * q] * t.x + pv[2 * q] * t.y : v[2 * q] * t.x - pv[2 * q] * t.y;
      v[2 * q + 1] = lo ? v[2 * q + 1] * t.z + pv[2 * q + 1] * t.w : v[2 * q + 1] * t.z - pv[2 * q + 1] * t.w;
    }
  }
  store_vec(out + int64_t(m) * (int64_t(cpr) * 8) + col0, v);
}

hipError_t launch_rope_bwd(const float* dq, const float* dk, const float* dv, const float* table, const int32_t* idx,
                           int B, int kk, int T, int Hq, int Hkv, int hd, int R, void* out, hipStream_t s) {
  const int64_t n = int64_t(B) * kk * (Hq + 2 * Hkv) * hd;
  if (n == 0) return hipSuccess;
  const int64_t chunks = n / 8;
  if (R % 16 == 0 && (hd & (hd - 1)) == 0 && hd >= 8 && chunks < (int64_t(1) << 31) &&
      (reinterpret_cast<uintptr_t>(out) & 15) == 0 && (reinterpret_cast<uintptr_t>(dq) & 15) == 0 &&
      (reinterpret_cast<uintptr_t>(dk) & 15) == 0 && (reinterpret_cast<uintptr_t>(dv) & 15) == 0 &&
      (reinterpret_cast<uintptr_t>(table) & 15) == 0) {
    int hshift = 0;
    while ((1 << hshift) < hd) ++hshift;
    rope_bwd_vec_kernel<<<unsigned((chunks + 255) / 256), 256, 0, s>>>(dq, dk, dv, table, idx, kk, T, Hq, Hkv, hshift,
                                                                        R, uint32_t(chunks), (uint16_t*)out);
    return hipGetLastError();
  }
  rope_bwd_kernel<<<int((n + 255) / 256), 256, 0, s>>>(dq, dk, dv, table, idx, kk, T, Hq, Hkv, hd, R, B * kk,
                                                       (uint16_t*)out);
  return hipGetLastError();
}

// ----------------------------------------------------- the final scatter

// x_grad[b][idx[m]][:] = dy[b][idx[m]][:] + acc[m][:] (fp32 add, one rounding);
// the other rows of x_grad were copied from dy before.
__global__ __launch_bounds__(256) void scatter_grad_kernel(const uint16_t* __restrict__ dy,
                                                           const float* __restrict__ acc, int T, int d,
                                                           const int32_t* __restrict__ idx, int kk, int M,
                                                           uint16_t* __restrict__ dx) {
  const int nv = d / 8;
  const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= int64_t(M) * nv) return;
  const int m = int(e / nv), c = int(e - int64_t(m) * nv) * 8;
  const int b = m / kk;
  const int64_t row = (int64_t(b) * T + clamp_pos(idx[m], T)) * d + c;
  float v[8];
  load_vec(dy + row, v);
  const float* a = acc + int64_t(m) * d + c;
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] += a[i];
  store_vec(dx + row, v);
}

hipError_t launch_scatter_grad(const void* dy, const float* acc, int B, int T, int d, const int32_t* idx, int kk,
                               void* dx, hipStream_t s) {
  const int64_t n = int64_t(B) * kk * (d / 8);
  if (n == 0) return hipSuccess;
  scatter_grad_kernel<<<int((n + 255) / 256), 256, 0, s>>>((const uint16_t*)dy, acc, T, d, idx, kk, B * kk,
                                                           (uint16_t*)dx);
  return hipGetLastError();
}

// ------------------------------------------------- attention backward

// Shapes: q [B, Hq, n, HD], k and v [B, Hkv, n, HD] (bf16, RoPE applied, as
// the forward's QKV epilogue writes them); o and dout [B n, Hq HD] (bf16,
// token-major: the attention output and its gradient); lse [B, Hq, n], the
// log of each query's softmax normaliser as the forward computed it. Query
// head h reads kv head h / (Hq / Hkv). scale = 1 / sqrt(HD).
//
// MFMA operand layout (v_mfma_f32_16x16x32_bf16): lane l supplies row l % 16
// of each operand and its 8 consecutive k slots 8 (l / 16) .. + 7; output
// element e of lane l is D[4 (l / 16) + e][l % 16]. A contraction may assign
// its 32 summed indices to the k slots in any order, the same for both
// operands: the probabilities and score gradients are used in the order a
// lane holds them after the score MFMA (index 16 blk + 4 grp + e of the two
// 16-blocks of the step), and the other operand is read with the LDS
// transpose load in that order (AttnTrans).
//
// Tiles of 64 rows go global -> LDS by buffer DMA into a ring of two stages
// (attn_tiles.h): the next tile's DMA is issued after the barrier that
// publishes the current one, and runs under its products.

constexpr int kAB = kAttnTileRows;  // queries or keys per block

__device__ __forceinline__ bf16x8 pack8(const float* v) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (__bf16)v[i];
  return r;
}

// Pass 1: one workgroup per (sequence, query head, 64-query block); wave w
// owns queries q0 + 16 w .. + 15 (lane l: query 16 w + l % 16). Scores are
// formed transposed (S^T = K Q^T, keys as MFMA rows), so a lane holds 16
// scores of its own query per 64-key block. With P = exp(S scale - lse):
// writes D = sum_c dout * o for pass 2, and dQ = scale * sum_keys dS K with
// dS = P (dP - D), dP = dout V^T.
template <int HD>
__global__ __launch_bounds__(256) void attn_bwd_dq_kernel(const uint16_t* __restrict__ Q,
                                                          const uint16_t* __restrict__ K,
                                                          const uint16_t* __restrict__ V,
                                                          const uint16_t* __restrict__ O,
                                                          const uint16_t* __restrict__ dO, int n, int Hq, int Hkv,
                                                          const float* __restrict__ lse,
                                                          float* __restrict__ dvec_out, float* __restrict__ dq_out) {
  using A = AttnTile<HD>;
  constexpr int NS = HD / 32, NC = HD / 16;
  __shared__ __attribute__((aligned(16))) char smem[2 * 2 * A::kTileBytes];  // stage: K tile, then V tile
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, grp = lane >> 4;
  const int nqb = (n + kAB - 1) / kAB;
  const int qb = blockIdx.x % nqb, bh = blockIdx.x / nqb;
  const int h = bh % Hq, b = bh / Hq, kvh = h / (Hq / Hkv);
  const int q0 = qb * kAB;
  const int query = q0 + 16 * wave + r16;
  const bool qok = query < n;
  const float scale = 1.f / sqrtf(float(HD));
  const uint16_t* Kh = K + (int64_t(b) * Hkv + kvh) * n * HD;
  const uint16_t* Vh = V + (int64_t(b) * Hkv + kvh) * n * HD;
  const int64_t orow = (int64_t(b) * n + (qok ? query : 0)) * (int64_t(Hq) * HD) + int64_t(h) * HD;
  const int nkb = qb + 1;
  auto issue = [&](int kt) {
    char* st = smem + (kt & 1) * 2 * A::kTileBytes;
    attn_tile_dma<HD>(Kh, HD, kt * kAB, n, st, wave, lane);
    attn_tile_dma<HD>(Vh, HD, kt * kAB, n, st + A::kTileBytes, wave, lane);
  };
  issue(0);

  // this lane's query as MFMA B operand: Q and dout rows, k slots 32 s + 8 grp ..
  bf16x8 qf[NS], df[NS];
  float dsum = 0.f;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    u32x4 z = {0u, 0u, 0u, 0u};
    u32x4 qv = z, dv = z, ov = z;
    if (qok) {
      qv = *reinterpret_cast<const u32x4*>(Q + ((int64_t(bh) * n + query) * HD) + 32 * s + 8 * grp);
      dv = *reinterpret_cast<const u32x4*>(dO + orow + 32 * s + 8 * grp);
      ov = *reinterpret_cast<const u32x4*>(O + orow + 32 * s + 8 * grp);
    }
    qf[s] = __builtin_bit_cast(bf16x8, qv);
    df[s] = __builtin_bit_cast(bf16x8, dv);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      dsum += __uint_as_float(dv[i] << 16) * __uint_as_float(ov[i] << 16);
      dsum += __uint_as_float(dv[i] & 0xffff0000u) * __uint_as_float(ov[i] & 0xffff0000u);
    }
  }
  const float Dq = rows4_sum(dsum);
  const float lq = qok ? lse[int64_t(bh) * n + query] : 0.f;
  if (qok && grp == 0) dvec_out[int64_t(bh) * n + query] = Dq;

  // dQ^T[c][query] = scale * sum_keys K^T[c][key] dS^T[key][query]
  const AttnTrans<HD> tr(lane);
  f32x4 acc[NC];
#pragma unroll
  for (int cb = 0; cb < NC; ++cb) acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int kt = 0; kt < nkb; ++kt) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's share of tile kt has landed
    __syncthreads();                                   // ... and every wave's; tile kt - 1 is retired
    if (kt + 1 < nkb) issue(kt + 1);
    const char* Kt = smem + (kt & 1) * 2 * A::kTileBytes;
    const char* Vt = Kt + A::kTileBytes;
    float ds[4][4];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      f32x4 st = {0.f, 0.f, 0.f, 0.f}, dp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const bf16x8 kf = attn_row_frag<HD>(Kt, 16 * blk + r16, 4 * s + grp);
        const bf16x8 vf = attn_row_frag<HD>(Vt, 16 * blk + r16, 4 * s + grp);
        st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[s], st, 0, 0, 0);
        dp = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, df[s], dp, 0, 0, 0);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = kt * kAB + 16 * blk + 4 * grp + e;
        const float p = (key <= query && key < n && qok) ? __expf(st[e] * scale - lq) : 0.f;
        ds[blk][e] = p * (dp[e] - Dq) * scale;
      }
    }
    bf16x8 dsb[2];
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] = ds[2 * s2][e];
        v[4 + e] = ds[2 * s2 + 1][e];
      }
      dsb[s2] = pack8(v);
    }
#pragma unroll
    for (int cb = 0; cb < NC; ++cb) {
      bf16x8 kt2[2];
      tr.read(Kt, cb, kt2);
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt2[s2], dsb[s2], acc[cb], 0, 0, 0);
    }
  }
  // lane holds dQ^T[16 cb + 4 grp + e][query]
  if (qok) {
    float* dst = dq_out + (int64_t(bh) * n + query) * HD;
#pragma unroll
    for (int cb = 0; cb < NC; ++cb) *reinterpret_cast<f32x4*>(dst + 16 * cb + 4 * grp) = acc[cb];
  }
}

// Pass 2: one workgroup per (sequence, kv head, 64-key block); wave w owns
// keys k0 + 16 w .. + 15 (lane l: key 16 w + l % 16). For every query head of
// the kv head's group and every query block at or after the key block (one
// work item each, in that order), scores are formed with keys as MFMA
// columns (S = Q K^T), so a lane holds the probabilities of its own key, and
//   dV^T[c][key] += sum_queries dout^T[c][query] P[query][key],
//   dK^T[c][key] += scale * sum_queries Q^T[c][query] dS[query][key].
// Each item's lse and D are loaded by wave 0 one item ahead and published in
// LDS with the item's tiles.
template <int HD>
__global__ __launch_bounds__(256) void attn_bwd_dkv_kernel(const uint16_t* __restrict__ Q,
                                                           const uint16_t* __restrict__ K,
                                                           const uint16_t* __restrict__ V,
                                                           const uint16_t* __restrict__ dO,
                                                           const float* __restrict__ lse,
                                                           const float* __restrict__ dvec, int n, int Hq, int Hkv,
                                                           float* __restrict__ dk_out, float* __restrict__ dv_out) {
  using A = AttnTile<HD>;
  constexpr int NS = HD / 32, NC = HD / 16;
  __shared__ __attribute__((aligned(16))) char smem[2 * 2 * A::kTileBytes];  // stage: Q tile, then dout tile
  __shared__ float lse_s[2][kAB], dvec_s[2][kAB];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, grp = lane >> 4;
  const int nkb = (n + kAB - 1) / kAB;
  const int kb = blockIdx.x % nkb, bkv = blockIdx.x / nkb;
  const int kvh = bkv % Hkv, b = bkv / Hkv;
  const int G = Hq / Hkv;
  const int key = kb * kAB + 16 * wave + r16;
  const bool kok = key < n;
  const float scale = 1.f / sqrtf(float(HD));
  const uint16_t* Kh = K + int64_t(bkv) * n * HD;
  const uint16_t* Vh = V + int64_t(bkv) * n * HD;
  const int nq = nkb - kb;  // query blocks at or after the key block
  const int items = G * nq;
  // item i: query head kvh G + i / nq, query block kb + i % nq
  auto issue = [&](int i) {
    const int h = kvh * G + i / nq, qb = kb + i % nq;
    const int64_t bh = int64_t(b) * Hq + h;
    char* st = smem + (i & 1) * 2 * A::kTileBytes;
    attn_tile_dma<HD>(Q + bh * n * HD, HD, qb * kAB, n, st, wave, lane);
    attn_tile_dma<HD>(dO + int64_t(b) * n * (int64_t(Hq) * HD) + int64_t(h) * HD, int64_t(Hq) * HD, qb * kAB, n,
                      st + A::kTileBytes, wave, lane);
  };
  float pl = 0.f, pd = 0.f;  // wave 0, lane = query of the next item: its lse and D
  auto fetch_stats = [&](int i) {
    const int h = kvh * G + i / nq, qq = (kb + i % nq) * kAB + lane;
    const int64_t bh = int64_t(b) * Hq + h;
    pl = qq < n ? lse[bh * n + qq] : 0.f;
    pd = qq < n ? dvec[bh * n + qq] : 0.f;
  };
  issue(0);
  if (wave == 0) fetch_stats(0);

  bf16x8 kf[NS], vf[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    u32x4 z = {0u, 0u, 0u, 0u}, kv = z, vv = z;
    if (kok) {
      kv = *reinterpret_cast<const u32x4*>(Kh + int64_t(key) * HD + 32 * s + 8 * grp);
      vv = *reinterpret_cast<const u32x4*>(Vh + int64_t(key) * HD + 32 * s + 8 * grp);
    }
    kf[s] = __builtin_bit_cast(bf16x8, kv);
    vf[s] = __builtin_bit_cast(bf16x8, vv);
  }
  const AttnTrans<HD> tr(lane);
  f32x4 adk[NC], adv[NC];
#pragma unroll
  for (int cb = 0; cb < NC; ++cb) {
    adk[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    adv[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int i = 0; i < items; ++i) {
    const int slot = i & 1;
    if (wave == 0) {  // slot's previous readers finished item i - 2 before the last barrier
      lse_s[slot][lane] = pl;
      dvec_s[slot][lane] = pd;
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's share of item i's tiles has landed
    __syncthreads();                                   // ... and every wave's; item i - 1 is retired
    if (i + 1 < items) {
      issue(i + 1);
      if (wave == 0) fetch_stats(i + 1);
    }
    const int qb = kb + i % nq;
    const char* Qt = smem + slot * 2 * A::kTileBytes;
    const char* Dt = Qt + A::kTileBytes;
    float p[4][4], ds[4][4];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      f32x4 st = {0.f, 0.f, 0.f, 0.f}, dp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const bf16x8 qa = attn_row_frag<HD>(Qt, 16 * blk + r16, 4 * s + grp);
        const bf16x8 da = attn_row_frag<HD>(Dt, 16 * blk + r16, 4 * s + grp);
        st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa, kf[s], st, 0, 0, 0);
        dp = __builtin_amdgcn_mfma_f32_16x16x32_bf16(da, vf[s], dp, 0, 0, 0);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int ql = 16 * blk + 4 * grp + e;
        const int qq = qb * kAB + ql;
        const float pv = (kok && qq < n && key <= qq) ? __expf(st[e] * scale - lse_s[slot][ql]) : 0.f;
        p[blk][e] = pv;
        ds[blk][e] = pv * (dp[e] - dvec_s[slot][ql]) * scale;
      }
    }
    bf16x8 pb[2], db[2];
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      float pv[8], dv[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pv[e] = p[2 * s2][e];
        pv[4 + e] = p[2 * s2 + 1][e];
        dv[e] = ds[2 * s2][e];
        dv[4 + e] = ds[2 * s2 + 1][e];
      }
      pb[s2] = pack8(pv);
      db[s2] = pack8(dv);
    }
#pragma unroll
    for (int cb = 0; cb < NC; ++cb) {
      bf16x8 dt2[2], qt2[2];
      tr.read(Dt, cb, dt2);
      tr.read(Qt, cb, qt2);
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        adv[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(dt2[s2], pb[s2], adv[cb], 0, 0, 0);
        adk[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qt2[s2], db[s2], adk[cb], 0, 0, 0);
      }
    }
  }
  if (kok) {
    float* dk = dk_out + (int64_t(bkv) * n + key) * HD;
    float* dv = dv_out + (int64_t(bkv) * n + key) * HD;
#pragma unroll
    for (int cb = 0; cb < NC; ++cb) {
      *reinterpret_cast<f32x4*>(dk + 16 * cb + 4 * grp) = adk[cb];
      *reinterpret_cast<f32x4*>(dv + 16 * cb + 4 * grp) = adv[cb];
    }
  }
}

hipError_t launch_attention_bwd(const void* q, const void* k, const void* v, const void* o, const void* dout, int B,
                                int Hq, int Hkv, int n, int hd, const float* lse, float* dvec, float* dq, float* dk,
                                float* dv, hipStream_t s) {
  if (B == 0 || n == 0) return hipSuccess;
  const int nb = (n + kAB - 1) / kAB;
  const auto *Qp = (const uint16_t*)q, *Kp = (const uint16_t*)k, *Vp = (const uint16_t*)v;
  const auto *Op = (const uint16_t*)o, *Dp = (const uint16_t*)dout;
  const dim3 g1(B * Hq * nb), g2(B * Hkv * nb);
  switch (hd) {
#define DSF_ATTN_BWD(H)                                                                         \
  case H:                                                                                       \
    attn_bwd_dq_kernel<H><<<g1, 256, 0, s>>>(Qp, Kp, Vp, Op, Dp, n, Hq, Hkv, lse, dvec, dq);   \
    attn_bwd_dkv_kernel<H><<<g2, 256, 0, s>>>(Qp, Kp, Vp, Dp, lse, dvec, n, Hq, Hkv, dk, dv); \
    break;
    DSF_ATTN_BWD(32)
    DSF_ATTN_BWD(64)
    DSF_ATTN_BWD(128)
#undef DSF_ATTN_BWD
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dsf
