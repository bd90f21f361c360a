// Streaming kernels of the depth-sparse layer on gfx950: RoPE table,
// similarity statistic (Eq. 4), per-sequence Top-K (Section 3.4),
// gather / scatter of hidden rows, and fused gather + LayerNorm / RMSNorm.
//
// These kernels move far more bytes than they compute on, so they are written
// for HBM: 16-byte vector accesses, one wavefront per row, deterministic
// fixed-order reductions (no floating-point atomics).
#include "dsf_device.h"
#include "dsf_internal.h"
#include "topk_block.h"

namespace dsf {

// --------------------------------------------------------------------- RoPE

__global__ void rope_table_kernel(float* table, int T, int half, int R, double theta) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= T * half) return;
  int p = i / half, j = i % half;
  double ang = double(p) * pow(theta, -2.0 * double(j) / double(R));
  double sn, cs;
  sincos(ang, &sn, &cs);
  table[2 * i] = float(cs);
  table[2 * i + 1] = float(sn);
}

hipError_t launch_rope_table(float* table, int T, int R, double theta, hipStream_t s) {
  int half = R / 2, n = T * half;
  if (n == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_OTHER, s);
  rope_table_kernel<<<(n + 255) / 256, 256, 0, s>>>(table, T, half, R, theta);
  return hipGetLastError();
}

// ------------------------------------------------ similarity statistic, Eq. 4

constexpr int kSimMaxGrid = 16384;

int sim_grid(int64_t n_tokens) {
  int64_t g = (n_tokens + 3) / 4;
  return int(g < 1 ? 1 : (g > kSimMaxGrid ? kSimMaxGrid : g));
}

// fp64 sum over the L-lane group of a lane (aligned groups; xor offsets
// below L stay inside the group).
template <int L>
__device__ __forceinline__ double group_sum_f64(double v) {
#pragma unroll
  for (int o = L / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// L lanes per token row, 64 / L rows per wavefront (grid-stride over rows);
// lane l of a row holds its 16-byte vectors l, l + L, ... (C of them; EXACT:
// the row splits evenly, no per-lane guards). Products and sums in fp64
// (products of bf16 or fp32 values are exact in fp64). Each block writes the
// sum of its rows' cosines, in a fixed order, to partial[blockIdx.x].
template <typename T, int L, int C, bool EXACT>
__global__ __launch_bounds__(256) void sim_partial_kernel(const T* a, const T* c, int64_t n, int d,
                                                          float* per_tok, double* partial) {
  constexpr int V = Elem<T>::kVec, RW = 64 / L;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hl = lane % L;
  const int nvec = d / V;
  auto in = [&](int ch) { return EXACT || hl + L * ch < nvec; };
  double wave_acc = 0.0;
  for (int64_t t0 = (int64_t(blockIdx.x) * 4 + w) * RW; t0 < n; t0 += int64_t(gridDim.x) * 4 * RW) {
    const int64_t t = t0 + lane / L;
    const int64_t tt = t < n ? t : n - 1;  // rows past the end are read again and dropped
    const T* ra = a + tt * d;
    const T* rc = c + tt * d;
    float va[C][V], vc[C][V];
#pragma unroll
    for (int ch = 0; ch < C; ++ch)
      if (in(ch)) {
        load_vec(ra + (hl + L * ch) * V, va[ch]);
        load_vec(rc + (hl + L * ch) * V, vc[ch]);
      }
    double dot = 0.0, aa = 0.0, cc = 0.0;
#pragma unroll
    for (int ch = 0; ch < C; ++ch)
      if (in(ch))
#pragma unroll
        for (int i = 0; i < V; ++i) {
          const double x = va[ch][i], y = vc[ch][i];
          dot = fma(x, y, dot);
          aa = fma(x, x, aa);
          cc = fma(y, y, cc);
        }
    dot = group_sum_f64<L>(dot);
    aa = group_sum_f64<L>(aa);
    cc = group_sum_f64<L>(cc);
    const double den = sqrt(aa) * sqrt(cc);
    const double cs = dot / (den > 1e-8 ? den : 1e-8);
    const bool lead = hl == 0 && t < n;
    if (lead && per_tok) per_tok[t] = float(cs);
    wave_acc += lead ? cs : 0.0;
  }
  wave_acc = wave_sum(wave_acc);  // the rows' leaders, in a fixed order
  __shared__ double wsum[4];
  if (lane == 0) wsum[w] = wave_acc;
  __syncthreads();
  if (threadIdx.x == 0) partial[blockIdx.x] = ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
}

// Single block: fixed-order sum of the partials, then accum += (sum, n).
__global__ __launch_bounds__(256) void sim_finish_kernel(const double* partial, int np, int64_t n,
                                                         double* accum) {
  __shared__ double red[256];
  // eight loads in flight per thread, then added in index order (the order
  // depends only on np)
  double v = 0.0;
  for (int base = 0; base < np; base += 8 * 256) {
    double t[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int i = base + 256 * j + int(threadIdx.x);
      t[j] = i < np ? partial[i] : 0.0;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) v += t[j];
  }
  red[threadIdx.x] = v;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    accum[0] += red[0];
    accum[1] += double(n);
  }
}

// Rows of any width: one wavefront per token row, the lanes stepping through
// its vectors; products and sums in fp64 (products of bf16 or
// fp32 values are exact in fp64). Each block writes the sum of its tokens'
// cosines, in a fixed order, to partial[blockIdx.x].
template <typename T>
__global__ __launch_bounds__(256) void sim_wide_kernel(const T* a, const T* c, int64_t n, int d,
                                                          float* per_tok, double* partial) {
  constexpr int V = Elem<T>::kVec;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nvec = d / V;
  double wave_acc = 0.0;
  for (int64_t t = int64_t(blockIdx.x) * 4 + w; t < n; t += int64_t(gridDim.x) * 4) {
    const T* ra = a + t * d;
    const T* rc = c + t * d;
    double dot = 0.0, aa = 0.0, cc = 0.0;
    for (int ch = lane; ch < nvec; ch += 64) {
      float va[V], vc[V];
      load_vec(ra + ch * V, va);
      load_vec(rc + ch * V, vc);
#pragma unroll
      for (int i = 0; i < V; ++i) {
        double x = va[i], y = vc[i];
        dot = fma(x, y, dot);
        aa = fma(x, x, aa);
        cc = fma(y, y, cc);
      }
    }
    dot = wave_sum(dot);
    aa = wave_sum(aa);
    cc = wave_sum(cc);
    double den = sqrt(aa) * sqrt(cc);
    double cs = dot / (den > 1e-8 ? den : 1e-8);
    if (lane == 0 && per_tok) per_tok[t] = float(cs);
    wave_acc += cs;
  }
  __shared__ double wsum[4];
  if (lane == 0) wsum[w] = wave_acc;
  __syncthreads();
  if (threadIdx.x == 0) partial[blockIdx.x] = ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
}

template <typename T, int L, bool EXACT>
static void launch_sim_l(const T* a, const T* c, int64_t n, int d, float* per_tok, double* partial, int& g,
                         int chunks, hipStream_t s) {
  // one row group per wavefront: 4 * (64 / L) rows per block (at most the
  // sim_grid blocks the workspace holds partials for)
  const int64_t need = (n + 4 * (64 / L) - 1) / (4 * (64 / L));
  if (need < g) g = int(need);
  switch (chunks) {
    case 1: sim_partial_kernel<T, L, 1, EXACT><<<g, 256, 0, s>>>(a, c, n, d, per_tok, partial); break;
    case 2: sim_partial_kernel<T, L, 2, EXACT><<<g, 256, 0, s>>>(a, c, n, d, per_tok, partial); break;
    case 3: sim_partial_kernel<T, L, 3, EXACT><<<g, 256, 0, s>>>(a, c, n, d, per_tok, partial); break;
    case 4: sim_partial_kernel<T, L, 4, EXACT><<<g, 256, 0, s>>>(a, c, n, d, per_tok, partial); break;
    case 5: sim_partial_kernel<T, L, 5, EXACT><<<g, 256, 0, s>>>(a, c, n, d, per_tok, partial); break;
    case 6: sim_partial_kernel<T, L, 6, EXACT><<<g, 256, 0, s>>>(a, c, n, d, per_tok, partial); break;
    case 7: sim_partial_kernel<T, L, 7, EXACT><<<g, 256, 0, s>>>(a, c, n, d, per_tok, partial); break;
    default: sim_partial_kernel<T, L, 8, EXACT><<<g, 256, 0, s>>>(a, c, n, d, per_tok, partial); break;
  }
}

// Lanes per row as for the norm kernel: the widest of 64, 32, 16 that splits
// the row evenly into at most 8 vectors per lane; otherwise 64 lanes looping
// over groups of 8 vectors.
template <typename T>
static void launch_sim_t(const T* a, const T* c, int64_t n, int d, float* per_tok, double* partial, int& g,
                         hipStream_t s) {
  const int nvec = d / Elem<T>::kVec;
  if (nvec % 64 == 0 && nvec / 64 <= 8) launch_sim_l<T, 64, true>(a, c, n, d, per_tok, partial, g, nvec / 64, s);
  else if (nvec % 32 == 0 && nvec / 32 <= 8) launch_sim_l<T, 32, true>(a, c, n, d, per_tok, partial, g, nvec / 32, s);
  else if (nvec % 16 == 0 && nvec / 16 <= 8) launch_sim_l<T, 16, true>(a, c, n, d, per_tok, partial, g, nvec / 16, s);
  else sim_wide_kernel<T><<<g, 256, 0, s>>>(a, c, n, d, per_tok, partial);
}

hipError_t launch_sim_stats(int dtype, const void* a, const void* c, int64_t n, int d, float* per_tok,
                            double* partial, double* accum, hipStream_t s) {
  if (n == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_SIM, s);
  int g = sim_grid(n);
  if (dtype == DSF_BF16)
    launch_sim_t<uint16_t>((const uint16_t*)a, (const uint16_t*)c, n, d, per_tok, partial, g, s);
  else
    launch_sim_t<float>((const float*)a, (const float*)c, n, d, per_tok, partial, g, s);
  sim_finish_kernel<<<1, 256, 0, s>>>(partial, g, n, accum);
  return hipGetLastError();
}

// -------------------------------------------------------- Top-K, Section 3.4

constexpr int kTopkThreads = 1024;

// One block per sequence (topk_block.h).
template <bool KEYS_IN_LDS>
__global__ __launch_bounds__(kTopkThreads) void topk_kernel(const float* __restrict__ scores, int T, int k,
                                                            int32_t* __restrict__ idx) {
  __shared__ TopkShared<kTopkThreads, KEYS_IN_LDS> sh;
  const float* sc = scores + int64_t(blockIdx.x) * T;
  topk_block<kTopkThreads, KEYS_IN_LDS>([&](int t) { return sc[t]; }, T, k, idx + int64_t(blockIdx.x) * k, sh);
}

hipError_t launch_topk(const float* scores, int B, int T, int k, int32_t* idx, hipStream_t s) {
  if (k == 0 || B == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_TOPK, s, true);
  if (T <= kTopkLdsKeys) launch_with_timing(topk_kernel<true>, dim3(B), dim3(kTopkThreads), s, scores, T, k, idx);
  else launch_with_timing(topk_kernel<false>, dim3(B), dim3(kTopkThreads), s, scores, T, k, idx);
  return hipGetLastError();
}

// ------------------------------------------------------- gather / scatter

template <typename T>
__global__ __launch_bounds__(256) void gather_kernel(const T* __restrict__ x, int Tlen, int d,
                                                     const int32_t* __restrict__ idx, int k,
                                                     T* __restrict__ out, int64_t nvec) {
  constexpr int V = Elem<T>::kVec;
  const int vpr = d / V;
  for (int64_t v = int64_t(blockIdx.x) * 256 + threadIdx.x; v < nvec; v += int64_t(gridDim.x) * 256) {
    int64_t row = v / vpr;
    int c = int(v - row * vpr);
    int64_t b = row / k;
    const T* src = x + (b * Tlen + clamp_pos(idx[row], Tlen)) * d + c * V;
    *reinterpret_cast<u32x4*>(out + row * d + c * V) = *reinterpret_cast<const u32x4*>(src);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void scatter_kernel(T* __restrict__ x, const T* __restrict__ delta, int Tlen,
                                                      int d, const int32_t* __restrict__ idx, int k,
                                                      int64_t nvec) {
  constexpr int V = Elem<T>::kVec;
  const int vpr = d / V;
  for (int64_t v = int64_t(blockIdx.x) * 256 + threadIdx.x; v < nvec; v += int64_t(gridDim.x) * 256) {
    int64_t row = v / vpr;
    int c = int(v - row * vpr);
    int64_t b = row / k;
    T* dst = x + (b * Tlen + clamp_pos(idx[row], Tlen)) * d + c * V;
    float a[V], e[V];
    load_vec(dst, a);
    load_vec(delta + row * d + c * V, e);
#pragma unroll
    for (int i = 0; i < V; ++i) a[i] += e[i];
    store_vec(dst, a);
  }
}

static unsigned stream_grid(int64_t nvec) {
  int64_t g = (nvec + 255) / 256;
  return unsigned(g > 8192 ? 8192 : (g < 1 ? 1 : g));
}

hipError_t launch_gather(int dtype, const void* x, int B, int T, int d, const int32_t* idx, int k,
                         void* out, hipStream_t s) {
  int64_t rows = int64_t(B) * k;
  if (rows == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_GATHER, s, true);
  if (dtype == DSF_BF16) {
    int64_t nvec = rows * (d / 8);
    launch_with_timing(gather_kernel<uint16_t>, dim3(stream_grid(nvec)), dim3(256), s, (const uint16_t*)x, T, d, idx,
                       k, (uint16_t*)out, nvec);
  } else {
    int64_t nvec = rows * (d / 4);
    launch_with_timing(gather_kernel<float>, dim3(stream_grid(nvec)), dim3(256), s, (const float*)x, T, d, idx, k,
                       (float*)out, nvec);
  }
  return hipGetLastError();
}

hipError_t launch_scatter(int dtype, void* x, const void* delta, int B, int T, int d, const int32_t* idx,
                          int k, hipStream_t s) {
  int64_t rows = int64_t(B) * k;
  if (rows == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_SCATTER, s, true);
  if (dtype == DSF_BF16) {
    int64_t nvec = rows * (d / 8);
    launch_with_timing(scatter_kernel<uint16_t>, dim3(stream_grid(nvec)), dim3(256), s, (uint16_t*)x,
                       (const uint16_t*)delta, T, d, idx, k, nvec);
  } else {
    int64_t nvec = rows * (d / 4);
    launch_with_timing(scatter_kernel<float>, dim3(stream_grid(nvec)), dim3(256), s, (float*)x, (const float*)delta, T,
                       d, idx, k, nvec);
  }
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void copy_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) dst[i] = src[i];
}

hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t s) {
  int64_t n = int64_t(bytes / 16);
  if (n == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_OTHER, s);
  copy_kernel<<<stream_grid(n), 256, 0, s>>>((const u32x4*)src, (u32x4*)dst, n);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void zero_u32_kernel(uint32_t* __restrict__ dst, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) dst[i] = 0u;
}

hipError_t launch_zero_u32(uint32_t* dst, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  zero_u32_kernel<<<stream_grid(n), 256, 0, s>>>(dst, n);
  return hipGetLastError();
}

// ------------------------------------------- gather + LayerNorm / RMSNorm

// Sum over the L-lane group of a lane (L = 16, 32 or 64; groups are aligned),
// with the row-swap permutes of gfx950 (VALU only): within 16-lane rows,
// then rows 0+1 and 2+3, then the two halves.
template <int L>
__device__ __forceinline__ float group_sum(float v) {
  v = row16_sum(v);
  if constexpr (L >= 32) {
    auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(b[0]) + __uint_as_float(b[1]);
  }
  if constexpr (L == 64) {
    auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  }
  return v;
}

// The forms the layer uses: LayerNorm with gain and bias into two outputs
// (NeoX: LN1 and LN2 of the same rows), the same without biases or with only
// one of them, and RMSNorm with gain into one output (Qwen).
enum NormMode { kNormLnBias2 = 0, kNormLn2 = 1, kNormRms1 = 2, kNormLnBiasMixed = 3 };

// L lanes per row, 64 / L rows per wavefront; lane l of a row holds its
// 16-byte vectors l, l + L, ... (C of them, the row in registers), so it is
// read from HBM once for both normalisations. L is chosen so that the row's
// vectors split evenly over the lanes (EXACT): no lane idles through the
// loads and sums. One row per wavefront at d = 768 left half the lanes one
// vector short and measured 1.6x slower. Short of an even split, trailing
// lanes skip their last vector. The straight-line form (no branches around
// loads, modes fixed at compile time) matters: the same steps with runtime
// branches measured 1.2x slower.
template <typename T, int L, int C, bool EXACT, int MODE>
__global__ __launch_bounds__(256) void norm_kernel(NormArgs a) {
  constexpr int V = Elem<T>::kVec, RW = 64 / L;
  constexpr bool kRms = MODE == kNormRms1, kBias = MODE == kNormLnBias2 || MODE == kNormLnBiasMixed;
  constexpr int NO = MODE == kNormRms1 ? 1 : 2;  // outputs
  constexpr bool kHoist = C <= 3;
  constexpr int HC = kHoist ? C : 1;
  const int lane = threadIdx.x & 63, hl = lane % L;
  const int64_t rows = int64_t(a.B) * a.kk;
  const int64_t r = (int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6)) * RW + lane / L;
  const int64_t rr = r < rows ? r : rows - 1;  // dead rows re-read the last row, write nothing
  const int d = a.d, nvec = d / V;
  auto in = [&](int c) { return EXACT || hl + L * c < nvec; };
  const int64_t b = rr / a.kk, j = rr - b * a.kk;
  const int64_t pos = a.idx ? clamp_pos(a.idx[rr], a.src_rows) : j;
  // src_rows == 0: compact rows (source row = output row)
  const T* src = (const T*)a.src + (a.src_rows ? b * a.src_rows + pos : rr) * d;
  float v[C][V];
#pragma unroll
  for (int c = 0; c < C; ++c)
    if (in(c)) load_vec(src + (hl + L * c) * V, v[c]);
  float wv[NO][HC][V], bv[NO][HC][V];
  auto load_wb = [&](int o, int c, float* w_out, float* b_out) {
    const int ch = hl + L * c;
    const T* wp = (const T*)(o == 0 ? a.w1 : a.w2);
    load_vec(wp + ch * V, w_out);
    if constexpr (MODE == kNormLnBias2) load_vec((const T*)(o == 0 ? a.b1 : a.b2) + ch * V, b_out);
    if constexpr (MODE == kNormLnBiasMixed) {  // a missing bias reads the gain and is discarded
      const T* bp = (const T*)(o == 0 ? a.b1 : a.b2);
      const bool hb = bp != nullptr;
      load_vec((hb ? bp : wp) + ch * V, b_out);
#pragma unroll
      for (int i = 0; i < V; ++i) b_out[i] = hb ? b_out[i] : 0.f;
    }
  };
  if constexpr (kHoist) {
#pragma unroll
    for (int o = 0; o < NO; ++o)
#pragma unroll
      for (int c = 0; c < C; ++c)
        if (in(c)) load_wb(o, c, wv[o][c], bv[o][c]);
  }
  float m = 0.f;
  if constexpr (!kRms) {
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c)
      if (in(c))
#pragma unroll
        for (int i = 0; i < V; ++i) sum += v[c][i];
    m = group_sum<L>(sum) / float(d);
  }
  float sq = 0.f;
#pragma unroll
  for (int c = 0; c < C; ++c)
    if (in(c))
#pragma unroll
      for (int i = 0; i < V; ++i) {
        const float t = v[c][i] - m;
        sq += t * t;
      }
  const float rstd = 1.0f / sqrtf(group_sum<L>(sq) / float(d) + a.eps);
  if (r >= rows) return;
#pragma unroll
  for (int o = 0; o < NO; ++o) {
    T* out = (T*)(o == 0 ? a.out1 : a.out2);
#pragma unroll
    for (int c = 0; c < C; ++c) {
      if (!in(c)) continue;
      float wl[V], bl[V];
      const float* wc = wl;
      const float* bc = bl;
      if constexpr (kHoist) {
        wc = wv[o][c];
        bc = bv[o][c];
      } else {
        load_wb(o, c, wl, bl);
      }
      float y[V];
#pragma unroll
      for (int i = 0; i < V; ++i) y[i] = (v[c][i] - m) * rstd * wc[i] + (kBias ? bc[i] : 0.f);
      store_vec(out + r * d + (hl + L * c) * V, y);
    }
  }
}

template <typename T, int L, bool EXACT, int MODE>
static hipError_t launch_norm_lm(const NormArgs& a, int chunks, hipStream_t s) {
  const int64_t rows = int64_t(a.B) * a.kk;
  const unsigned grid = unsigned((rows + 4 * (64 / L) - 1) / (4 * (64 / L)));
  switch (chunks) {
    case 1: launch_with_timing(norm_kernel<T, L, 1, EXACT, MODE>, dim3(grid), dim3(256), s, a); break;
    case 2: launch_with_timing(norm_kernel<T, L, 2, EXACT, MODE>, dim3(grid), dim3(256), s, a); break;
    case 3: launch_with_timing(norm_kernel<T, L, 3, EXACT, MODE>, dim3(grid), dim3(256), s, a); break;
    case 4: launch_with_timing(norm_kernel<T, L, 4, EXACT, MODE>, dim3(grid), dim3(256), s, a); break;
    case 5: launch_with_timing(norm_kernel<T, L, 5, EXACT, MODE>, dim3(grid), dim3(256), s, a); break;
    case 6: launch_with_timing(norm_kernel<T, L, 6, EXACT, MODE>, dim3(grid), dim3(256), s, a); break;
    case 7: launch_with_timing(norm_kernel<T, L, 7, EXACT, MODE>, dim3(grid), dim3(256), s, a); break;
    case 8: launch_with_timing(norm_kernel<T, L, 8, EXACT, MODE>, dim3(grid), dim3(256), s, a); break;
    default:
      if constexpr (EXACT) return hipErrorInvalidValue;
      if (chunks <= 12) launch_with_timing(norm_kernel<T, L, 12, false, MODE>, dim3(grid), dim3(256), s, a);
      else if (chunks <= 16) launch_with_timing(norm_kernel<T, L, 16, false, MODE>, dim3(grid), dim3(256), s, a);
      else return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T, int L, bool EXACT>
static hipError_t launch_norm_l(const NormArgs& a, int chunks, hipStream_t s) {
  if (a.rms) {
    if (a.out2 || a.b1) return hipErrorInvalidValue;
    return launch_norm_lm<T, L, EXACT, kNormRms1>(a, chunks, s);
  }
  if (!a.out2) return hipErrorInvalidValue;
  if (a.b1 && a.b2) return launch_norm_lm<T, L, EXACT, kNormLnBias2>(a, chunks, s);
  if (!a.b1 && !a.b2) return launch_norm_lm<T, L, EXACT, kNormLn2>(a, chunks, s);
  return launch_norm_lm<T, L, EXACT, kNormLnBiasMixed>(a, chunks, s);
}

// Lanes per row: the widest of 64, 32, 16 that splits the row's vectors
// evenly into at most 8 per lane (fewer vectors per lane keep the weights in
// registers); otherwise 64 lanes, the last vectors of the row on the first
// lanes only.
template <typename T>
static hipError_t launch_norm_t(const NormArgs& a, hipStream_t s) {
  const int nvec = a.d / Elem<T>::kVec;
  if (nvec % 64 == 0 && nvec / 64 <= 8) return launch_norm_l<T, 64, true>(a, nvec / 64, s);
  if (nvec % 32 == 0 && nvec / 32 <= 8) return launch_norm_l<T, 32, true>(a, nvec / 32, s);
  if (nvec % 16 == 0 && nvec / 16 <= 8) return launch_norm_l<T, 16, true>(a, nvec / 16, s);
  return launch_norm_l<T, 64, false>(a, (nvec + 63) / 64, s);
}

hipError_t launch_norm(const NormArgs& a, hipStream_t s) {
  if (int64_t(a.B) * a.kk == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_NORM, s, true);
  return a.dtype == DSF_BF16 ? launch_norm_t<uint16_t>(a, s) : launch_norm_t<float>(a, s);
}

}  // namespace dsf
