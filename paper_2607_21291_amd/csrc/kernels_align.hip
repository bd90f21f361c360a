// The feature-preserving alignment objective of Section 3.5 on gfx950:
// the hidden-state distance of Eq. 9 (softmax over each token's hidden
// dimension, squared differences summed) and the per-row KL divergence of
// Eq. 10 over a row of logits. Both stream their inputs once from HBM.
//
// The exponentials run on the hardware exp2 in fp32; the normalisers,
// probabilities' differences and every sum across vectors are fp64, and every
// reduction runs in an order fixed by the shape, so results repeat bitwise.
#include <cmath>

#include "dsf_device.h"
#include "dsf_internal.h"

namespace dsf {

// e^x as 2^(x log2 e) on the hardware exponential (v_exp_f32, about 1 ulp).
// Rounding x log2 e adds a relative error of about |x| 2^-24 to the result;
// the callers' arguments are differences to a row maximum, so |x| is the
// distance of a logit from the largest one.
__device__ __forceinline__ float exp_hw(float x) { return __builtin_amdgcn_exp2f(x * 1.44269504088896341f); }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// --------------------------------------------------------------- Eq. 9

constexpr int kAlignMaxGrid = 16384;  // one token per wavefront up to 65536 tokens

int align_grid(int64_t n_tokens) {
  const int64_t g = (n_tokens + 3) / 4;
  return int(g < 1 ? 1 : (g > kAlignMaxGrid ? kAlignMaxGrid : g));
}

// One wavefront per token: both rows stay in registers (MAXC 16-byte vectors
// per lane) through the three steps max, exponentials and their sums, and
// the squared differences of the two softmaxes. Each block writes the sum
// of its tokens' distances, in a fixed order, to partial[blockIdx.x].
template <typename T, int MAXC>
__global__ __launch_bounds__(256) void align_hidden_kernel(const T* __restrict__ hs, const T* __restrict__ hd,
                                                           int64_t n, int d, float* __restrict__ per_tok,
                                                           double* __restrict__ partial) {
  constexpr int V = Elem<T>::kVec;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nvec = d / V;
  double wave_acc = 0.0;
  for (int64_t t = int64_t(blockIdx.x) * 4 + w; t < n; t += int64_t(gridDim.x) * 4) {
    float a[MAXC][V], b[MAXC][V];
    float ma = -INFINITY, mb = -INFINITY;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int ch = lane + 64 * i;
      if (ch < nvec) {
        load_vec(hs + t * d + ch * V, a[i]);
        load_vec(hd + t * d + ch * V, b[i]);
#pragma unroll
        for (int e = 0; e < V; ++e) {
          ma = fmaxf(ma, a[i][e]);
          mb = fmaxf(mb, b[i][e]);
        }
      }
    }
    ma = wave_max(ma);
    mb = wave_max(mb);
    double za = 0.0, zb = 0.0;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      if (lane + 64 * i < nvec) {
#pragma unroll
        for (int e = 0; e < V; ++e) {
          a[i][e] = exp_hw(a[i][e] - ma);
          b[i][e] = exp_hw(b[i][e] - mb);
          za += a[i][e];
          zb += b[i][e];
        }
      }
    }
    za = wave_sum(za);
    zb = wave_sum(zb);
    const double ia = 1.0 / za, ib = 1.0 / zb;
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      if (lane + 64 * i < nvec) {
#pragma unroll
        for (int e = 0; e < V; ++e) {
          // both products rounded alike (no fused multiply-add), so that
          // identical rows give exactly zero
#pragma clang fp contract(off)
          const double pa = double(a[i][e]) * ia;
          const double pb = double(b[i][e]) * ib;
          const double diff = pa - pb;
          acc = fma(diff, diff, acc);
        }
      }
    }
    acc = wave_sum(acc);
    if (lane == 0 && per_tok) per_tok[t] = float(acc);
    wave_acc += acc;
  }
  __shared__ double wsum[4];
  if (lane == 0) wsum[w] = wave_acc;
  __syncthreads();
  if (threadIdx.x == 0) partial[blockIdx.x] = ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
}

// The same over L-lane groups, 64 / L rows per wavefront, when the row splits
// evenly into C <= 8 vectors per lane (no lane idles; one row per wavefront at
// d = 768 left half the lanes a vector short).
template <int L>
__device__ __forceinline__ float group_max(float v) {
#pragma unroll
  for (int o = L / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
template <int L>
__device__ __forceinline__ double group_sum_d(double v) {
#pragma unroll
  for (int o = L / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

template <typename T, int L, int C>
__global__ __launch_bounds__(256) void align_hidden_group_kernel(const T* __restrict__ hs, const T* __restrict__ hd,
                                                                 int64_t n, int d, float* __restrict__ per_tok,
                                                                 double* __restrict__ partial) {
  constexpr int V = Elem<T>::kVec, RW = 64 / L;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hl = lane % L;
  double wave_acc = 0.0;
  for (int64_t t0 = (int64_t(blockIdx.x) * 4 + w) * RW; t0 < n; t0 += int64_t(gridDim.x) * 4 * RW) {
    const int64_t t = t0 + lane / L;
    const int64_t tt = t < n ? t : n - 1;  // rows past the end are read again and dropped
    float a[C][V], b[C][V];
    float ma = -INFINITY, mb = -INFINITY;
#pragma unroll
    for (int i = 0; i < C; ++i) {
      load_vec(hs + tt * d + (hl + L * i) * V, a[i]);
      load_vec(hd + tt * d + (hl + L * i) * V, b[i]);
    }
#pragma unroll
    for (int i = 0; i < C; ++i)
#pragma unroll
      for (int e = 0; e < V; ++e) {
        ma = fmaxf(ma, a[i][e]);
        mb = fmaxf(mb, b[i][e]);
      }
    ma = group_max<L>(ma);
    mb = group_max<L>(mb);
    double za = 0.0, zb = 0.0;
#pragma unroll
    for (int i = 0; i < C; ++i)
#pragma unroll
      for (int e = 0; e < V; ++e) {
        a[i][e] = exp_hw(a[i][e] - ma);
        b[i][e] = exp_hw(b[i][e] - mb);
        za += a[i][e];
        zb += b[i][e];
      }
    za = group_sum_d<L>(za);
    zb = group_sum_d<L>(zb);
    const double ia = 1.0 / za, ib = 1.0 / zb;
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < C; ++i)
#pragma unroll
      for (int e = 0; e < V; ++e) {
        // both products rounded alike (no fused multiply-add), so that
        // identical rows give exactly zero
#pragma clang fp contract(off)
        const double pa = double(a[i][e]) * ia;
        const double pb = double(b[i][e]) * ib;
        const double diff = pa - pb;
        acc = fma(diff, diff, acc);
      }
    acc = group_sum_d<L>(acc);
    const bool lead = hl == 0 && t < n;
    if (lead && per_tok) per_tok[t] = float(acc);
    wave_acc += lead ? acc : 0.0;
  }
  wave_acc = wave_sum(wave_acc);  // the rows' leaders, in a fixed order
  __shared__ double wsum[4];
  if (lane == 0) wsum[w] = wave_acc;
  __syncthreads();
  if (threadIdx.x == 0) partial[blockIdx.x] = ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
}

// Single block: accum[0] += the partials, summed in a fixed order.
__global__ __launch_bounds__(256) void sum_finish_kernel(const double* __restrict__ partial, int64_t np,
                                                         double* __restrict__ accum) {
  __shared__ double red[256];
  // eight loads in flight per thread, then added in index order (the order
  // depends only on np)
  double v = 0.0;
  for (int64_t base = 0; base < np; base += 8 * 256) {
    double t[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t i = base + 256 * j + threadIdx.x;
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
  if (threadIdx.x == 0) accum[0] += red[0];
}

int align_max_d(int dtype) { return 64 * 16 * (dtype == DSF_BF16 ? 8 : 4); }

template <typename T, int L>
static void launch_align_group(const T* hs, const T* hd, int64_t n, int d, float* per_tok, double* partial, int g,
                               int c, hipStream_t s) {
  switch (c) {
    case 1: align_hidden_group_kernel<T, L, 1><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial); break;
    case 2: align_hidden_group_kernel<T, L, 2><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial); break;
    case 3: align_hidden_group_kernel<T, L, 3><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial); break;
    case 4: align_hidden_group_kernel<T, L, 4><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial); break;
    case 5: align_hidden_group_kernel<T, L, 5><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial); break;
    case 6: align_hidden_group_kernel<T, L, 6><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial); break;
    case 7: align_hidden_group_kernel<T, L, 7><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial); break;
    default: align_hidden_group_kernel<T, L, 8><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial); break;
  }
}

template <typename T>
static void launch_align_hidden_t(const T* hs, const T* hd, int64_t n, int d, float* per_tok, double* partial,
                                  int g, hipStream_t s) {
  const int nvec = d / Elem<T>::kVec;
  if (nvec % 64 == 0 && nvec / 64 <= 8) return launch_align_group<T, 64>(hs, hd, n, d, per_tok, partial, g, nvec / 64, s);
  if (nvec % 32 == 0 && nvec / 32 <= 8) return launch_align_group<T, 32>(hs, hd, n, d, per_tok, partial, g, nvec / 32, s);
  if (nvec % 16 == 0 && nvec / 16 <= 8) return launch_align_group<T, 16>(hs, hd, n, d, per_tok, partial, g, nvec / 16, s);
  const int chunks = (nvec + 63) / 64;
  if (chunks <= 1) align_hidden_kernel<T, 1><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial);
  else if (chunks <= 2) align_hidden_kernel<T, 2><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial);
  else if (chunks <= 4) align_hidden_kernel<T, 4><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial);
  else if (chunks <= 8) align_hidden_kernel<T, 8><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial);
  else align_hidden_kernel<T, 16><<<g, 256, 0, s>>>(hs, hd, n, d, per_tok, partial);
}

hipError_t launch_align_hidden(int dtype, const void* hs, const void* hd, int64_t n, int d, float* per_tok,
                               double* partial, double* accum, hipStream_t s) {
  if (n == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_ALIGN, s);
  const int g = align_grid(n);
  if (dtype == DSF_BF16)
    launch_align_hidden_t<uint16_t>((const uint16_t*)hs, (const uint16_t*)hd, n, d, per_tok, partial, g, s);
  else
    launch_align_hidden_t<float>((const float*)hs, (const float*)hd, n, d, per_tok, partial, g, s);
  sum_finish_kernel<<<1, 256, 0, s>>>(partial, g, accum);
  return hipGetLastError();
}

// -------------------------------------------------------------- Eq. 10

// Online log-sum-exp state of one softmax, with the running sum of
// e^(z - m) (z_dense - z_sparse) for the dense row.
struct KlState {
  float md, ms;       // running maxima of the dense and sparse logits
  double zd, zs, s;   // sum e^(ld - md), sum e^(ls - ms), sum e^(ld - md) (ld - ls)
};

// e^(from - to) for from <= to, with e^(-inf) = 0 (an empty state)
__device__ __forceinline__ double rescale(float from, float to) {
  return from == -INFINITY ? 0.0 : double(exp_hw(from - to));
}

__device__ __forceinline__ KlState kl_combine(const KlState& a, const KlState& b) {
  KlState r;
  r.md = fmaxf(a.md, b.md);
  r.ms = fmaxf(a.ms, b.ms);
  const double fa = rescale(a.md, r.md), fb = rescale(b.md, r.md);
  r.zd = a.zd * fa + b.zd * fb;
  r.s = a.s * fa + b.s * fb;
  r.zs = a.zs * rescale(a.ms, r.ms) + b.zs * rescale(b.ms, r.ms);
  return r;
}

// One workgroup per row of C logits (dense and sparse): each thread runs the
// online state over its 16-byte vectors (strided by the workgroup), then the
// states meet in a fixed tree. KL = s / zd - (md + log zd) + (ms + log zs).
template <typename T>
__global__ __launch_bounds__(256) void kl_row_kernel(const T* __restrict__ ld, const T* __restrict__ ls, int C,
                                                     float* __restrict__ per_row, double* __restrict__ partial) {
  constexpr int V = Elem<T>::kVec;
  const int64_t row = blockIdx.x;
  const T* pd = ld + row * C;
  const T* ps = ls + row * C;
  KlState st{-INFINITY, -INFINITY, 0.0, 0.0, 0.0};
  const int nvec = C / V;
  for (int ch = threadIdx.x; ch < nvec; ch += 256) {
    float a[V], b[V];
    load_vec(pd + ch * V, a);
    load_vec(ps + ch * V, b);
    float va = a[0], vb = b[0];
#pragma unroll
    for (int e = 1; e < V; ++e) {
      va = fmaxf(va, a[e]);
      vb = fmaxf(vb, b[e]);
    }
    if (va > st.md) {
      const double f = rescale(st.md, va);
      st.zd *= f;
      st.s *= f;
      st.md = va;
    }
    if (vb > st.ms) {
      st.zs *= rescale(st.ms, vb);
      st.ms = vb;
    }
    // the vector's eight terms in fp32, then into the fp64 sums
    float zd8 = 0.f, s8 = 0.f, zs8 = 0.f;
#pragma unroll
    for (int e = 0; e < V; ++e) {
      const float ea = exp_hw(a[e] - st.md);
      zd8 += ea;
      s8 = fmaf(ea, a[e] - b[e], s8);
      zs8 += exp_hw(b[e] - st.ms);
    }
    st.zd += zd8;
    st.s += s8;
    st.zs += zs8;
  }
  __shared__ KlState red[256];
  red[threadIdx.x] = st;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] = kl_combine(red[threadIdx.x], red[threadIdx.x + o]);
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const KlState& f = red[0];
    const double kl = f.s / f.zd - (double(f.md) + log(f.zd)) + (double(f.ms) + log(f.zs));
    if (per_row) per_row[row] = float(kl);
    partial[row] = kl;
  }
}

hipError_t launch_kl_align(int dtype, const void* ld, const void* ls, int64_t rows, int C, float* per_row,
                           double* partial, double* accum, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_ALIGN, s);
  if (dtype == DSF_BF16)
    kl_row_kernel<uint16_t><<<unsigned(rows), 256, 0, s>>>((const uint16_t*)ld, (const uint16_t*)ls, C, per_row,
                                                           partial);
  else
    kl_row_kernel<float><<<unsigned(rows), 256, 0, s>>>((const float*)ld, (const float*)ls, C, per_row, partial);
  sum_finish_kernel<<<1, 256, 0, s>>>(partial, rows, accum);
  return hipGetLastError();
}

}  // namespace dsf
