// Incremental decoding with per-layer caches of the kept tokens' keys and
// values (the paper treats prefill only; the decode-time routing rule is a
// threshold on the new token's router score, and a kept token attends
// causally over the layer's cached kept tokens).
//
// The projections of a decode step reuse the prefill GEMMs on B rows; the
// kernels here are the pieces decoding adds:
// - the routing flags of the new tokens (threshold, cache capacity);
// - the append of the kept tokens' keys and values to the caches;
// - attention of one query per (sequence, head) over its cache, split into
//   chunks of keys with a fixed-order combine (memory-bound: it reads the
//   cache once);
// - for a prefill: copying each layer's kept keys/values into the caches and
//   the lowest kept score per sequence (the threshold that continues the
//   prompt's selection).
#include <algorithm>

#include "dsf_device.h"
#include "dsf_internal.h"

namespace dsf {

// keep = score >= thr (NaN: not kept); a kept token whose cache is full is
// skipped and reported as 2. gate = +inf / -inf for the gated residual update
// (sigmoid gives exactly 1 / 0).
__global__ void decode_route_kernel(const float* __restrict__ scores, const float* __restrict__ thr, int B,
                                    const int32_t* __restrict__ cache_len, int cap, int32_t* __restrict__ keep,
                                    float* __restrict__ gate, int32_t* __restrict__ keep_out) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const bool want = scores[b] >= thr[b];
  const bool room = cache_len[b] < cap;
  const int k = want && room;
  keep[b] = k;
  gate[b] = k ? INFINITY : -INFINITY;
  if (keep_out) keep_out[b] = want ? (room ? 1 : 2) : 0;
}

hipError_t launch_decode_route(const float* scores, const float* thr, int B, const int32_t* cache_len, int cap,
                               int32_t* keep, float* gate, int32_t* keep_out, hipStream_t s) {
  if (B == 0) return hipSuccess;
  decode_route_kernel<<<(B + 255) / 256, 256, 0, s>>>(scores, thr, B, cache_len, cap, keep, gate, keep_out);
  return hipGetLastError();
}

// One workgroup per sequence: a kept token's key and value rows (all kv heads)
// go to slot cache_len[b] of its caches, then the length grows by one (after
// every head has been written, so readers of the length see whole rows).
__global__ __launch_bounds__(256) void kv_append_kernel(const u32x4* __restrict__ knew, const u32x4* __restrict__ vnew,
                                                        const int32_t* __restrict__ keep, u32x4* __restrict__ ck,
                                                        u32x4* __restrict__ cv, int32_t* __restrict__ cache_len,
                                                        int Hkv, int row_vecs, int cap) {
  const int b = blockIdx.x;
  if (!keep[b]) return;  // uniform over the workgroup
  const int slot = cache_len[b];
  const int n = Hkv * row_vecs;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int h = i / row_vecs, e = i - h * row_vecs;
    const int64_t src = (int64_t(b) * Hkv + h) * row_vecs + e;
    const int64_t dst = ((int64_t(b) * Hkv + h) * cap + slot) * row_vecs + e;
    ck[dst] = knew[src];
    cv[dst] = vnew[src];
  }
  __syncthreads();
  if (threadIdx.x == 0) cache_len[b] = slot + 1;
}

hipError_t launch_kv_append(int dtype, const void* knew, const void* vnew, const int32_t* keep, void* ck, void* cv,
                            int32_t* cache_len, int B, int Hkv, int hd, int cap, hipStream_t s) {
  if (B == 0) return hipSuccess;
  const int row_vecs = hd * (dtype == DSF_BF16 ? 2 : 4) / 16;
  kv_append_kernel<<<B, 256, 0, s>>>((const u32x4*)knew, (const u32x4*)vnew, keep, (u32x4*)ck, (u32x4*)cv,
                                     cache_len, Hkv, row_vecs, cap);
  return hipGetLastError();
}

// ------------------------------------------------------- decode attention

template <typename T>
struct DecElem;
template <>
struct DecElem<float> {
  static __device__ __forceinline__ float to_f(float v) { return v; }
  static __device__ __forceinline__ float from_f(float v) { return v; }
};
template <>
struct DecElem<uint16_t> {
  static __device__ __forceinline__ float to_f(uint16_t v) { return bf2f(v); }
  static __device__ __forceinline__ uint16_t from_f(float v) { return f2bf(v); }
};

__device__ __forceinline__ float wave_max_dec(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide max / sum over 256 threads (4 wavefronts) through LDS.
__device__ __forceinline__ float block4_max(float v, float* red) {
  v = wave_max_dec(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  const float r = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  return r;
}
__device__ __forceinline__ float block4_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  const float r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

constexpr int kDecChunk = 256;  // keys per workgroup of the decode attention

// Workgroup (chunk c, head h, sequence b): keys c*256 .. of the first
// cache_len[b] slots of kv head h / (Hq / Hkv). Key and value rows are read as
// 16-byte vectors, HD / 8 (bf16) or HD / 4 (fp32) lanes per row, so a group
// of lanes reads one whole row: scores q . k / sqrt(hd) in fp32 (the group
// adds its lanes' products with xor shuffles), the chunk's max m and sum l of
// exp(s - m), then o = sum_t exp(s_t - m) v_t with each lane owning one
// vector of dims and the row groups added in order through LDS.
// part[(b, h, c)] = {m, l, o[0..HD)}; an empty chunk stores m = -inf, l = 0.
template <typename T, int HD>
__global__ __launch_bounds__(256) void decode_attn_part_kernel(const T* __restrict__ q, const T* __restrict__ ck,
                                                               const T* __restrict__ cv,
                                                               const int32_t* __restrict__ cache_len, int Hq,
                                                               int Hkv, int cap, float* __restrict__ part) {
  constexpr int VEC = 16 / int(sizeof(T));  // elements per 16-byte vector
  constexpr int LPK = HD / VEC;             // lanes per key row
  constexpr int KPP = 256 / LPK;            // rows per pass
  constexpr int NPASS = kDecChunk / KPP;
  static_assert(LPK <= 64 && 64 % LPK == 0, "row groups within a wavefront");
  __shared__ float ps[kDecChunk];
  __shared__ float red[4];
  __shared__ float osum[KPP][HD];
  const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int nch = gridDim.x;
  const int tid = threadIdx.x, sub = tid % LPK, row = tid / LPK;
  const int len = min(cache_len[b], cap);
  const int k0 = c * kDecChunk;
  float* dst = part + ((int64_t(b) * Hq + h) * nch + c) * (HD + 2);
  if (k0 >= len) {  // uniform
    if (tid == 0) {
      dst[0] = -INFINITY;
      dst[1] = 0.f;
    }
    if (tid < HD) dst[2 + tid] = 0.f;
    return;
  }
  const int kvh = h / (Hq / Hkv);
  const T* qr = q + (int64_t(b) * Hq + h) * HD + sub * VEC;
  float qv[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) qv[i] = DecElem<T>::to_f(qr[i]);
  const T* kbase = ck + ((int64_t(b) * Hkv + kvh) * cap) * HD + sub * VEC;
  const T* vbase = cv + ((int64_t(b) * Hkv + kvh) * cap) * HD + sub * VEC;
  const float scale = 1.0f / sqrtf(float(HD));
#pragma unroll 4
  for (int pass = 0; pass < NPASS; ++pass) {
    const int j = pass * KPP + row, key = k0 + j;
    float acc = 0.f;
    if (key < len) {
      T kv[VEC];
      *reinterpret_cast<u32x4*>(kv) = *reinterpret_cast<const u32x4*>(kbase + int64_t(key) * HD);
#pragma unroll
      for (int i = 0; i < VEC; ++i) acc = fmaf(qv[i], DecElem<T>::to_f(kv[i]), acc);
    }
#pragma unroll
    for (int o = LPK / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (sub == 0) ps[j] = key < len ? acc * scale : -INFINITY;
  }
  __syncthreads();
  const float sv = ps[tid];
  const float m = block4_max(sv, red);
  const float p = sv == -INFINITY ? 0.f : expf(sv - m);
  ps[tid] = p;
  const float l = block4_sum(p, red);  // its barriers also publish ps
  float o[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) o[i] = 0.f;
#pragma unroll 4
  for (int pass = 0; pass < NPASS; ++pass) {
    const int j = pass * KPP + row, key = k0 + j;
    if (key < len) {
      T vv[VEC];
      *reinterpret_cast<u32x4*>(vv) = *reinterpret_cast<const u32x4*>(vbase + int64_t(key) * HD);
      const float pp = ps[j];
#pragma unroll
      for (int i = 0; i < VEC; ++i) o[i] = fmaf(pp, DecElem<T>::to_f(vv[i]), o[i]);
    }
  }
#pragma unroll
  for (int i = 0; i < VEC; ++i) osum[row][sub * VEC + i] = o[i];
  __syncthreads();
  if (tid < HD) {
    float acc = 0.f;
#pragma unroll 8
    for (int r = 0; r < KPP; ++r) acc += osum[r][tid];
    dst[2 + tid] = acc;
    if (tid == 0) {
      dst[0] = m;
      dst[1] = l;
    }
  }
}

// out[b, h*HD + d] = sum_c o_c[d] e^(m_c - M) / sum_c l_c e^(m_c - M), chunks in
// order (0 when the cache is empty).
template <typename T, int HD>
__global__ __launch_bounds__(HD) void decode_attn_combine_kernel(const float* __restrict__ part, int Hq, int nch,
                                                                 T* __restrict__ out) {
  const int bh = blockIdx.x, d = threadIdx.x;
  const float* p = part + int64_t(bh) * nch * (HD + 2);
  float M = -INFINITY;
  for (int c = 0; c < nch; ++c) M = fmaxf(M, p[c * (HD + 2)]);
  float L = 0.f, O = 0.f;
  if (M != -INFINITY) {
    for (int c = 0; c < nch; ++c) {
      const float* pc = p + c * (HD + 2);
      const float w = pc[0] == -INFINITY ? 0.f : expf(pc[0] - M);
      L = fmaf(pc[1], w, L);
      O = fmaf(pc[2 + d], w, O);
    }
  }
  out[int64_t(bh) * HD + d] = DecElem<T>::from_f(L > 0.f ? O / L : 0.f);
}

int decode_attn_chunks(int cap) { return (cap + kDecChunk - 1) / kDecChunk; }

hipError_t launch_decode_attention(int dtype, const void* q, const void* ck, const void* cv,
                                   const int32_t* cache_len, int B, int Hq, int Hkv, int hd, int cap, float* part,
                                   void* out, hipStream_t s) {
  if (B == 0) return hipSuccess;
  const int nch = decode_attn_chunks(cap);
  const dim3 grid(nch, Hq, B);
  auto run = [&](auto tag, auto hdc) -> hipError_t {
    using T = decltype(tag);
    constexpr int HD = decltype(hdc)::value;
    decode_attn_part_kernel<T, HD><<<grid, 256, 0, s>>>((const T*)q, (const T*)ck, (const T*)cv, cache_len, Hq, Hkv,
                                                        cap, part);
    decode_attn_combine_kernel<T, HD><<<B * Hq, HD, 0, s>>>(part, Hq, nch, (T*)out);
    return hipGetLastError();
  };
  const bool bf = dtype == DSF_BF16;
  switch (hd) {
    case 32: return bf ? run(uint16_t(), std::integral_constant<int, 32>()) : run(float(), std::integral_constant<int, 32>());
    case 64: return bf ? run(uint16_t(), std::integral_constant<int, 64>()) : run(float(), std::integral_constant<int, 64>());
    case 128:
      return bf ? run(uint16_t(), std::integral_constant<int, 128>()) : run(float(), std::integral_constant<int, 128>());
    default: return hipErrorInvalidValue;
  }
}

// ------------------------------------------------------------- prefill

// Rows j < k of src [B, Hkv, k, hd] -> slots 0..k-1 of the caches [B, Hkv, cap, hd];
// cache_len[b] = k for every sequence (written by the first workgroup).
__global__ void kv_fill_kernel(const u32x4* __restrict__ ks, const u32x4* __restrict__ vs, u32x4* __restrict__ ck,
                               u32x4* __restrict__ cv, int32_t* __restrict__ cache_len, int B, int Hkv, int k, int cap,
                               int row_vecs) {
  const int64_t n = int64_t(B) * Hkv * k * row_vecs;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x) {
    const int64_t e = i % row_vecs, r = i / row_vecs;  // r = (b * Hkv + h) * k + j
    const int64_t j = r % k, bh = r / k;
    ck[(bh * cap + j) * row_vecs + e] = ks[i];
    cv[(bh * cap + j) * row_vecs + e] = vs[i];
  }
  if (blockIdx.x == 0)
    for (int b = threadIdx.x; b < B; b += blockDim.x) cache_len[b] = k;
}

hipError_t launch_kv_fill(int dtype, const void* ks, const void* vs, void* ck, void* cv, int32_t* cache_len, int B,
                          int Hkv, int hd, int k, int cap, hipStream_t s) {
  if (B == 0) return hipSuccess;
  const int row_vecs = hd * (dtype == DSF_BF16 ? 2 : 4) / 16;
  const int64_t n = int64_t(B) * Hkv * k * row_vecs;
  const int blocks = int(std::min<int64_t>(std::max<int64_t>((n + 255) / 256, 1), 4096));
  kv_fill_kernel<<<blocks, 256, 0, s>>>((const u32x4*)ks, (const u32x4*)vs, (u32x4*)ck, (u32x4*)cv, cache_len, B, Hkv,
                                        k, cap, row_vecs);
  return hipGetLastError();
}

// thr[b] = min over the kept tokens of scores[b, idx[b, j]] (+inf for k = 0).
__global__ __launch_bounds__(256) void kept_min_score_kernel(const float* __restrict__ scores,
                                                             const int32_t* __restrict__ idx, int T, int k,
                                                             float* __restrict__ thr) {
  __shared__ float red[4];
  const int b = blockIdx.x;
  float v = INFINITY;
  for (int j = threadIdx.x; j < k; j += 256) v = fminf(v, scores[int64_t(b) * T + clamp_pos(idx[int64_t(b) * k + j], T)]);
  v = -block4_max(-v, red);
  if (threadIdx.x == 0) thr[b] = v;
}

hipError_t launch_kept_min_score(const float* scores, const int32_t* idx, int B, int T, int k, float* thr,
                                 hipStream_t s) {
  if (B == 0) return hipSuccess;
  kept_min_score_kernel<<<B, 256, 0, s>>>(scores, idx, T, k, thr);
  return hipGetLastError();
}

}  // namespace dsf
