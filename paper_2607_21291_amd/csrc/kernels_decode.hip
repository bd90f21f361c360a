// Incremental decoding with per-layer caches of the kept tokens' keys and
// values (the paper treats prefill only; the decode-time routing rule is a
// threshold on the new token's router score, and a kept token attends
// causally over the layer's cached kept tokens).
//
// The projections of a decode step run on the few-row GEMM and the routing
// flags come from the router kernel; the kernels here are the other pieces
// decoding adds:
// - attention of one query per (sequence, head) over its cache and the new
//   token, split into chunks of keys whose last-arriving workgroup combines
//   them in chunk order (memory-bound: it reads the cache once), which also
//   appends the kept tokens' keys and values to the caches;
// - for a prefill: copying each layer's kept keys/values into the caches and
//   the lowest kept score per sequence (the threshold that continues the
//   prompt's selection).
#include <algorithm>

#include "dsf_device.h"
#include "dsf_internal.h"

namespace dsf {

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
// vector of dims and the row groups added in order through LDS. The chunk
// publishes {m, l, o[0..HD)} with device-coherent stores (an empty chunk:
// m = -inf, l = 0, o = 0) and counts itself on a device-scope counter; the
// last chunk of (b, h) to arrive resets the counter and combines the chunks in
// chunk order: out = sum_c o_c e^(m_c - M) / sum_c l_c e^(m_c - M), M the
// largest m_c (0 for an empty cache). No workgroup waits for another.
//
// With keep non-null the launch also appends the step's new key and value
// rows (knew, vnew [B, Hkv, HD]) of every kept sequence: attention runs over
// the cache_len[b] cached slots plus the new token, whose rows every
// workgroup reads from knew / vnew (so no workgroup reads the slot being
// written); the workgroup of the first query head of each kv head whose
// chunk holds slot cache_len[b] copies them into that slot; and once the
// last head of sequence b has combined (a second counter, count[B Hq + b]),
// cache_len[b] grows by one. Every workgroup of b has read cache_len[b]
// before it counted itself, so none sees the new length.
template <typename T, int HD>
__global__ __launch_bounds__(256) void decode_attn_kernel(const T* __restrict__ q, const T* __restrict__ ck,
                                                          const T* __restrict__ cv,
                                                          int32_t* __restrict__ cache_len, const T* __restrict__ knew,
                                                          const T* __restrict__ vnew,
                                                          const int32_t* __restrict__ keep, int Hq, int Hkv,
                                                          int cap, float* __restrict__ part,
                                                          uint32_t* __restrict__ count, T* __restrict__ out) {
  constexpr int VEC = 16 / int(sizeof(T));  // elements per 16-byte vector
  constexpr int LPK = HD / VEC;             // lanes per key row
  constexpr int KPP = 256 / LPK;            // rows per pass
  constexpr int NPASS = kDecChunk / KPP;
  constexpr int kMaxChunks = kDecodeMaxCap / kDecChunk;
  static_assert(LPK <= 64 && 64 % LPK == 0, "row groups within a wavefront");
  __shared__ float ps[kDecChunk];
  __shared__ float red[4];
  __shared__ float osum[KPP][HD];
  __shared__ float cw[kMaxChunks];
  __shared__ int is_last;
  const int c = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int nch = gridDim.x;
  const int tid = threadIdx.x, sub = tid % LPK, row = tid / LPK;
  const int len_old = min(cache_len[b], cap);
  const int kp = keep && keep[b] && len_old < cap ? 1 : 0;  // the new token joins at slot len_old
  const int len = len_old + kp;
  const int k0 = c * kDecChunk;
  const int64_t bh = int64_t(b) * Hq + h;
  const int kvh = h / (Hq / Hkv);
  const T* qr = q + bh * HD + sub * VEC;
  float qv[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) qv[i] = DecElem<T>::to_f(qr[i]);
  const T* kbase = ck + ((int64_t(b) * Hkv + kvh) * cap) * HD + sub * VEC;
  const T* vbase = cv + ((int64_t(b) * Hkv + kvh) * cap) * HD + sub * VEC;
  // the new token's rows (read only when kp)
  const T* knb = knew + (int64_t(b) * Hkv + kvh) * HD + sub * VEC;
  const T* vnb = vnew + (int64_t(b) * Hkv + kvh) * HD + sub * VEC;
  // key row `key` (< len): a cached slot, or the new token at slot len_old
  auto krow = [&](int key) { return key < len_old ? kbase + int64_t(key) * HD : knb; };
  auto vrow = [&](int key) { return key < len_old ? vbase + int64_t(key) * HD : vnb; };
  if (kp && c == len_old / kDecChunk && h % (Hq / Hkv) == 0 && row == 0) {
    // one row group copies the new rows into slot len_old (nobody reads that slot here)
    T* kd = const_cast<T*>(kbase) + int64_t(len_old) * HD;
    T* vd = const_cast<T*>(vbase) + int64_t(len_old) * HD;
    *reinterpret_cast<u32x4*>(kd) = *reinterpret_cast<const u32x4*>(knb);
    *reinterpret_cast<u32x4*>(vd) = *reinterpret_cast<const u32x4*>(vnb);
  }
  const float scale = 1.0f / sqrtf(float(HD));
  float o[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) o[i] = 0.f;
  float m, l;
  if constexpr (NPASS <= 16) {
    // every key and value vector of this thread's rows is requested before
    // the first is used (up to 32 16-byte loads in flight per thread)
    u32x4 kr[NPASS], vr[NPASS];
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      const int key = k0 + pass * KPP + row;
      kr[pass] = key < len ? *reinterpret_cast<const u32x4*>(krow(key)) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      const int key = k0 + pass * KPP + row;
      vr[pass] = key < len ? *reinterpret_cast<const u32x4*>(vrow(key)) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      const int j = pass * KPP + row, key = k0 + j;
      const T* kv = reinterpret_cast<const T*>(&kr[pass]);
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < VEC; ++i) acc = fmaf(qv[i], DecElem<T>::to_f(kv[i]), acc);
#pragma unroll
      for (int sh = LPK / 2; sh > 0; sh >>= 1) acc += __shfl_xor(acc, sh, 64);
      if (sub == 0) ps[j] = key < len ? acc * scale : -INFINITY;
    }
    __syncthreads();
    const float sv = ps[tid];
    m = block4_max(sv, red);
    const float p = sv == -INFINITY ? 0.f : expf(sv - m);
    ps[tid] = p;
    l = block4_sum(p, red);  // its barriers also publish ps
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      const int j = pass * KPP + row;
      if (k0 + j < len) {
        const T* vv = reinterpret_cast<const T*>(&vr[pass]);
        const float pp = ps[j];
#pragma unroll
        for (int i = 0; i < VEC; ++i) o[i] = fmaf(pp, DecElem<T>::to_f(vv[i]), o[i]);
      }
    }
  } else {
#pragma unroll 4
    for (int pass = 0; pass < NPASS; ++pass) {
      const int j = pass * KPP + row, key = k0 + j;
      float acc = 0.f;
      if (key < len) {
        T kv[VEC];
        *reinterpret_cast<u32x4*>(kv) = *reinterpret_cast<const u32x4*>(krow(key));
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc = fmaf(qv[i], DecElem<T>::to_f(kv[i]), acc);
      }
#pragma unroll
      for (int sh = LPK / 2; sh > 0; sh >>= 1) acc += __shfl_xor(acc, sh, 64);
      if (sub == 0) ps[j] = key < len ? acc * scale : -INFINITY;
    }
    __syncthreads();
    const float sv = ps[tid];
    m = block4_max(sv, red);
    const float p = sv == -INFINITY ? 0.f : expf(sv - m);
    ps[tid] = p;
    l = block4_sum(p, red);  // its barriers also publish ps
#pragma unroll 4
    for (int pass = 0; pass < NPASS; ++pass) {
      const int j = pass * KPP + row, key = k0 + j;
      if (key < len) {
        T vv[VEC];
        *reinterpret_cast<u32x4*>(vv) = *reinterpret_cast<const u32x4*>(vrow(key));
        const float pp = ps[j];
#pragma unroll
        for (int i = 0; i < VEC; ++i) o[i] = fmaf(pp, DecElem<T>::to_f(vv[i]), o[i]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < VEC; ++i) osum[row][sub * VEC + i] = o[i];
  __syncthreads();
  float* dst = part + (bh * nch + c) * (HD + 2);
  if (tid < HD) {
    float acc = 0.f;
#pragma unroll 8
    for (int r = 0; r < KPP; ++r) acc += osum[r][tid];
    __hip_atomic_store(dst + 2 + tid, acc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (tid == 0) {
      __hip_atomic_store(dst, m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(dst + 1, l, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  // the device-coherent stores complete before the counter moves; the last
  // chunk reads them back with device-coherent loads
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0) {
    const uint32_t old = __hip_atomic_fetch_add(count + bh, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    is_last = old == uint32_t(nch - 1);
    if (is_last) __hip_atomic_store(count + bh, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!is_last) return;
  const float* pb = part + bh * nch * (HD + 2);
  for (int cc = tid; cc < nch; cc += 256) {
    ps[cc] = __hip_atomic_load(pb + int64_t(cc) * (HD + 2), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    cw[cc] = __hip_atomic_load(pb + int64_t(cc) * (HD + 2) + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  // every thread forms M and L in chunk order from LDS; ps[] holds m_c
  float M = -INFINITY;
  for (int cc = 0; cc < nch; ++cc) M = fmaxf(M, ps[cc]);
  float L = 0.f;
  if (M != -INFINITY)
    for (int cc = 0; cc < nch; ++cc) L = fmaf(cw[cc], ps[cc] == -INFINITY ? 0.f : expf(ps[cc] - M), L);
  if (tid < HD) {
    float O = 0.f;
    if (M != -INFINITY) {
      for (int c0 = 0; c0 < nch; c0 += 8) {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
          v[j] = __hip_atomic_load(pb + int64_t(min(c0 + j, nch - 1)) * (HD + 2) + 2 + tid, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (c0 + j < nch && ps[c0 + j] != -INFINITY) O = fmaf(v[j], expf(ps[c0 + j] - M), O);
      }
    }
    out[bh * HD + tid] = DecElem<T>::from_f(L > 0.f ? O / L : 0.f);
  }
  if (keep && tid == 0) {
    // the last head of sequence b to combine moves its cache length
    uint32_t* cb = count + int64_t(gridDim.z) * Hq + b;
    const uint32_t old = __hip_atomic_fetch_add(cb, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old == uint32_t(Hq - 1)) {
      __hip_atomic_store(cb, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (kp) cache_len[b] = len;
    }
  }
}

int decode_attn_chunks(int cap) { return (cap + kDecChunk - 1) / kDecChunk; }

hipError_t launch_decode_attention(int dtype, const void* q, const void* ck, const void* cv, int32_t* cache_len,
                                   const void* knew, const void* vnew, const int32_t* keep, int B, int Hq, int Hkv,
                                   int hd, int cap, float* part, uint32_t* count, void* out, hipStream_t s) {
  if (B == 0) return hipSuccess;
  if (cap > kDecodeMaxCap) return hipErrorInvalidValue;
  const int nch = decode_attn_chunks(cap);
  const dim3 grid(nch, Hq, B);
  auto run = [&](auto tag, auto hdc) -> hipError_t {
    using T = decltype(tag);
    constexpr int HD = decltype(hdc)::value;
    decode_attn_kernel<T, HD><<<grid, 256, 0, s>>>((const T*)q, (const T*)ck, (const T*)cv, cache_len,
                                                   (const T*)knew, (const T*)vnew, keep, Hq, Hkv, cap, part, count,
                                                   (T*)out);
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
