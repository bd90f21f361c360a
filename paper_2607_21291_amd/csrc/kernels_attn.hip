// Causal attention among the kept tokens (Eq. 1 over the compacted set) for
// gfx950.
//
// bf16 paths (flash-style, online softmax in fp32). A workgroup of four
// wavefronts owns 64*NQ consecutive queries of one (sequence, query head); each
// wavefront owns NQ groups of 16 queries. Key/value tiles of 64 tokens are
// staged in LDS.
//
// Scores are formed transposed, S^T = K Q^T, with v_mfma_f32_16x16x32_bf16, so
// a lane holds 16 scores of ONE query (its column): the row max needs only two
// cross-lane steps, and the probabilities already sit in the layout of the B
// operand of O^T += V^T P^T. The MFMA's k slots there are filled with keys in
// the order the lane holds them, and V^T is read in the same order, so the
// contraction over keys is unchanged. The row sums of P come from the matrix
// cores as well: an A operand of ones gives, in every row of its output block,
// sum_k P[query][k] over the same bf16 probabilities that weight V.
//
// K and V tiles go global -> LDS by buffer DMA (no registers, no VALU), both
// row-major with each row's 16-byte chunks XOR-swizzled by the row index, in
// a ring of two stages; V^T is read with the LDS transpose load
// (ds_read_b64_tr_b16). Two forms of the kernel (attn_bf16_dma_kernel):
// - one query group per wave, the tile's V^T fragments read before the next
//   tile's DMA is issued (short sequences: more, shorter workgroups);
// - two query groups per wave (each K and V fragment serves 32 queries), the
//   next tile's DMA issued first and V^T read block by block in the
//   product, four transpose loads and their wait at a time: two waves per
//   SIMD at head dim 128, where holding a whole tile's V^T fragments would
//   not fit.
//
// Kept positions ascend, so causal order over compacted indices is causal
// order over original positions.
#include <hip/hip_ext.h>

#include <cstdlib>
#include <cstring>

#include "attn_sched.h"
#include "attn_tiles.h"
#include "dsf_device.h"
#include "dsf_internal.h"

namespace dsf {

constexpr int kKV = 64;  // keys per tile

// ------------------------------------------------------------------- DMA ring
template <int HD>
struct DmaTile : AttnTile<HD> {
  static constexpr int kStage = 2 * AttnTile<HD>::kTileBytes;  // K tile, then V tile
};

// LDS transpose load: within each 16-lane group G, lane 16G + 4a + b receives
// element b of the 8-byte rows addressed by lanes 16G + a + 4j, j = 0..3.
__device__ __forceinline__ bf16x4 lds_read_tr(const uint16_t* p) {
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4*)((__attribute__((address_space(3))) uint16_t*)(p)));
}

template <int HD, int NQ, bool LATE = false>
__global__ __launch_bounds__(256) void attn_bf16_dma_kernel(const uint16_t* __restrict__ Q,
                                                            const uint16_t* __restrict__ K,
                                                            const uint16_t* __restrict__ V, int Hq, int Hkv,
                                                            int n, uint16_t* __restrict__ out,
                                                            float* __restrict__ lse_out) {
  using A = DmaTile<HD>;
  constexpr int QB = 64 * NQ;          // queries per workgroup
  constexpr int NS = HD / 32;          // MFMA k steps over the head dim
  constexpr int ND = HD / 16;          // 16-row blocks of the head dim
  __shared__ __attribute__((aligned(16))) char smem[2 * A::kStage];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: keeps tile tests scalar
  const int r16 = lane & 15, grp = lane >> 4;
  // one work item per (sequence, head, query block); the query blocks of one
  // (sequence, head) share K/V, so they are kept on one XCD, and each XCD
  // starts its longest blocks first
  const int nqb = (n + QB - 1) / QB;
  const AttnItem it = attn_item(int(blockIdx.x), int(gridDim.x), nqb);
  const int bh = it.bh, qblk = it.qblk;
  const int h = bh % Hq, b = bh / Hq;
  const int kvh = h / (Hq / Hkv);
  const int q0 = qblk * QB;
  const int qw0 = q0 + wave * 16 * NQ;

  const uint16_t* Qh = Q + (int64_t(b) * Hq + h) * n * HD;
  const uint16_t* Kh = K + (int64_t(b) * Hkv + kvh) * n * HD;
  const uint16_t* Vh = V + (int64_t(b) * Hkv + kvh) * n * HD;

  const int kend = min(n, q0 + QB);
  const int ntiles = (kend + kKV - 1) / kKV;

  // DMA of tile t into stage t & 1. The buffer resources start at the tile's
  // first key and end at key n - 1, so rows past the last key land as zeros
  // (their scores are masked to -inf, their V rows weighted by zero). Lane
  // `lane` of this wave's e-th DMA fills 16 bytes at tile byte
  // 1024 (wave kDmaPerWave + e) + 16 lane: row r, chunk position c, which
  // holds the row's global chunk c ^ (r & kSwz).
  uint32_t dma_off[A::kDmaPerWave];
#pragma unroll
  for (int e = 0; e < A::kDmaPerWave; ++e) {
    const int byte = 1024 * (wave * A::kDmaPerWave + e) + 16 * lane;
    const int r = byte / A::kRowBytes, c = (byte % A::kRowBytes) / 16;
    dma_off[e] = uint32_t(r * A::kRowBytes + ((c ^ (r & A::kSwz)) * 16));
  }
  auto issue = [&](int t) {
    const int kb0 = t * kKV;
    const int bytes = (n - kb0) * A::kRowBytes;
    const auto kr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(Kh + int64_t(kb0) * HD), (short)0,
                                                      bytes, 0x00020000);
    const auto vr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(Vh + int64_t(kb0) * HD), (short)0,
                                                      bytes, 0x00020000);
    char* st = smem + (t & 1) * A::kStage + 1024 * (wave * A::kDmaPerWave);
#pragma unroll
    for (int e = 0; e < A::kDmaPerWave; ++e) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (__attribute__((address_space(3))) void*)(st + 1024 * e), 16,
                                               int(dma_off[e]), 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          vr, (__attribute__((address_space(3))) void*)(st + A::kTileBytes + 1024 * e), 16, int(dma_off[e]), 0, 0, 0);
    }
  };
  issue(0);

  // Q^T operand: lane (query r16, group grp) holds Q[query][32 s + 8 grp .. +8]
  bf16x8 qf[NQ][NS];
#pragma unroll
  for (int qi = 0; qi < NQ; ++qi) {
    int qrow = qw0 + 16 * qi + r16;
    if (qrow > n - 1) qrow = n - 1;
#pragma unroll
    for (int s = 0; s < NS; ++s)
      qf[qi][s] = *reinterpret_cast<const bf16x8*>(Qh + int64_t(qrow) * HD + 32 * s + 8 * grp);
  }

  // all-ones A operand: l_run accumulates the row sums of P on the matrix cores
  bf16x8 ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = (__bf16)1.0f;
  f32x4 o[NQ][ND], l_run[NQ];
  float m_run[NQ];
#pragma unroll
  for (int qi = 0; qi < NQ; ++qi) {
    m_run[qi] = -INFINITY;
    l_run[qi] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int db = 0; db < ND; ++db) o[qi][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const float sc = 1.4426950408889634f / sqrtf(float(HD));  // log2(e) / sqrt(hd)
  const int wave_qmax = qw0 + 16 * NQ - 1;

  // lane-constant parts of the V^T transpose reads: lane (16 G + a + 4 j)
  // addresses V row 4 G + j (+ 32 ks + 16 half) at dims 16 db + 4 a .. + 3,
  // i.e. chunk (2 db + a / 2) ^ swz at byte (a & 1) * 8 of it
  const int tg = lane >> 4, ta = lane & 3, tj = (lane >> 2) & 3;
  const int vrow = 4 * tg + tj;
  const int vbase = vrow * A::kRowBytes + (ta & 1) * 8;
  const int vu = (ta >> 1) ^ (vrow & A::kSwz);

  // V^T fragments of tile t: lane (dim r16 of block db, group grp) gets
  // V[32 ks + 4 grp + j][16 db + r16] (j = 0..3) and the same 16 keys later
  auto read_v = [&](int t, bf16x8 (&vf)[ND][2]) {
    const uint16_t* Vs = reinterpret_cast<const uint16_t*>(smem + (t & 1) * A::kStage + A::kTileBytes + vbase);
#pragma unroll
    for (int db = 0; db < ND; ++db) {
      const int coff = ((2 * db) ^ vu) * 8;  // elements
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x4 lo = lds_read_tr(Vs + (32 * ks) * HD + coff);
        const bf16x4 hi = lds_read_tr(Vs + (32 * ks + 16) * HD + coff);
        vf[db][ks] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    }
  };
  // one tile: scores, online softmax and P V over LDS stage t & 1
  auto tile = [&](int t, const bf16x8 (&vf)[ND][2]) {
    const int kb0 = t * kKV;
    const char* stage = smem + (t & 1) * A::kStage;
    const uint16_t* Ks = reinterpret_cast<const uint16_t*>(stage);
    {
      // S^T blocks: lane holds S[query 16 qi + r16][key kb0 + 16 kb + 4 grp + i]
      f32x4 s[NQ][4];
#pragma unroll
      for (int qi = 0; qi < NQ; ++qi)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) s[qi][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const int row = 16 * kb + r16;
#pragma unroll
        for (int st = 0; st < NS; ++st) {
          const int ch = 4 * st + grp;
          bf16x8 kf = *reinterpret_cast<const bf16x8*>(Ks + row * HD + ((ch ^ (row & A::kSwz)) << 3));
#pragma unroll
          for (int qi = 0; qi < NQ; ++qi)
            s[qi][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[qi][st], s[qi][kb], 0, 0, 0);
        }
      }
      const bool diag = kb0 + kKV - 1 > qw0 || kb0 + kKV > n;  // wave-uniform
      bf16x8 pb[NQ][2];
#pragma unroll
      for (int qi = 0; qi < NQ; ++qi) {
        if (diag) {
          // key kb0 + 4 grp + (16 kb + i) is visible to query qg iff 16 kb + i <= lim
          const int qg = qw0 + 16 * qi + r16;
          const int lim = min(qg, n - 1) - (kb0 + 4 * grp);
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) s[qi][kb][i] = (16 * kb + i > lim) ? -INFINITY : s[qi][kb][i];
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) mx = fmaxf(mx, s[qi][kb][i]);
        // running max in log2 units of the scaled scores (sc > 0 keeps the order)
        const float m_new = fmaxf(m_run[qi], rows4_max(mx) * sc);
        const float base = m_new == -INFINITY ? 0.f : m_new;
        float p[4][4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) p[kb][i] = __builtin_amdgcn_exp2f(fmaf(s[qi][kb][i], sc, -base));
        // rescale the running sums only when some lane's max moved (rare after the first tiles)
        if (__builtin_amdgcn_ballot_w64(m_new != m_run[qi])) {
          const float alpha = __builtin_amdgcn_exp2f(m_run[qi] - base);
          l_run[qi] *= alpha;
#pragma unroll
          for (int db = 0; db < ND; ++db) o[qi][db] *= alpha;
        }
        m_run[qi] = m_new;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            pb[qi][ks][i] = (__bf16)p[2 * ks][i];
            pb[qi][ks][4 + i] = (__bf16)p[2 * ks + 1][i];
          }
      }
      // O^T[dim 16 db + r16 .. ][query] += V^T P^T over this tile's 64 keys
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int qi = 0; qi < NQ; ++qi)
          l_run[qi] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb[qi][ks], l_run[qi], 0, 0, 0);
      if constexpr (LATE) {
        // V^T fragments read block by block, the next block's loads issued
        // after this block's MFMAs
        const uint32_t vs = uint32_t(size_t((__attribute__((address_space(3))) char*)(
                                smem + (t & 1) * A::kStage + A::kTileBytes + vbase)));
        u32x2 cur[4];
        lds_read_tr4<HD>(vs + uint32_t(((0 ^ vu) * 8) * 2), cur);
#pragma unroll
        for (int db = 0; db < ND; ++db) {
          bf16x8 vv[2];
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            const u32x4 raw = {cur[2 * ks][0], cur[2 * ks][1], cur[2 * ks + 1][0], cur[2 * ks + 1][1]};
            vv[ks] = __builtin_bit_cast(bf16x8, raw);
          }
#pragma unroll
          for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int qi = 0; qi < NQ; ++qi)
              o[qi][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vv[ks], pb[qi][ks], o[qi][db], 0, 0, 0);
          if (db + 1 < ND) {
            __builtin_amdgcn_sched_barrier(0);
            lds_read_tr4<HD>(vs + uint32_t((((2 * (db + 1)) ^ vu) * 8) * 2), cur);
          }
        }
      } else {
#pragma unroll
        for (int db = 0; db < ND; ++db)
#pragma unroll
          for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int qi = 0; qi < NQ; ++qi)
              o[qi][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[db][ks], pb[qi][ks], o[qi][db], 0, 0, 0);
      }
    }
  };
  // The barrier at the top of tile t publishes tile t and retires tile
  // t - 1, whose stage the DMA of tile t + 1 then refills. Each wave first
  // waits for its own DMA (__syncthreads does not wait for LDS DMA), so after
  // the barrier every wave's share of the tile is in LDS. The V fragments are
  // read before the next DMA is issued: a transpose read after it would wait
  // for that DMA to land.
  // tiles this wave computes: t kKV <= wave_qmax (every key of a later tile
  // is in the future of all its queries); the rest only keep the barriers
  // and the DMA going for the other waves
  const int tc = min(ntiles, wave_qmax / kKV + 1);
  int t = 0;
  for (; t < tc; ++t) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if constexpr (LATE) {
      if (t + 1 < ntiles) issue(t + 1);
      bf16x8 none[ND][2];
      tile(t, none);
    } else {
      bf16x8 vf[ND][2];
      read_v(t, vf);
      if (t + 1 < ntiles) issue(t + 1);
      tile(t, vf);
    }
  }
  for (; t < ntiles; ++t) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (t + 1 < ntiles) issue(t + 1);
  }
  // lane holds O^T[dim 16 db + 4 grp + i][query r16]
#pragma unroll
  for (int qi = 0; qi < NQ; ++qi) {
    const int qg = qw0 + 16 * qi + r16;
    if (qg >= n) continue;
    const float inv = 1.0f / l_run[qi][0];
    uint16_t* orow = out + (int64_t(b) * n + qg) * (int64_t(Hq) * HD) + int64_t(h) * HD;
#pragma unroll
    for (int db = 0; db < ND; ++db) {
      u32x2 pk;
      pk[0] = uint32_t(f2bf(o[qi][db][0] * inv)) | (uint32_t(f2bf(o[qi][db][1] * inv)) << 16);
      pk[1] = uint32_t(f2bf(o[qi][db][2] * inv)) | (uint32_t(f2bf(o[qi][db][3] * inv)) << 16);
      *reinterpret_cast<u32x2*>(orow + 16 * db + 4 * grp) = pk;
    }
    // log of the softmax normaliser in natural units of q.k / sqrt(hd):
    // (max in log2 units + log2 of the row sum) ln 2
    if (lse_out && grp == 0)
      lse_out[(int64_t(b) * Hq + h) * n + qg] = (m_run[qi] + __log2f(l_run[qi][0])) * 0.6931471805599453f;
  }
}


// fp32: one thread per query, online softmax over its causal prefix.
template <int HD>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ Q, const float* __restrict__ K,
                                                      const float* __restrict__ V, int Hq, int Hkv, int n,
                                                      float* __restrict__ out) {
  const int qi = blockIdx.x * 64 + threadIdx.x, h = blockIdx.y, b = blockIdx.z;
  if (qi >= n) return;
  const int kvh = h / (Hq / Hkv);
  const float* qr = Q + ((int64_t(b) * Hq + h) * n + qi) * HD;
  const float* Kh = K + (int64_t(b) * Hkv + kvh) * n * HD;
  const float* Vh = V + (int64_t(b) * Hkv + kvh) * n * HD;
  float qv[HD], o[HD];
  for (int d = 0; d < HD; ++d) {
    qv[d] = qr[d];
    o[d] = 0.f;
  }
  const float scale = 1.0f / sqrtf(float(HD));
  float m = -INFINITY, l = 0.f;
  for (int j = 0; j <= qi; ++j) {
    const float* kr = Kh + int64_t(j) * HD;
    float s = 0.f;
    for (int d = 0; d < HD; ++d) s = fmaf(qv[d], kr[d], s);
    s *= scale;
    const float mn = fmaxf(m, s);
    const float c = expf(m - mn), p = expf(s - mn);
    l = l * c + p;
    const float* vr = Vh + int64_t(j) * HD;
    for (int d = 0; d < HD; ++d) o[d] = o[d] * c + p * vr[d];
    m = mn;
  }
  float* orow = out + (int64_t(b) * n + qi) * (int64_t(Hq) * HD) + int64_t(h) * HD;
  for (int d = 0; d < HD; ++d) orow[d] = o[d] / l;
}

// Launch kern<<<grid, block>>>(args...), through hipExtLaunchKernelGGL when
// the enclosing timing scope hands over its events.
template <typename K, typename... A>
static void launch_timed(K kern, dim3 grid, dim3 block, hipStream_t s, A... args) {
  hipEvent_t e0, e1;
  if (timing_claim(&e0, &e1)) hipExtLaunchKernelGGL(kern, grid, block, 0, s, e0, e1, 0, args...);
  else kern<<<grid, block, 0, s>>>(args...);
}

// Keys per sequence up to which one query group per wave is faster
// (measured, per head dim): at head dim 64 the two forms are within 2 % up to
// 2k keys and two groups win beyond (-10 % at 2362); at head dim 128 one group
// wins at 512 keys (-20 %), two groups from about 1k (-3 % at 1024, -17 % at
// 1638, -9 % at 4118).
constexpr int kAttnOneGroupMaxKeys64 = 2048;
constexpr int kAttnOneGroupMaxKeys128 = 768;

hipError_t launch_attention(int dtype, const void* q, const void* k, const void* v, int B, int Hq, int Hkv,
                            int n, int hd, void* out, hipStream_t s, float* lse) {
  if (n == 0 || B == 0) return hipSuccess;
  TimedScope ts(DSF_KIND_ATTN, s, true);
  if (dtype == DSF_F32) {
    dim3 grid((n + 63) / 64, Hq, B);
    auto Qp = (const float*)q; auto Kp = (const float*)k; auto Vp = (const float*)v; auto O = (float*)out;
    switch (hd) {
      case 32: launch_timed(attn_f32_kernel<32>, grid, dim3(64), s, Qp, Kp, Vp, Hq, Hkv, n, O); break;
      case 64: launch_timed(attn_f32_kernel<64>, grid, dim3(64), s, Qp, Kp, Vp, Hq, Hkv, n, O); break;
      case 128: launch_timed(attn_f32_kernel<128>, grid, dim3(64), s, Qp, Kp, Vp, Hq, Hkv, n, O); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  auto grid = [&](int nq) { return dim3(((n + 64 * nq - 1) / (64 * nq)) * Hq * B); };
  auto Qp = (const uint16_t*)q; auto Kp = (const uint16_t*)k; auto Vp = (const uint16_t*)v; auto O = (uint16_t*)out;
  // DSF_ATTN_GROUPS=1 or =2 (read at every launch) forces one form (testing)
  int groups = hd == 32 ? 1 : n <= (hd == 64 ? kAttnOneGroupMaxKeys64 : kAttnOneGroupMaxKeys128) ? 1 : 2;
  if (const char* e = getenv("DSF_ATTN_GROUPS")) {
    if (!strcmp(e, "1")) groups = 1;
    if (!strcmp(e, "2")) groups = 2;
  }
  switch (hd) {
#define DSF_ATTN_LAUNCH(H)                                                                                      \
  case H:                                                                                                       \
    if (groups == 1) launch_timed(attn_bf16_dma_kernel<H, 1>, grid(1), dim3(256), s, Qp, Kp, Vp, Hq, Hkv, n, O, lse); \
    else launch_timed(attn_bf16_dma_kernel<H, 2, true>, grid(2), dim3(256), s, Qp, Kp, Vp, Hq, Hkv, n, O, lse);      \
    break;
    DSF_ATTN_LAUNCH(32)
    DSF_ATTN_LAUNCH(64)
    DSF_ATTN_LAUNCH(128)
#undef DSF_ATTN_LAUNCH
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dsf
