// Projection GEMMs of the decoder block on the kept tokens (Eqs. 1-2),
// C[M, N] = A[M, K] . B[N, K]^T with fused epilogues, for gfx950.
//
// bf16 path: 128 x 128 x 64 workgroup tiles, four wavefronts of 64 x 64, each
// built from v_mfma_f32_16x16x32_bf16. Global tiles are staged through LDS
// (double buffered, 16-byte chunks XOR-swizzled by row so that the 16 rows an
// MFMA operand read touches fall in distinct bank groups). The next tile's
// global loads are in flight while the current tile is multiplied.
//
// After the K loop the fp32 tile is written to LDS and the epilogue reads it
// back row-wise, so every epilogue (RoPE pairs dims i and i + R/2; SwiGLU
// pairs gate and up columns) sees whole rows and stores 16-byte vectors.
//
// fp32 path: a plain LDS-tiled FMA kernel (32 x 128 tiles) that shares the
// epilogue. It exists for the fp32 workload and is not tuned.
#include <algorithm>
#include <atomic>
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include <hip/hip_ext.h>

#include "dsf_device.h"
#include "dsf_internal.h"
#include "gemm_sched.h"

namespace dsf {

// ------------------------------------------------------------- epilogue

template <typename T>
__device__ __forceinline__ void load8(const T* p, float* v) {
  if constexpr (sizeof(T) == 2) {
    load_vec(p, v);
  } else {
    load_vec(p, v);
    load_vec(p + 4, v + 4);
  }
}
template <typename T>
__device__ __forceinline__ void store8(T* p, const float* v) {
  if constexpr (sizeof(T) == 2) {
    store_vec(p, v);
  } else {
    store_vec(p, v);
    store_vec(p + 4, v + 4);
  }
}

// Eight elements of a row as raw 16-byte vectors (one for bf16, two for
// fp32), widened to fp32 only where they are used.
template <typename T>
struct Raw8 {
  u32x4 v[sizeof(T) / 2];
};
template <typename T>
__device__ __forceinline__ Raw8<T> load_raw8(const T* p) {
  Raw8<T> r;
#pragma unroll
  for (int i = 0; i < int(sizeof(T)) / 2; ++i) r.v[i] = reinterpret_cast<const u32x4*>(p)[i];
  return r;
}
template <typename T>
__device__ __forceinline__ void unpack8(const Raw8<T>& r, float* out) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if constexpr (sizeof(T) == 2) {
      out[2 * i] = __uint_as_float(r.v[0][i] << 16);
      out[2 * i + 1] = __uint_as_float(r.v[0][i] & 0xffff0000u);
    } else {
      out[i] = __uint_as_float(r.v[0][i]);
      out[4 + i] = __uint_as_float(r.v[1][i]);
    }
  }
}

// Rows of one thread in an epilogue of BM rows, BN columns, NT threads: its
// chunk column, then rows rr0, rr0 + RSTEP, ... with their sequence, slot in
// the kept list and position, and (residual kinds) the residual rows, read
// ahead of the staged tile by epi_prefetch so that their memory latency
// overlaps other work.
template <typename T, int BM, int BN, int NT>
struct EpiPre {
  static constexpr int CPR = BN / 8, RSTEP = NT / CPR, RPT = (BM + RSTEP - 1) / RSTEP;
  int bq[RPT], jq[RPT], pq[RPT];
  bool live[RPT];
  Raw8<T> xr[RPT];
};

// Kinds whose epilogue reads the rows' sequence positions.
constexpr bool epi_uses_positions(int epi) {
  return epi == EPI_QKV_ROPE || epi == EPI_RESID_STORE || epi == EPI_RESID_SCATTER || epi == EPI_RESID_SCATTER_GATE;
}

// EPI: the kind whose rows are read; RES: also read its residual rows
// (residual kinds).
template <typename T, int BM, int BN, int NT, int EPI, bool RES>
__device__ __forceinline__ void epi_prefetch(const GemmArgs& g, int m0, int tn, int tid, EpiPre<T, BM, BN, NT>& e) {
  using E = EpiPre<T, BM, BN, NT>;
  const int rr0 = tid / E::CPR, n = tn * BN + (tid % E::CPR) * 8;
#pragma unroll
  for (int q = 0; q < E::RPT; ++q) {
    const int m = m0 + rr0 + q * E::RSTEP;
    e.live[q] = rr0 + q * E::RSTEP < BM && m < g.M;
    // a dead slot reads the last row (M > 0); m0 itself can be past M where
    // a wave's part of a ragged tile holds no row at all
    const int mm = e.live[q] ? m : g.M - 1;
    e.bq[q] = mm / g.kk;
    e.jq[q] = mm - e.bq[q] * g.kk;
    e.pq[q] = epi_uses_positions(EPI) && g.idx ? clamp_pos(g.idx[mm], g.T) : e.jq[q];
  }
  if constexpr (RES && (EPI == EPI_RESID_STORE || EPI == EPI_RESID_SCATTER)) {
    if (n < g.N) {
#pragma unroll
      for (int q = 0; q < E::RPT; ++q) {
        if (!e.live[q]) continue;  // residual rows of live slots only
        const int m = m0 + rr0 + q * E::RSTEP;
        const T* src = (EPI == EPI_RESID_SCATTER && g.res)
                           ? (const T*)g.res + int64_t(m) * g.N + n
                           : (const T*)g.x + (int64_t(e.bq[q]) * g.T + e.pq[q]) * g.N + n;
        e.xr[q] = load_raw8(src);
      }
    }
  }
}

// stage: fp32 tile [BM][BN + 4] in LDS; tile origin (m0, tn). Each thread owns
// one 8-column chunk and walks the tile's rows, so everything that depends
// only on the column (bias, head, RoPE partner) is computed once. EPI is an
// EpiKind. rows: the thread's rows as epi_prefetch read them for this
// (m0, tn, tid); PRE: they include the residual rows (else these are loaded
// here).
template <typename T, int BM, int BN, int NT, int EPI, bool PRE>
__device__ __forceinline__ void gemm_epilogue_rows(const GemmArgs& g, const float* stage, int m0, int tn, int tid,
                                                   const EpiPre<T, BM, BN, NT>& rows) {
  constexpr int LD = BN + 4;
  if constexpr (EPI == EPI_SWIGLU) {
    // tile columns [0, BN/2) are gate units, [BN/2, BN) the matching up units
    constexpr int H = BN / 2, CPR = H / 8, RSTEP = NT / CPR;
    static_assert(NT % CPR == 0, "threads must tile the chunk columns");
    const int cc = (tid % CPR) * 8;
    for (int rr = tid / CPR; rr < BM; rr += RSTEP) {
      const int m = m0 + rr;
      if (m >= g.M) break;
      float y[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float gt = stage[rr * LD + cc + i];
        y[i] = (sizeof(T) == 2 ? silu_bf16(gt) : silu(gt)) * stage[rr * LD + H + cc + i];
      }
      store8((T*)g.out + int64_t(m) * g.ldo + tn * H + cc, y);
    }
    return;
  }
  constexpr int CPR = BN / 8, RSTEP = NT / CPR;
  static_assert(NT % CPR == 0, "threads must tile the chunk columns");
  const int cc = (tid % CPR) * 8;
  const int n = tn * BN + cc;
  if (n >= g.N) return;
  float bias[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) bias[i] = 0.f;
  if (g.bias) load8((const T*)g.bias + n, bias);
  if constexpr (EPI == EPI_RESID_SCATTER || EPI == EPI_RESID_SCATTER_GATE) {
    if (g.bias2) {
      float b2[8];
      load8((const T*)g.bias2 + n, b2);
#pragma unroll
      for (int i = 0; i < 8; ++i) bias[i] += b2[i];
    }
  }
  // QKV: which section (q, k, v), head and dims this chunk holds; hd is a power of two
  T* sec = nullptr;
  int heads = 0, head = 0, dim0 = 0, hshift = 0;
  bool rot = false;
  float pbias[8];
  if constexpr (EPI == EPI_QKV_ROPE) {
    hshift = 31 - __clz(g.hd);
    const int qcols = g.Hq << hshift, kcols = g.Hkv << hshift;
    int c = n;
    if (c < qcols) {
      sec = (T*)g.q; heads = g.Hq; rot = true;
    } else if (c < qcols + kcols) {
      sec = (T*)g.k; heads = g.Hkv; c -= qcols; rot = true;
    } else {
      sec = (T*)g.v; heads = g.Hkv; c -= qcols + kcols;
    }
    head = c >> hshift;
    dim0 = c & (g.hd - 1);
    rot = rot && dim0 < g.R;
    if (rot) {  // bias of each element's rotation partner (dims i and i + R/2)
      const int half = g.R / 2;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int dim = dim0 + i;
        const int pdim = dim < half ? dim + half : dim - half;
        pbias[i] = (g.bias && dim < g.R) ? Elem<T>::to_f(((const T*)g.bias)[n - dim0 + pdim]) : 0.f;
      }
    }
  }
  // Rows of this thread: rr0, rr0 + RSTEP, ... All their positions, and for
  // the residual kinds all their residual rows, are requested before any row
  // is finished, so the rows' memory latencies overlap instead of adding up.
  constexpr int RPT = (BM + RSTEP - 1) / RSTEP;
  const int rr0 = tid / CPR;
  const int(&bq)[RPT] = rows.bq;
  const int(&jq)[RPT] = rows.jq;
  const int(&pq)[RPT] = rows.pq;
  const bool(&live)[RPT] = rows.live;
  if constexpr (EPI == EPI_RESID_SCATTER_GATE) {
    // Gated scatter (Section 3.4): the block's update of each kept row,
    // delta = (resid + C + biases) - x[b, pos], is scaled by sigmoid of the
    // token's router score before it is added to x[b, pos]. The rows are held
    // as raw 16-byte vectors until used, which keeps this variant within the
    // register budget of the plain scatter.
    Raw8<T> rr[RPT], ro[RPT];
    float gs[RPT];
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      if (!live[q]) continue;
      const int m = m0 + rr0 + q * RSTEP;
      const int64_t xrow = int64_t(bq[q]) * g.T + pq[q];
      rr[q] = load_raw8(g.res ? (const T*)g.res + int64_t(m) * g.N + n : (const T*)g.x + xrow * g.N + n);
      if (g.res) ro[q] = load_raw8((const T*)g.x + xrow * g.N + n);
      gs[q] = g.gate[xrow];
    }
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      if (!live[q]) continue;
      const float* row = stage + (rr0 + q * RSTEP) * LD;
      const float sg = 1.f / (1.f + expf(-gs[q]));
      float r[8], v[8];
      unpack8(rr[q], r);
      if (g.res) {
        float o[8];
        unpack8(ro[q], o);
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = o[i] + sg * ((row[cc + i] + bias[i]) + (r[i] - o[i]));
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = r[i] + sg * (row[cc + i] + bias[i]);
      }
      store8((T*)g.x + (int64_t(bq[q]) * g.T + pq[q]) * g.N + n, v);
    }
    return;
  }
  if constexpr (EPI == EPI_RESID_STORE || EPI == EPI_RESID_SCATTER) {
    float xr[RPT][8];
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      if (!live[q]) continue;
      if constexpr (PRE) {
        unpack8(rows.xr[q], xr[q]);
        continue;
      }
      const int m = m0 + rr0 + q * RSTEP;
      const T* src = (EPI == EPI_RESID_SCATTER && g.res) ? (const T*)g.res + int64_t(m) * g.N + n
                                                         : (const T*)g.x + (int64_t(bq[q]) * g.T + pq[q]) * g.N + n;
      load8(src, xr[q]);
    }
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      if (!live[q]) continue;
      const int m = m0 + rr0 + q * RSTEP;
      const float* row = stage + (rr0 + q * RSTEP) * LD;
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = row[cc + i] + bias[i] + xr[q][i];
      if constexpr (EPI == EPI_RESID_STORE) store8((T*)g.out + int64_t(m) * g.ldo + n, v);
      else store8((T*)g.x + (int64_t(bq[q]) * g.T + pq[q]) * g.N + n, v);
    }
    return;
  }
  if constexpr (EPI == EPI_STORE_F32) {
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      if (!live[q]) continue;
      const int m = m0 + rr0 + q * RSTEP;
      const float* row = stage + (rr0 + q * RSTEP) * LD;
      float* dst = (float*)g.out + int64_t(m) * g.ldo + n;
      store_vec(dst, row + cc);
      store_vec(dst + 4, row + cc + 4);
    }
    return;
  }
  if constexpr (EPI == EPI_GELU_BWD || EPI == EPI_SWIGLU_BWD) {
    // gradient at the activation's input from the gradient at its output (C)
    // and the forward pre-activation(s) in res
    Raw8<T> ra[RPT], rb[RPT];
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      if (!live[q]) continue;
      const T* aux = (const T*)g.res + int64_t(m0 + rr0 + q * RSTEP) * g.ldo + n;
      ra[q] = load_raw8(aux);
      if constexpr (EPI == EPI_SWIGLU_BWD) rb[q] = load_raw8(aux + g.f);
    }
#pragma unroll
    for (int q = 0; q < RPT; ++q) {
      if (!live[q]) continue;
      const int m = m0 + rr0 + q * RSTEP;
      const float* row = stage + (rr0 + q * RSTEP) * LD;
      float a[8], v[8];
      unpack8(ra[q], a);
      T* dst = (T*)g.out + int64_t(m) * g.ldo + n;
      if constexpr (EPI == EPI_GELU_BWD) {
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = row[cc + i] * gelu_grad_bf16(a[i]);
        store8(dst, v);
      } else {
        float up[8], w[8];
        unpack8(rb[q], up);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          v[i] = row[cc + i] * up[i] * silu_grad_bf16(a[i]);
          w[i] = row[cc + i] * silu_bf16(a[i]);
        }
        store8(dst, v);
        store8(dst + g.f, w);
      }
    }
    return;
  }
#pragma unroll
  for (int q = 0; q < RPT; ++q) {
    if (!live[q]) continue;
    const int m = m0 + rr0 + q * RSTEP;
    const float* row = stage + (rr0 + q * RSTEP) * LD;
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = row[cc + i] + bias[i];
    if constexpr (EPI == EPI_STORE) {
      store8((T*)g.out + int64_t(m) * g.ldo + n, v);
    } else if constexpr (EPI == EPI_QKV_ROPE) {
      // columns: Q heads, then K heads, then V heads; written head-major [B, H, kk, hd]
      T* dst = sec + ((int64_t(bq[q]) * heads + head) * g.kk + jq[q]) * g.hd + dim0;
      if (rot) {
        const int half = g.R / 2;
        float out[8];
        if ((g.R & 15) == 0) {
          // the chunk's 8 dims lie in one half: their (cos, sin) pairs are 64
          // contiguous bytes of the table, their partners the chunk half a span away
          const bool lo = dim0 < half;
          const int off = lo ? half : -half;
          const float4* cs = reinterpret_cast<const float4*>(g.rope + (int64_t(pq[q]) * half + (lo ? dim0 : dim0 - half)) * 2);
#pragma unroll
          for (int p2 = 0; p2 < 4; ++p2) {
            const float4 c = cs[p2];
#pragma unroll
            for (int e = 0; e < 2; ++e) {
              const int i = 2 * p2 + e;
              const float cv = e ? c.z : c.x, sv = e ? c.w : c.y;
              const float xp = row[cc + off + i] + pbias[i];
              out[i] = lo ? v[i] * cv - xp * sv : v[i] * cv + xp * sv;
            }
          }
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const int dim = dim0 + i;
            if (dim >= g.R) {
              out[i] = v[i];
              continue;
            }
            const bool lo = dim < half;
            const int pdim = lo ? dim + half : dim - half;
            const float xp = row[cc - dim0 + pdim] + pbias[i];
            const float* cs = g.rope + (int64_t(pq[q]) * half + (lo ? dim : dim - half)) * 2;
            out[i] = lo ? v[i] * cs[0] - xp * cs[1] : v[i] * cs[0] + xp * cs[1];
          }
        }
        store8(dst, out);
      } else {
        store8(dst, v);
      }
    } else {  // EPI_BIAS_GELU
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = sizeof(T) == 2 ? gelu_bf16(v[i]) : gelu_erf(v[i]);
      store8((T*)g.out + int64_t(m) * g.ldo + n, v);
    }
  }
}

template <typename T, int BM, int BN, int NT, int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& g, const float* stage, int m0, int tn, int tid) {
  EpiPre<T, BM, BN, NT> rows;
  if constexpr (EPI != EPI_SWIGLU) epi_prefetch<T, BM, BN, NT, EPI, false>(g, m0, tn, tid, rows);  // rows only
  gemm_epilogue_rows<T, BM, BN, NT, EPI, false>(g, stage, m0, tn, tid, rows);
}

// ----------------------------------------------------------- bf16 MFMA GEMM

constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kWM = 64, kWN = 64;
constexpr int kThreads = 256;
constexpr int kStageLD = kBN + 4;
constexpr int kTileBytes = 2 * (kBM + kBN) * kBK * 2;       // double-buffered A and B tiles
constexpr int kStageBytes = kBM * kStageLD * 4;             // fp32 epilogue tile
constexpr int kSmemBytes = kTileBytes > kStageBytes ? kTileBytes : kStageBytes;

// Row of the B operand (weight matrix) that tile row r of column tile tn reads.
template <int EPI>
__device__ __forceinline__ int b_row(const GemmArgs& g, int tn, int r) {
  if constexpr (EPI == EPI_SWIGLU) {
    constexpr int H = kBN / 2;
    return r < H ? tn * H + r : g.f + tn * H + (r - H);
  }
  int n = tn * kBN + r;
  return n < g.N ? n : g.N - 1;
}

template <int EPI>
__global__ __launch_bounds__(kThreads, 2) void gemm_bf16_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) char smem[kSmemBytes];
  uint16_t* As = reinterpret_cast<uint16_t*>(smem);
  uint16_t* Bs = As + 2 * kBM * kBK;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int r16 = lane & 15, grp = lane >> 4;
  const int tn = blockIdx.x, tm = blockIdx.y;
  const int m0 = tm * kBM;

  // this thread's four A rows and four B rows (tile rows tid/8 + 32 i), chunk tid%8
  const int lrow = tid >> 3, lch = tid & 7;
  const uint16_t* arow[4];
  const uint16_t* arow2[4];
  const uint16_t* brow[4];
  const uint16_t* brow2[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int m = m0 + lrow + 32 * i;
    if (m > g.M - 1) m = g.M - 1;
    arow[i] = (const uint16_t*)g.a + int64_t(m) * g.lda;
    arow2[i] = g.a2 ? (const uint16_t*)g.a2 + int64_t(m) * g.lda2 : nullptr;
    const int n = b_row<EPI>(g, tn, lrow + 32 * i);
    brow[i] = (const uint16_t*)g.b + int64_t(n) * g.ldb;
    brow2[i] = g.b2 ? (const uint16_t*)g.b2 + int64_t(n) * g.ldb2 : nullptr;
  }

  u32x4 ra[4], rb[4];
  auto gload = [&](int kt) {
    const int k0 = kt * kBK;
    const bool second = k0 >= g.K1;
    const int kc = (second ? k0 - g.K1 : k0) + lch * 8;
    const bool ok = k0 + lch * 8 < g.K;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint16_t* pa = (second ? arow2[i] : arow[i]) + kc;
      const uint16_t* pb = (second ? brow2[i] : brow[i]) + kc;
      ra[i] = ok ? *reinterpret_cast<const u32x4*>(pa) : u32x4{0, 0, 0, 0};
      rb[i] = ok ? *reinterpret_cast<const u32x4*>(pb) : u32x4{0, 0, 0, 0};
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = lrow + 32 * i;
      const int off = row * kBK + ((lch ^ (row & 7)) << 3);
      *reinterpret_cast<u32x4*>(As + buf * kBM * kBK + off) = ra[i];
      *reinterpret_cast<u32x4*>(Bs + buf * kBN * kBK + off) = rb[i];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = (g.K + kBK - 1) / kBK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    const uint16_t* At = As + cur * kBM * kBK;
    const uint16_t* Bt = Bs + cur * kBN * kBK;
#pragma unroll
    for (int ks = 0; ks < kBK / 32; ++ks) {
      bf16x8 af[4], bfr[4];
      const int ch = ks * 4 + grp;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int ar = wm * kWM + i * 16 + r16;
        af[i] = *reinterpret_cast<const bf16x8*>(At + ar * kBK + ((ch ^ (ar & 7)) << 3));
        const int br = wn * kWN + i * 16 + r16;
        bfr[i] = *reinterpret_cast<const bf16x8*>(Bt + br * kBK + ((ch ^ (br & 7)) << 3));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // accumulator element (i, j, e) is C[wm*64 + 16 i + 4 grp + e][wn*64 + 16 j + r16]
  float* stage = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        stage[(wm * kWM + 16 * i + 4 * grp + e) * kStageLD + wn * kWN + 16 * j + r16] = acc[i][j][e];
  __syncthreads();
  gemm_epilogue<uint16_t, kBM, kBN, kThreads, EPI>(g, stage, m0, tn, threadIdx.x);
}

// ------------------------------------------- bf16 MFMA GEMM, LDS-DMA ring

// Tiles arrive in LDS straight from global memory (global_load_lds_dwordx4:
// each lane moves 16 bytes, a wavefront fills 1 KiB of consecutive tile rows
// at a wave-uniform LDS address). The lane picks WHICH global chunk it loads,
// so the LDS copy comes out XOR-swizzled without passing through registers.
// NS stages of BK columns form a ring: while tile kt is multiplied, tiles
// kt+1 .. kt+NS-1 are in flight. Requires K % BK == 0 and K1 % BK == 0.
//
// Swizzle: a tile row is BK/8 chunks of 16 bytes. With BK = 64 (128-byte rows)
// chunk c of row r sits at c ^ (r & 7); with BK = 32 (64-byte rows, two rows
// per 128-byte bank line) at c ^ ((r >> 1) & 3). Either way the 8 lanes that
// one 128-byte LDS cycle serves (8 consecutive rows, one logical chunk) hit 8
// distinct bank groups.
template <int BK>
__device__ __forceinline__ int swz(int row, int ch) {
  if constexpr (BK == 64) return ch ^ (row & 7);
  else return ch ^ ((row >> 1) & 3);
}

template <int BM, int BN, int WM, int WN, int NS, int BK>
struct DmaCfg {
  static constexpr int kWaves = (BM / WM) * (BN / WN);
  static constexpr int kThreads = kWaves * 64;
  static constexpr int kRowBytes = BK * 2;
  static constexpr int kRowsPerLoad = 1024 / kRowBytes;             // tile rows one wavefront load fills
  static constexpr int kStage = (BM + BN) * kRowBytes;              // bytes per stage
  static constexpr int kLoadsA = BM / kRowsPerLoad / kWaves;        // loads per wave per tile
  static constexpr int kLoadsB = BN / kRowsPerLoad / kWaves;
  static constexpr int kLoads = kLoadsA + kLoadsB;
  // Epilogue staging: the whole fp32 tile, or (wave tiles 128 wide) each wave
  // stages 32 rows x WN of its own tile at a time.
  static constexpr bool kWaveEpi = WN == 128;
  static constexpr int kStageLD = (kWaveEpi ? WN : BN) + 4;
  static constexpr int kStageBytes = kWaveEpi ? kWaves * 32 * kStageLD * 4 : BM * kStageLD * 4;
  static constexpr int kSmem = NS * kStage > kStageBytes ? NS * kStage : kStageBytes;
  static_assert(BK == 32 || BK == 64, "BK");
  static_assert(BM % (kRowsPerLoad * kWaves) == 0 && BN % (kRowsPerLoad * kWaves) == 0,
                "tile rows must split evenly over waves");
  static_assert(NS >= 2 && (NS - 1) * kLoads < 64, "vmcnt range");
};

// Scheduling fence (no instruction moves across it), used to keep the next
// substep's LDS reads ahead of the current substep's MFMAs.
#ifndef DSF_SCHED_FENCES
#define DSF_SCHED_FENCES 1
#endif
#if DSF_SCHED_FENCES
#define DSF_SCHED_FENCE() __builtin_amdgcn_sched_barrier(0)
#else
#define DSF_SCHED_FENCE() ((void)0)
#endif

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // the memory clobber orders the compiler's LDS reads after the DMA has landed
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier of the DMA ring. __syncthreads() would also wait for every
// outstanding global access (vmcnt(0)), draining the tiles still in flight and
// reducing any ring to double buffering; here each wave has already waited for
// its own share of the tile it needs. The memory clobber keeps the compiler's
// LDS reads of the new tile below the barrier.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// A row-major bf16 matrix as a DMA source: a buffer resource covering its
// rows x ld elements (range-checked: loads past the end read as zeros).
struct RowSrc {
  __amdgpu_buffer_rsrc_t rsrc;
  int ld;
  __device__ RowSrc(const void* p, int rows, int ld_) : ld(ld_) {
    const int64_t bytes = p ? int64_t(rows) * ld_ * 2 : 0;
    rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, int(bytes), 0x00020000);
  }
};

// 16 bytes per lane from byte offset voff + soff of src into LDS at
// lds + 16 * lane (lds and soff are wave-uniform). Kept out of lambdas: the
// builtin exists only for the device.
__device__ __forceinline__ void dma16(const RowSrc& src, uint32_t voff, uint32_t soff, char* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(src.rsrc, (__attribute__((address_space(3))) void*)lds, 16, int(voff),
                                           int(soff), 0, 0);
}

// Device-side pieces of the LDS-DMA GEMM: the main loop over a range of
// k-tiles of one output tile, and the fused epilogue of a finished tile.
// Tile configurations of the LDS-DMA GEMM (DSF_GEMM_USE_DMA=0 keeps every
// bf16 GEMM on the register-staged kernel). Small: 128 x 128 tiles of four
// 64 x 64 waves, two workgroups per CU. Large: 256 x 256 tiles of eight
// 64 x 128 waves, one workgroup per CU; per flop it loads half the tile
// bytes from L2 and reads half the fragment bytes from LDS, which pays when
// there are enough tiles to fill the chip (the large projections).
#ifndef DSF_GEMM_USE_DMA
#define DSF_GEMM_USE_DMA 1
#endif
struct TileSmall {
  static constexpr int BM = 128, BN = 128, WM = 64, WN = 64, NS = 2, BK = 64;
};
struct TileLarge {
  static constexpr int BM = 256, BN = 256, WM = 64, WN = 128, NS = 2, BK = 64;
};

// Stream-K partial tiles: one slot per workgroup of a persistent grid, at
// most kSkMaxSlots workgroups (2 per CU on a 256-CU device with small tiles,
// 1 with large tiles).
constexpr int kSkMaxSlots = 512;
constexpr int kSkMinIters = 8;  // mean k-iterations per workgroup below which one tile per workgroup is kept
constexpr int kSkMinK = 32;    // k-iterations per tile below which the partial sums cost more than they save
// Split last round (choose_tail): at most this many pieces per tile, each at
// least this many k-iterations long.
constexpr int kTailMaxSplit = 4;
constexpr int kTailMinK = 8;
constexpr int kGroupM = 4;      // tile rows per band of the grouped tile order
constexpr int kGroupMinCols = 8;  // below this many tile columns row-major order is already compact
constexpr size_t kSkPartBytes = size_t(kSkMaxSlots) / 2 * TileLarge::BM * TileLarge::BN * sizeof(float);
static_assert(kSkPartBytes >= size_t(kSkMaxSlots) * TileSmall::BM * TileSmall::BN * sizeof(float),
              "partial-tile slots of the small tiles");

template <int EPI, int BM, int BN, int WM, int WN, int NS, int BK>
struct DmaGemm {
  using C = DmaCfg<BM, BN, WM, WN, NS, BK>;
  static constexpr int MI = WM / 16, NI = WN / 16;
  static constexpr int CPR = BK / 8;  // chunks per tile row
  static constexpr int RPL = C::kRowsPerLoad;
  typedef f32x4 Acc[MI][NI];

  // acc = A[rows of tile tm, k-tiles kb..ke-1] . B[rows of tile tn, same]^T.
  // Starts with a barrier, so the ring may still hold the previous tile.
  __device__ static __forceinline__ void mainloop(const GemmArgs& g, char* smem, int tm, int tn, int kb, int ke,
                                                  Acc& acc) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / (BN / WN), wn = wave % (BN / WN);
    const int r16 = lane & 15, grp = lane >> 4;
    const int m0 = tm * BM;
    // DMA sources are buffer resources over A, A2, B, B2 whose size is the
    // matrix's rows x leading dimension: a row beyond M (or N) is out of range
    // and reads as zeros, so ragged tiles need no clamping. Load i of this
    // wave fills tile rows RPL (wave + kWaves i) .. + RPL; the lane part of
    // the offset (row lane / CPR, physical chunk lane % CPR holding logical
    // chunk swz^-1) is the same for every load, the row base is uniform.
    const int lr = lane / CPR;
    const int lc = swz<BK>(lr, lane % CPR);  // swz is an involution for a fixed row
    const RowSrc sa{g.a, g.M, g.lda}, sa2{g.a2, g.M, g.lda2};
    const int nrows_b = EPI == EPI_SWIGLU ? 2 * g.f : g.N;
    const RowSrc sb{g.b, nrows_b, g.ldb}, sb2{g.b2, nrows_b, g.ldb2};
    const uint32_t va = uint32_t(lr * g.lda + lc * 8) * 2u, va2 = uint32_t(lr * g.lda2 + lc * 8) * 2u;
    const uint32_t vb = uint32_t(lr * g.ldb + lc * 8) * 2u, vb2 = uint32_t(lr * g.ldb2 + lc * 8) * 2u;
    // first B row of load i (uniform)
    auto brow = [&](int i) {
      const int r = RPL * (wave + C::kWaves * i);
      if constexpr (EPI == EPI_SWIGLU) {
        // each 128-row block of the B tile holds 64 gate units then the same 64 up units
        const int blk = r / 128, rr = r % 128, u0 = (tn * (BN / 128) + blk) * 64;
        return rr < 64 ? u0 + rr : g.f + u0 + (rr - 64);
      } else {
        return tn * BN + r;
      }
    };
    auto issue = [&](int kt) {
      const int k0 = kt * BK;
      const bool second = k0 >= g.K1;
      const int kc = second ? k0 - g.K1 : k0;
      char* st = smem + (kt % NS) * C::kStage;
      const RowSrc& A = second ? sa2 : sa;
      const RowSrc& Bm = second ? sb2 : sb;
      const uint32_t vA = second ? va2 : va, vB = second ? vb2 : vb;
#pragma unroll
      for (int i = 0; i < C::kLoadsA; ++i)
        dma16(A, vA, uint32_t((m0 + RPL * (wave + C::kWaves * i)) * A.ld + kc) * 2u,
              st + 1024 * (wave + C::kWaves * i));
#pragma unroll
      for (int i = 0; i < C::kLoadsB; ++i)
        dma16(Bm, vB, uint32_t(brow(i) * Bm.ld + kc) * 2u, st + BM * C::kRowBytes + 1024 * (wave + C::kWaves * i));
    };

#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Every wave is done with the LDS before the ring is refilled. Stores of
    // an earlier tile may still be in flight: they only add to the counter,
    // so each wait below still covers the loads it is for (whether or not the
    // stores retire in order), and they drain under this tile's first loads.
    ring_barrier();
    // Ring of NS buffers, all filled ahead: tile kt lives in buffer kt % NS,
    // and tile kt + NS is issued into it as soon as tile kt has been read.
#pragma unroll
    for (int s = 0; s < NS; ++s)
      if (kb + s < ke) issue(kb + s);
    if (kb + NS - 1 < ke) wait_vmcnt<(NS - 1) * C::kLoads>();  // tile kb has landed
    else wait_vmcnt<0>();
    ring_barrier();

    constexpr int KS = BK / 32;   // 32-deep MFMA substeps per tile
    constexpr int G = KS * MI;    // MFMA groups per tile (one A fragment each)
    auto tileA = [&](int kt) { return reinterpret_cast<const uint16_t*>(smem + (kt % NS) * C::kStage); };
    bf16x8 bq[2][NI];             // B fragments of the current and the next substep
    auto read_b = [&](const uint16_t* At, int ks, int buf) {
      const uint16_t* Bt = At + BM * BK;
      const int ch = ks * 4 + grp;
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int br = wn * WN + j * 16 + r16;
        bq[buf][j] = *reinterpret_cast<const bf16x8*>(Bt + br * BK + (swz<BK>(br, ch) << 3));
      }
    };
    auto read_a = [&](const uint16_t* At, int ks, int i) -> bf16x8 {
      const int ar = wm * WM + i * 16 + r16;
      return *reinterpret_cast<const bf16x8*>(At + ar * BK + (swz<BK>(ar, ks * 4 + grp) << 3));
    };
    read_b(tileA(kb), 0, 0);
    bf16x8 a_cur = read_a(tileA(kb), 0, 0);

    // One tile. Software pipeline over its MFMA groups: the next A fragment is
    // read before the NI MFMAs of the current one, and the next substep's B
    // fragments halfway through the current substep. In the last group the
    // workgroup moves on to tile kt + 1: wait for its loads, one barrier (all
    // reads of tile kt are complete, so its buffer takes tile kt + NS), and
    // read tile kt + 1's first fragments under the group's remaining MFMAs,
    // so no tile starts with an exposed LDS wait. B fragments alternate
    // between the two register sets by substep; P is the tile's parity
    // relative to kb, which makes every index below a compile-time constant.
    auto step = [&](int kt, auto Pc) {
      constexpr int P = decltype(Pc)::value;
      const uint16_t* At = tileA(kt);
      const bool has_next = kt + 1 < ke;
#pragma unroll
      for (int gi = 0; gi < G; ++gi) {
        const int ks = gi / MI, i = gi % MI;
        const int cb = (P * KS + ks) & 1;
        acc[i][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_cur, bq[cb][0], acc[i][0], 0, 0, 0);
        DSF_SCHED_FENCE();
        bf16x8 a_nxt = a_cur;
        if (gi + 1 < G) {
          a_nxt = read_a(At, (gi + 1) / MI, (gi + 1) % MI);
          if (i == MI / 2 && ks + 1 < KS) read_b(At, ks + 1, (P * KS + ks + 1) & 1);
        } else if (has_next) {
          // tile kt + 1 has landed once the tiles issued after it are all that remain
          if (kt + NS - 1 < ke) wait_vmcnt<(NS - 2) * C::kLoads>();
          else wait_vmcnt<0>();
          ring_barrier();
          if (kt + NS < ke) issue(kt + NS);
          const uint16_t* An = tileA(kt + 1);
          read_b(An, 0, ((P + 1) * KS) & 1);
          a_nxt = read_a(An, 0, 0);
        }
        DSF_SCHED_FENCE();
#pragma unroll
        for (int j = 1; j < NI; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_cur, bq[cb][j], acc[i][j], 0, 0, 0);
        DSF_SCHED_FENCE();
        a_cur = a_nxt;
      }
    };
    if constexpr (KS % 2 == 0) {
      for (int kt = kb; kt < ke; ++kt) step(kt, std::integral_constant<int, 0>());
    } else {
      int kt = kb;
      for (; kt + 1 < ke; kt += 2) {
        step(kt, std::integral_constant<int, 0>());
        step(kt + 1, std::integral_constant<int, 1>());
      }
      if (kt < ke) step(kt, std::integral_constant<int, 0>());
    }
  }

  // Stage the finished tile (tm, tn) through LDS and apply the fused epilogue.
  // NP > 0 (wave-staged tiles only): the tile's sum also takes the partials
  // in slots slot0 .. slot0 + np - 1 (np <= NP, published before the call),
  // added in slot order to each fragment as it is staged, a few fragments'
  // loads in flight at a time; a partial beyond np is read beyond the end of
  // the buffer, out of the resource's range, where every load returns zeros.
  // PF: request the rows' positions and residual rows before the barrier
  // (off in the persistent stream-K kernel, whose registers are taken).
  template <int NP = 0, bool PF = true>
  __device__ static __forceinline__ void epilogue(const GemmArgs& g, char* smem, int tm, int tn, Acc& acc,
                                                  int slot0 = 0, int np = 0) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / (BN / WN), wn = wave % (BN / WN);
    const int r16 = lane & 15, grp = lane >> 4;
    const int m0 = tm * BM;
    // wave-staged tiles: the rows' positions (and residual rows) of every
    // round are requested first, so that their latency overlaps the barrier
    // and the staging instead of starting each round (not beside the
    // partials' loads, which take those registers)
    using Pre = EpiPre<uint16_t, 32, 128, 64>;
    constexpr bool kPre = C::kWaveEpi && PF && epi_uses_positions(EPI) && NP == 0;
    Pre pre[kPre ? MI / 2 : 1];
    if constexpr (kPre) {
#pragma unroll
      for (int rnd = 0; rnd < MI / 2; ++rnd)
        epi_prefetch<uint16_t, 32, 128, 64, EPI, true>(g, m0 + wm * WM + 32 * rnd, tn * (BN / 128) + wn, lane, pre[rnd]);
    }
    // workgroup-staged tiles: the same for the thread's rows of the whole tile
    using PreT = EpiPre<uint16_t, BM, BN, C::kThreads>;
    constexpr bool kPreT = !C::kWaveEpi && PF && epi_uses_positions(EPI) && NP == 0;
    PreT pre_t;
    if constexpr (kPreT) epi_prefetch<uint16_t, BM, BN, C::kThreads, EPI, true>(g, m0, tn, tid, pre_t);
    __syncthreads();  // all waves are done reading the ring before it becomes the epilogue tile
    if constexpr (C::kWaveEpi) {
      // each wave stages and finishes its own tile, 32 rows at a time, as a
      // 32 x 128 virtual tile whose column index is 2 tn + wn (BN = 256) or tn
      float* stage = reinterpret_cast<float*>(smem) + wave * 32 * C::kStageLD;
      const int vtn = tn * (BN / 128) + wn;
#pragma unroll
      for (int rnd = 0; rnd < MI / 2; ++rnd) {
#pragma unroll
        for (int ii = 0; ii < 2; ++ii)
#pragma unroll
          for (int j0 = 0; j0 < NI; j0 += kAddGroup) {
            if constexpr (NP > 0) {
              const auto r = part_rsrc(g);
              const int vo = lane_offset();
#pragma unroll
              for (int pp = 0; pp < NP; ++pp) {
                const int so = __builtin_amdgcn_readfirstlane(pp < np ? (slot0 + pp) * kSlotBytes : int(kSkPartBytes));
#pragma unroll
                for (int j = j0; j < j0 + kAddGroup; ++j)
                  acc[2 * rnd + ii][j] += __builtin_bit_cast(
                      f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, vo + ((2 * rnd + ii) * NI + j) * kFragBytes, so,
                                                                   kCoherent));
              }
            }
#pragma unroll
            for (int j = j0; j < j0 + kAddGroup; ++j)
#pragma unroll
              for (int e = 0; e < 4; ++e)
                stage[(16 * ii + 4 * grp + e) * C::kStageLD + 16 * j + r16] = acc[2 * rnd + ii][j][e];
            if constexpr (NP > 0) __builtin_amdgcn_sched_barrier(0);
          }
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
        __builtin_amdgcn_wave_barrier();
        if constexpr (kPre)
          gemm_epilogue_rows<uint16_t, 32, 128, 64, EPI, true>(g, stage, m0 + wm * WM + 32 * rnd, vtn, lane, pre[rnd]);
        else
          gemm_epilogue<uint16_t, 32, 128, 64, EPI>(g, stage, m0 + wm * WM + 32 * rnd, vtn, lane);
        __builtin_amdgcn_s_waitcnt(0xc07f);
        __builtin_amdgcn_wave_barrier();
      }
    } else {
      float* stage = reinterpret_cast<float*>(smem);
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            stage[(wm * WM + 16 * i + 4 * grp + e) * C::kStageLD + wn * WN + 16 * j + r16] = acc[i][j][e];
      __syncthreads();
      if constexpr (kPreT)
        gemm_epilogue_rows<uint16_t, BM, BN, C::kThreads, EPI, true>(g, stage, m0, tn, tid, pre_t);
      else
        gemm_epilogue<uint16_t, BM, BN, C::kThreads, EPI>(g, stage, m0, tn, threadIdx.x);
    }
  }

  // Partial tiles of the stream-K schedule live in slot-major order, each in
  // the accumulators' own register layout: (slot, wave, i, j, lane) -> f32x4,
  // so fragment f = i * NI + j of a wave's partial sits kFragBytes * f after
  // the lane's first one, and slot s starts kSlotBytes * s into the buffer.
  static constexpr int kFragBytes = 64 * 16;
  static constexpr int kSlotBytes = C::kWaves * MI * NI * kFragBytes;

  // The partial sums go from one workgroup to another, possibly on another
  // XCD (each XCD has its own L2). They are stored and loaded with
  // device-scope coherent accesses (sc1 in the buffer instructions' cache
  // policy), which is what the relaxed device-scope atomics on the flags use
  // as well, so the hand-over needs only a completion wait: no write-back of
  // the writer's whole L2 before the flag, no invalidation of the reader's L2
  // after it (both would cost every other workgroup on those XCDs its cached
  // tiles). The accesses are compiler intrinsics, so the compiler places the
  // waits for the loads and overlaps as many of them as registers allow.
  static constexpr int kCoherent = 16;  // cache policy: sc1
  static constexpr int kAddGroup = 8;
  __device__ static __forceinline__ __amdgpu_buffer_rsrc_t part_rsrc(const GemmArgs& g) {
    return __builtin_amdgcn_make_buffer_rsrc(g.part, (short)0, int(kSkPartBytes), 0x00020000);
  }
  __device__ static __forceinline__ int lane_offset() {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    return wave * (MI * NI * kFragBytes) + lane * 16;
  }

  // Store the partial into slot; returns once every store has completed. The
  // slot offset goes into the vector offset and the scalar offset is the
  // constant 0: the compiler then keeps the store-data hazard of 128-bit
  // buffer stores (a VALU write to a store's data registers right after it
  // changes what the later lanes store) with a wait state. With a register
  // scalar offset it assumes no hazard and reuses the data registers at
  // once, which corrupted a few elements of some partials.
  __device__ static __forceinline__ void store_partial(const GemmArgs& g, const Acc& acc, int slot) {
    const f32x4* a = &acc[0][0];
    const auto r = part_rsrc(g);
    const int vo = lane_offset() + slot * kSlotBytes;
#pragma unroll
    for (int f = 0; f < MI * NI; ++f)
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, a[f]), r, vo + f * kFragBytes, 0, kCoherent);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }

  // acc += the partials in slots slot0 .. slot0 + n - 1 (published before
  // this call), added in slot order, n <= NMAX. Straight-line code over NMAX
  // partials, so that the accumulators stay in place and the loads overlap:
  // a partial beyond n is read at the end of the buffer, out of the
  // resource's range, where every load returns zeros.
  template <int NMAX>
  __device__ static __forceinline__ void add_partials(const GemmArgs& g, int slot0, int n, Acc& acc) {
    f32x4* a = &acc[0][0];
    const auto r = part_rsrc(g);
    const int vo = lane_offset();
    int so[NMAX];
#pragma unroll
    for (int pp = 0; pp < NMAX; ++pp)
      so[pp] = __builtin_amdgcn_readfirstlane(pp < n ? (slot0 + pp) * kSlotBytes : int(kSkPartBytes));
    // kAddGroup fragments of every partial in flight at a time (their loads
    // are not hoisted past the group boundary, which would spill)
#pragma unroll
    for (int f0 = 0; f0 < MI * NI; f0 += kAddGroup) {
#pragma unroll
      for (int f = f0; f < f0 + kAddGroup; ++f)
#pragma unroll
        for (int pp = 0; pp < NMAX; ++pp)
          a[f] += __builtin_bit_cast(f32x4,
                                     __builtin_amdgcn_raw_buffer_load_b128(r, vo + f * kFragBytes, so[pp], kCoherent));
      __builtin_amdgcn_sched_barrier(0);
    }
  }
};

// One output tile per workgroup (grid = tiles). Each XCD takes one contiguous
// range of the tile order (gemm_sched.h): row-major, or bands of g.group_m
// tile rows walked column by column when the grid has more tiles than
// resident workgroups.
template <int EPI, int BM, int BN, int WM, int WN, int NS, int BK>
__global__ __launch_bounds__((DmaCfg<BM, BN, WM, WN, NS, BK>::kThreads)) void gemm_bf16_dma_kernel(GemmArgs g) {
  using G = DmaGemm<EPI, BM, BN, WM, WN, NS, BK>;
  __shared__ __attribute__((aligned(1024))) char smem[G::C::kSmem];
  // the grid covers the first gridDim.x tiles of the order (all of them, or
  // all but a split last round)
  const GemmTile t = gemm_tile(xcd_remap(int(blockIdx.x), int(gridDim.x)), g.ntm, g.ntn, g.group_m);
  const int tm = t.tm, tn = t.tn;
  typename G::Acc acc;
  G::mainloop(g, smem, tm, tn, 0, g.K / BK, acc);
  G::epilogue(g, smem, tm, tn, acc);
}

// The last round of a one-tile-per-workgroup grid, split along K: tiles
// tail0 .. tail0 + tail_r - 1 of the tile order, each cut into tail_s
// contiguous pieces of its k-tiles, tail_s * tail_r pieces for at most as many
// resident workgroups, so the round takes about 1 / tail_s of a tile. The
// pieces of a tile run on one XCD (tile t on XCD t % 8, its pieces at
// launch indices 8 (tail_s q + p) + t % 8 with q = t / 8), the last piece
// at the highest index. The other pieces publish partial sums (slot
// t (tail_s - 1) + p) with device-coherent stores and a flag; the last piece
// waits for them in piece order, adds them and runs the fused epilogue. Only
// the last piece waits, and only for workgroups of its XCD dispatched before
// it that never wait: the waits end. The bounded spin of the stream-K kernel
// guards them the same way (status word on a give-up).
template <int EPI, int BM, int BN, int WM, int WN, int NS, int BK>
__global__ __launch_bounds__((DmaCfg<BM, BN, WM, WN, NS, BK>::kThreads)) void gemm_bf16_tail_kernel(GemmArgs g) {
  using G = DmaGemm<EPI, BM, BN, WM, WN, NS, BK>;
  __shared__ __attribute__((aligned(1024))) char smem[G::C::kSmem];
  __shared__ int n_seen;
  const int s = g.tail_s;
  const int x = int(blockIdx.x) % kXcds, m = int(blockIdx.x) / kXcds;
  const int q = m / s, p = m - q * s, t = x + kXcds * q;
  if (t >= g.tail_r) return;  // padding of the last group (uniform)
  const int nk = g.K / BK;
  const int kb = int(int64_t(nk) * p / s), ke = int(int64_t(nk) * (p + 1) / s);
  const GemmTile tt = gemm_tile(g.tail0 + t, g.ntm, g.ntn, g.group_m);
  typename G::Acc acc;
  G::mainloop(g, smem, tt.tm, tt.tn, kb, ke, acc);
  if (p < s - 1) {
    const int slot = t * (s - 1) + p;
    G::store_partial(g, acc, slot);
    __syncthreads();  // every wave's partial stores have completed
    if (threadIdx.x == 0) __hip_atomic_store(g.flags + slot, g.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  // the finisher (highest workgroup id of its tile) waits for the partials
  // in piece order, then adds those it has seen
  if (threadIdx.x == 0) {
    int seen = 0;
    for (; seen < s - 1; ++seen) {
      int it = 0;
      while (it < g.spin_limit &&
             __hip_atomic_load(g.flags + t * (s - 1) + seen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != g.epoch) {
        __builtin_amdgcn_s_sleep(2);
        ++it;
      }
      if (it == g.spin_limit) break;
    }
    n_seen = seen;
    if (seen < s - 1 && g.status)
      __hip_atomic_fetch_or(g.status, uint32_t(DSF_WS_STATUS_SK_TIMEOUT), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();  // the partials' loads below are issued after their flags were seen
  // a partial not seen is left out (and reported) rather than waited for
  G::template epilogue<kTailMaxSplit - 1>(g, smem, tt.tm, tt.tn, acc, t * (s - 1),
                                          __builtin_amdgcn_readfirstlane(n_seen));
}

// Persistent grid of 8 * px workgroups (workgroup w runs on XCD w % 8 as the
// hardware deals workgroups to the 8 XCDs in turn). The tiles, in the order
// of gemm_sched.h (bands of g.group_m tile rows), are cut into 8 contiguous
// ranges, one per XCD, and each XCD's px
// workgroups share its range as an independent problem. With g.split == 0
// they take whole tiles only (tile j, j + px, ...): a workgroup moves on to
// its next tile while its last tile's stores drain. With g.split == 1
// (stream-K) they take whole tiles while at least two full rounds remain,
// then the remaining k-iterations (tiles x K/BK) in px equal contiguous
// pieces.
// A piece that covers only part of a tile leaves a partial sum: the
// workgroup holding the tile's last k-iteration finishes it, adding the
// partials of the lower-numbered workgroups that hold its earlier iterations
// (a fixed order, so results do not depend on timing). Each workgroup walks
// its piece from the end backwards, so the one partial it can leave (at the
// top of its piece) is written first, and it waits only for lower-numbered
// workgroups of its own XCD, which are dispatched before it and never wait
// before writing their partial: the waits always end. A bounded spin keeps
// even a broken dispatch order from hanging the device: a finisher that gives
// up leaves its tile without the missing partials and reports it in the
// call's status word (g.status), which the host reads back.
template <int EPI, int BM, int BN, int WM, int WN, int NS, int BK>
__global__ __launch_bounds__((DmaCfg<BM, BN, WM, WN, NS, BK>::kThreads)) void gemm_bf16_sk_kernel(GemmArgs g) {
  using G = DmaGemm<EPI, BM, BN, WM, WN, NS, BK>;
  __shared__ __attribute__((aligned(1024))) char smem[G::C::kSmem];
  __shared__ int spin_failed;
  const int ntn = EPI == EPI_SWIGLU ? g.f / (BN / 2) : (g.N + BN - 1) / BN;
  const int nt = g.ntm * ntn, nk = g.K / BK, px = g.px;
  const int x = int(blockIdx.x) % kXcds, j = int(blockIdx.x) / kXcds;
  const int t0 = int(int64_t(nt) * x / kXcds), ntx = int(int64_t(nt) * (x + 1) / kXcds) - t0;
  const int full = ntx / px, rem = ntx % px;
  // whole tiles only (g.split == 0), or whole tiles while two or more rounds remain
  const int dp = (!g.split || rem == 0) ? ntx : (full >= 1 ? (full - 1) * px : 0);
  typename G::Acc acc;
  for (int t = j; t < dp; t += px) {
    const GemmTile tt = gemm_tile(t0 + t, g.ntm, ntn, g.group_m);
    const int tm = tt.tm, tn = tt.tn;
    G::mainloop(g, smem, tm, tn, 0, nk, acc);
    G::template epilogue<0, false>(g, smem, tm, tn, acc);
  }
  const int64_t usk = int64_t(ntx - dp) * nk;
  auto piece = [&](int w) { return usk * w / px; };  // first k-iteration of workgroup w's piece
  const int64_t a = piece(j);
  int64_t u = piece(j + 1);
  while (u > a) {
    const int st = int((u - 1) / nk);
    const int64_t tb = int64_t(st) * nk;
    const int kb = int((a > tb ? a : tb) - tb), ke = int(u - tb);
    const GemmTile tt = gemm_tile(t0 + dp + st, g.ntm, ntn, g.group_m);
    const int tm = tt.tm, tn = tt.tn;
    G::mainloop(g, smem, tm, tn, kb, ke, acc);
    if (ke < nk) {
      // top of the piece, short of the tile's end: publish the partial sum
      G::store_partial(g, acc, int(blockIdx.x));
      __syncthreads();  // every wave's partial stores have completed
      if (threadIdx.x == 0) __hip_atomic_store(g.flags + blockIdx.x, g.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      // this workgroup holds the tile's last iteration: add the earlier pieces
      for (int w = j - 1; kb > 0 && w >= 0; --w) {
        const int64_t pw = piece(w), pe = piece(w + 1);
        if (pe <= tb) break;     // w's piece ends before this tile, and so do all below it
        if (pw == pe) continue;  // empty piece: no partial
        const int slot = w * kXcds + x;
        if (threadIdx.x == 0) {
          int ok = 0;
          for (int it = 0; it < g.spin_limit; ++it) {
            if (__hip_atomic_load(g.flags + slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == g.epoch) {
              ok = 1;
              break;
            }
            __builtin_amdgcn_s_sleep(2);
          }
          spin_failed = !ok;
          if (!ok && g.status)
            __hip_atomic_fetch_or(g.status, uint32_t(DSF_WS_STATUS_SK_TIMEOUT), __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT);
        }
        __syncthreads();  // the partial's loads below are issued after its flag was seen
        if (spin_failed) break;  // left unfinished (and reported) rather than hang
        G::template add_partials<1>(g, slot, 1, acc);
      }
      G::template epilogue<0, false>(g, smem, tm, tn, acc);
    }
    u = tb + kb;
  }
}

// ------------------------------------------------------------ fp32 GEMM

constexpr int kFBM = 32, kFBN = 128, kFBK = 32;

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs g) {
  __shared__ float As[kFBK][kFBM + 4];
  __shared__ float Bs[kFBK][kFBN + 4];
  __shared__ float stage[kFBM * (kFBN + 4)];
  const int tid = threadIdx.x;
  const int tn = blockIdx.x, tm = blockIdx.y, m0 = tm * kFBM;
  const int tr = tid / 32, tc = tid % 32;  // 4 rows x 4 cols per thread
  float acc[4][4] = {};
  for (int k0 = 0; k0 < g.K; k0 += kFBK) {
    const bool second = k0 >= g.K1;
    {  // A: 32 rows x 32 k, one float4 per thread
      const int row = tid / 8, c4 = (tid % 8) * 4;
      int m = m0 + row;
      if (m > g.M - 1) m = g.M - 1;
      float v[4] = {0.f, 0.f, 0.f, 0.f};
      if (k0 + c4 < g.K) {
        const float* p = second ? (const float*)g.a2 + int64_t(m) * g.lda2 + (k0 - g.K1) + c4
                                : (const float*)g.a + int64_t(m) * g.lda + k0 + c4;
        load_vec(p, v);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) As[c4 + i][row] = v[i];
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {  // B: 128 rows x 32 k
      const int e = tid + 256 * t;
      const int row = e / 8, c4 = (e % 8) * 4;
      int n;
      if constexpr (EPI == EPI_SWIGLU) n = row < kFBN / 2 ? tn * (kFBN / 2) + row : g.f + tn * (kFBN / 2) + row - kFBN / 2;
      else n = min(tn * kFBN + row, g.N - 1);
      float v[4] = {0.f, 0.f, 0.f, 0.f};
      if (k0 + c4 < g.K) {
        const float* p = second ? (const float*)g.b2 + int64_t(n) * g.ldb2 + (k0 - g.K1) + c4
                                : (const float*)g.b + int64_t(n) * g.ldb + k0 + c4;
        load_vec(p, v);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) Bs[c4 + i][row] = v[i];
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < kFBK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        av[i] = As[kk][tr * 4 + i];
        bv[i] = Bs[kk][tc * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) stage[(tr * 4 + i) * (kFBN + 4) + tc * 4 + j] = acc[i][j];
  __syncthreads();
  gemm_epilogue<float, kFBM, kFBN, 256, EPI>(g, stage, m0, tn, threadIdx.x);
}

size_t gemm_partial_bytes() { return kSkPartBytes; }
int gemm_flag_count() { return kSkMaxSlots; }

// Polls of a stream-K flag before a finisher gives up (2^22, each followed
// by a short sleep). DSF_SK_SPIN_LIMIT, read at every launch, overrides it:
// a test sets 0 so that every finisher with a predecessor gives up at once
// and the status report can be checked without any wait being broken.
static int spin_limit() {
  const char* e = getenv("DSF_SK_SPIN_LIMIT");
  if (!e || !*e) return 1 << 22;
  const long v = strtol(e, nullptr, 10);
  return v < 0 ? 0 : (v > (1L << 30) ? (1 << 30) : int(v));
}

// DSF_GEMM_SCHEDULE=classic|streamk overrides the automatic choice (tests and
// tuning); read at every launch so that a process can switch between calls.
static int schedule_override() {
  const char* e = getenv("DSF_GEMM_SCHEDULE");
  if (!e) return 0;
  if (!strcmp(e, "classic")) return 1;
  if (!strcmp(e, "streamk")) return 2;
  if (!strcmp(e, "persistent")) return 3;
  return 0;
}

// Resident workgroups of kernel fn on the current device, capped at
// kSkMaxSlots (one cache per instantiation: each kernel has its own count).
template <typename Tag>
static int resident_slots(const void* fn, int threads) {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v) return v;
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, 0) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  v = std::min(per_cu * cus, kSkMaxSlots);
  cache[dev].store(v, std::memory_order_relaxed);
  return v;
}

// Schedule of a launch: px = workgroups per XCD of a persistent grid (0: one
// tile per workgroup) and split (1: stream-K split of the last round).
//  - Long reductions (at least kSkMinK k-iterations per tile) whose last
//    round of tiles would be at most a quarter full: stream-K. Then most CUs
//    would idle through that round, whereas a partial first round (fewer
//    tiles than slots) already runs its lone workgroups faster.
//  - Otherwise one tile per workgroup. For short reductions a persistent
//    grid over whole tiles (forced with DSF_GEMM_SCHEDULE=persistent) was
//    6 % faster alone but 10-15 % slower inside the layer stack, and stream-K
//    pieces cost more than the idle tail saves.
// Stream-K is also left out when the pieces would be too short to pay for
// their partial sums.
struct Schedule {
  int px, split;
};
// underfilled: also split a grid of at most half as many tiles as slots
// whose reduction is long (the backward's weight gradients: few output
// tiles, a reduction over every kept token), every workgroup taking an equal
// piece of all the tiles' k-iterations.
static Schedule choose_schedule(int nt, int nk, int slots, bool underfilled = false) {
  const int px = slots / kXcds;
  if (px < 1) return {0, 0};
  const int mode = schedule_override();
  if (mode == 1) return {0, 0};
  if (mode == 2) return {px, 1};
  if (mode == 3) return {px, 0};
  const int64_t P = int64_t(px) * kXcds;
  const int64_t last = nt % P;
  if (nk >= kSkMinK) {
    if (underfilled && 2 * int64_t(nt) <= P && int64_t(nt) * nk >= P * kSkMinIters) return {px, 1};
    if (nt <= P || last == 0 || 4 * last > P) return {0, 0};
    if (int64_t(nt) * nk < P * kSkMinIters) return {0, 0};
    return {px, 1};
  }
  return {0, 0};
}

// Split last round of a one-tile-per-workgroup grid of large tiles: with nt
// tiles on P resident workgroups, the last nt mod P tiles would run alone in
// a last round that leaves most CUs idle (the 3584-wide O and down
// projections of the Qwen2.5-7B shape end 3.2-4.1 rounds). They go to a
// second launch, each cut along K into s pieces, the largest s <= 4 with
// s * r <= P and at least kTailMinK k-tiles per piece, so that round takes
// about 1 / s of a tile. DSF_GEMM_TAIL (read at every launch): 0 turns the
// split off; force splits as if 8 workgroups were resident (tests on small
// grids).
struct TailSplit {
  int r, s;
};
static TailSplit choose_tail(int nt, int nk, int slots, int part_slots, bool avail) {
  const char* e = getenv("DSF_GEMM_TAIL");
  if (!avail || (e && e[0] == '0')) return {0, 1};
  const bool force = e && !strcmp(e, "force");
  const int P = force ? kXcds : slots;
  if (P <= 0 || nt <= P) return {0, 1};
  const int r = nt % P;
  if (r == 0) return {0, 1};
  for (int sp = kTailMaxSplit; sp >= 2; --sp)
    if (sp * r <= P && r * (sp - 1) <= part_slots && nk / sp >= kTailMinK) return {r, sp};
  return {0, 1};
}

// The DMA kernels address each operand through a buffer resource with a
// 32-bit byte range and 32-bit offsets: every operand, padded to whole tiles,
// must stay below 4 GiB.
template <class TC>
static bool dma_addressable(const GemmArgs& g, int rows_b) {
  const int64_t lim = (int64_t(1) << 32) - 1024;
  const int64_t mp = int64_t(g.M + TC::BM), np = int64_t(rows_b + TC::BN);
  return mp * g.lda * 2 < lim && (!g.a2 || mp * g.lda2 * 2 < lim) && np * g.ldb * 2 < lim &&
         (!g.b2 || np * g.ldb2 * 2 < lim);
}

// Launch kern<<<grid, block>>>(g), through hipExtLaunchKernelGGL when an
// enclosing timing scope hands over its events.
template <typename K, typename... A>
static void launch_timed(K kern, dim3 grid, dim3 block, hipStream_t s, const A&... args) {
  hipEvent_t e0, e1;
  if (timing_claim(&e0, &e1)) hipExtLaunchKernelGGL(kern, grid, block, 0, s, e0, e1, 0, args...);
  else kern<<<grid, block, 0, s>>>(args...);
}

// ------------------------------------------- few-row GEMM (decode steps)

// For M <= 16 rows the tile GEMMs leave most of the chip idle (N / 128
// workgroups). Here a workgroup takes 128 output columns and one slice of K:
// each of its four wavefronts computes a 16 x 32 block (two
// v_mfma_f32_16x16x32_bf16 blocks) from operands loaded straight from global
// memory (16 bytes per lane, 64 contiguous bytes per weight row and k-step),
// so the weights stream once over ~256-512 workgroups. With one slice the
// workgroup finishes its tile; otherwise it publishes its fp32 partial tile
// with device-coherent stores, and the last of the tile's workgroups to
// arrive (a device-scope counter, reset by that workgroup) adds the slices in
// slice order (deterministic) and runs the same fused epilogue as the tile
// GEMMs. No workgroup waits for another.
constexpr int kSkinnyRows = 16, kSkinnyBN = 128;
constexpr int kSkinnyMaxParts = 1024;   // partial tiles per launch
constexpr int kSkinnyCounters = 1024;   // column tiles per launch

size_t gemm_skinny_partial_bytes() { return size_t(kSkinnyMaxParts) * kSkinnyRows * kSkinnyBN * sizeof(float); }
int gemm_skinny_counters() { return kSkinnyCounters; }

template <int EPI>
__global__ __launch_bounds__(256) void gemm_skinny_kernel(GemmArgs g, int splits, int kc) {
  constexpr int LD = kSkinnyBN + 4;
  __shared__ float stage[kSkinnyRows * LD];
  __shared__ int is_last;
  const int tn = int(blockIdx.x) / splits, sl = int(blockIdx.x) - tn * splits;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, grp = lane >> 4;
  const int k0 = sl * kc, k1 = min(g.K, k0 + kc);
  // the B rows (output columns) of this lane in the wave's two 16-column blocks
  const uint16_t* brow[2];
  const uint16_t* brow2[2];
  bool bok[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int c = wave * 32 + nb * 16 + r16;  // column within the tile
    int r;
    if constexpr (EPI == EPI_SWIGLU) {
      // tile columns [0, 64) are gate units, [64, 128) the matching up units
      r = c < kSkinnyBN / 2 ? tn * (kSkinnyBN / 2) + c : g.f + tn * (kSkinnyBN / 2) + (c - kSkinnyBN / 2);
      bok[nb] = true;
    } else {
      r = tn * kSkinnyBN + c;
      bok[nb] = r < g.N;
      if (!bok[nb]) r = 0;
    }
    brow[nb] = (const uint16_t*)g.b + int64_t(r) * g.ldb;
    brow2[nb] = g.b2 ? (const uint16_t*)g.b2 + int64_t(r) * g.ldb2 : nullptr;
  }
  const bool aok = r16 < g.M;
  const uint16_t* arow = (const uint16_t*)g.a + int64_t(aok ? r16 : 0) * g.lda;
  const uint16_t* arow2 = g.a2 ? (const uint16_t*)g.a2 + int64_t(aok ? r16 : 0) * g.lda2 : nullptr;
  f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  const bf16x8 zero = {};
  // k-steps of 32 (the slice is a multiple of 32; k chunks of 8 never
  // straddle K1, a multiple of 32), up to 8 at a time: every load of a group
  // is issued before its MFMAs
  constexpr int kGroup = 8;
  const int nsteps = (k1 - k0) / 32;
  for (int st0 = 0; st0 < nsteps; st0 += kGroup) {
    bf16x8 af[kGroup], bf[kGroup][2];
#pragma unroll
    for (int it = 0; it < kGroup; ++it) {
      const int k = k0 + 32 * min(st0 + it, nsteps - 1) + 8 * grp;  // past the end: repeat the last step (unused)
      const bool first = k < g.K1;
      const int kk = first ? k : k - g.K1;
      af[it] = aok ? *reinterpret_cast<const bf16x8*>((first ? arow : arow2) + kk) : zero;
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        bf[it][nb] = bok[nb] ? *reinterpret_cast<const bf16x8*>((first ? brow[nb] : brow2[nb]) + kk) : zero;
    }
#pragma unroll
    for (int it = 0; it < kGroup; ++it)
      if (st0 + it < nsteps)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[it], bf[it][nb], acc[nb], 0, 0, 0);
  }
  // lane holds C[m = 4 grp + i][column wave*32 + nb*16 + r16]
  if (splits == 1) {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int i = 0; i < 4; ++i) stage[(4 * grp + i) * LD + wave * 32 + nb * 16 + r16] = acc[nb][i];
    __syncthreads();
    gemm_epilogue<uint16_t, kSkinnyRows, kSkinnyBN, 256, EPI>(g, stage, 0, tn, tid);
    return;
  }
  float* part = g.spart + (int64_t(tn) * splits + sl) * (kSkinnyRows * kSkinnyBN);
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      __hip_atomic_store(part + (4 * grp + i) * kSkinnyBN + wave * 32 + nb * 16 + r16, acc[nb][i], __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  // The device-coherent (sc1) stores have completed before the counter moves,
  // and the last workgroup reads the partials with device-coherent loads, so
  // no cache write-back or invalidate is needed (as in the stream-K GEMM).
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (tid == 0) {
    const uint32_t old = __hip_atomic_fetch_add(g.scount + tn, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    is_last = old == uint32_t(splits - 1);
    if (is_last) __hip_atomic_store(g.scount + tn, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!is_last) return;
  // 16 x 128 sums, 8 per thread, slices added in order; the slices' loads
  // are issued four at a time (device-coherent) before one wait
  const float* base = g.spart + int64_t(tn) * splits * (kSkinnyRows * kSkinnyBN);
  const int e0 = tid * 8, m = e0 / kSkinnyBN, c0 = e0 % kSkinnyBN;
  f32x4 vlo = {0.f, 0.f, 0.f, 0.f}, vhi = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < splits; s0 += 4) {
    f32x4 lo[4], hi[4];
    const float* p[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) p[j] = base + int64_t(min(s0 + j, splits - 1)) * (kSkinnyRows * kSkinnyBN) + e0;
    // the loads and their wait in one statement: no register they write is
    // touched before the data has arrived
    asm volatile(
        "global_load_dwordx4 %0, %8, off sc1\n\t"
        "global_load_dwordx4 %1, %8, off offset:16 sc1\n\t"
        "global_load_dwordx4 %2, %9, off sc1\n\t"
        "global_load_dwordx4 %3, %9, off offset:16 sc1\n\t"
        "global_load_dwordx4 %4, %10, off sc1\n\t"
        "global_load_dwordx4 %5, %10, off offset:16 sc1\n\t"
        "global_load_dwordx4 %6, %11, off sc1\n\t"
        "global_load_dwordx4 %7, %11, off offset:16 sc1\n\t"
        "s_waitcnt vmcnt(0)"
        : "=&v"(lo[0]), "=&v"(hi[0]), "=&v"(lo[1]), "=&v"(hi[1]), "=&v"(lo[2]), "=&v"(hi[2]), "=&v"(lo[3]),
          "=&v"(hi[3])
        : "v"(p[0]), "v"(p[1]), "v"(p[2]), "v"(p[3])
        : "memory");
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (s0 + j < splits) {
        vlo += lo[j];
        vhi += hi[j];
      }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    stage[m * LD + c0 + i] = vlo[i];
    stage[m * LD + c0 + 4 + i] = vhi[i];
  }
  __syncthreads();
  gemm_epilogue<uint16_t, kSkinnyRows, kSkinnyBN, 256, EPI>(g, stage, 0, tn, tid);
}

// Slices of K for a few-row launch: enough workgroups to cover the chip
// (~384) where the reduction allows, each slice a multiple of 32 and at least
// 128 deep, at most 16 slices (the last workgroup adds them), within the
// partial-tile budget.
static void skinny_split(int ntn, int K, int* splits, int* kc) {
  int s = std::max(1, (384 + ntn - 1) / ntn);
  s = std::min(s, std::max(1, K / 128));
  s = std::min(s, 16);
  s = std::min(s, std::max(1, kSkinnyMaxParts / ntn));
  int c = (K + s - 1) / s;
  c = (c + 31) / 32 * 32;
  *kc = c;
  *splits = (K + c - 1) / c;
}

// Large tiles when the grid of 256 x 256 tiles still fills the chip for more
// than a round (at least kLargeMinTiles tiles), and the SwiGLU units split
// into whole 128-unit tiles; small tiles otherwise. Measured on one layer of
// each workload: the large tiles win on every Qwen2.5-7B projection (gate/up
// 0.38 -> 0.47 of peak, down 0.32 -> 0.46), on the NeoX-1.4B QKV and up, and
// on the NeoX-160M QKV alone; the small ones on the 768- to 2048-wide down
// projections, whose grids of large tiles cover the chip once or less. In
// the stacks, forward projections with shallow reductions (K below
// kLargeMinDepth: 896 and 1536 on the Qwen2.5-0.5B and -1.5B shapes) keep
// the small tiles up to kLargeShallowMinTiles tiles, where a large tile's
// short main loop leaves its epilogue a bigger share (stacks 1.5 and 0.6 %
// faster). A caller that runs two projections side by side on two streams
// picks one size for both (GemmArgs::tile_hint, gemm_pair_tile_hint): a
// 256 x 256 workgroup takes most of a CU's LDS and cannot share the CU with
// a 128 x 128 one, so mixed sizes starve the large-tile launch.
// DSF_GEMM_TILE=small|large (read at every launch) forces one of them.
constexpr int kLargeMinTiles = 320;
constexpr int kLargeMinDepth = 2048;
constexpr int kLargeShallowMinTiles = 640;
constexpr int kLargePairMinTiles = 400;

// The tile size for a pair of forward projections that share the chip,
// from the leading one's shape (M x N, reduction K): deep reductions keep
// each launch's own rule (large from kLargeMinTiles tiles for both NeoX-1.4B
// projections); shallow ones take one size for both, large from
// kLargePairMinTiles tiles of the leading grid. NeoX-130M shape (QKV grids
// of 405-522 large tiles): large for both 2-8 % faster than small for both;
// NeoX-160M (171-441): small for both 1.5 % faster than the sizes chosen
// one launch at a time.
int gemm_pair_tile_hint(int M, int N, int K) {
  if (K >= kLargeMinDepth) return 0;
  const int64_t nt = int64_t((M + TileLarge::BM - 1) / TileLarge::BM) * ((N + TileLarge::BN - 1) / TileLarge::BN);
  return nt >= kLargePairMinTiles ? 2 : 1;
}

template <int EPI>
static bool use_large_tiles(const GemmArgs& g) {
  if (EPI == EPI_SWIGLU && g.f % (TileLarge::BN / 2) != 0) return false;
  const char* e = getenv("DSF_GEMM_TILE");
  if (e && !strcmp(e, "small")) return false;
  if (e && !strcmp(e, "large")) return true;
  if (g.tile_hint) return g.tile_hint == 2;
  const int64_t ntm = (g.M + TileLarge::BM - 1) / TileLarge::BM;
  const int64_t ntn = EPI == EPI_SWIGLU ? g.f / (TileLarge::BN / 2) : (g.N + TileLarge::BN - 1) / TileLarge::BN;
  const int64_t nt = ntm * ntn;
  if (EPI < EPI_STORE && g.K < kLargeMinDepth) return nt >= kLargeShallowMinTiles;
  return nt >= kLargeMinTiles;
}

template <int EPI, class TC>
static void launch_dma(const GemmArgs& g, hipStream_t s) {
  {
    constexpr int BM = TC::BM, BN = TC::BN, WM = TC::WM, WN = TC::WN, NS = TC::NS, BK = TC::BK;
    using Cfg = DmaCfg<BM, BN, WM, WN, NS, BK>;
    // partial-tile slots the workspace holds for this tile size
    constexpr int kPartSlots = int(kSkPartBytes / (size_t(BM) * BN * sizeof(float)));
    const int ntn = EPI == EPI_SWIGLU ? g.f / (BN / 2) : (g.N + BN - 1) / BN;
    GemmArgs ga = g;
    ga.ntm = (g.M + BM - 1) / BM;
    ga.px = 0;
    // Persistent and stream-K grids only with small tiles: the large tiles'
    // grids run many rounds (a short last round costs a few percent), and the
    // stream-K kernel's partial-sum hand-over does not fit their register
    // budget beside 128 accumulators per lane. Among the backward kinds only
    // the weight gradients (fp32 output) take them.
    if constexpr (BM == TileSmall::BM && BN == TileSmall::BN && (EPI < EPI_STORE || EPI == EPI_STORE_F32)) {
      if (g.part && g.flags) {
        auto fn = gemm_bf16_sk_kernel<EPI, BM, BN, WM, WN, NS, BK>;
        const int slots = std::min(kPartSlots, resident_slots<std::integral_constant<int, EPI * 2 + (BM > 128)>>(
                                                   (const void*)fn, Cfg::kThreads));
        const Schedule sch = choose_schedule(ntn * ga.ntm, g.K / BK, slots, EPI == EPI_STORE_F32);
        ga.px = sch.px;
        ga.split = sch.split;
        ga.spin_limit = spin_limit();
        // tile order as for one tile per workgroup
        ga.group_m = ntn >= kGroupMinCols ? kGroupM : 0;
        if (ga.px > 0) {
          launch_timed(fn, dim3(ga.px * kXcds), dim3(Cfg::kThreads), s, ga);
          return;
        }
      }
    }
    // More tiles than resident workgroups: walk bands of kGroupM tile rows
    // column by column, so that the workgroups resident on an XCD at one
    // time cover a compact block of tiles (A rows and B rows both reused
    // from its L2). A single round, or a grid fewer than kGroupMinCols tiles
    // wide (an XCD's row-major range is then already a compact block; banding
    // it measured more L2 misses on the 768-wide down projection), keeps
    // row-major order.
    auto fn = gemm_bf16_dma_kernel<EPI, BM, BN, WM, WN, NS, BK>;
    const int slots = resident_slots<std::integral_constant<int, 32 + EPI * 2 + (BM > 128)>>((const void*)fn, Cfg::kThreads);
    const int nt = ntn * ga.ntm;
    ga.ntn = ntn;
    ga.group_m = nt > slots && ntn >= kGroupMinCols ? kGroupM : 0;
    // Large tiles of the forward epilogues, on a call's stream-K workspace:
    // the last round of tiles split along K in a second launch. SwiGLU keeps
    // one launch, so that a launch of that kind is always the whole gate|up
    // projection (the duration its roofline figure is computed from).
    if constexpr (BM == TileLarge::BM && BN == TileLarge::BN && EPI < EPI_STORE && EPI != EPI_SWIGLU) {
      const TailSplit ts = choose_tail(nt, g.K / BK, slots, std::min(kPartSlots, gemm_flag_count()), g.part && g.flags);
      if (ts.s > 1) {
        ga.tail0 = nt - ts.r;
        ga.tail_r = ts.r;
        ga.tail_s = ts.s;
        ga.spin_limit = spin_limit();
        launch_timed(fn, dim3(nt - ts.r), dim3(Cfg::kThreads), s, ga);
        timing_continue();
        launch_timed(gemm_bf16_tail_kernel<EPI, BM, BN, WM, WN, NS, BK>,
                     dim3(kXcds * ts.s * ((ts.r + kXcds - 1) / kXcds)), dim3(Cfg::kThreads), s, ga);
        return;
      }
    }
    launch_timed(fn, dim3(nt), dim3(Cfg::kThreads), s, ga);
  }
}

template <int EPI>
static void launch_gemm_t(const GemmArgs& g, hipStream_t s) {
  if constexpr (EPI >= EPI_STORE) {
    // backward kinds: bf16 only, one output tile per workgroup
    const int rows_b = g.N;
    if (g.K % 64 == 0 && g.K1 % 64 == 0) {
      if (use_large_tiles<EPI>(g) && dma_addressable<TileLarge>(g, rows_b)) {
        launch_dma<EPI, TileLarge>(g, s);
        return;
      }
      if (dma_addressable<TileSmall>(g, rows_b)) {
        launch_dma<EPI, TileSmall>(g, s);
        return;
      }
    }
    launch_timed(gemm_bf16_kernel<EPI>, dim3((g.N + kBN - 1) / kBN, (g.M + kBM - 1) / kBM), dim3(kThreads), s, g);
    return;
  } else {
  if (g.dtype == DSF_BF16 && g.M <= kSkinnyRows && g.spart && g.scount && g.K % 32 == 0 && g.K1 % 32 == 0 &&
      g.lda % 8 == 0 && g.ldb % 8 == 0 && (!g.a2 || g.lda2 % 8 == 0) && (!g.b2 || g.ldb2 % 8 == 0)) {
    const int ntn = EPI == EPI_SWIGLU ? g.f / (kSkinnyBN / 2) : (g.N + kSkinnyBN - 1) / kSkinnyBN;
    if (ntn <= kSkinnyCounters && (EPI != EPI_SWIGLU || g.f % (kSkinnyBN / 2) == 0)) {
      int splits = 1, kc = g.K;
      skinny_split(ntn, g.K, &splits, &kc);
      launch_timed(gemm_skinny_kernel<EPI>, dim3(ntn * splits), dim3(256), s, g, splits, kc);
      return;
    }
  }

  if (DSF_GEMM_USE_DMA && g.dtype == DSF_BF16 && g.K % 64 == 0 && g.K1 % 64 == 0) {
    const int rows_b = EPI == EPI_SWIGLU ? 2 * g.f : g.N;
    if (use_large_tiles<EPI>(g) && dma_addressable<TileLarge>(g, rows_b)) {
      launch_dma<EPI, TileLarge>(g, s);
      return;
    }
    if (dma_addressable<TileSmall>(g, rows_b)) {
      launch_dma<EPI, TileSmall>(g, s);
      return;
    }
  }
  if (g.dtype == DSF_BF16) {
    const int ntn = EPI == EPI_SWIGLU ? g.f / (kBN / 2) : (g.N + kBN - 1) / kBN;
    launch_timed(gemm_bf16_kernel<EPI>, dim3(ntn, (g.M + kBM - 1) / kBM), dim3(kThreads), s, g);
  } else {
    const int ntn = EPI == EPI_SWIGLU ? g.f / (kFBN / 2) : (g.N + kFBN - 1) / kFBN;
    launch_timed(gemm_f32_kernel<EPI>, dim3(ntn, (g.M + kFBM - 1) / kFBM), dim3(256), s, g);
  }
  }
}

hipError_t launch_gemm(const GemmArgs& g, hipStream_t s) {
  if (g.M == 0 || g.N == 0) return hipSuccess;
  switch (g.epi) {
    case EPI_QKV_ROPE: launch_gemm_t<EPI_QKV_ROPE>(g, s); break;
    case EPI_BIAS_GELU: launch_gemm_t<EPI_BIAS_GELU>(g, s); break;
    case EPI_SWIGLU: launch_gemm_t<EPI_SWIGLU>(g, s); break;
    case EPI_RESID_STORE: launch_gemm_t<EPI_RESID_STORE>(g, s); break;
    case EPI_RESID_SCATTER: launch_gemm_t<EPI_RESID_SCATTER>(g, s); break;
    case EPI_RESID_SCATTER_GATE: launch_gemm_t<EPI_RESID_SCATTER_GATE>(g, s); break;
    case EPI_STORE: launch_gemm_t<EPI_STORE>(g, s); break;
    case EPI_STORE_F32: launch_gemm_t<EPI_STORE_F32>(g, s); break;
    case EPI_GELU_BWD: launch_gemm_t<EPI_GELU_BWD>(g, s); break;
    case EPI_SWIGLU_BWD: launch_gemm_t<EPI_SWIGLU_BWD>(g, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace dsf
