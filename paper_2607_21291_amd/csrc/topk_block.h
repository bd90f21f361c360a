// Per-sequence Top-K of Section 3.4 as a device routine for one block of NT
// threads, shared by the standalone Top-K kernel and the router kernel that
// selects in its last-arriving workgroup of each sequence.
#pragma once

#include "dsf_device.h"

namespace dsf {

// Order-preserving key: larger score -> larger key; -0 == +0; NaN -> 0 (lowest).
__device__ __forceinline__ uint32_t score_key(float f) {
  if (f != f) return 0u;
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kTopkLdsKeys = 16384;  // sequences up to this length keep their keys in LDS

template <int NT, bool KEYS_IN_LDS>
struct TopkShared {
  static constexpr int NW = NT / 64;
  uint32_t keys[KEYS_IN_LDS ? kTopkLdsKeys : 1];
  uint32_t whist[2][NW][256];  // per-wave digit histograms, two buffers used by alternate passes
  uint32_t wave_tot[NW];
  uint32_t digit, remaining, whole;
};

// Exclusive prefix sum of v over the block in thread order; `total` gets the
// block's sum. A wave-level scan, then the wave totals through LDS.
template <int NW>
__device__ __forceinline__ uint32_t block_excl_sum(uint32_t v, uint32_t* wave_tot, uint32_t& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t u = __shfl_up(incl, o, 64);
    if (lane >= o) incl += u;
  }
  if (lane == 63) wave_tot[w] = incl;
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint32_t c = wave_tot[i];
    before += (i < w) ? c : 0u;
    tot += c;
  }
  __syncthreads();
  total = tot;
  return before + incl - v;
}

// Top-K of one sequence of T scores (score(t) returns score t) by one block of
// NT threads (NT >= 128); writes the k kept positions (1 <= k <= T) to out in
// ascending order. The order-preserving keys are kept in LDS when
// KEYS_IN_LDS (T <= kTopkLdsKeys), read from global memory once.
//
// Radix select, 8 bits per pass, most significant first, finds the key of the
// k-th largest score and how many of the keys equal to it are kept. Each
// wavefront counts into its own histogram, so that equal digits (frequent in
// the top byte) do not serialise on one LDS address; wave 0 then adds the
// wave histograms and scans them while the other waves clear the buffer the
// next pass counts into: two barriers per pass. The final pass gives each
// thread a contiguous run of positions: a block scan of the equal keys
// before each run decides which of them are kept (the lowest positions), a
// second block scan places each run's kept positions in the output.
template <int NT, bool KEYS_IN_LDS, typename Score>
__device__ void topk_block(Score score, int T, int k, int32_t* __restrict__ out, TopkShared<NT, KEYS_IN_LDS>& sh) {
  constexpr int NW = NT / 64;
  static_assert(NW >= 2, "the histogram scan and the buffer clearing run on different waves");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  auto key_at = [&](int t) -> uint32_t { return KEYS_IN_LDS ? sh.keys[t] : score_key(score(t)); };

  for (int i = tid; i < 2 * NW * 256; i += NT) (&sh.whist[0][0][0])[i] = 0;
  if constexpr (KEYS_IN_LDS) {
    // eight scores per thread in flight before the first is used
    for (int t0 = tid; t0 < T; t0 += 8 * NT) {
      float v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = t0 + j * NT < T ? score(t0 + j * NT) : 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (t0 + j * NT < T) sh.keys[t0 + j * NT] = score_key(v[j]);
    }
  }
  __syncthreads();
  uint32_t prefix = 0, mask = 0, remaining = uint32_t(k);
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass, cur = pass & 1;
    for (int t = tid; t < T; t += NT) {
      const uint32_t key = key_at(t);
      if ((key & mask) == prefix) atomicAdd(&sh.whist[cur][wave][(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (wave == 0) {
      // lane L owns digits 255-4L .. 252-4L (descending); exclusive scan over lanes
      uint32_t c[4], tot = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint32_t v = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w) v += sh.whist[cur][w][255 - 4 * lane - e];
        c[e] = v;
        tot += v;
      }
      uint32_t incl = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t v = __shfl_up(incl, o, 64);
        if (lane >= o) incl += v;
      }
      uint32_t cum = incl - tot;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (cum < remaining && remaining <= cum + c[e]) {
          sh.digit = uint32_t(255 - 4 * lane - e);
          sh.remaining = remaining - cum;
          sh.whole = remaining == cum + c[e];  // every key of the digit's bucket is kept
        }
        cum += c[e];
      }
    } else if (pass < 3) {
      // the other buffer was last read by the previous pass's scan
      for (int i = tid - 64; i < NW * 256; i += NT - 64) (&sh.whist[cur ^ 1][0][0])[i] = 0;
    }
    __syncthreads();
    prefix |= sh.digit << shift;
    mask |= 255u << shift;
    remaining = sh.remaining;
    if (sh.whole) break;  // the bucket holding the k-th key is kept whole: no more digits needed
  }
  // The keys' top bits under mask select: those above prefix are kept, and of
  // those equal to it (after four passes: the k-th largest key itself) the
  // `remaining` lowest-positioned ones. Thread tid owns positions [t0, t1).
  const int run = (T + NT - 1) / NT;
  const int t0 = min(T, tid * run), t1 = min(T, t0 + run);
  uint32_t n_gt = 0, n_eq = 0;
  for (int t = t0; t < t1; ++t) {
    const uint32_t key = key_at(t) & mask;
    n_gt += key > prefix;
    n_eq += key == prefix;
  }
  uint32_t tot;
  const uint32_t eq_before = block_excl_sum<NW>(n_eq, sh.wave_tot, tot);
  const uint32_t eq_kept = eq_before >= remaining ? 0u : min(n_eq, remaining - eq_before);
  const uint32_t sel_before = block_excl_sum<NW>(n_gt + eq_kept, sh.wave_tot, tot);
  uint32_t o = sel_before, eq_seen = 0;
  for (int t = t0; t < t1; ++t) {
    const uint32_t key = key_at(t) & mask;
    const bool eq = key == prefix;
    const bool sel = key > prefix || (eq && eq_seen < eq_kept);
    eq_seen += eq;
    if (sel && o < uint32_t(k)) out[o++] = t;
  }
}

}  // namespace dsf
