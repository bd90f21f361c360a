// Work order of the causal attention grid (host- and device-callable so that
// the mapping can be checked exhaustively on the CPU).
//
// A work item is one block of queries of one (sequence, query head) pair; a
// block b costs b + 1 key tiles under the causal mask, so the blocks of a
// head range from one tile to the whole prefix. Workgroup ids are dispatched
// round-robin over the 8 XCDs, each with its own L2, so XCD x receives the
// launch indices x, x + 8, x + 16, ... in that order.
//
// Each XCD owns one contiguous range of the head-major item list (all blocks
// of a head on one L2, except where a range boundary splits a head between two
// XCDs), and walks its range longest block first across all of its heads:
// list scheduling in decreasing order of cost, so no long block starts late
// behind the short ones of an earlier head.
#pragma once

#ifndef DSF_HD
#define DSF_HD __host__ __device__
#endif

namespace dsf {

struct AttnItem {
  int bh;    // (sequence, query head) pair, b * Hq + h
  int qblk;  // query block, 0 = the first queries of the sequence
};

// Launch index L of W = nqb * BH workgroups -> its work item. A bijection of
// [0, W) onto all (bh, qblk) pairs with bh < W / nqb and qblk < nqb.
DSF_HD inline AttnItem attn_item(int L, int W, int nqb) {
  constexpr int X = 8;
  const int x = L % X, j0 = L / X;
  const int q = W / X, r = W % X;
  const int s = x * q + (x < r ? x : r);           // range [s, e) of head-major items
  const int e = s + q + (x < r ? 1 : 0);
  // head-major item i = bh * nqb + u is block nqb - 1 - u of head bh
  const int bs = s / nqb, us = s - bs * nqb;       // first head: blocks 0 .. nqb - 1 - us
  const int be = (e - 1) / nqb, ue = (e - 1) - be * nqb;  // last head: blocks nqb - 1 - ue .. nqb - 1
  if (bs == be) return {bs, nqb - 1 - (us + j0)};
  const int first_hi = nqb - 1 - us, last_lo = nqb - 1 - ue, nmid = be - bs - 1;
  int j = j0;
  for (int b = nqb - 1; b >= 0; --b) {
    const int f = b <= first_hi ? 1 : 0, l = b >= last_lo ? 1 : 0;
    const int c = f + nmid + l;
    if (j < c) return {(f && j == 0) ? bs : bs + 1 + (j - f), b};
    j -= c;
  }
  return {-1, -1};  // only for L >= W
}

}  // namespace dsf
