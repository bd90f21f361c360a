// Tile order of the one-tile-per-workgroup GEMM grid (host- and
// device-callable so that the mapping can be checked exhaustively on the CPU).
//
// Workgroup ids are dispatched round-robin over the 8 XCDs, each with its own
// L2; xcd_remap (dsf_device.h) first turns launch index L into a work index
// so that every XCD receives one contiguous range of work indices. The work
// index then names a tile:
//  - group_m == 0: row-major (M-tile, N-tile) order;
//  - group_m > 0: bands of group_m tile rows, each band walked column by
//    column, so that the workgroups resident on one XCD at a time cover a
//    compact block of tiles and reuse both A rows and B rows from its L2.
#pragma once

#ifndef DSF_HD
#define DSF_HD __host__ __device__
#endif

namespace dsf {

struct GemmTile {
  int tm, tn;
};

// Work index i of ntm * ntn -> its tile; a bijection onto [0, ntm) x [0, ntn).
DSF_HD inline GemmTile gemm_tile(int i, int ntm, int ntn, int group_m) {
  if (group_m <= 0) return {i / ntn, i % ntn};
  const int per = group_m * ntn, band = i / per, r = i - band * per;
  const int m0 = band * group_m;
  const int gm = ntm - m0 < group_m ? ntm - m0 : group_m;  // the last band may be shorter
  return {m0 + r % gm, r / gm};
}

}  // namespace dsf
