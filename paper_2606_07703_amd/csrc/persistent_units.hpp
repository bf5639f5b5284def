// Work split of the persistent block-indexer grid, shared by the kernel and
// the host (the launch counts units; a host test replays the split).
//
// Work is the sequence of units (query group qg, key tile t) for
// t < tiles(qg), ordered by group, then tile; tiles(qg) counts the key tiles
// at or below the group's last query (causal, Section 4.2). The grid splits
// the sequence into equal contiguous runs, one per workgroup: run r covers
// units [r*n/grid, (r+1)*n/grid). Workgroup i, which the hardware places on
// XCD i % 8, takes run xcd_run(i, grid), so each XCD's runs are contiguous
// and its L2 sees a contiguous range of groups and the key tiles they share.
// g0 is the first query group (a chunked call starting at g0 * QG covers
// groups g0 ..).
#pragma once

#include <hip/hip_runtime.h>

namespace sp {

constexpr int kXcds = 8;   // XCDs of the chip; workgroup i runs on XCD i % 8

__host__ __device__ constexpr int imin(int a, int b) { return a < b ? a : b; }

template <int QG, int KT>
struct UnitCursor {
  int S, qg, t, nt;   // sequence length, current group, tile, tiles of the group
  __host__ __device__ static int tiles(int S, int g) {
    return (imin((g + 1) * QG, S) + KT - 1) / KT;
  }
  // position the cursor on unit u, counted from the first unit of group g0
  __host__ __device__ void seek(int g0, long long u) {
    qg = g0;
    for (;;) {
      nt = tiles(S, qg);
      if (u < nt) break;
      u -= nt;
      ++qg;
    }
    t = (int)u;
  }
  // first unit of the next group
  __host__ __device__ void next_group() {
    ++qg;
    t = 0;
    nt = tiles(S, qg);
  }
};

// Run of workgroup i of n: XCD x = i % 8 takes the x-th contiguous share of
// the runs (the remainder spread over the first XCDs).
__host__ __device__ inline int xcd_run(int i, int n) {
  const int x = i % kXcds, j = i / kXcds;
  return x * (n / kXcds) + imin(x, n % kXcds) + j;
}

// Units [u0, u1) of run r of a grid of n workgroups over n_units units.
__host__ __device__ inline void run_units(long long n_units, int r, int n, int &u0, int &u1) {
  u0 = (int)(n_units * r / n);
  u1 = (int)(n_units * (r + 1) / n);
}

template <int QG, int KT>
long long count_units(int S, int g0) {
  long long n = 0;
  for (int g = g0; g * QG < S; ++g) n += UnitCursor<QG, KT>::tiles(S, g);
  return n;
}

}  // namespace sp
