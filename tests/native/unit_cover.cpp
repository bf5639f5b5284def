// Replays the persistent block-indexer work split on the host: for many
// sequence lengths, first groups and grid sizes, every (query group, key
// tile) unit must be visited by exactly one workgroup, and each workgroup
// must walk its run in the order the kernel does (seek, tiles of the group,
// next group). Prints "cover ok" and exits 0 when every case holds.
#include <stdio.h>

#include <vector>

#include "persistent_units.hpp"

using namespace sp;

template <int QG, int KT>
static int check(int S, int g0, int grid) {
  const long long n = count_units<QG, KT>(S, g0);
  // unit index of (group, tile), counted from group g0
  std::vector<long long> first;
  for (int g = g0; g * QG < S; ++g)
    first.push_back(g == g0 ? 0 : first.back() + UnitCursor<QG, KT>::tiles(S, g - 1));
  std::vector<int> seen(n, 0);
  std::vector<int> runs(grid, 0);
  for (int i = 0; i < grid; ++i) {
    const int run = xcd_run(i, grid);
    if (run < 0 || run >= grid) return 1;
    ++runs[run];
    int u0, u1;
    run_units(n, run, grid, u0, u1);
    if (u0 == u1) continue;
    UnitCursor<QG, KT> uc;
    uc.S = S;
    uc.seek(g0, u0);
    for (int u = u0; u < u1;) {
      const int group = uc.qg, nt = uc.nt;
      if (group * QG >= S) return 2;   // walked past the last group
      const int t_end = imin(nt, uc.t + (u1 - u));
      for (int t = uc.t; t < t_end; ++t, ++u) {
        const long long id = first[group - g0] + t;
        if (id != u) return 3;          // the walk and the unit numbering disagree
        if (t * KT > imin((group + 1) * QG, S) - 1) return 4;   // a tile past the group
        ++seen[id];
      }
      uc.next_group();
    }
  }
  for (int r = 0; r < grid; ++r)
    if (runs[r] != 1) return 5;         // xcd_run is not a permutation
  for (long long u = 0; u < n; ++u)
    if (seen[u] != 1) return 6;
  return 0;
}

int main() {
  const int lens[] = {1, 2, 63, 64, 127, 128, 129, 511, 512, 513, 1000, 4096, 16384, 32768,
                      32769, 102400};
  const int grids[] = {1, 3, 7, 8, 9, 17, 255, 256, 257, 512, 1024, 4000};
  int cases = 0;
  for (int S : lens)
    for (int g0 = 0; g0 * 512 < S && g0 < 3; ++g0)
      for (int grid : grids) {
        int rc = check<512, 128>(S, g0, grid);
        if (!rc) rc = check<512, 64>(S, g0, grid);
        if (rc) {
          fprintf(stderr, "coverage failed (code %d): S=%d g0=%d grid=%d\n", rc, S, g0, grid);
          return 1;
        }
        ++cases;
      }
  printf("cover ok (%d cases)\n", cases);
  return 0;
}
