// Checks the broadcast pass's grid (plan.hpp bcast_grid, bcast_tile): reads
// lines "nbytes lane_bytes p span_bytes" on stdin and writes per line
// "n ts nspan rows total covered padded bad", where covered counts the
// (row, tile) pairs inside y_0 that some workgroup writes, padded the
// workgroups whose tile lies past y_0's end, and bad the workgroups that hit
// a pair already written or a row outside 1 .. p-1.  Test infrastructure.
#include <cstdio>
#include <vector>

#include "plan.hpp"

int main() {
  unsigned long long nbytes, lane, span;
  int p;
  while (std::scanf("%llu %llu %d %llu", &nbytes, &lane, &p, &span) == 4) {
    const dpar::BcastGrid g = dpar::bcast_grid(nbytes, lane, p, span);
    const uint64_t tiles = (g.n + 255) / 256;
    std::vector<unsigned char> seen(g.rows * tiles, 0);
    uint64_t covered = 0, padded = 0, bad = 0;
    for (uint64_t w = 0; w < g.total; ++w) {
      uint64_t row, tile;
      dpar::bcast_tile(g, w, &row, &tile);
      if (row < 1 || row > g.rows) {
        ++bad;
        continue;
      }
      if (tile >= tiles) {
        ++padded;
        continue;
      }
      unsigned char& s = seen[(row - 1) * tiles + tile];
      if (s) ++bad;
      s = 1;
      ++covered;
    }
    std::printf("%llu %llu %llu %llu %llu %llu %llu %llu\n",
                (unsigned long long)g.n, (unsigned long long)g.ts,
                (unsigned long long)g.nspan, (unsigned long long)g.rows,
                (unsigned long long)g.total, (unsigned long long)covered,
                (unsigned long long)padded, (unsigned long long)bad);
  }
  return 0;
}
