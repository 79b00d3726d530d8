// Checks the broadcast pass's grid (plan.hpp bcast_grid, bcast_tile): reads
// lines "nbytes lane_bytes p span_bytes" on stdin and writes per line
// "n ts nspan rows total covered padded bad", where covered counts the
// (row, tile) pairs inside y_0 that some workgroup writes, padded the
// workgroups whose tile lies past y_0's end, and bad the workgroups that hit
// a pair already written or a row outside 1 .. p-1.  Test infrastructure.
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "plan.hpp"

static void split(unsigned long long dst, unsigned long long ndw) {
  uint64_t h, nbody;
  dpar::bcast_row_split(dst, ndw, &h, &nbody);
  std::vector<int> seen(ndw, 0);
  uint64_t twice = 0, outside = 0, misaligned = 0;
  auto put = [&](uint64_t k) {
    if (k >= ndw) {
      ++outside;
      return;
    }
    if (seen[k]++) ++twice;
  };
  for (uint64_t l = 0; l < nbody; ++l) {   // body: one 16-byte store each
    if ((dst + 4 * (h + 4 * l)) & 15) ++misaligned;
    if (l % 256 == 0 && ((dst + 4 * (h + 4 * l)) & 4095)) ++misaligned;
    for (uint64_t d = 0; d < 4; ++d) put(h + 4 * l + d);
  }
  for (uint64_t k = 0; k < h; ++k) put(k);  // the tile-0 workgroup's dwords
  for (uint64_t t = 0; t < 4; ++t)
    if (h + 4 * nbody + t < ndw) put(h + 4 * nbody + t);
  uint64_t covered = 0;
  for (uint64_t k = 0; k < ndw; ++k) covered += seen[k] != 0;
  std::printf("%llu %llu %llu %llu %llu %llu\n", (unsigned long long)h,
              (unsigned long long)nbody, (unsigned long long)covered,
              (unsigned long long)twice, (unsigned long long)outside,
              (unsigned long long)misaligned);
}

int main() {
  char tag[32];
  while (std::scanf("%31s", tag) == 1) {
    if (std::string(tag) == "split") {
      unsigned long long dst, ndw;
      if (std::scanf("%llu %llu", &dst, &ndw) != 2) return 1;
      split(dst, ndw);
      continue;
    }
    const unsigned long long nbytes = std::strtoull(tag, nullptr, 10);
    unsigned long long lane, span;
    int p;
    if (std::scanf("%llu %d %llu", &lane, &p, &span) != 3) return 1;
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
