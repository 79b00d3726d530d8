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

// "div d": floor(n / d) by fastdiv against the divide instruction for n
// near 0, near 2^32, around multiples of d and at pseudo-random points;
// prints the number of mismatches.
static void divcheck(unsigned long long d) {
  const uint64_t M = dpar::fastdiv_magic(d);
  uint64_t bad = 0;
  auto one = [&](uint64_t n) {
    if (n > 0xFFFFFFFFull) return;
    if (dpar::fastdiv((uint32_t)n, M, d) != n / d) ++bad;
  };
  for (uint64_t n = 0; n < 4096; ++n) one(n);
  for (uint64_t n = 0xFFFFFFFFull - 4096; n <= 0xFFFFFFFFull; ++n) one(n);
  for (uint64_t k = 1; k < 4096; ++k) {
    const uint64_t top = 0xFFFFFFFFull / d;
    for (uint64_t q : {k, top >= k ? top - k : 0, top / 2 + k})
      for (int e = -1; e <= 1; ++e) one(q * d + e);
  }
  uint64_t s = 0x9E3779B97F4A7C15ull ^ d;
  for (int k = 0; k < 200000; ++k) {
    s ^= s << 13; s ^= s >> 7; s ^= s << 17;
    one(s & 0xFFFFFFFFull);
  }
  std::printf("%llu\n", (unsigned long long)bad);
}

int main() {
  char tag[32];
  while (std::scanf("%31s", tag) == 1) {
    if (std::string(tag) == "div") {
      unsigned long long d;
      if (std::scanf("%llu", &d) != 1) return 1;
      divcheck(d);
      continue;
    }
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
    dpar::BcastGrid g = dpar::bcast_grid(nbytes, lane, p, span);
    g.fast = 1;   // the division-free mapping, checked against division
    const uint64_t tiles = (g.n + 255) / 256;
    std::vector<unsigned char> seen(g.rows * tiles, 0);
    uint64_t covered = 0, padded = 0, bad = 0;
    for (uint64_t w = 0; w < g.total; ++w) {
      uint64_t row, tile, row_d, tile_d;
      dpar::bcast_tile<true>(g, w, &row, &tile);
      dpar::bcast_tile<false>(g, w, &row_d, &tile_d);
      if (row != row_d || tile != tile_d) ++bad;
      // the same pair by plain division
      const uint64_t per_span = g.rows * g.ts, sp = w / per_span;
      if (row != 1 + (w - sp * per_span) / g.ts ||
          tile != sp * g.ts + (w - sp * per_span) % g.ts)
        ++bad;
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
