// Checks plan.hpp xcd_run_index: for each n read from stdin prints
// "n ok" when workgroups 0..n-1 map one-to-one onto work items 0..n-1 and
// the workgroups of each XCD (w mod 8) take one contiguous run of items in
// increasing order, else "n bad <reason>".  Test infrastructure.
#include <cstdio>
#include <vector>

#include "plan.hpp"

int main() {
  unsigned n;
  while (std::scanf("%u", &n) == 1) {
    std::vector<int> seen(n, 0);
    const char* bad = nullptr;
    std::vector<long long> last(8, -1), count(8, 0);
    for (unsigned w = 0; w < n && !bad; ++w) {
      const uint64_t t = dpar::xcd_run_index(w, n);
      if (t >= n) {
        bad = "out_of_range";
        break;
      }
      if (seen[t]++) bad = "twice";
      const unsigned k = w & 7u;
      if (last[k] >= 0 && (long long)t != last[k] + 1) bad = "not_contiguous";
      last[k] = (long long)t;
      ++count[k];
    }
    // runs in XCD order: XCD k's run starts where XCD k-1's ends
    if (!bad) {
      long long start = 0;
      for (unsigned k = 0; k < 8 && !bad; ++k) {
        if (count[k] == 0) continue;
        if (last[k] - count[k] + 1 != start) bad = "runs_out_of_order";
        start = last[k] + 1;
      }
    }
    if (bad)
      std::printf("%u bad %s\n", n, bad);
    else
      std::printf("%u ok\n", n);
  }
  return 0;
}
