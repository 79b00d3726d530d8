// Prints the host's block grouping for one-launch executors: reads lines
// "m b g lq" on stdin, writes "Q NL C G" per line (plan.hpp make_schedule,
// block_group).
#include <cstdio>

#include "plan.hpp"

int main() {
  unsigned long long m;
  int b, g, lq;
  while (std::scanf("%llu %d %d %d", &m, &b, &g, &lq) == 4) {
    const dpar::Schedule s = dpar::make_schedule(m, b, g, lq);
    std::printf("%llu %llu %d %d\n", (unsigned long long)s.Q,
                (unsigned long long)s.NL, s.C, dpar::block_group(s));
  }
  return 0;
}
