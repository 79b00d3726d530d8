/* A plain C99 program against include/dpar.h and libdpar.so: the boundary is
 * a C ABI, usable without C++ or Python.  It calls only the entry points that
 * do no device work (tree tables, round counts, block rule, decomposition,
 * argument errors) and prints one line per check, "ok <name>" or
 * "FAIL <name>".  Test infrastructure. */
#include <stdio.h>
#include <stdlib.h>

#include "dpar.h"

static int failures = 0;

static void check(int cond, const char* name) {
  printf("%s %s\n", cond ? "ok" : "FAIL", name);
  if (!cond) ++failures;
}

int main(void) {
  dpar_node_t n;
  /* p = 7: tree A = ranks 0..3 (root 3), tree B = 4..6 (root 6) */
  check(dpar_tree_info(7, 1, &n) == DPAR_SUCCESS && n.parent == 3 &&
            n.child0 == 0 && n.child1 == -1 && n.depth == 1 &&
            n.subtree_lo == 0 && n.dual == -1,
        "tree_info_p7_rank1");
  check(dpar_tree_info(7, 3, &n) == DPAR_SUCCESS && n.parent == -1 &&
            n.child0 == 2 && n.child1 == 1 && n.depth == 0 && n.dual == 6,
        "tree_info_p7_root_a");
  check(dpar_tree_info(7, 7, &n) == DPAR_ERR_INVALID_ARG, "tree_info_bad_rank");
  check(dpar_rounds(7, 4, 0) == 6 && dpar_rounds(7, 4, 2) == 5 &&
            dpar_rounds(7, 4, -1) == 6,
        "rounds_p7_b4");
  check(dpar_block_rule(1152, (size_t)1 << 22, 0.0, 0.0) == 6532,
        "block_rule_p1152");
  check(dpar_schedule_rounds(7, 4, DPAR_ALG_DUAL_ROOT) == 6, "schedule_rounds");
  {
    dpar_schedule_t s;
    size_t a = 0, e = 0;
    check(dpar_schedule_info(1152, (size_t)1 << 22, DPAR_FLOAT32, 0, 1, &s) ==
                  DPAR_SUCCESS &&
              s.b == 6532 && s.quantum == 4 && s.granularity == 32 &&
              s.height == 9,
          "schedule_info_p1152");
    check(dpar_block_bounds(&s, (size_t)1 << 22, 0, &a, &e) == DPAR_SUCCESS &&
              a == 0 && e > 0 && e % 32 == 0,
          "block_bounds_first");
  }
  {
    /* argument errors come back before any device work */
    const void* x[2] = {(const void*)0x100000, (const void*)0x200000};
    void* y[2] = {(void*)0x300000, (void*)0x400000};
    check(dpar_allreduce(NULL, y, 2, 16, DPAR_INT32, DPAR_SUM, 0, NULL) ==
              DPAR_ERR_INVALID_ARG,
          "null_array");
    check(dpar_allreduce(x, y, 2, 16, DPAR_FLOAT32, DPAR_MAX, 0, NULL) ==
              DPAR_ERR_UNSUPPORTED,
          "unsupported_pair");
    check(dpar_allreduce(x, y, 2, 16, DPAR_INT32, DPAR_SUM, 17, NULL) ==
              DPAR_ERR_INVALID_ARG && dpar_last_error()[0] != '\0',
          "b_above_m");
  }
  check(dpar_finalize() == DPAR_SUCCESS, "finalize");
  return failures ? 1 : 0;
}
