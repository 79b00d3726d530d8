/* Plain C oracle of the reduction-to-all: test infrastructure only (the
 * tests, the smoke check and the benchmark's CPU baseline use it; the
 * library never does).  All pointers are host memory. */
#ifndef DPAR_ORACLE_H
#define DPAR_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* element operators (Section 1: any associative operator; these four) */
enum {
  DPO_I32_SUM = 0,       /* int32, two's-complement wrap */
  DPO_I32_MAX = 1,       /* int32 */
  DPO_F32_SUM = 2,       /* IEEE binary32, round to nearest even */
  DPO_U32MAT_MATMUL = 3  /* 2x2 uint32 row-major (16 bytes), mod 2^32 */
};

/* tree layouts */
enum {
  DPO_DUAL = 2,   /* two trees with dual roots (Section 1.1) */
  DPO_SINGLE = 1  /* one tree over all ranks (Section 1.2; Section 2) */
};

/* The post-order numbered, heap-shaped trees of Section 1.1 for p ranks:
 * p entries each of parent, first child (rank - 1 when there is one),
 * second child and depth (root 0); -1 where there is none.  roots[0] is
 * the root of tree A (or of the one tree), roots[1] that of tree B or -1.
 * Returns 0, -1 on a bad argument, -2 when out of memory. */
int dpo_trees(int p, int layout, int32_t* parent, int32_t* child0,
              int32_t* child1, int32_t* depth, int32_t* roots);

/* y = x_0 (.) ... (.) x_{p-1} over m elements, in the association of the
 * trees (Algorithm 1).  x: p row pointers, each m elements of the
 * operator's type; y: m elements.  threads >= 1: the columns are cut into
 * that many contiguous ranges, one thread each.  Returns 0, -1 on a bad
 * argument, -2 when out of memory.  m == 0 does nothing. */
int dpo_allreduce(int kind, int layout, const void* const* x, int p, size_t m,
                  void* y, int threads);

/* The same, y written into each of the p output rows (the broadcast half
 * of the reduction-to-all).  Outputs must not overlap the inputs. */
int dpo_allreduce_all(int kind, int layout, const void* const* x,
                      void* const* out, int p, size_t m, int threads);

#ifdef __cplusplus
}
#endif

#endif
