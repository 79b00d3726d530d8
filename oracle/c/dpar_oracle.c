/* Plain C oracle of the reduction-to-all (Traeff 2021).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path links, loads or
 * calls this file: only the tests, the smoke check and the CPU baseline of
 * the benchmark do.  It shares no code, header, table or helper with the
 * HIP library and includes nothing from it.
 *
 * What it computes (Section 1, problem statement): p ranks each hold m
 * elements x_i; every rank receives y = x_0 (.) x_1 (.) ... (.) x_{p-1},
 * element by element.  For fp32 SUM the association is part of the result;
 * it is the one the two trees of Section 1.1 impose under Algorithm 1:
 *
 *   - Tree A holds ranks [0, ceil(p/2)), tree B the rest.  Each is the
 *     heap-shaped complete binary tree on its n ranks (heap indices 1..n,
 *     children 2h and 2h+1, last level filled from the left), numbered in
 *     post-order from its first rank, so that its root is its last rank.
 *   - The first child of a rank i is i-1 (the right heap child, or the only
 *     child); the second child is the left heap child when there are two.
 *   - A rank combines the value of its first child's subtree into its own
 *     block with the child's value on the left, then the value of its second
 *     child's subtree the same way:  S(i) = S(c1) (.) (S(c0) (.) x_i).
 *   - The two roots exchange their tree values; both end with
 *     y = S(root A) (.) S(root B).
 *   - The one-tree layout (Section 1.2's single doubly-pipelined tree and the
 *     tree of Section 2's reduce-then-broadcast) is one heap-shaped tree over
 *     all p ranks, y = S(p-1).
 *
 * Evaluation: ranks are visited in increasing order (post-order), keeping a
 * stack of subtree values; every column is independent, so each stack entry
 * is a vector over the columns a thread owns.  A rank with no child pushes
 * its x_i; a rank with children combines x_i into the top entry (its first
 * child's value), then, if it has a second child, combines the top entry
 * into the one beneath it (the second child's value) and pops.  Columns are
 * cut into contiguous ranges only to run them on several threads; nothing is
 * blocked, fused or reordered within a column.
 *
 * Operators: int32 SUM with two's-complement wrap (computed in uint32),
 * int32 MAX, fp32 SUM in IEEE binary32 with round to nearest even (build
 * without fast-math and without FMA contraction), and the product of 2x2
 * uint32 matrices (row-major, 16 bytes) modulo 2^32, which is not
 * commutative.
 *
 * DPO_MUTANT (0 unless a test builds a copy with a planted mistake): 1 takes
 * the second child before the first, 2 puts the child's value on the right,
 * 3 combines the two roots the other way round, 4 combines the two children
 * with each other first, (S(c1) (.) S(c0)) (.) x_i.
 */

#include "dpar_oracle.h"

#include <pthread.h>
#include <stdlib.h>
#include <string.h>

#ifndef DPO_MUTANT
#define DPO_MUTANT 0
#endif

/* ------------------------------------------------------------- operators */

static size_t elem_bytes(int kind) { return kind == DPO_U32MAT_MATMUL ? 16 : 4; }

/* a[k] = a[k] (.) b[k] for k in [0, n): the left operand is overwritten. */
static void combine_left(int kind, void* a, const void* b, size_t n) {
  size_t k;
  if (kind == DPO_I32_SUM) {
    uint32_t* u = (uint32_t*)a;
    const uint32_t* v = (const uint32_t*)b;
    for (k = 0; k < n; ++k) u[k] = u[k] + v[k];
  } else if (kind == DPO_I32_MAX) {
    int32_t* u = (int32_t*)a;
    const int32_t* v = (const int32_t*)b;
    for (k = 0; k < n; ++k) u[k] = u[k] > v[k] ? u[k] : v[k];
  } else if (kind == DPO_F32_SUM) {
    float* u = (float*)a;
    const float* v = (const float*)b;
    for (k = 0; k < n; ++k) u[k] = u[k] + v[k];
  } else {
    uint32_t* u = (uint32_t*)a;
    const uint32_t* v = (const uint32_t*)b;
    for (k = 0; k < n; ++k, u += 4, v += 4) {
      const uint32_t r0 = u[0] * v[0] + u[1] * v[2];
      const uint32_t r1 = u[0] * v[1] + u[1] * v[3];
      const uint32_t r2 = u[2] * v[0] + u[3] * v[2];
      const uint32_t r3 = u[2] * v[1] + u[3] * v[3];
      u[0] = r0;
      u[1] = r1;
      u[2] = r2;
      u[3] = r3;
    }
  }
}

#if DPO_MUTANT == 2 || DPO_MUTANT == 3
/* a[k] = b[k] (.) a[k]: the right operand is overwritten (planted
 * mistakes only). */
static void combine_right(int kind, void* a, const void* b, size_t n) {
  size_t k;
  if (kind != DPO_U32MAT_MATMUL) {
    /* SUM and MAX commute bit for bit, fp32 addition included */
    combine_left(kind, a, b, n);
    return;
  }
  {
    uint32_t* u = (uint32_t*)a;
    const uint32_t* v = (const uint32_t*)b;
    for (k = 0; k < n; ++k, u += 4, v += 4) {
      const uint32_t r0 = v[0] * u[0] + v[1] * u[2];
      const uint32_t r1 = v[0] * u[1] + v[1] * u[3];
      const uint32_t r2 = v[2] * u[0] + v[3] * u[2];
      const uint32_t r3 = v[2] * u[1] + v[3] * u[3];
      u[0] = r0;
      u[1] = r1;
      u[2] = r2;
      u[3] = r3;
    }
  }
}
#endif

/* ------------------------------------------------------------------ trees */

/* One heap-shaped tree on n ranks starting at `first`, numbered in
 * post-order.  The ranks of a subtree are contiguous: the subtree of heap
 * node h starts at lo[h], its left subtree comes first, then its right
 * subtree, then h itself, so rank(h) = lo[h] + size(h) - 1. */
static int heap_tree(int n, int first, int32_t* parent, int32_t* child0,
                     int32_t* child1, int32_t* depth) {
  int h;
  int32_t* size = (int32_t*)calloc((size_t)n + 2, sizeof(int32_t));
  int32_t* lo = (int32_t*)calloc((size_t)n + 2, sizeof(int32_t));
  int32_t* rank = (int32_t*)calloc((size_t)n + 2, sizeof(int32_t));
  if (!size || !lo || !rank) {
    free(size);
    free(lo);
    free(rank);
    return -2;
  }
  for (h = n; h >= 1; --h) {
    size[h] = 1;
    if (2 * h <= n) size[h] += size[2 * h];
    if (2 * h + 1 <= n) size[h] += size[2 * h + 1];
  }
  lo[1] = first;
  for (h = 1; h <= n; ++h) {
    if (2 * h <= n) lo[2 * h] = lo[h];
    if (2 * h + 1 <= n) lo[2 * h + 1] = lo[h] + size[2 * h];
    rank[h] = lo[h] + size[h] - 1;
  }
  for (h = 1; h <= n; ++h) {
    const int r = rank[h];
    int d = 0, g = h;
    while (g > 1) {
      g /= 2;
      ++d;
    }
    depth[r] = d;
    parent[r] = h > 1 ? rank[h / 2] : -1;
    if (2 * h + 1 <= n) {        /* two children: the right one is first */
      child0[r] = rank[2 * h + 1];
      child1[r] = rank[2 * h];
    } else if (2 * h <= n) {     /* only a left child: it is the first */
      child0[r] = rank[2 * h];
      child1[r] = -1;
    } else {
      child0[r] = -1;
      child1[r] = -1;
    }
  }
  free(size);
  free(lo);
  free(rank);
  return 0;
}

int dpo_trees(int p, int layout, int32_t* parent, int32_t* child0,
              int32_t* child1, int32_t* depth, int32_t* roots) {
  int n_a, rc;
  if (p < 1 || (layout != DPO_DUAL && layout != DPO_SINGLE) || !parent ||
      !child0 || !child1 || !depth || !roots)
    return -1;
  n_a = layout == DPO_DUAL ? (p + 1) / 2 : p;
  rc = heap_tree(n_a, 0, parent, child0, child1, depth);
  if (rc) return rc;
  roots[0] = n_a - 1;
  roots[1] = -1;
  if (n_a < p) {
    rc = heap_tree(p - n_a, n_a, parent, child0, child1, depth);
    if (rc) return rc;
    roots[1] = p - 1;
  }
  return 0;
}

/* --------------------------------------------------------------- reduction */

struct job {
  int kind;
  int p;
  const void* const* x;
  void* y;                  /* m elements, or NULL when only `out` is wanted */
  void* const* out;         /* p output rows, or NULL */
  size_t k0, k1;            /* this thread's columns */
  const int32_t* child0;
  const int32_t* child1;
  int nroots;
  int depth_max;            /* stack entries the evaluation can need */
  int rc;
};

static void* run_job(void* arg) {
  struct job* j = (struct job*)arg;
  const size_t e = elem_bytes(j->kind);
  const size_t n = j->k1 - j->k0;
  const size_t row = n * e;
  unsigned char* stack;
  int top = 0, i;
  j->rc = 0;
  if (n == 0) return NULL;
  stack = (unsigned char*)malloc((size_t)j->depth_max * row);
  if (!stack) {
    j->rc = -2;
    return NULL;
  }
  for (i = 0; i < j->p; ++i) {
    const unsigned char* xi = (const unsigned char*)j->x[i] + j->k0 * e;
    const int c0 = j->child0[i], c1 = j->child1[i];
    if (c0 < 0) {                       /* leaf: its own block */
      memcpy(stack + (size_t)top * row, xi, row);
      ++top;
      continue;
    }
#if DPO_MUTANT == 1
    if (c1 >= 0) {
      /* planted mistake: the second child's value (beneath) is taken first */
      unsigned char* tmp = (unsigned char*)malloc(row);
      if (!tmp) {
        free(stack);
        j->rc = -2;
        return NULL;
      }
      memcpy(tmp, stack + (size_t)(top - 1) * row, row);
      memcpy(stack + (size_t)(top - 1) * row, stack + (size_t)(top - 2) * row,
             row);
      memcpy(stack + (size_t)(top - 2) * row, tmp, row);
      free(tmp);
    }
#endif
#if DPO_MUTANT == 4
    if (c1 >= 0) {
      /* planted mistake: (S(c1) (.) S(c0)) (.) x_i */
      combine_left(j->kind, stack + (size_t)(top - 2) * row,
                   stack + (size_t)(top - 1) * row, n);
      --top;
      combine_left(j->kind, stack + (size_t)(top - 1) * row, xi, n);
      continue;
    }
#endif
    /* first child: Y <- S(c0) (.) x_i, in the first child's entry */
#if DPO_MUTANT == 2
    {
      unsigned char* t = stack + (size_t)(top - 1) * row;
      combine_right(j->kind, t, xi, n);   /* planted mistake: x_i (.) S(c0) */
    }
#else
    combine_left(j->kind, stack + (size_t)(top - 1) * row, xi, n);
#endif
    if (c1 >= 0) {
      /* second child: Y <- S(c1) (.) Y, in the second child's entry */
#if DPO_MUTANT == 2
      combine_right(j->kind, stack + (size_t)(top - 2) * row,
                    stack + (size_t)(top - 1) * row, n);
#else
      combine_left(j->kind, stack + (size_t)(top - 2) * row,
                   stack + (size_t)(top - 1) * row, n);
#endif
      --top;
    }
  }
  /* top == number of roots: [S(root A)] or [S(root A), S(root B)] */
  if (top != j->nroots) {
    free(stack);
    j->rc = -3;
    return NULL;
  }
  if (top == 2) {
#if DPO_MUTANT == 3
    combine_right(j->kind, stack, stack + row, n);   /* planted: T_B (.) T_A */
#else
    combine_left(j->kind, stack, stack + row, n);    /* T_A (.) T_B */
#endif
  }
  if (j->y) memcpy((unsigned char*)j->y + j->k0 * e, stack, row);
  if (j->out) {
    for (i = 0; i < j->p; ++i)
      memcpy((unsigned char*)j->out[i] + j->k0 * e, stack, row);
  }
  free(stack);
  return NULL;
}

static int reduce(int kind, int layout, const void* const* x, int p, size_t m,
                  void* y, void* const* out, int threads) {
  int32_t *parent, *child0, *child1, *depth;
  int32_t roots[2];
  struct job* jobs;
  pthread_t* tids;
  int rc = 0, t, i, top = 0, top_max = 0, started = 0;
  if (kind < DPO_I32_SUM || kind > DPO_U32MAT_MATMUL || p < 1 || !x ||
      threads < 1 || (layout != DPO_DUAL && layout != DPO_SINGLE))
    return -1;
  if (m == 0) return 0;
  for (i = 0; i < p; ++i)
    if (!x[i] || (out && !out[i])) return -1;
  if ((size_t)threads > m) threads = (int)m;
  parent = (int32_t*)malloc((size_t)p * sizeof(int32_t));
  child0 = (int32_t*)malloc((size_t)p * sizeof(int32_t));
  child1 = (int32_t*)malloc((size_t)p * sizeof(int32_t));
  depth = (int32_t*)malloc((size_t)p * sizeof(int32_t));
  jobs = (struct job*)calloc((size_t)threads, sizeof(struct job));
  tids = (pthread_t*)calloc((size_t)threads, sizeof(pthread_t));
  if (!parent || !child0 || !child1 || !depth || !jobs || !tids) {
    rc = -2;
    goto done;
  }
  rc = dpo_trees(p, layout, parent, child0, child1, depth, roots);
  if (rc) goto done;
  /* the largest stack the walk reaches (one more entry for a leaf) */
  for (i = 0; i < p; ++i) {
    if (child0[i] < 0) {
      ++top;
    } else if (child1[i] >= 0) {
      --top;
    }
    if (top > top_max) top_max = top;
  }
  for (t = 0; t < threads; ++t) {
    struct job* j = &jobs[t];
    j->kind = kind;
    j->p = p;
    j->x = x;
    j->y = y;
    j->out = out;
    j->k0 = m * (size_t)t / (size_t)threads;
    j->k1 = m * (size_t)(t + 1) / (size_t)threads;
    j->child0 = child0;
    j->child1 = child1;
    j->nroots = roots[1] >= 0 ? 2 : 1;
    j->depth_max = top_max;
  }
  if (threads == 1) {
    run_job(&jobs[0]);
  } else {
    for (t = 0; t < threads; ++t) {
      if (pthread_create(&tids[t], NULL, run_job, &jobs[t]) != 0) {
        rc = -2;
        break;
      }
      ++started;
    }
    for (t = 0; t < started; ++t) pthread_join(tids[t], NULL);
  }
  for (t = 0; t < threads && !rc; ++t) rc = jobs[t].rc;
done:
  free(parent);
  free(child0);
  free(child1);
  free(depth);
  free(jobs);
  free(tids);
  return rc;
}

int dpo_allreduce(int kind, int layout, const void* const* x, int p, size_t m,
                  void* y, int threads) {
  if (!y && m) return -1;
  return reduce(kind, layout, x, p, m, y, NULL, threads);
}

int dpo_allreduce_all(int kind, int layout, const void* const* x,
                      void* const* out, int p, size_t m, int threads) {
  if (!out) return -1;
  return reduce(kind, layout, x, p, m, NULL, out, threads);
}
