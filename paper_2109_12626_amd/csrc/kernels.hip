// gfx950 kernels for the doubly-pipelined, dual-root reduction-to-all
// (Traeff 2021, Algorithm 1), all p virtual ranks on one GPU.
//
// Work item = one chunk (<= 64 quanta) of one pipeline block Y[j].  For its
// columns a workgroup runs the whole round of Algorithm 1 on chip:
//
//   * receive-reduce-forward up both trees: the ranks are visited in
//     post-order; rank i's block is loaded once from HBM (16-byte lanes),
//     combined as Y <- t (.) Y with its first child's block (held in a
//     register, "current") and then with its second child's block (waiting in
//     a per-depth LDS slot), and forwarded to its parent by staying in the
//     register or by being parked in the slot of its own depth;
//   * dual-root exchange: with two wavefronts per workgroup, wavefront 0 owns
//     tree A and wavefront 1 tree B; the two root blocks meet in LDS and both
//     compute y = T_A (.) T_B, the lower root's value on the left;
//   * write-out: y goes from registers to all p output buffers (fused), or
//     to y_0 only, from where a broadcast pass copies it on (split), or to
//     the roots' outputs only, from where the round-structured down-step
//     passes it from parent to child one depth per round.
//
// Short chunks can instead be evaluated level by level with the chunk staged
// in LDS (run_unit_lv).  Round sequencing: all work items in round order in
// one launch (split: the hardware dispatcher hands them out), one launch per
// round, a persistent kernel with a grid barrier per round, a persistent
// kernel that claims work items from atomic tickets in round order, or the
// full round structure including the down-phase (k_rounds,
// k_rounds_barrier).  One tree (Sections 1.2, 2) runs through the same code
// in a two-part form (plan.hpp kernel_single_tree).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <map>
#include <type_traits>
#include <utility>

#include "kernels.hpp"
#include "plan.hpp"

namespace dpar {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// The same 16 bytes in global memory, where a row may start at any 4-byte
// boundary: gfx950 loads and stores 16 bytes at 4-byte aligned addresses in
// one instruction (the HSA runtime runs the GPU in unaligned access mode, so
// the compiler emits global_load/store_dwordx4 for this type as well).
typedef uint32_t u32x4g __attribute__((ext_vector_type(4), aligned(4)));

// Global-memory pointers (address space 1): lets the compiler emit global_*
// instructions with a scalar base and a 32-bit per-lane offset instead of
// flat accesses.
#define DPAR_GLOBAL __attribute__((address_space(1)))

#ifndef DPAR_NT_LOAD
#define DPAR_NT_LOAD 1
#endif
#ifndef DPAR_NT_STORE
#define DPAR_NT_STORE 1
#endif

template <class T>
__device__ inline T ld(const DPAR_GLOBAL T* p) {
#if DPAR_NT_LOAD
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}
template <class T>
__device__ inline void st(DPAR_GLOBAL T* p, T v) {
#if DPAR_NT_STORE
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

template <class T>
__device__ inline const DPAR_GLOBAL T* gptr(uint64_t row, uint32_t off) {
  return reinterpret_cast<const DPAR_GLOBAL T*>(
      reinterpret_cast<const DPAR_GLOBAL char*>(row) + off);
}
template <class T>
__device__ inline DPAR_GLOBAL T* gptr_w(uint64_t row, uint32_t off) {
  return reinterpret_cast<DPAR_GLOBAL T*>(
      reinterpret_cast<DPAR_GLOBAL char*>(row) + off);
}

// ------------------------------------------------------------ operators

struct I32Sum {
  __device__ static uint32_t ap(uint32_t a, uint32_t b) { return a + b; }
};
struct I32Max {
  __device__ static uint32_t ap(uint32_t a, uint32_t b) {
    return (int32_t)a > (int32_t)b ? a : b;
  }
};
struct F32Sum {
  __device__ static uint32_t ap(uint32_t a, uint32_t b) {
    return __float_as_uint(__fadd_rn(__uint_as_float(a), __uint_as_float(b)));
  }
};

// 2x2 matrix product mod 2^32, row-major [a00, a01, a10, a11]; a on the left.
__device__ inline u32x4 mat_mul(u32x4 a, u32x4 b) {
  u32x4 c;
  c.x = a.x * b.x + a.y * b.z;
  c.y = a.x * b.y + a.y * b.w;
  c.z = a.z * b.x + a.w * b.z;
  c.w = a.z * b.y + a.w * b.w;
  return c;
}

// ------------------------------------------------------------ lane layouts
// A lane owns one quantum: `bytes` contiguous bytes of every rank row.

template <class E>
struct Lane4 {  // four scalars, one 16-byte access (4-byte aligned)
  using T = u32x4;
  static constexpr uint32_t bytes = 16;
  __device__ static T ap(T a, T b) {
    T r;
    r.x = E::ap(a.x, b.x);
    r.y = E::ap(a.y, b.y);
    r.z = E::ap(a.z, b.z);
    r.w = E::ap(a.w, b.w);
    return r;
  }
  __device__ static T load(uint64_t row, uint32_t off) {
    return ld(gptr<u32x4g>(row, off));
  }
  __device__ static void store(uint64_t row, uint32_t off, T v) {
    st(gptr_w<u32x4g>(row, off), (u32x4g)v);
  }
};

template <class E>
struct Lane1 {  // one scalar
  using T = uint32_t;
  static constexpr uint32_t bytes = 4;
  __device__ static T ap(T a, T b) { return E::ap(a, b); }
  __device__ static T load(uint64_t row, uint32_t off) {
    return ld(gptr<T>(row, off));
  }
  __device__ static void store(uint64_t row, uint32_t off, T v) {
    st(gptr_w<T>(row, off), v);
  }
};

struct LaneMat {  // one matrix, one 16-byte access (4-byte aligned)
  using T = u32x4;
  static constexpr uint32_t bytes = 16;
  __device__ static T ap(T a, T b) { return mat_mul(a, b); }
  __device__ static T load(uint64_t row, uint32_t off) {
    return ld(gptr<u32x4g>(row, off));
  }
  __device__ static void store(uint64_t row, uint32_t off, T v) {
    st(gptr_w<u32x4g>(row, off), (u32x4g)v);
  }
};

// ------------------------------------------------------------ one work item

// Lines [ls, le) of work item t's blocks and the item's chunk c within them:
// work item t belongs to group g = t / C, which holds the whole blocks
// [g G, min(g G + G, b)) (G = prm.grp consecutive blocks; 1 except in the
// one-launch executors when blocks are shorter than half a chunk); block j
// is the run of lines [floor(j NL / b), floor((j + 1) NL / b)) of Section
// 1.1's partition into b blocks.
__device__ inline void item_lines(const Params& prm, uint64_t t, uint64_t* ls,
                                  uint64_t* le, uint64_t* c) {
  const uint64_t g = t / (uint64_t)prm.C;
  *c = t % (uint64_t)prm.C;
  const uint64_t j0 = g * (uint64_t)prm.grp;
  const uint64_t j1 = min(j0 + (uint64_t)prm.grp, (uint64_t)prm.b);
  *ls = prm.NL * j0 / (uint64_t)prm.b;
  *le = prm.NL * j1 / (uint64_t)prm.b;
}

// Work-item groups of a one-launch run (b when every group is one block).
__device__ __host__ inline uint64_t item_groups(const Params& prm) {
  return ((uint64_t)prm.b + (uint64_t)prm.grp - 1) / (uint64_t)prm.grp;
}

// Ranks whose loads are in flight per wavefront.  The host pads the pointer
// and opcode tables by kTablePad >= 2 * kU entries.
#ifndef DPAR_KU
#define DPAR_KU 8
#endif
constexpr int kU = DPAR_KU;
static_assert(2 * kU <= kTablePad, "tables are padded for 2 * kU reads");
// The subtree work item's deep variant (Params::sub_deep): 16 loads in flight
// per wavefront, for calls whose items all run at once, one per CU.
constexpr int kUDeep = 16;
static_assert(2 * kUDeep <= kTablePad, "tables are padded for 2 * kU reads");

// Up-step of one chunk over the ranks [r0, r1) in post-order (Algorithm 1's
// "Y <- t (.) Y" with the first child's block, then with the second
// child's): rank i's block is loaded, combined with its first child's value
// (`cur`, a register) and its second child's (waiting in slot d + 1), and
// then waits in slot d (a second child) or becomes `cur`; d is the opcode's
// slot depth, slots are my[(d - base) * 64].  Loads run in a rotating
// pipeline of kU: slot k of `buf` holds rank base + k; it is consumed and at
// once refilled with rank base + kU + k.  The tables are padded by kU
// entries, so reading kU entries ahead stays inside them; ranks past r1
// re-read row r1 - 1 (cache hits) and are not processed.  TAIL (fused work
// items, whose write-out follows at once): no load is issued for a rank
// past r1; the full rounds of KU ranks run branch-free and only the last
// ones test for the end.  Returns the value of the last rank walked.
template <class L, int KU = kU, bool TAIL = false>
__device__ __forceinline__ typename L::T walk(const uint64_t* __restrict__ xp,
                                              const uint32_t* __restrict__ ops,
                                              int r0, int r1,
                                              uint64_t unit_off,
                                              uint32_t lane_off,
                                              typename L::T* my, int base,
                                              typename L::T& cur) {
  using T = typename L::T;
  T last = T{};
  auto step = [&](T v, uint32_t op) {
    const int d = (int)(op & OP_DEPTH_MASK) - base;
    if (op & OP_C0) v = L::ap(cur, v);                 // first child
    if (op & OP_C1) v = L::ap(my[(d + 1) * 64], v);    // second child
    if (op & OP_SAVE)
      my[d * 64] = v;
    else
      cur = v;
    last = v;
  };
  const uint64_t last_row = xp[r1 - 1] + unit_off;
  T buf[KU];
  if constexpr (TAIL) {
#pragma unroll
    for (int k = 0; k < KU; ++k) {
      buf[k] = T{};
      if (r0 + k < r1) buf[k] = L::load(xp[r0 + k] + unit_off, lane_off);
      __builtin_amdgcn_sched_barrier(0);
    }
    int rb = r0;
    // full rounds: every rank consumed and every refill a rank below r1
    for (; rb + 2 * KU <= r1; rb += KU) {
      uint64_t next_row[KU];
      uint32_t op[KU];
#pragma unroll
      for (int k = 0; k < KU; ++k) {
        next_row[k] = xp[rb + KU + k] + unit_off;
        op[k] = ops[rb + k];
      }
#pragma unroll
      for (int k = 0; k < KU; ++k) {
        const T v = buf[k];
        buf[k] = L::load(next_row[k], lane_off);
        __builtin_amdgcn_sched_barrier(0);
        step(v, op[k]);
      }
    }
    for (; rb < r1; rb += KU) {
      uint64_t next_row[KU];
      uint32_t op[KU];
#pragma unroll
      for (int k = 0; k < KU; ++k) {
        next_row[k] = xp[rb + KU + k] + unit_off;
        op[k] = ops[rb + k];
      }
#pragma unroll
      for (int k = 0; k < KU; ++k) {
        const T v = buf[k];
        if (rb + KU + k < r1) buf[k] = L::load(next_row[k], lane_off);
        __builtin_amdgcn_sched_barrier(0);
        if (rb + k < r1) step(v, op[k]);
      }
    }
    return last;
  }
#pragma unroll
  for (int k = 0; k < KU; ++k) {
    const uint64_t row = xp[r0 + k] + unit_off;
    buf[k] = L::load(r0 + k < r1 ? row : last_row, lane_off);
    // keep the loads in slot order: the wait before consuming slot k then
    // only needs the oldest load, in the prologue and in the loop alike
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int rb = r0; rb < r1; rb += KU) {
    uint64_t next_row[KU];
    uint32_t op[KU];
#pragma unroll
    for (int k = 0; k < KU; ++k) {
      next_row[k] = xp[rb + KU + k] + unit_off;
      op[k] = ops[rb + k];
    }
#pragma unroll
    for (int k = 0; k < KU; ++k) {
      const T v = buf[k];
      buf[k] = L::load(rb + KU + k < r1 ? next_row[k] : last_row, lane_off);
      __builtin_amdgcn_sched_barrier(0);
      if (rb + k < r1) step(v, op[k]);
    }
  }
  return last;
}

// Processes work item t (block j = t / C, chunk c = t % C).  FUSED: y goes
// straight to all p outputs; otherwise only to y_0, from where a separate
// broadcast pass copies it to the other p - 1 outputs.
template <class L, int W, bool FUSED>
__device__ __forceinline__ void run_unit(const uint64_t* __restrict__ xp,
                                         const uint64_t* __restrict__ yp,
                                         const uint32_t* __restrict__ ops,
                                         const Params& prm, uint64_t t,
                                         typename L::T* slots) {
  using T = typename L::T;
  const int lane = threadIdx.x & 63;
  // wave-uniform by construction; readfirstlane tells the compiler so, which
  // keeps every rank index, table read and branch below in scalar registers
  const int wave =
      (W == 1) ? 0 : __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));

  // chunk -> quanta [cs, ce): the item's blocks are a run of lines, cut
  // into C chunks at line boundaries
  uint64_t cs, ce;
  item_quanta(prm.NL, (uint64_t)prm.b, (uint64_t)prm.C, (uint64_t)prm.grp,
              prm.lq, prm.Q, t, &cs, &ce);
  const uint32_t count = (uint32_t)(ce - cs);
  if (count == 0) return;  // uniform; cannot happen for b <= Q
  const uint64_t unit_off = (prm.qbase + cs) * (uint64_t)L::bytes;
  // lanes past the chunk re-read the last quantum (no branch on the loads)
  const uint32_t lane_off =
      (uint32_t)(lane < (int)count ? lane : (int)count - 1) * L::bytes;
  const bool active = lane < (int)count;

  int r0 = 0, r1 = prm.p;
  if (W == 2) {
    r0 = wave == 0 ? 0 : prm.n_a;
    r1 = wave == 0 ? prm.n_a : prm.p;
  }
  T* my = slots + (size_t)wave * prm.nslots * 64 + lane;

  T cur = T{};
  walk<L, kU, FUSED>(xp, ops, r0, r1, unit_off, lane_off, my, 0, cur);

  // Dual-root exchange.
  T y;
  if (W == 1) {
    y = prm.dual ? L::ap(my[0], cur) : my[0];
  } else {
    if (wave == 1) my[0] = cur;  // tree B's root value
    __syncthreads();
    y = L::ap(slots[lane], slots[(size_t)prm.nslots * 64 + lane]);
  }

  // Fused broadcast of y to this wavefront's ranks, or y to the outputs of
  // ranks out0 and out1 only.
  if (!FUSED) {
    if (active) {
      if (W == 1) {
        L::store(yp[prm.out0] + unit_off, lane_off, y);
        if (prm.out1 >= 0) L::store(yp[prm.out1] + unit_off, lane_off, y);
      } else {
        const int o = wave == 0 ? prm.out0 : prm.out1;
        if (o >= 0) L::store(yp[o] + unit_off, lane_off, y);
      }
    }
  } else if (active) {
    for (int base = r0; base < r1; base += kU) {
      uint64_t row[kU];
#pragma unroll
      for (int k = 0; k < kU; ++k) row[k] = yp[base + k] + unit_off;
#pragma unroll
      for (int k = 0; k < kU; ++k)
        if (base + k < r1) L::store(row[k], lane_off, y);
    }
  }
  if (W == 2) __syncthreads();  // slots are reused by the next work item
}

// ------------------------------------------------------------ level units
// Level-synchronous work item, for chunks too small to keep a GPU busy with
// one post-order walk per chunk.  1024 threads load every rank's quanta of a
// chunk of at most T quanta into LDS at once, then evaluate the two trees one
// depth level at a time from the deepest up: every (node, quantum) pair of a
// level computes S(i) = S(child1) (.) (S(child0) (.) x_i) from children
// finished in the previous level, then a barrier.  Same association as the
// post-order walk; the dependent chain is H + 1 levels instead of p loads.
//
// LDS: S [p][T] lane values | Y [T] | ptr [p] row addresses | lvl [p]
// level-ordered entries | off [H + 2] level boundaries.
constexpr int kLvThreads = 1024;
constexpr int kLvBatch = 8;  // loads in flight per thread

__host__ __device__ inline size_t align16(size_t v) { return (v + 15) & ~(size_t)15; }

template <class L>
struct LvLayout {
  size_t s, y, ptr, lvl, off, total;
  __host__ __device__ LvLayout(int p, int T, int nlev) {
    s = 0;
    y = align16(s + (size_t)p * T * sizeof(typename L::T));
    ptr = align16(y + (size_t)T * sizeof(typename L::T));
    lvl = align16(ptr + (size_t)p * 8);
    off = align16(lvl + (size_t)p * 4);
    total = align16(off + (size_t)(nlev + 1) * 4);
  }
};

template <class L, bool FUSED>
__device__ __forceinline__ void run_unit_lv(const uint64_t* __restrict__ xp,
                                            const uint64_t* __restrict__ yp,
                                            const uint32_t* __restrict__ lvl_g,
                                            const Params& prm, uint64_t t,
                                            char* lds) {
  using T = typename L::T;
  const int tid = threadIdx.x;
  const int p = prm.p, sh = prm.lv_log2t, TQ = 1 << sh, nlev = prm.nlev;
  const LvLayout<L> lay(p, TQ, nlev);
  T* S = reinterpret_cast<T*>(lds + lay.s);
  T* Y = reinterpret_cast<T*>(lds + lay.y);
  uint64_t* ptr = reinterpret_cast<uint64_t*>(lds + lay.ptr);
  uint32_t* lvl = reinterpret_cast<uint32_t*>(lds + lay.lvl);
  uint32_t* off = reinterpret_cast<uint32_t*>(lds + lay.off);

  // chunk -> quanta [cs, ce): the item's blocks are cut at lines, the chunk
  // at quanta
  uint64_t ls, le, c;
  item_lines(prm, t, &ls, &le, &c);
  const uint64_t qs = min(ls * prm.lq, prm.Q);
  const uint64_t qe = min(le * prm.lq, prm.Q);
  const uint64_t n = qe - qs;
  const uint64_t cs = qs + c * n / (uint64_t)prm.C;
  const uint64_t ce = qs + (c + 1) * n / (uint64_t)prm.C;
  const int count = (int)(ce - cs);
  if (count == 0) return;  // uniform
  const uint64_t unit_off = (prm.qbase + cs) * (uint64_t)L::bytes;

  for (int i = tid; i < p; i += kLvThreads) {
    ptr[i] = xp[i] + unit_off;
    lvl[i] = lvl_g[i];
  }
  for (int i = tid; i <= nlev; i += kLvThreads) off[i] = lvl_g[p + i];
  __syncthreads();

  // all loads of the chunk, kLvBatch per thread in flight
  const int total = p << sh;
  for (int base = 0; base < total; base += kLvThreads * kLvBatch) {
    T v[kLvBatch];
#pragma unroll
    for (int k = 0; k < kLvBatch; ++k) {
      const int idx = base + k * kLvThreads + tid;
      const bool ok = idx < total && (idx & (TQ - 1)) < count;
      // items past the chunk re-read quantum 0 of rank 0 (always in range)
      const int i = ok ? (idx >> sh) : 0;
      const uint32_t q = ok ? (uint32_t)(idx & (TQ - 1)) : 0u;
      v[k] = L::load(ptr[i], q * L::bytes);
    }
#pragma unroll
    for (int k = 0; k < kLvBatch; ++k) {
      const int idx = base + k * kLvThreads + tid;
      if (idx < total && (idx & (TQ - 1)) < count) S[idx] = v[k];
    }
  }
  __syncthreads();

  // levels, deepest first; entry = node << 16 | code, code 0xFFFF: leaf,
  // 0xFFFE: first child only (node - 1), else the second child's rank
  for (int lv = 0; lv < nlev; ++lv) {
    const int o0 = (int)off[lv];
    const int items = ((int)off[lv + 1] - o0) << sh;
    for (int idx = tid; idx < items; idx += kLvThreads) {
      const int q = idx & (TQ - 1);
      if (q >= count) continue;
      const uint32_t e = lvl[o0 + (idx >> sh)];
      const int node = (int)(e >> 16);
      const uint32_t code = e & 0xFFFFu;
      T v = S[(node << sh) + q];
      if (code != 0xFFFFu) v = L::ap(S[((node - 1) << sh) + q], v);
      if (code < 0xFFFEu) v = L::ap(S[((int)code << sh) + q], v);
      S[(node << sh) + q] = v;
    }
    __syncthreads();
  }

  // dual-root step, then the write-out
  if (tid < count) {
    const int ra = prm.n_a - 1;
    Y[tid] = prm.dual ? L::ap(S[(ra << sh) + tid], S[((p - 1) << sh) + tid])
                      : S[(ra << sh) + tid];
  }
  if (FUSED)
    for (int i = tid; i < p; i += kLvThreads) ptr[i] = yp[i] + unit_off;
  __syncthreads();
  if (FUSED) {
    for (int idx = tid; idx < total; idx += kLvThreads) {
      const int q = idx & (TQ - 1);
      if (q < count) L::store(ptr[idx >> sh], (uint32_t)q * L::bytes, Y[q]);
    }
  } else if (tid < count) {
    L::store(yp[prm.out0] + unit_off, (uint32_t)tid * L::bytes, Y[tid]);
    if (prm.out1 >= 0)
      L::store(yp[prm.out1] + unit_off, (uint32_t)tid * L::bytes, Y[tid]);
  }
  __syncthreads();  // LDS is reused by the next work item
}

size_t sub_lds_bytes(size_t lane_bytes, int ns) {
  return ((size_t)kSubParts * ns + kSubParts + 2 * kSubSpineRanks) * 64 *
         lane_bytes;
}

// ------------------------------------------------------------ subtree units
// Work item for chunks too few to keep a GPU busy when p is large: the trees
// are cut kSubParts ways (plan.hpp make_sub), wavefront w walks part w (a
// whole subtree, a contiguous rank range) with the post-order walk above,
// and then wavefront 0 (tree A) and 1 (tree B) walk their spines in the same
// post-order, taking each part's value where the part's root would come.
// The chains are p / kSubParts loads long instead of p / 2.  Same
// association, same operations as the post-order work item.
//
// LDS: slots [kSubParts][NS][64] | part values [kSubParts][64] | spine
// blocks [2][kSubSpineRanks][64].
template <class L, bool FUSED, int KU>
__device__ __forceinline__ void run_unit_sub(const uint64_t* __restrict__ xp,
                                             const uint64_t* __restrict__ yp,
                                             const uint32_t* __restrict__ ops,
                                             const uint32_t* __restrict__ sub,
                                             const Params& prm, uint64_t t,
                                             typename L::T* lds) {
  using T = typename L::T;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));

  // chunk -> quanta [cs, ce), as in run_unit
  uint64_t cs, ce;
  item_quanta(prm.NL, (uint64_t)prm.b, (uint64_t)prm.C, (uint64_t)prm.grp,
              prm.lq, prm.Q, t, &cs, &ce);
  const uint32_t count = (uint32_t)(ce - cs);
  if (count == 0) return;  // uniform
  const uint64_t unit_off = (prm.qbase + cs) * (uint64_t)L::bytes;
  const uint32_t lane_off =
      (uint32_t)(lane < (int)count ? lane : (int)count - 1) * L::bytes;
  const bool active = lane < (int)count;

  const int nparts = (int)sub[0];
  const int NS = (int)sub[3];
  const uint32_t* parts = sub + 4;
  const uint32_t* sranks = parts + 3 * nparts;   // [2][kSubSpineRanks]
  const uint32_t* spine = sranks + 2 * kSubSpineRanks;
  T* my = lds + (size_t)wave * NS * 64 + lane;
  T* pval = lds + (size_t)kSubParts * NS * 64;
  T* sx = pval + (size_t)kSubParts * 64;

  // the spine wavefronts start the loads of their spine ranks' blocks first
  T pre[kSubSpineRanks];
  if (wave < 2) {
#pragma unroll
    for (int k = 0; k < kSubSpineRanks; ++k)
      pre[k] = L::load(xp[sranks[wave * kSubSpineRanks + k]] + unit_off,
                       lane_off);
  }
  if (wave < nparts) {
    const int lo = (int)parts[3 * wave], hi = (int)parts[3 * wave + 1];
    const int base = (int)parts[3 * wave + 2];
    T cur = T{};
    pval[(size_t)wave * 64 + lane] =
        walk<L, KU, FUSED>(xp, ops, lo, hi + 1, unit_off, lane_off, my, base,
                           cur);
  }
  if (wave < 2) {
#pragma unroll
    for (int k = 0; k < kSubSpineRanks; ++k)
      sx[(size_t)(wave * kSubSpineRanks + k) * 64 + lane] = pre[k];
  }
  __syncthreads();

  // spines: the post-order of the top levels, parts taken from pval
  if (wave < 2) {
    const int n0 = (int)sub[1];
    const int n = wave == 0 ? n0 : (int)sub[2];
    const uint32_t* e = spine + (wave == 0 ? 0 : 2 * n0);
    T cur = T{};
    for (int k = 0; k < n; ++k) {
      const uint32_t code = e[2 * k], op = e[2 * k + 1];
      T v = (code & 0x80000000u)
                ? pval[(size_t)(code & 0xFFFFu) * 64 + lane]
                : sx[(size_t)(wave * kSubSpineRanks + code) * 64 + lane];
      const int d = (int)(op & OP_DEPTH_MASK);
      if (op & OP_C0) v = L::ap(cur, v);
      if (op & OP_C1) v = L::ap(my[(d + 1) * 64], v);
      if (op & OP_SAVE)
        my[d * 64] = v;
      else
        cur = v;
    }
    if (wave == 1) my[0] = cur;  // tree B's root value; tree A's is in slot 0
  }
  __syncthreads();
  const T y = L::ap(lds[lane], lds[(size_t)NS * 64 + lane]);

  if (!FUSED) {
    if (active) {
      if (wave == 0) L::store(yp[prm.out0] + unit_off, lane_off, y);
      if (wave == 1 && prm.out1 >= 0)
        L::store(yp[prm.out1] + unit_off, lane_off, y);
    }
  } else if (active) {
    // every wavefront writes its share of the p outputs
    const int r0 = (int)((int64_t)prm.p * wave / kSubParts);
    const int r1 = (int)((int64_t)prm.p * (wave + 1) / kSubParts);
    for (int rb = r0; rb < r1; rb += kU) {
      uint64_t row[kU];
#pragma unroll
      for (int k = 0; k < kU; ++k) row[k] = yp[rb + k] + unit_off;
#pragma unroll
      for (int k = 0; k < kU; ++k)
        if (rb + k < r1) L::store(row[k], lane_off, y);
    }
  }
  __syncthreads();  // LDS is reused by the next work item
}

// ------------------------------------------------------------ wide units
// Post-order work item for short walks over long rows.  A wavefront carries
// kWideQ quanta per lane (lane l: quanta l, l + 64, ...), so each rank
// visit reads kWideQ contiguous pieces of 64 quanta (kWideQ KB of the row
// on 16-byte lanes), with kWideKF visits in flight; the workgroup's
// kWideWaves wavefronts take neighbouring column ranges of its chunk, and
// each walks both trees (all p ranks, tree A then tree B) for its own
// columns, so the wavefronts never wait for each other.  Same association,
// same operations as the post-order work item, per column.  Only the
// one-launch executors run it, over chunks of kWideChunk quanta.
//
// Why: with few ranks every work item's walk is short, all the items of a
// call run at once and proceed in step, and one-KB pieces with many ranks
// in flight per wavefront then read HBM slowly (p = 36, rows of 4 MB:
// 5.5 TB/s with 1 KB per visit and 8 visits in flight; 6.5 TB/s with
// 4 KB per visit and 2 in flight, as fast as contiguous 16 KB tiles).
//
// A wide item holds its CU for a chain of p / kWideKF dependent visits,
// long next to its share of the bandwidth once fewer items than CUs are
// left; so the columns past the call's last whole round of full items (one
// item per CU) go to tail items of kWideTailQ quanta per lane with
// kWideTailKF visits in flight, whose chains are shorter (the host makes
// that cut).
//
// LDS: per wavefront nslots depth slots of QW x 64 lanes, slot d's piece u
// at [(d QW + u) 64 + lane] (one 16-byte access per lane, conflict-free);
// a tail item uses the first part of the full item's allocation.

// The scalars a wide work item reads: 64 bytes, loaded together at the
// start of its kernel.
struct WideArgs {
  const uint64_t* xp;
  const uint64_t* yp;
  const uint32_t* ops;
  uint64_t Q;
  uint64_t qbase;
  int p;
  int nslots;
  int out0;
  int out1;
  int dual;
  uint32_t nfull;  // items [0, nfull) are full, later ones tail items
};

__host__ __device__ inline WideArgs wide_args(const uint64_t* xp,
                                              const uint64_t* yp,
                                              const uint32_t* ops,
                                              const Params& prm) {
  return WideArgs{xp,       yp,          ops,       prm.Q,    prm.qbase,
                  prm.p,    prm.nslots,  prm.out0,  prm.out1, prm.dual,
                  prm.wide_full};
}

// One wide or tail work item whose columns start at quantum q0 of the
// call, QW quanta per lane, KF visits in flight per wavefront.
template <class L, bool FUSED, int QW, int KF>
__device__ __forceinline__ void run_unit_wide(const WideArgs& a, uint64_t q0,
                                              typename L::T* slots) {
  using T = typename L::T;
  const uint64_t* __restrict__ xp = a.xp;
  const uint64_t* __restrict__ yp = a.yp;
  const uint32_t* __restrict__ ops = a.ops;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));

  // this wavefront's share [ws, we) of the item's 64 QW kWideWaves quanta
  const uint64_t ws = min(q0 + (uint64_t)wave * 64 * QW, a.Q);
  const uint64_t we = min(ws + 64 * QW, a.Q);
  const uint32_t count = (uint32_t)(we - ws);
  // wave-uniform; the unit has no workgroup barrier, so a wavefront without
  // columns may leave at once
  if (count == 0) return;
  const uint64_t unit_off = (a.qbase + ws) * (uint64_t)L::bytes;
  // piece u of this lane: quantum lane + 64 u; lanes past the wavefront's
  // columns re-read its last quantum (no branch on the loads)
  uint32_t off[QW];
  bool act[QW];
#pragma unroll
  for (int u = 0; u < QW; ++u) {
    const uint32_t q = (uint32_t)lane + 64u * u;
    act[u] = q < count;
    off[u] = (act[u] ? q : count - 1) * L::bytes;
  }
  T* my = slots + (size_t)wave * a.nslots * QW * 64 + lane;

  const int p = a.p;
  T cur[QW];
#pragma unroll
  for (int u = 0; u < QW; ++u) cur[u] = T{};
  // rank visit: rank i's pieces combined with its first child's value
  // (cur) and its second child's (slot d + 1), then parked in slot d (a
  // second child) or kept as cur
  auto step = [&](T (&v)[QW], uint32_t op) {
    const int d = (int)(op & OP_DEPTH_MASK);
#pragma unroll
    for (int u = 0; u < QW; ++u) {
      T w = v[u];
      if (op & OP_C0) w = L::ap(cur[u], w);
      if (op & OP_C1) w = L::ap(my[((d + 1) * QW + u) * 64], w);
      if (op & OP_SAVE)
        my[(d * QW + u) * 64] = w;
      else
        cur[u] = w;
    }
  };
  // Rotating pipeline of KF visits: buffer slot k % KF holds visit k and
  // is refilled with visit k + KF once its step is done.  The row
  // addresses and opcodes come from the tables a group of G visits ahead
  // (scalar loads issued a group before they are needed; entries past p
  // name row p - 1, the opcode table is padded).
  constexpr int G = KF > 8 ? KF : 8;
  static_assert(G % KF == 0 && KF <= G, "groups hold whole pipelines");
  static_assert(2 * G <= kTablePad, "the walk reads two groups ahead");
  // (ranks past p read row p - 1 through a clamped index: a table load
  // under a condition would become a branch around a scalar load that waits
  // for it)
  uint64_t row_cur[G];
  uint32_t op_cur[G];
#pragma unroll
  for (int k = 0; k < G; ++k) {
    row_cur[k] = xp[min(k, p - 1)] + unit_off;
    op_cur[k] = ops[k];
  }
  T buf[KF][QW];
#pragma unroll
  for (int k = 0; k < KF; ++k) {
#pragma unroll
    for (int u = 0; u < QW; ++u) buf[k][u] = L::load(row_cur[k], off[u]);
    __builtin_amdgcn_sched_barrier(0);
  }
  // One group of G visits from gb.  STEP: a visit may lie past the last
  // rank (then it is not processed); LOAD: a refill may (then it is not
  // issued).  Groups that need neither run without a per-visit branch.
  auto group = [&](int gb, auto step_c, auto load_c) {
    constexpr bool STEP = decltype(step_c)::value;
    constexpr bool LOAD = decltype(load_c)::value;
    uint64_t row_nxt[G];
    uint32_t op_nxt[G];
#pragma unroll
    for (int k = 0; k < G; ++k) {
      row_nxt[k] = xp[min(gb + G + k, p - 1)] + unit_off;
      op_nxt[k] = ops[gb + G + k];
    }
#pragma unroll
    for (int k = 0; k < G; ++k) {
      const uint64_t nrow = k + KF < G ? row_cur[k + KF] : row_nxt[k + KF - G];
      // consumed before refilled: at most KF visits in flight (measured
      // 0-2% faster than refilling first, with one visit more in flight)
      if (!STEP || gb + k < p) step(buf[k % KF], op_cur[k]);
      if (!LOAD || gb + k + KF < p) {
#pragma unroll
        for (int u = 0; u < QW; ++u) buf[k % KF][u] = L::load(nrow, off[u]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int k = 0; k < G; ++k) {
      row_cur[k] = row_nxt[k];
      op_cur[k] = op_nxt[k];
    }
  };
  using yes = std::true_type;
  using no = std::false_type;
  int gb = 0;
  if constexpr (FUSED) {
    // The write-out follows the walk at once: loads issued past the last
    // rank would hold it up (they still count in the wavefront's memory
    // counter), and with few ranks outnumber the real ones (p = 2,
    // m = 2^22, one fused launch: 25.8 -> 17.3 us; p = 36, m = 2^20:
    // 56.6 -> 54.4 us).  So the full groups run branch-free and only the
    // last visits test for the end.
    for (; gb + G + KF <= p; gb += G) group(gb, no{}, no{});
    for (; gb < p; gb += G) group(gb, yes{}, yes{});
  } else {
    // Split up-phase: the last group re-reads row p - 1 for the visits past
    // the end (cache hits) rather than branch around those loads, whose
    // waits at the branches cost more there (p = 64 and 128: 1.5-2.3%).
    for (; gb < p; gb += G) group(gb, yes{}, no{});
  }

  // dual-root combine: tree A's root waits in slot 0, tree B's is cur
  T y[QW];
#pragma unroll
  for (int u = 0; u < QW; ++u)
    y[u] = a.dual ? L::ap(my[u * 64], cur[u]) : my[u * 64];

  if (!FUSED) {
#pragma unroll
    for (int u = 0; u < QW; ++u) {
      if (!act[u]) continue;
      L::store(yp[a.out0] + unit_off, off[u], y[u]);
      if (a.out1 >= 0) L::store(yp[a.out1] + unit_off, off[u], y[u]);
    }
  } else {
    for (int base = 0; base < p; base += kU) {
      uint64_t row[kU];
#pragma unroll
      for (int k = 0; k < kU; ++k) row[k] = yp[base + k] + unit_off;
#pragma unroll
      for (int k = 0; k < kU; ++k) {
        if (base + k >= p) continue;
#pragma unroll
        for (int u = 0; u < QW; ++u)
          if (act[u]) L::store(row[k], off[u], y[u]);
      }
    }
  }
}

// Work item t of a wide call: full items first (kWideChunk quanta each,
// from the call's first column), then tail items (kWideTailChunk each); the
// host cuts the columns this way whatever the blocks.  TAIL: the call has
// tail items (without them the kernel holds only the full items' walk: the
// combined kernel ran calls of full items only 1.5-3.5% slower).
template <class L, bool FUSED, bool TAIL>
__device__ __forceinline__ void run_wide_item(const WideArgs& a, uint64_t t,
                                              typename L::T* slots) {
  if (!TAIL || t < (uint64_t)a.nfull)
    run_unit_wide<L, FUSED, kWideQ, kWideKF>(a, t * kWideChunk, slots);
  else
    run_unit_wide<L, FUSED, kWideTailQ, kWideTailKF>(
        a, (uint64_t)a.nfull * kWideChunk + (t - a.nfull) * kWideTailChunk,
        slots);
}

// ------------------------------------------------------------ unit policies

template <class L, int W, bool FUSED>
struct SeqUnit {
  using Lane = L;
  static constexpr int kThreads = 64 * W;
  __device__ static void run(const uint64_t* __restrict__ xp,
                             const uint64_t* __restrict__ yp,
                             const uint32_t* __restrict__ ops,
                             const uint32_t* __restrict__ lvl,
                             const Params& prm, uint64_t t, char* lds) {
    (void)lvl;
    run_unit<L, W, FUSED>(xp, yp, ops, prm, t,
                          reinterpret_cast<typename L::T*>(lds));
  }
  static size_t lds(const Params& prm) {
    return (size_t)W * prm.nslots * 64 * sizeof(typename L::T);
  }
};

template <class L, bool FUSED, int KU = kU>
struct SubUnit {
  using Lane = L;
  static constexpr int kThreads = 64 * kSubParts;
  __device__ static void run(const uint64_t* __restrict__ xp,
                             const uint64_t* __restrict__ yp,
                             const uint32_t* __restrict__ ops,
                             const uint32_t* __restrict__ lvl,
                             const Params& prm, uint64_t t, char* lds) {
    run_unit_sub<L, FUSED, KU>(xp, yp, ops, lvl, prm, t,
                               reinterpret_cast<typename L::T*>(lds));
  }
  static size_t lds(const Params& prm) {
    return sub_lds_bytes(sizeof(typename L::T), prm.nslots);
  }
};

template <class L, bool FUSED>
struct LvUnit {
  using Lane = L;
  static constexpr int kThreads = kLvThreads;
  __device__ static void run(const uint64_t* __restrict__ xp,
                             const uint64_t* __restrict__ yp,
                             const uint32_t* __restrict__ ops,
                             const uint32_t* __restrict__ lvl,
                             const Params& prm, uint64_t t, char* lds) {
    (void)ops;
    run_unit_lv<L, FUSED>(xp, yp, lvl, prm, t, lds);
  }
  static size_t lds(const Params& prm) {
    return LvLayout<L>(prm.p, 1 << prm.lv_log2t, prm.nlev).total;
  }
};

template <class L, bool FUSED, bool TAIL>
struct WideUnit {
  using Lane = L;
  static constexpr int kThreads = 64 * kWideWaves;
  __device__ static void run(const uint64_t* __restrict__ xp,
                             const uint64_t* __restrict__ yp,
                             const uint32_t* __restrict__ ops,
                             const uint32_t* __restrict__ lvl,
                             const Params& prm, uint64_t t, char* lds) {
    (void)lvl;
    run_wide_item<L, FUSED, TAIL>(wide_args(xp, yp, ops, prm), t,
                                  reinterpret_cast<typename L::T*>(lds));
  }
  static size_t lds(const Params& prm) {
    return wide_lds_bytes(sizeof(typename L::T), prm.nslots);
  }
};

// ------------------------------------------------------------ executors

#define DPAR_KARGS                                                     \
  const uint64_t *__restrict__ xp, const uint64_t *__restrict__ yp,   \
      const uint32_t *__restrict__ ops, const uint32_t *__restrict__ lvl, \
      Params prm

template <class U>
__global__ __launch_bounds__(U::kThreads) void k_round(DPAR_KARGS, int round,
                                                      uint64_t first) {
  extern __shared__ char lds_raw[];
  // in launch order, or each XCD a contiguous run of the launch's items
  const uint64_t w =
      prm.xcd_runs ? xcd_run_index(blockIdx.x, gridDim.x) : blockIdx.x;
  U::run(xp, yp, ops, lvl, prm, (uint64_t)round * prm.C + first + w, lds_raw);
}

// One launch of wide work items (split up-phase, one fused launch): item
// first + blockIdx.x, its scalars in one 64-byte argument.
template <class L, bool FUSED, bool TAIL>
__global__ __launch_bounds__(64 * kWideWaves) void k_wide(WideArgs a,
                                                         uint64_t first) {
  extern __shared__ char lds_raw[];
  run_wide_item<L, FUSED, TAIL>(a, first + blockIdx.x,
                                reinterpret_cast<typename L::T*>(lds_raw));
}

__device__ inline void grid_barrier(const Params& prm) {
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned g =
        __hip_atomic_load(prm.bar_gen, __ATOMIC_RELAXED,
                          __HIP_MEMORY_SCOPE_AGENT);
    const unsigned arrived = __hip_atomic_fetch_add(
        prm.bar_count, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (arrived == gridDim.x - 1) {
      __hip_atomic_store(prm.bar_count, 0u, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_fetch_add(prm.bar_gen, 1u, __ATOMIC_RELEASE,
                             __HIP_MEMORY_SCOPE_AGENT);
    } else if (__hip_atomic_load(prm.bar_quit, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT) == 0) {
      // (once a wait of this call has given up, its later barriers do not
      // wait; the word belongs to this call alone)
      // Poll with relaxed loads: on this multi-XCD part an agent-scope
      // acquire invalidates the XCD's L2, and polling with it from many
      // workgroups would keep every L2 invalidating under the workgroups
      // still working.  One acquire after the wait is enough.
      unsigned long long spins = 0;
      while (__hip_atomic_load(prm.bar_gen, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT) == g) {
        __builtin_amdgcn_s_sleep(2);
        if (++spins > prm.spin_limit) {  // watchdog: give up, report
          atomicOr(prm.bar_quit, 1u);
          atomicOr(prm.err, 1u);
          break;
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
}

template <class U>
__global__ __launch_bounds__(U::kThreads) void k_barrier(DPAR_KARGS) {
  extern __shared__ char lds_raw[];
  for (int j = 0; j < prm.b; ++j) {
    for (uint64_t c = blockIdx.x; c < (uint64_t)prm.C; c += gridDim.x)
      U::run(xp, yp, ops, lvl, prm, (uint64_t)j * prm.C + c, lds_raw);
    if (j + 1 < prm.b) grid_barrier(prm);
  }
}

// ------------------------------------------------------------ round-structured executor
// Algorithm 1's round structure made explicit on the device.  Round r runs
// the up-step of block r (r < b) for all ranks, writing y[r] to the roots'
// outputs only, and the down-step: every rank at depth d >= 1 receives block
// r - d - dshift from its parent, i.e. copies it from the parent's output,
// which the parent received in round r - 1 (dshift = 0: the doubly-pipelined
// schedule of Algorithm 1; dshift = b - 1: the broadcast that follows a
// completed reduction, Section 2's reduce-then-broadcast).

// Down-step for the ranks at positions [a0, a1) of the depth-ordered rank
// table, piece k (kDownPiece quanta) of their blocks: the workgroup's
// wavefronts take the ranks in turn; a lane copies 4 quanta, all loads in
// flight before the stores.
template <class L, int TH>
__device__ __forceinline__ void down_copy(const uint64_t* __restrict__ yp,
                                          const uint32_t* __restrict__ dn,
                                          const uint32_t* __restrict__ ranks,
                                          const Params& prm, int round,
                                          uint32_t a0, uint32_t a1,
                                          uint64_t k) {
  constexpr int kWaves = TH / 64;
  constexpr int kQ = kDownPiece / 64;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  for (uint32_t a = a0 + wave; a < a1; a += kWaves) {
    const uint32_t i = ranks[a];
    const uint32_t e = dn[i];
    const uint32_t par = e >> 8;
    const int64_t j = (int64_t)round - (int64_t)(e & 0xFFu) - prm.dshift;
    if (par == 0xFFFFFFu || j < 0 || j >= prm.b) continue;  // not in range
    const uint64_t ls = prm.NL * (uint64_t)j / (uint64_t)prm.b;
    const uint64_t le = prm.NL * (uint64_t)(j + 1) / (uint64_t)prm.b;
    const uint64_t qs = min(ls * prm.lq, prm.Q);
    const uint64_t qe = min(le * prm.lq, prm.Q);
    const uint64_t ps = qs + k * kDownPiece;
    if (ps >= qe) continue;
    const uint64_t src = yp[par] + prm.qbase * L::bytes;
    const uint64_t dst = yp[i] + prm.qbase * L::bytes;
    typename L::T v[kQ];
#pragma unroll
    for (int u = 0; u < kQ; ++u) {
      const uint64_t q = ps + (uint64_t)u * 64 + lane;
      if (q < qe) v[u] = L::load(src + q * L::bytes, 0);
    }
#pragma unroll
    for (int u = 0; u < kQ; ++u) {
      const uint64_t q = ps + (uint64_t)u * 64 + lane;
      if (q < qe) L::store(dst + q * L::bytes, 0, v[u]);
    }
  }
}

// The ranks receiving a block in round r have depths [dlo, dhi]; their
// positions in the depth-ordered table are [*a0, *a0 + *n).
__host__ __device__ inline void active_ranks(const uint32_t* doff, int H,
                                             int b, int dshift, int r,
                                             uint32_t* a0, uint32_t* n) {
  const int dlo = max(1, r - dshift - (b - 1));
  const int dhi = min(H, r - dshift);
  if (dlo > dhi) {
    *a0 = 0;
    *n = 0;
    return;
  }
  *a0 = doff[dlo];
  *n = doff[dhi + 1] - doff[dlo];
}

// Work item `item` of round r: the first C items (r < b) are the up-step's
// chunks of block r; then, for each slice of dslice active ranks, npieces
// down-step pieces.
template <class U>
__device__ __forceinline__ void round_item(DPAR_KARGS,
                                           const uint32_t* __restrict__ dn,
                                           const uint32_t* __restrict__ ranks,
                                           int r, uint32_t act0, uint32_t nact,
                                           uint64_t item, char* lds) {
  const uint64_t nup = r < prm.b ? (uint64_t)prm.C : 0;
  if (item < nup) {
    U::run(xp, yp, ops, lvl, prm, (uint64_t)r * prm.C + item, lds);
    return;
  }
  const uint64_t d = item - nup;
  const uint32_t a0 = act0 + (uint32_t)(d / (uint64_t)prm.npieces) * prm.dslice;
  const uint32_t a1 = min(act0 + nact, a0 + (uint32_t)prm.dslice);
  down_copy<typename U::Lane, U::kThreads>(yp, dn, ranks, prm, r, a0, a1,
                                           d % (uint64_t)prm.npieces);
}

template <class U>
__global__ __launch_bounds__(U::kThreads) void k_rounds(
    DPAR_KARGS, const uint32_t* __restrict__ dn,
    const uint32_t* __restrict__ dord, int round, uint32_t act0,
    uint32_t nact, uint64_t first) {
  extern __shared__ char lds_raw[];
  round_item<U>(xp, yp, ops, lvl, prm, dn, dord + prm.dheight + 2, round,
                act0, nact, first + blockIdx.x, lds_raw);
}

template <class U>
__global__ __launch_bounds__(U::kThreads) void k_rounds_barrier(
    DPAR_KARGS, const uint32_t* __restrict__ dn,
    const uint32_t* __restrict__ dord) {
  extern __shared__ char lds_raw[];
  const int H = prm.dheight;
  for (int r = prm.r0; r < prm.r1; ++r) {
    uint32_t act0, nact;
    active_ranks(dord, H, prm.b, prm.dshift, r, &act0, &nact);
    const uint64_t items =
        (r < prm.b ? (uint64_t)prm.C : 0) +
        (uint64_t)((nact + prm.dslice - 1) / prm.dslice) * prm.npieces;
    for (uint64_t it = blockIdx.x; it < items; it += gridDim.x)
      round_item<U>(xp, yp, ops, lvl, prm, dn, dord + H + 2, r, act0, nact,
                    it, lds_raw);
    if (r + 1 < prm.r1) {
      // the next round reads blocks other workgroups (other XCDs, other L2s)
      // wrote in this one: every wavefront releases its stores at agent
      // scope before the barrier; the barrier acquires for the workgroup
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      grid_barrier(prm);
    }
  }
}

template <class U>
__global__ __launch_bounds__(U::kThreads) void k_ticket(DPAR_KARGS) {
  extern __shared__ char lds_raw[];
  __shared__ unsigned s_ticket;
  const uint64_t nunits = item_groups(prm) * prm.C;
  const uint64_t K = prm.batch;
  // Batch k (work items [k K, k K + K)) belongs to counter k % NC.  A
  // workgroup serves one counter: its first batch is its own index, later
  // ones come from that counter in increasing order, so every counter hands
  // out its batches in round order and the atomics are spread NC ways.
  const unsigned NC = min((unsigned)kTicketCounters, gridDim.x);
  const unsigned c = blockIdx.x % NC;
  const unsigned served = (gridDim.x - c + NC - 1) / NC;  // WGs on counter c
  unsigned* ctr = prm.ticket + (size_t)c * kCounterStride;
  uint64_t batch = blockIdx.x;
  // the next batch is claimed before the current one is processed, so the
  // atomic's round trip overlaps the work
  unsigned next = 0;
  if (threadIdx.x == 0 && batch * K < nunits) next = atomicAdd(ctr, 1u);
  for (;;) {
    const uint64_t first = batch * K;
    if (first >= nunits) break;
    const uint64_t last = min(first + K, nunits);
    for (uint64_t t = first; t < last; ++t)
      U::run(xp, yp, ops, lvl, prm, t, lds_raw);
    if (threadIdx.x == 0) s_ticket = next;
    __syncthreads();
    batch = ((uint64_t)served + s_ticket) * NC + c;
    __syncthreads();
    if (threadIdx.x == 0 && batch * K < nunits) next = atomicAdd(ctr, 1u);
  }
  // the last workgroup of each counter resets it for the next call
  if (threadIdx.x == 0) {
    unsigned* dn = prm.done + (size_t)c * kCounterStride;
    __threadfence();
    if (atomicAdd(dn, 1u) == served - 1) {
      atomicExch(ctr, 0u);
      atomicExch(dn, 0u);
    }
  }
}

// Broadcast pass of the split executor: y_0 -> y_1 .. y_{p-1}.  One
// workgroup per (output row, tile of 256 lanes), in the order of plan.hpp
// bcast_tile: y_0 in spans, every row of a span with its tiles on
// consecutive workgroups, then the next span.  Each thread loads one lane of
// y_0 and writes it with one streaming store.  The load is an L2 hit: every
// XCD reads the same eighth of a span for every row, and a span is sized so
// that this eighth stays in the XCD's L2 while the stores stream past it
// (taken as one span, a 32 MB y_0 fell out of L2 and the pass ran at half
// speed).  Many short workgroups with one store per thread write HBM faster
// on this part than long-running workgroups with many stores each (measured
// at p = 1152, m = 2^22 fp32: 7.1 vs 5.7 TB/s).  Works on bytes, whatever
// the element type.
template <class T, bool FAST>
__global__ __launch_bounds__(256) void k_bcast(const uint64_t* __restrict__ yp,
                                               BcastGrid g, uint64_t first) {
  uint64_t row, tile;
  bcast_tile<FAST>(g, first + blockIdx.x, &row, &tile);  // workgroup-uniform
  const uint64_t lane = tile * 256 + threadIdx.x;
  if (lane >= g.n) return;
  const uint64_t off = lane * sizeof(T);
  const T v = *reinterpret_cast<const DPAR_GLOBAL T*>(yp[0] + off);
  __builtin_nontemporal_store(v,
                              reinterpret_cast<DPAR_GLOBAL T*>(yp[row] + off));
}
// (T = u32x4g: 16-byte lanes on rows that all start on 128-byte lines;
// uint32_t: 4-byte lanes)

// The same pass with 16-byte lanes for output rows that do not all start on
// a 128-byte line.  The body of row i starts at the row's own first 4 KB
// boundary, h dwords in (plan.hpp bcast_row_split), so that every store
// fills 16 aligned bytes and every workgroup's tile is whole cache lines of
// one page; lane l of the body copies dwords [h + 4 l, h + 4 l + 4), reading
// them from y_0 at any 4-byte alignment (an L2 hit).  The row's tile-0
// workgroup also copies the h leading and the (up to 3) trailing dwords,
// one dword per thread.  At p = 1152, m = 2^22 with rows 4 bytes off a
// 16-byte boundary this pass takes 3.0 ms, against 3.7 ms with stores that
// straddle 16-byte boundaries, 3.3 ms with the body shifted to the next
// 16-byte boundary and 3.06 ms to the next 128-byte line (tiles straddling
// cache lines leave partial lines to two workgroups); on rows that start on
// 128-byte lines (the headline's, 16 MB apart) the plain pass is faster
// (2.6 against 3.1 ms), so the library picks this one only when some output
// row needs it.  Rows on 16-byte boundaries but off the 128-byte lines need
// it too: their plain tiles leave partial lines to two workgroups
// (p = 1152, m = 2^22, rows 16 bytes past a line: 3.50 ms plain, 3.01 ms
// with this pass).
template <bool FAST>
__global__ __launch_bounds__(256) void k_bcast16_rows(
    const uint64_t* __restrict__ yp, BcastGrid g, uint64_t first) {
  uint64_t row, tile;
  bcast_tile<FAST>(g, first + blockIdx.x, &row, &tile);  // workgroup-uniform
  const uint64_t src = yp[0], dst = yp[row];
  const uint64_t ndw = g.n * 4;                       // dwords per row
  uint64_t h, nbody;
  bcast_row_split(dst, ndw, &h, &nbody);
  const uint64_t lane = tile * 256 + threadIdx.x;
  if (lane < nbody) {
    const uint64_t off = (h + 4 * lane) * 4;
    const u32x4g v = *reinterpret_cast<const DPAR_GLOBAL u32x4g*>(src + off);
    __builtin_nontemporal_store((u32x4)v,
                                reinterpret_cast<DPAR_GLOBAL u32x4*>(dst + off));
  }
  if (tile == 0) {
    const DPAR_GLOBAL uint32_t* a =
        reinterpret_cast<const DPAR_GLOBAL uint32_t*>(src);
    DPAR_GLOBAL uint32_t* d = reinterpret_cast<DPAR_GLOBAL uint32_t*>(dst);
    for (uint64_t k = threadIdx.x; k < h; k += 256)    // leading dwords
      __builtin_nontemporal_store(a[k], d + k);
    const uint64_t k = h + 4 * nbody + threadIdx.x;    // trailing dwords
    if (threadIdx.x < 4 && k < ndw) __builtin_nontemporal_store(a[k], d + k);
  }
}

// One rank (p = 1): y_0 <- x_0.  Lane `first * 256 + t` of n copies one T
// (16 bytes, or 4) with a streaming store: the broadcast pass's shape with
// the source row in place of y_0.
template <class T>
__global__ __launch_bounds__(256) void k_copy(uint64_t src, uint64_t dst,
                                              uint64_t n, uint64_t first) {
  const uint64_t lane = (first + blockIdx.x) * 256 + threadIdx.x;
  if (lane >= n) return;
  const uint64_t off = lane * sizeof(T);
  // streaming load and store: every byte moves once (a copy of 19.3 GB
  // each way: 6.46 TB/s, with an ordinary load 6.32 TB/s)
  const T v = __builtin_nontemporal_load(
      reinterpret_cast<const DPAR_GLOBAL T*>(src + off));
  __builtin_nontemporal_store(v, reinterpret_cast<DPAR_GLOBAL T*>(dst + off));
}

// ------------------------------------------------------------ host launch

namespace {

// Workgroups per CU for (kernel, LDS bytes), cached: the query costs more than
// a launch.  Callers hold the library lock.
hipError_t occupancy(const void* kfn, int threads, size_t lds, int* out) {
  static std::map<std::pair<const void*, size_t>, int> cache;
  const auto key = std::make_pair(kfn, lds);
  auto it = cache.find(key);
  if (it != cache.end()) {
    *out = it->second;
    return hipSuccess;
  }
  hipError_t e =
      hipOccupancyMaxActiveBlocksPerMultiprocessor(out, kfn, threads, lds);
  if (e == hipSuccess) cache[key] = *out;
  return e;
}

// The persistent ticketed executor: per_cu workgroups per CU, no more than
// there are batches of work items.
template <class U>
hipError_t launch_ticket(const Tables& tab, const Params& prm,
                         hipStream_t stream, int num_cus, size_t lds,
                         int per_cu) {
  // no workgroup fits (dynamic plus static LDS beyond a CU's): never launch
  if (per_cu < 1) return hipErrorInvalidConfiguration;
  const uint64_t nunits = item_groups(prm) * prm.C;
  uint64_t grid = (uint64_t)per_cu * num_cus;
  const uint64_t batches = (nunits + prm.batch - 1) / prm.batch;
  if (grid > batches) grid = batches;
  hipLaunchKernelGGL((k_ticket<U>), dim3((unsigned)grid), dim3(U::kThreads),
                     lds, stream, tab.xp, tab.yp, tab.ops, tab.lvl, prm);
  return hipGetLastError();
}

template <class U>
hipError_t launch_u(Exec exec, const Tables& tab, const Params& prm,
                    hipStream_t stream, int num_cus, size_t lds_floor) {
  // a larger request than the work item needs only lowers the number of
  // workgroups resident per CU (see launch())
  const size_t lds = U::lds(prm) > lds_floor ? U::lds(prm) : lds_floor;
  const dim3 block(U::kThreads);
  const uint64_t nunits = item_groups(prm) * prm.C;
  // One workgroup per work item: a launch's total thread count must stay
  // below 2^32, so a grid of more than kMaxGrid workgroups goes out as
  // several launches, each given the index of its first item.
  const uint64_t kMaxGrid = (1ull << 31) / U::kThreads;
  if (exec == Exec::DISPATCH) {  // work item t = first + blockIdx.x
    for (uint64_t first = 0; first < nunits; first += kMaxGrid) {
      const uint64_t n = min(kMaxGrid, nunits - first);
      hipLaunchKernelGGL((k_round<U>), dim3((unsigned)n), block, lds, stream,
                         tab.xp, tab.yp, tab.ops, tab.lvl, prm, 0, first);
    }
    return hipGetLastError();
  }
  if (exec == Exec::LAUNCH_PER_ROUND) {
    for (int j = 0; j < prm.b; ++j)
      for (uint64_t first = 0; first < (uint64_t)prm.C; first += kMaxGrid) {
        const uint64_t n = min(kMaxGrid, (uint64_t)prm.C - first);
        hipLaunchKernelGGL((k_round<U>), dim3((unsigned)n), block, lds,
                           stream, tab.xp, tab.yp, tab.ops, tab.lvl, prm, j,
                           first);
      }
    return hipGetLastError();
  }
  // down-step items of the busiest round: every non-root rank active
  const int H = prm.dheight;
  const uint64_t ndown =
      tab.doff_host
          ? (uint64_t)((tab.doff_host[H + 1] + prm.dslice - 1) / prm.dslice) *
                (uint64_t)prm.npieces
          : 0;
  if (exec == Exec::ROUNDS) {
    for (int r = prm.r0; r < prm.r1; ++r) {
      uint32_t act0, nact;
      active_ranks(tab.doff_host, H, prm.b, prm.dshift, r, &act0, &nact);
      const uint64_t items =
          (r < prm.b ? (uint64_t)prm.C : 0) +
          (uint64_t)((nact + prm.dslice - 1) / prm.dslice) * prm.npieces;
      for (uint64_t first = 0; first < items; first += kMaxGrid) {
        const uint64_t n = min(kMaxGrid, items - first);
        hipLaunchKernelGGL((k_rounds<U>), dim3((unsigned)n), block, lds,
                           stream, tab.xp, tab.yp, tab.ops, tab.lvl, prm,
                           tab.dn, tab.dord, r, act0, nact, first);
      }
    }
    return hipGetLastError();
  }
  const void* kfn =
      exec == Exec::GRID_BARRIER     ? reinterpret_cast<const void*>(&k_barrier<U>)
      : exec == Exec::ROUNDS_BARRIER ? reinterpret_cast<const void*>(&k_rounds_barrier<U>)
                                     : reinterpret_cast<const void*>(&k_ticket<U>);
  int per_cu = 0;
  hipError_t e = occupancy(kfn, U::kThreads, lds, &per_cu);
  if (e != hipSuccess) return e;
  if (exec == Exec::GRID_BARRIER || exec == Exec::ROUNDS_BARRIER) {
    if (per_cu < 1) return hipErrorInvalidConfiguration;
    // every workgroup must be resident at once; leave one slot per CU free
    // rather than fill the machine to the last slot
    if (per_cu > 1) --per_cu;
    // the round-structured rounds are short: two workgroups per CU keep the
    // waiting (polling) workgroups few
    if (exec == Exec::ROUNDS_BARRIER && per_cu > 2) per_cu = 2;
    uint64_t grid = (uint64_t)per_cu * num_cus;
    // more than the largest round's work items would only wait
    const uint64_t most =
        exec == Exec::GRID_BARRIER ? (uint64_t)prm.C : (uint64_t)prm.C + ndown;
    if (grid > most) grid = most;
    const uint64_t* xp = tab.xp;
    const uint64_t* yp = tab.yp;
    const uint32_t* ops = tab.ops;
    const uint32_t* lvl = tab.lvl;
    const uint32_t* dn = tab.dn;
    const uint32_t* dord = tab.dord;
    Params p2 = prm;
    void* args[] = {&xp, &yp, &ops, &lvl, &p2, &dn, &dord};
    return hipLaunchCooperativeKernel(kfn, dim3((unsigned)grid), block, args,
                                      (unsigned)lds, stream);
  }
  return launch_ticket<U>(tab, prm, stream, num_cus, lds, per_cu);
}

// Wide work items: one launch of k_wide, one workgroup per item (split
// up-phase, one fused launch), or the persistent ticketed executor.
template <class L, bool FUSED, bool TAIL>
hipError_t launch_wide(Exec exec, const Tables& tab, const Params& prm,
                       hipStream_t stream, int num_cus) {
  using U = WideUnit<L, FUSED, TAIL>;
  const size_t lds = U::lds(prm);
  const uint64_t nunits = item_groups(prm) * prm.C;
  if (exec == Exec::DISPATCH) {
    const WideArgs a = wide_args(tab.xp, tab.yp, tab.ops, prm);
    const uint64_t kMaxGrid = (1ull << 31) / U::kThreads;
    for (uint64_t first = 0; first < nunits; first += kMaxGrid) {
      const uint64_t n = min(kMaxGrid, nunits - first);
      hipLaunchKernelGGL((k_wide<L, FUSED, TAIL>), dim3((unsigned)n),
                         dim3(U::kThreads), lds, stream, a, first);
    }
    return hipGetLastError();
  }
  if (exec != Exec::TICKET) return hipErrorInvalidValue;
  int per_cu = 0;
  const hipError_t e = occupancy(reinterpret_cast<const void*>(&k_ticket<U>),
                                 U::kThreads, lds, &per_cu);
  if (e != hipSuccess) return e;
  return launch_ticket<U>(tab, prm, stream, num_cus, lds, per_cu);
}

template <class L>
hipError_t launch_l(Unit unit, int waves, Exec exec, const Tables& tab,
                    const Params& prm, hipStream_t stream, int num_cus,
                    size_t lds_floor) {
  const bool fused = exec != Exec::TICKET_SPLIT && exec != Exec::SPLIT &&
                     exec != Exec::ROUNDS && exec != Exec::ROUNDS_BARRIER;
  const Exec ex = exec == Exec::TICKET_SPLIT ? Exec::TICKET
                  : exec == Exec::SPLIT      ? Exec::DISPATCH
                                             : exec;
#define DPAR_LAUNCH_U(...) \
  launch_u<__VA_ARGS__>(ex, tab, prm, stream, num_cus, lds_floor)
  if (unit == Unit::LEVEL)
    return fused ? DPAR_LAUNCH_U(LvUnit<L, true>)
                 : DPAR_LAUNCH_U(LvUnit<L, false>);
  if (unit == Unit::SUB) {
    if (prm.sub_deep)
      return fused ? DPAR_LAUNCH_U(SubUnit<L, true, kUDeep>)
                   : DPAR_LAUNCH_U(SubUnit<L, false, kUDeep>);
    return fused ? DPAR_LAUNCH_U(SubUnit<L, true>)
                 : DPAR_LAUNCH_U(SubUnit<L, false>);
  }
  if (unit == Unit::WIDE) {
    // 16-byte lanes and one-launch executors only (the host asks for
    // nothing else)
    if constexpr (L::bytes == 16) {
      const bool tail = (uint64_t)prm.wide_full < item_groups(prm) * prm.C;
      if (tail)
        return fused ? launch_wide<L, true, true>(ex, tab, prm, stream, num_cus)
                     : launch_wide<L, false, true>(ex, tab, prm, stream,
                                                   num_cus);
      return fused ? launch_wide<L, true, false>(ex, tab, prm, stream, num_cus)
                   : launch_wide<L, false, false>(ex, tab, prm, stream,
                                                  num_cus);
    } else
      return hipErrorInvalidValue;
  }
  if (waves == 2)
    return fused ? DPAR_LAUNCH_U(SeqUnit<L, 2, true>)
                 : DPAR_LAUNCH_U(SeqUnit<L, 2, false>);
  return fused ? DPAR_LAUNCH_U(SeqUnit<L, 1, true>)
               : DPAR_LAUNCH_U(SeqUnit<L, 1, false>);
#undef DPAR_LAUNCH_U
}

}  // namespace

hipError_t launch(Kind kind, Path path, Unit unit, int waves, Exec exec,
                  const Tables& tab, const Params& prm, hipStream_t stream,
                  int num_cus, size_t lds_floor) {
  const bool vec = path == Path::VEC16;
#define DPAR_LAUNCH_L(L) \
  launch_l<L>(unit, waves, exec, tab, prm, stream, num_cus, lds_floor)
  switch (kind) {
    case Kind::I32_SUM:
      return vec ? DPAR_LAUNCH_L(Lane4<I32Sum>) : DPAR_LAUNCH_L(Lane1<I32Sum>);
    case Kind::I32_MAX:
      return vec ? DPAR_LAUNCH_L(Lane4<I32Max>) : DPAR_LAUNCH_L(Lane1<I32Max>);
    case Kind::F32_SUM:
      return vec ? DPAR_LAUNCH_L(Lane4<F32Sum>) : DPAR_LAUNCH_L(Lane1<F32Sum>);
    case Kind::MAT:
      return DPAR_LAUNCH_L(LaneMat);  // 16-byte lanes on either path
  }
#undef DPAR_LAUNCH_L
  return hipErrorInvalidValue;
}

size_t level_lds_bytes(Path path, Kind kind, int p, int log2t, int nlev) {
  const size_t lane = (path == Path::VEC16 || kind == Kind::MAT) ? 16 : 4;
  const size_t T = (size_t)1 << log2t;
  const size_t s = 0;
  const size_t y = align16(s + (size_t)p * T * lane);
  const size_t ptr = align16(y + T * lane);
  const size_t lvl = align16(ptr + (size_t)p * 8);
  const size_t off = align16(lvl + (size_t)p * 4);
  return align16(off + (size_t)(nlev + 1) * 4);
}

template <bool FAST>
hipError_t broadcast_t(const Tables& tab, const BcastGrid& g, bool vec16,
                       bool rows_lines, hipStream_t stream) {
  // a launch's thread count stays below 2^32: pieces of at most 2^23
  // workgroups (a multiple of 8, so workgroup w stays on XCD w mod 8)
  const uint64_t kMaxGrid = (1ull << 31) / 256;
  for (uint64_t first = 0; first < g.total; first += kMaxGrid) {
    const unsigned n = (unsigned)min(kMaxGrid, g.total - first);
    if (vec16 && rows_lines)
      hipLaunchKernelGGL((k_bcast<u32x4g, FAST>), dim3(n), dim3(256), 0,
                         stream, tab.yp, g, first);
    else if (vec16)
      hipLaunchKernelGGL((k_bcast16_rows<FAST>), dim3(n), dim3(256), 0,
                         stream, tab.yp, g, first);
    else
      hipLaunchKernelGGL((k_bcast<uint32_t, FAST>), dim3(n), dim3(256), 0,
                         stream, tab.yp, g, first);
  }
  return hipGetLastError();
}

hipError_t broadcast(const Tables& tab, int p, uint64_t nbytes, bool vec16,
                     bool rows_lines, uint64_t span_bytes, bool fastdiv_tiles,
                     hipStream_t stream) {
  BcastGrid g = bcast_grid(nbytes, vec16 ? 16 : 4, p, span_bytes);
  g.fast = fastdiv_tiles && g.total <= 0xFFFFFFFFull;
  return g.fast ? broadcast_t<true>(tab, g, vec16, rows_lines, stream)
                : broadcast_t<false>(tab, g, vec16, rows_lines, stream);
}

size_t wide_lds_bytes(size_t lane_bytes, int nslots) {
  return (size_t)kWideWaves * nslots * kWideQ * 64 * lane_bytes;
}

size_t lds_bytes(Path path, Kind kind, int waves, int nslots) {
  const size_t lane = (path == Path::VEC16 || kind == Kind::MAT) ? 16 : 4;
  return (size_t)waves * nslots * 64 * lane;
}

hipError_t copy_row(uint64_t src, uint64_t dst, uint64_t bytes,
                    hipStream_t stream) {
  const uint64_t kMaxGrid = (1ull << 31) / 256;  // threads per launch < 2^32
  const uint64_t n16 = bytes / 16;
  for (uint64_t first = 0; first * 256 < n16; first += kMaxGrid) {
    const uint64_t wg = min(kMaxGrid, (n16 + 255) / 256 - first);
    hipLaunchKernelGGL((k_copy<u32x4g>), dim3((unsigned)wg), dim3(256), 0,
                       stream, src, dst, n16, first);
  }
  const uint64_t n4 = (bytes - n16 * 16) / 4;  // at most 3 dwords
  if (n4)
    hipLaunchKernelGGL((k_copy<uint32_t>), dim3(1), dim3(256), 0, stream,
                       src + n16 * 16, dst + n16 * 16, n4, (uint64_t)0);
  return hipGetLastError();
}

// ------------------------------------------------------------ fixed scratch

// Each GPU holds its own copy of this array until the process ends.  Host
// code never passes its name to a kernel: it asks the runtime for the
// device's address once (fixed_scratch_address) and uses that.
static __device__ __align__(256) unsigned char scratch[kFixedScratchBytes];

namespace {

// One launch carries this many payload bytes in its kernel arguments (the
// whole argument block stays below 4 KB).
constexpr int kStageWords = 480;

struct StagePacket {
  uint64_t* dst;
  uint32_t nwords;
  uint32_t unused;
  uint64_t w[kStageWords];
};

__global__ __launch_bounds__(256) void k_stage(StagePacket pk) {
  for (uint32_t i = threadIdx.x; i < pk.nwords; i += 256) pk.dst[i] = pk.w[i];
}

}  // namespace

hipError_t fixed_scratch_address(void** out) {
  return hipGetSymbolAddress(out, HIP_SYMBOL(scratch));
}

hipError_t stage_by_args(void* dst, const void* src, size_t nbytes,
                         hipStream_t stream) {
  const unsigned char* s = static_cast<const unsigned char*>(src);
  uint64_t* d = static_cast<uint64_t*>(dst);
  const size_t per = sizeof(uint64_t) * kStageWords;
  for (size_t off = 0; off < nbytes; off += per) {
    const size_t n = nbytes - off < per ? nbytes - off : per;
    StagePacket pk{};
    pk.dst = d + off / sizeof(uint64_t);
    pk.nwords = (uint32_t)((n + 7) / 8);
    memcpy(pk.w, s + off, n);  // the rest of the last word stays zero
    hipLaunchKernelGGL(k_stage, dim3(1), dim3(256), 0, stream, pk);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace dpar
