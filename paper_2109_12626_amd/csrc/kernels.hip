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
//   * fused broadcast: y goes from registers to all p output buffers.
//
// Round sequencing: one launch per round, a persistent kernel with a grid
// barrier per round, or a persistent kernel that claims work items from an
// atomic ticket in round order.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.hpp"
#include "plan.hpp"

namespace dpar {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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
struct Lane4 {  // four scalars, one 16-byte access
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
    return ld(gptr<T>(row, off));
  }
  __device__ static void store(uint64_t row, uint32_t off, T v) {
    st(gptr_w<T>(row, off), v);
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

struct LaneMat16 {  // one matrix, 16-byte aligned
  using T = u32x4;
  static constexpr uint32_t bytes = 16;
  __device__ static T ap(T a, T b) { return mat_mul(a, b); }
  __device__ static T load(uint64_t row, uint32_t off) {
    return ld(gptr<T>(row, off));
  }
  __device__ static void store(uint64_t row, uint32_t off, T v) {
    st(gptr_w<T>(row, off), v);
  }
};

struct LaneMat4 {  // one matrix, only 4-byte aligned: four dword accesses
  using T = u32x4;
  static constexpr uint32_t bytes = 16;
  __device__ static T ap(T a, T b) { return mat_mul(a, b); }
  __device__ static T load(uint64_t row, uint32_t off) {
    const DPAR_GLOBAL uint32_t* q = gptr<uint32_t>(row, off);
    T v;
    v.x = q[0];
    v.y = q[1];
    v.z = q[2];
    v.w = q[3];
    return v;
  }
  __device__ static void store(uint64_t row, uint32_t off, T v) {
    DPAR_GLOBAL uint32_t* q = gptr_w<uint32_t>(row, off);
    q[0] = v.x;
    q[1] = v.y;
    q[2] = v.z;
    q[3] = v.w;
  }
};

// ------------------------------------------------------------ one work item

// Ranks whose loads are in flight per wavefront.  The host pads the pointer
// and opcode tables by kTablePad >= 2 * kU entries.
#ifndef DPAR_KU
#define DPAR_KU 8
#endif
constexpr int kU = DPAR_KU;
static_assert(2 * kU <= kTablePad, "tables are padded for 2 * kU reads");

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

  // chunk -> quanta [cs, ce): block j is a run of lines (Section 1.1's
  // partition into b blocks), cut into C chunks at line boundaries
  const uint64_t j = t / (uint64_t)prm.C, c = t % (uint64_t)prm.C;
  const uint64_t ls = prm.NL * j / (uint64_t)prm.b;
  const uint64_t le = prm.NL * (j + 1) / (uint64_t)prm.b;
  const uint64_t nl = le - ls;
  const uint64_t cls = ls + c * nl / (uint64_t)prm.C;
  const uint64_t cle = ls + (c + 1) * nl / (uint64_t)prm.C;
  const uint64_t cs = min(cls * prm.lq, prm.Q);
  const uint64_t ce = min(cle * prm.lq, prm.Q);
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
  auto step = [&](T v, uint32_t op) {
    const uint32_t d = op & OP_DEPTH_MASK;
    if (op & OP_C0) v = L::ap(cur, v);                 // first child
    if (op & OP_C1) v = L::ap(my[(d + 1) * 64], v);    // second child
    if (op & OP_SAVE)
      my[d * 64] = v;
    else
      cur = v;
  };

  // Up-phase over ranks [r0, r1): a rotating pipeline of kU loads.  Slot k
  // of `buf` holds rank base + k; it is consumed and at once refilled with
  // rank base + kU + k, so kU loads stay in flight.  The tables are padded
  // by kU entries, so reading kU entries ahead stays inside them; ranks past
  // r1 re-read row r1 - 1 (cache hits) and are not processed.
  const uint64_t last_row = xp[r1 - 1] + unit_off;
  T buf[kU];
#pragma unroll
  for (int k = 0; k < kU; ++k) {
    const uint64_t row = xp[r0 + k] + unit_off;
    buf[k] = L::load(r0 + k < r1 ? row : last_row, lane_off);
    // keep the loads in slot order: the wait before consuming slot k then
    // only needs the oldest load, in the prologue and in the loop alike
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int base = r0; base < r1; base += kU) {
    uint64_t next_row[kU];
    uint32_t op[kU];
#pragma unroll
    for (int k = 0; k < kU; ++k) {
      next_row[k] = xp[base + kU + k] + unit_off;
      op[k] = ops[base + k];
    }
#pragma unroll
    for (int k = 0; k < kU; ++k) {
      const T v = buf[k];
      buf[k] = L::load(base + kU + k < r1 ? next_row[k] : last_row, lane_off);
      __builtin_amdgcn_sched_barrier(0);
      if (base + k < r1) step(v, op[k]);
    }
  }

  // Dual-root exchange.
  T y;
  if (W == 1) {
    y = prm.dual ? L::ap(my[0], cur) : my[0];
  } else {
    if (wave == 1) my[0] = cur;  // tree B's root value
    __syncthreads();
    y = L::ap(slots[lane], slots[(size_t)prm.nslots * 64 + lane]);
  }

  // Fused broadcast of y to this wavefront's ranks, or y to y_0 only.
  if (!FUSED) {
    if (active && wave == 0) L::store(yp[0] + unit_off, lane_off, y);
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

// ------------------------------------------------------------ executors

template <class L, int W>
__global__ __launch_bounds__(64 * W) void k_round(
    const uint64_t* __restrict__ xp, const uint64_t* __restrict__ yp,
    const uint32_t* __restrict__ ops, Params prm, int round) {
  extern __shared__ char lds_raw[];
  typename L::T* slots = reinterpret_cast<typename L::T*>(lds_raw);
  run_unit<L, W, true>(xp, yp, ops, prm,
                       (uint64_t)round * prm.C + blockIdx.x, slots);
}

__device__ inline void grid_barrier(const Params& prm) {
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned g =
        __hip_atomic_load(prm.bar_gen, __ATOMIC_ACQUIRE,
                          __HIP_MEMORY_SCOPE_AGENT);
    const unsigned arrived = __hip_atomic_fetch_add(
        prm.bar_count, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    if (arrived == gridDim.x - 1) {
      __hip_atomic_store(prm.bar_count, 0u, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_fetch_add(prm.bar_gen, 1u, __ATOMIC_RELEASE,
                             __HIP_MEMORY_SCOPE_AGENT);
    } else if (__hip_atomic_load(prm.err, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT) == 0) {
      // (once a wait has given up, later barriers of the call do not wait)
      unsigned long long spins = 0;
      while (__hip_atomic_load(prm.bar_gen, __ATOMIC_ACQUIRE,
                               __HIP_MEMORY_SCOPE_AGENT) == g) {
        __builtin_amdgcn_s_sleep(2);
        if (++spins > prm.spin_limit) {  // watchdog: give up, report
          atomicOr(prm.err, 1u);
          break;
        }
      }
    }
  }
  __syncthreads();
}

template <class L, int W>
__global__ __launch_bounds__(64 * W) void k_barrier(
    const uint64_t* __restrict__ xp, const uint64_t* __restrict__ yp,
    const uint32_t* __restrict__ ops, Params prm) {
  extern __shared__ char lds_raw[];
  typename L::T* slots = reinterpret_cast<typename L::T*>(lds_raw);
  for (int j = 0; j < prm.b; ++j) {
    for (uint64_t c = blockIdx.x; c < (uint64_t)prm.C; c += gridDim.x)
      run_unit<L, W, true>(xp, yp, ops, prm, (uint64_t)j * prm.C + c, slots);
    if (j + 1 < prm.b) grid_barrier(prm);
  }
}

template <class L, int W, bool FUSED>
__global__ __launch_bounds__(64 * W) void k_ticket(
    const uint64_t* __restrict__ xp, const uint64_t* __restrict__ yp,
    const uint32_t* __restrict__ ops, Params prm) {
  extern __shared__ char lds_raw[];
  typename L::T* slots = reinterpret_cast<typename L::T*>(lds_raw);
  __shared__ unsigned s_ticket;
  const uint64_t nunits = (uint64_t)prm.b * prm.C;
  for (;;) {
    if (threadIdx.x == 0) s_ticket = atomicAdd(prm.ticket, 1u);
    __syncthreads();
    const unsigned t = s_ticket;
    __syncthreads();
    if (t >= nunits) break;
    run_unit<L, W, FUSED>(xp, yp, ops, prm, t, slots);
  }
  if (threadIdx.x == 0) {
    __threadfence();
    if (atomicAdd(prm.done, 1u) == gridDim.x - 1) {
      atomicExch(prm.ticket, 0u);
      atomicExch(prm.done, 0u);
    }
  }
}

// Broadcast pass of the split executor: y_0 -> y_1 .. y_{p-1}.  A workgroup
// owns a tile of QPT * 256 lanes of y_0 (QPT * 4 KB on the 16-byte path) and
// a group of consecutive ranks; it reads its tile once (a cache hit: the
// up-phase has just written it) and streams it into each of its ranks' rows,
// so every row receives QPT * 4 KB contiguous bytes per visit.  Works on
// bytes, whatever the element type.
#ifndef DPAR_BCAST_NT
#define DPAR_BCAST_NT 0
#endif
constexpr int kBcastRows = 8;

template <class T, int QPT>
__global__ __launch_bounds__(256) void k_bcast(const uint64_t* __restrict__ yp,
                                               int p, uint64_t n,
                                               int rows_per_group) {
  const uint64_t tile_lanes = 256ull * QPT;
  const uint64_t tiles = (n + tile_lanes - 1) / tile_lanes;
  const int groups = (p - 1 + rows_per_group - 1) / rows_per_group;
  const uint64_t items = tiles * (uint64_t)groups;
  for (uint64_t it = blockIdx.x; it < items; it += gridDim.x) {
    // consecutive workgroups take neighbouring tiles of the same row group
    const uint64_t tile = it % tiles;
    const int grp = (int)(it / tiles);
    const int i0 = 1 + grp * rows_per_group;
    const int i1 = min(p, i0 + rows_per_group);
    const uint64_t tile_off = tile * tile_lanes * sizeof(T);
    T v[QPT];
    bool ok[QPT];
#pragma unroll
    for (int k = 0; k < QPT; ++k) {
      const uint64_t lane = tile * tile_lanes + (uint64_t)k * 256 + threadIdx.x;
      ok[k] = lane < n;
      // lanes past the end re-read lane 0 of the tile (always in range)
      const uint32_t off =
          ok[k] ? ((uint32_t)k * 256 + threadIdx.x) * (uint32_t)sizeof(T) : 0u;
      v[k] = *gptr<T>(yp[0] + tile_off, off);
    }
    for (int i = i0; i < i1; i += kBcastRows) {
      uint64_t row[kBcastRows];
#pragma unroll
      for (int r = 0; r < kBcastRows; ++r) row[r] = yp[i + r] + tile_off;
#pragma unroll
      for (int r = 0; r < kBcastRows; ++r) {
        if (i + r < i1) {
#pragma unroll
          for (int k = 0; k < QPT; ++k) {
            const uint32_t off =
                ((uint32_t)k * 256 + threadIdx.x) * (uint32_t)sizeof(T);
            if (ok[k]) {
#if DPAR_BCAST_NT
              __builtin_nontemporal_store(v[k], gptr_w<T>(row[r], off));
#else
              *gptr_w<T>(row[r], off) = v[k];
#endif
            }
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------ host launch

namespace {

template <class L, int W>
hipError_t launch_t(Exec exec, const Tables& tab, const Params& prm,
                    hipStream_t stream, int num_cus) {
  const size_t lds = (size_t)W * prm.nslots * 64 * sizeof(typename L::T);
  const dim3 block(64 * W);
  const uint64_t nunits = (uint64_t)prm.b * prm.C;
  if (exec == Exec::LAUNCH_PER_ROUND) {
    for (int j = 0; j < prm.b; ++j) {
      hipLaunchKernelGGL((k_round<L, W>), dim3(prm.C), block, lds, stream,
                         tab.xp, tab.yp, tab.ops, prm, j);
    }
    return hipGetLastError();
  }
  if (exec == Exec::GRID_BARRIER) {
    int per_cu = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &per_cu, reinterpret_cast<const void*>(&k_barrier<L, W>), 64 * W, lds);
    if (e != hipSuccess) return e;
    if (per_cu < 1) return hipErrorInvalidConfiguration;
    uint64_t grid = (uint64_t)per_cu * num_cus;
    if (grid > (uint64_t)prm.C) grid = prm.C;  // more would only wait
    const uint64_t* xp = tab.xp;
    const uint64_t* yp = tab.yp;
    const uint32_t* ops = tab.ops;
    Params p2 = prm;
    void* args[] = {&xp, &yp, &ops, &p2};
    return hipLaunchCooperativeKernel(
        reinterpret_cast<const void*>(&k_barrier<L, W>), dim3((unsigned)grid),
        block, args, (unsigned)lds, stream);
  }
  const bool fused = exec == Exec::TICKET;
  const void* kfn = fused
      ? reinterpret_cast<const void*>(&k_ticket<L, W, true>)
      : reinterpret_cast<const void*>(&k_ticket<L, W, false>);
  int per_cu = 0;
  hipError_t e =
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kfn, 64 * W, lds);
  if (e != hipSuccess) return e;
  if (per_cu < 1) per_cu = 1;
  uint64_t grid = (uint64_t)per_cu * num_cus;
  if (grid > nunits) grid = nunits;
  if (fused)
    hipLaunchKernelGGL((k_ticket<L, W, true>), dim3((unsigned)grid), block,
                       lds, stream, tab.xp, tab.yp, tab.ops, prm);
  else
    hipLaunchKernelGGL((k_ticket<L, W, false>), dim3((unsigned)grid), block,
                       lds, stream, tab.xp, tab.yp, tab.ops, prm);
  return hipGetLastError();
}

template <class L>
hipError_t launch_w(int waves, Exec exec, const Tables& tab,
                    const Params& prm, hipStream_t stream, int num_cus) {
  return waves == 2 ? launch_t<L, 2>(exec, tab, prm, stream, num_cus)
                    : launch_t<L, 1>(exec, tab, prm, stream, num_cus);
}

}  // namespace

hipError_t launch(Kind kind, Path path, int waves, Exec exec,
                  const Tables& tab, const Params& prm, hipStream_t stream,
                  int num_cus) {
  const bool vec = path == Path::VEC16;
  switch (kind) {
    case Kind::I32_SUM:
      return vec ? launch_w<Lane4<I32Sum>>(waves, exec, tab, prm, stream, num_cus)
                 : launch_w<Lane1<I32Sum>>(waves, exec, tab, prm, stream, num_cus);
    case Kind::I32_MAX:
      return vec ? launch_w<Lane4<I32Max>>(waves, exec, tab, prm, stream, num_cus)
                 : launch_w<Lane1<I32Max>>(waves, exec, tab, prm, stream, num_cus);
    case Kind::F32_SUM:
      return vec ? launch_w<Lane4<F32Sum>>(waves, exec, tab, prm, stream, num_cus)
                 : launch_w<Lane1<F32Sum>>(waves, exec, tab, prm, stream, num_cus);
    case Kind::MAT:
      return vec ? launch_w<LaneMat16>(waves, exec, tab, prm, stream, num_cus)
                 : launch_w<LaneMat4>(waves, exec, tab, prm, stream, num_cus);
  }
  return hipErrorInvalidValue;
}

hipError_t broadcast(const Tables& tab, int p, uint64_t nbytes, bool vec16,
                     hipStream_t stream, int num_cus, int qpt, int rows) {
  if (p < 2 || nbytes == 0) return hipSuccess;
  const uint64_t lane = vec16 ? 16 : 4;
  const uint64_t n = nbytes / lane;
  if (qpt != 1 && qpt != 2 && qpt != 4 && qpt != 8 && qpt != 16) qpt = 8;
  if (rows < 1) rows = p - 1;
  const uint64_t tiles = (n + 256ull * qpt - 1) / (256ull * qpt);
  const uint64_t groups = (uint64_t)(p - 1 + rows - 1) / rows;
  uint64_t grid = tiles * groups;
  const uint64_t cap = (uint64_t)num_cus * 64;  // grid-stride beyond this
  if (grid > cap) grid = cap;
#define DPAR_BCAST_CASE(Q)                                                  \
  if (qpt == Q) {                                                           \
    if (vec16)                                                              \
      hipLaunchKernelGGL((k_bcast<u32x4, Q>), dim3((unsigned)grid),        \
                         dim3(256), 0, stream, tab.yp, p, n, rows);         \
    else                                                                    \
      hipLaunchKernelGGL((k_bcast<uint32_t, Q>), dim3((unsigned)grid),     \
                         dim3(256), 0, stream, tab.yp, p, n, rows);         \
  }
  DPAR_BCAST_CASE(1)
  DPAR_BCAST_CASE(2)
  DPAR_BCAST_CASE(4)
  DPAR_BCAST_CASE(8)
  DPAR_BCAST_CASE(16)
#undef DPAR_BCAST_CASE
  return hipGetLastError();
}

size_t lds_bytes(Path path, Kind kind, int waves, int nslots) {
  const size_t lane = (path == Path::VEC16 || kind == Kind::MAT) ? 16 : 4;
  return (size_t)waves * nslots * 64 * lane;
}

}  // namespace dpar
