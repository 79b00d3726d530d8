// Read- and write-pattern probes for measurement only; the reduction never
// calls them.  Each read kernel reads a region of device memory, XORs what it
// reads and stores nothing unless the XOR hits a fixed 64-bit pattern (it
// never does for the probe's inputs, but the compiler cannot drop the
// loads), so its duration is the time to read that pattern from HBM.  The
// write kernels copy one row into the others in several workgroup shapes.
// Built as libdpar_probe.so.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
#define DPAR_GLOBAL __attribute__((address_space(1)))

constexpr int kInFlight = 8;  // row visits in flight per wavefront

template <class T>
__device__ inline const DPAR_GLOBAL T* at(uint64_t addr) {
  return reinterpret_cast<const DPAR_GLOBAL T*>(addr);
}

__device__ inline void sink_if_magic(u32x4 acc, uint64_t sink) {
  if (acc.x == 0x9e3779b9u && acc.y == 0x7f4a7c15u)
    reinterpret_cast<DPAR_GLOBAL u32x4*>(sink)[threadIdx.x & 63] = acc;
}

// The up-phase's pattern: workgroup c reads chunk c (64 * QPL quanta of 16
// bytes, i.e. QPL KB) of every one of the p rows; wavefront w takes the rows
// [p w / W, p (w + 1) / W) in order with kInFlight visits in flight.
template <int QPL, int W>
__global__ __launch_bounds__(64 * W) void k_rows(uint64_t base,
                                                uint64_t stride, int p,
                                                uint64_t sink) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int r0 = (int)((int64_t)p * wave / W);
  const int r1 = (int)((int64_t)p * (wave + 1) / W);
  const uint64_t off = ((uint64_t)blockIdx.x * 64 * QPL + lane) * 16;
  auto row = [&](int r) {
    return at<u32x4>(base + (uint64_t)(r < r1 ? r : r1 - 1) * stride + off);
  };
  u32x4 acc = {0, 0, 0, 0};
  u32x4 buf[kInFlight][QPL];
#pragma unroll
  for (int k = 0; k < kInFlight; ++k) {
#pragma unroll
    for (int u = 0; u < QPL; ++u)
      buf[k][u] = __builtin_nontemporal_load(row(r0 + k) + 64 * u);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int rb = r0; rb < r1; rb += kInFlight) {
#pragma unroll
    for (int k = 0; k < kInFlight; ++k) {
#pragma unroll
      for (int u = 0; u < QPL; ++u) acc ^= buf[k][u];
#pragma unroll
      for (int u = 0; u < QPL; ++u)
        buf[k][u] =
            __builtin_nontemporal_load(row(rb + kInFlight + k) + 64 * u);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  sink_if_magic(acc, sink);
}

// Short workgroups over 16 KB tiles: workgroup g reads tile (g * mul) mod
// ntiles, 4 loads of 16 bytes per thread (mul = 1: address order).
__global__ __launch_bounds__(256) void k_tiles(uint64_t base, uint64_t ntiles,
                                              uint64_t mul, uint64_t sink) {
  const DPAR_GLOBAL u32x4* a = at<u32x4>(base);
  const uint64_t tile = ((uint64_t)blockIdx.x * mul) % ntiles;
  const uint64_t t = tile * 1024 + threadIdx.x;
  u32x4 v[4];
#pragma unroll
  for (int k = 0; k < 4; ++k)
    v[k] = __builtin_nontemporal_load(a + t + 256 * k);
  sink_if_magic(v[0] ^ v[1] ^ v[2] ^ v[3], sink);
}

// Broadcast shapes (probe.h dpar_probe_bcast).  TPB threads per workgroup,
// each storing S lanes of 16 bytes (lane t and t + TPB, ...) into R rows;
// workgroup w takes row 1 + R (w / ntiles) (and the next R - 1 rows) and tile
// w mod ntiles of TPB * S lanes; XCDSPLIT: the tile comes from the eighth of
// the row that belongs to XCD w mod 8.
template <int TPB, int S, int R, bool XCDSPLIT, bool NT>
__global__ __launch_bounds__(TPB) void k_bcast_shape(uint64_t base,
                                                     uint64_t row_bytes,
                                                     uint64_t ntiles,
                                                     uint64_t rows) {
  const uint64_t w = blockIdx.x;
  uint64_t rg, tile;
  if (XCDSPLIT) {
    const uint64_t k = w & 7, q = w >> 3, per = ntiles / 8;
    rg = q / per;
    tile = k * per + q % per;
  } else {
    rg = w / ntiles;
    tile = w % ntiles;
  }
  const uint64_t lane0 = tile * TPB * S + threadIdx.x;
  u32x4 v[S];
#pragma unroll
  for (int s = 0; s < S; ++s)
    v[s] = *at<u32x4>(base + (lane0 + (uint64_t)s * TPB) * 16);
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const uint64_t row = 1 + rg * R + r;
    if (row > rows) break;
#pragma unroll
    for (int s = 0; s < S; ++s) {
      DPAR_GLOBAL u32x4* d = reinterpret_cast<DPAR_GLOBAL u32x4*>(
          base + row * row_bytes + (lane0 + (uint64_t)s * TPB) * 16);
      if (NT)
        __builtin_nontemporal_store(v[s], d);
      else
        *d = v[s];
    }
  }
}

uint64_t gcd(uint64_t a, uint64_t b) {
  while (b) {
    const uint64_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

}  // namespace

extern "C" int dpar_probe_rows(const void* base, unsigned long long stride,
                               int p, unsigned long long row_bytes, int qpl,
                               int waves, void* sink, hipStream_t stream) {
  if (!base || !sink || p < waves || qpl < 1 || row_bytes > stride)
    return -1;
  const uint64_t chunk = 1024ull * (uint64_t)qpl;
  if (row_bytes == 0 || row_bytes % chunk) return -1;
  const uint64_t grid = row_bytes / chunk;
  if (grid * 64 * (uint64_t)waves >= (1ull << 31)) return -1;
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint64_t s = reinterpret_cast<uint64_t>(sink);
#define DPAR_PROBE(Q, W)                                                 \
  hipLaunchKernelGGL((k_rows<Q, W>), dim3((unsigned)grid), dim3(64 * W), \
                     0, stream, b, (uint64_t)stride, p, s)
  if (waves == 2 && qpl == 1) DPAR_PROBE(1, 2);
  else if (waves == 2 && qpl == 2) DPAR_PROBE(2, 2);
  else if (waves == 2 && qpl == 4) DPAR_PROBE(4, 2);
  else if (waves == 8 && qpl == 1) DPAR_PROBE(1, 8);
  else return -1;
#undef DPAR_PROBE
  return hipGetLastError() == hipSuccess ? 0 : -2;
}

extern "C" int dpar_probe_tiles(const void* base, unsigned long long nbytes,
                                unsigned long long mul, void* sink,
                                hipStream_t stream) {
  constexpr uint64_t kTile = 16384;
  if (!base || !sink || nbytes == 0 || nbytes % kTile) return -1;
  const uint64_t ntiles = nbytes / kTile;
  if (ntiles * 256 >= (1ull << 31) || mul == 0 || gcd(mul, ntiles) != 1)
    return -1;
  hipLaunchKernelGGL(k_tiles, dim3((unsigned)ntiles), dim3(256), 0, stream,
                     reinterpret_cast<uint64_t>(base), ntiles, (uint64_t)mul,
                     reinterpret_cast<uint64_t>(sink));
  return hipGetLastError() == hipSuccess ? 0 : -2;
}

extern "C" int dpar_probe_bcast(void* base, unsigned long long row_bytes,
                                int p, int variant, hipStream_t stream) {
  if (!base || p < 2 || row_bytes == 0 || row_bytes % 32768) return -1;
  const uint64_t rows = (uint64_t)(p - 1);
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint64_t rb = row_bytes;
#define DPAR_SHAPE(TPB, S, R, X, NT)                                        \
  do {                                                                      \
    const uint64_t nt = rb / (16ull * TPB * S);                             \
    const uint64_t grid = nt * ((rows + R - 1) / R);                        \
    if (grid * TPB >= (1ull << 32)) return -1;                              \
    hipLaunchKernelGGL((k_bcast_shape<TPB, S, R, X, NT>), dim3((unsigned)grid), \
                       dim3(TPB), 0, stream, b, rb, nt, rows);              \
  } while (0)
  switch (variant) {
    case 0: DPAR_SHAPE(256, 1, 1, false, true); break;
    case 1: DPAR_SHAPE(256, 1, 1, true, true); break;
    case 2: DPAR_SHAPE(256, 2, 1, false, true); break;
    case 3: DPAR_SHAPE(256, 1, 2, false, true); break;
    case 4: DPAR_SHAPE(128, 1, 1, false, true); break;
    case 5: DPAR_SHAPE(256, 1, 1, false, false); break;
    case 6: DPAR_SHAPE(512, 1, 1, false, true); break;
    default: return -1;
  }
#undef DPAR_SHAPE
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
