// Read-pattern probes (libdpar_probe.so): measurement kernels that read HBM
// in the patterns the reduction's phases use, for comparison with them.  Not
// part of the reduction's interface.  Both calls enqueue one kernel on
// `stream` and return 0, -1 on invalid arguments (nothing launched) or -2 on
// a launch error.  `sink` is a device buffer of at least 1 KB that the
// kernels never write for inputs whose XOR is not the fixed pattern
// 0x9e3779b9, 0x7f4a7c15 in its first two words.
#pragma once

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

// Reads bytes [0, row_bytes) of p rows at base + r * stride (the buffer
// holds p * stride bytes; row_bytes <= stride, a multiple of qpl KB): one
// workgroup of `waves` wavefronts per qpl-KB chunk of the columns, each
// wavefront reading its share of the rows in order, 8 rows in flight.
// qpl in {1, 2, 4} with waves = 2, or qpl = 1 with waves = 8; p >= waves.
int dpar_probe_rows(const void* base, unsigned long long stride, int p,
                    unsigned long long row_bytes, int qpl, int waves,
                    void* sink, hipStream_t stream);

// Reads nbytes (a multiple of 16 KB) as 16 KB tiles, one 256-thread
// workgroup per tile, workgroup g taking tile (g * mul) mod ntiles; mul must
// be coprime to ntiles (mul = 1: address order).
int dpar_probe_tiles(const void* base, unsigned long long nbytes,
                     unsigned long long mul, void* sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif
