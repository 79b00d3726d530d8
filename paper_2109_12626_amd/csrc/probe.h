// Read- and write-pattern probes (libdpar_probe.so): measurement kernels
// that move HBM data in the patterns the reduction's phases use, or in
// alternatives to them, for comparison.  Not part of the reduction's
// interface.  Every call enqueues one kernel on `stream` and returns 0, -1 on
// invalid arguments (nothing launched) or -2 on a launch error.  The read
// probes take `sink`, a device buffer of at least 1 KB that the kernels never
// write for inputs whose XOR is not the fixed pattern 0x9e3779b9,
// 0x7f4a7c15 in its first two words.
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

// Broadcast shapes: copies row 0 of a [p][row_bytes] buffer at base into
// rows 1 .. p-1 (row_bytes a multiple of 32 KB, p >= 2), one workgroup per
// (row, tile), the tiles of a row on consecutive workgroups, with streaming
// stores unless stated:
//   0  256 threads, 4 KB tiles, one 16-byte store per thread (the library's
//      broadcast pass);
//   1  as 0, but workgroup w (XCD w mod 8) takes its tiles from its own
//      eighth of the row;
//   2  256 threads, 8 KB tiles, two stores per thread;
//   3  256 threads, 4 KB tiles, the same tile into two consecutive rows;
//   4  128 threads, 2 KB tiles;
//   5  as 0 with ordinary (non-streaming) stores;
//   6  512 threads, 8 KB tiles.
int dpar_probe_bcast(void* base, unsigned long long row_bytes, int p,
                     int variant, hipStream_t stream);

#ifdef __cplusplus
}
#endif
