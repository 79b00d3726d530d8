// Interface between the C ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

namespace dpar {

// Operator / lane-layout families compiled into the library.
enum class Kind : int { I32_SUM = 0, I32_MAX = 1, F32_SUM = 2, MAT = 3 };
// VEC16: 16-byte lanes (4 scalars or 1 matrix) on 16-byte aligned buffers.
// SCALAR: one 4-byte scalar (or one matrix read as 4 dwords) per lane.
enum class Path : int { VEC16 = 0, SCALAR = 1 };
// How one work item (a chunk of a block) is evaluated: a post-order walk per
// wavefront over 16-byte lanes (SEQ) or level by level with the whole chunk
// staged in LDS (LEVEL; short chunks, latency-bound cases).
// SUB: the trees cut into subtrees, one wavefront each, then the spines
// (few chunks, large p).  WIDE: the post-order walk with kWideQ quanta per
// lane and kWideWaves wavefronts on neighbouring columns (few ranks, long
// rows; 16-byte lanes).
enum class Unit : int { SEQ = 0, LEVEL = 1, SUB = 2, WIDE = 3 };
enum class Exec : int {
  LAUNCH_PER_ROUND = 1,
  GRID_BARRIER = 2,
  TICKET = 3,
  SPLIT = 4,         // up-phase of every chunk (DISPATCH order), y into y_0
                     // only, then the broadcast pass
  DISPATCH = 5,      // one launch, one workgroup per work item in round
                     // order (the hardware dispatcher hands them out)
  TICKET_SPLIT = 6,  // as SPLIT with a ticketed up-phase (experiments)
  ROUNDS = 7,        // the algorithm's full round structure, one launch per
                     // round: up-step of block r to the roots' outputs,
                     // down-step of every rank from its parent's output
  ROUNDS_BARRIER = 8,  // the same rounds in one persistent launch with a
                       // grid barrier (and agent-scope fences) per round
};

// Scalars every kernel needs.  The tables (device pointers to the x and y
// pointer arrays and the per-rank opcodes) are passed as separate restrict
// parameters so the compiler reads them through the scalar cache.
struct Params {
  int p;            // ranks
  int n_a;          // tree A = [0, n_a)
  int nslots;       // LDS slots per wavefront = H + 1
  int dual;         // 1 when there is a tree B (p >= 2)
  uint64_t Q;       // quanta split into blocks
  uint64_t NL;      // lines of lq quanta (the partition unit)
  uint32_t lq;      // quanta per line
  uint64_t qbase;   // first quantum index (the tail unit starts after Q)
  int b;            // blocks = rounds
  int C;            // chunks per block (per group of grp blocks)
  int grp;          // one-launch executors: consecutive whole blocks per
                    // work-item group (1: every block on its own; more when
                    // blocks are shorter than half a chunk)
  unsigned batch;   // TICKET: consecutive work items claimed per ticket
  int lv_log2t;     // LEVEL: log2 of the chunk capacity T in quanta
  int nlev;         // LEVEL: H + 1 depth levels
  unsigned* ticket;     // TICKET: kTicketCounters counters, kCounterStride
                        // words apart; each reset by the last WG it served
  unsigned* done;       // TICKET: per-counter count of WGs finished, same
                        // layout as `ticket`
  unsigned* bar_count;  // GRID_BARRIER, ROUNDS_BARRIER: arrivals
  unsigned* bar_gen;    // generation
  unsigned* bar_quit;   // nonzero once a wait of this call gave up (the
                        // host zeroes the three words before each call)
  unsigned* err;        // device-wide report: bit 0 set when any barrier
                        // wait gave up (cleared by the host's status check)
  unsigned long long spin_limit;
  int out0, out1;       // non-fused up-step: ranks whose outputs receive y
                        // (out1 < 0: none)
  int dshift;           // ROUNDS: depth-d rank receives block r - d - dshift
  int dslice;           // ROUNDS: ranks per down-step work item
  int npieces;          // ROUNDS: down-step pieces per block (kDownPiece
                        // quanta each)
  int dheight;          // ROUNDS: height of the real tree(s) (the kernel
                        // form of one tree with p <= 2 is lower)
  int r0, r1;           // ROUNDS: run rounds [r0, r1)
  int xcd_runs;         // k_round: each XCD takes a contiguous run of the
                        // launch's work items (else consecutive items go
                        // to consecutive XCDs)
  int sub_deep;         // SUB: the parts are walked with 16 loads in flight
                        // per wavefront instead of 8 (host-side choice of
                        // the kernel)
  uint32_t wide_full;   // WIDE: items [0, wide_full) take kWideChunk quanta
                        // each, later ones kWideTailChunk (the columns past
                        // the full items)
};

// Quanta per down-step piece: 64 lanes x 4 quanta per lane.
constexpr int kDownPiece = 256;

// Ticket counters per call (each on its own 128-byte line): work-item batch
// k belongs to counter k % kTicketCounters, which spreads the atomics.
constexpr int kTicketCounters = 16;
constexpr int kCounterStride = 32;  // uint32 words = 128 bytes

// Entries the host appends to the pointer and opcode tables so that the
// kernels may read a fixed number of entries past the last rank.
constexpr int kTablePad = 64;

struct Tables {
  const uint64_t* xp;   // [p] device addresses of x_i
  const uint64_t* yp;   // [p] device addresses of y_i
  const uint32_t* ops;  // [p] opcodes (plan.hpp)
  const uint32_t* lvl;  // LEVEL: [p] level-ordered entries, then H + 2
                        // offsets; SUB: the subtree plan (plan.hpp)
  const uint32_t* dn;   // [p] ROUNDS: parent << 8 | depth (plan.hpp)
  const uint32_t* dord;  // ROUNDS: H + 2 depth offsets, then the non-root
                         // ranks by depth (plan.hpp make_depth_order)
  const uint32_t* doff_host;  // the same offsets in host memory
};

// Enqueue one executor run over all b*C chunks of a schedule.
// `waves` is 1 or 2 (2 needs p >= 2).  `lds_floor`: bytes of LDS each
// workgroup requests at least (0: what the work item needs); a larger
// request caps the workgroups resident per CU.  Returns the first HIP error.
hipError_t launch(Kind kind, Path path, Unit unit, int waves, Exec exec,
                  const Tables& tab, const Params& prm, hipStream_t stream,
                  int num_cus, size_t lds_floor);

// LDS a work item's dynamic request must leave free for the kernels' own
// static LDS (the ticket executor's claim word): the host compares
// requests with the device limit minus this.  (A subtree plan needing
// exactly the 160 KB limit once went to the ticket kernel, whose claim word
// then did not fit; the launch ran with an invalid LDS allocation and
// faulted.)
constexpr size_t kStaticLdsReserve = 256;

// Bytes of dynamic LDS a LEVEL work item needs.
size_t level_lds_bytes(Path path, Kind kind, int p, int log2t, int nlev);

// WIDE work items: quanta per lane, wavefronts per workgroup (each on its
// own 64 kWideQ quanta of the chunk), rank visits in flight per wavefront.
#ifndef DPAR_WIDE_Q
#define DPAR_WIDE_Q 4
#endif
#ifndef DPAR_WIDE_WAVES
#define DPAR_WIDE_WAVES 4
#endif
#ifndef DPAR_WIDE_KF
#define DPAR_WIDE_KF 2
#endif
constexpr int kWideQ = DPAR_WIDE_Q;
constexpr int kWideWaves = DPAR_WIDE_WAVES;
constexpr int kWideKF = DPAR_WIDE_KF;
// Quanta of one WIDE work item.
constexpr uint64_t kWideChunk = 64ull * kWideQ * kWideWaves;
// Tail items of a WIDE call (the columns past its last whole round of
// full items): the same walk with kWideTailQ quanta per lane and
// kWideTailKF visits in flight per wavefront, kWideTailChunk quanta each.
#ifndef DPAR_WIDE_TAIL_Q
#define DPAR_WIDE_TAIL_Q 1
#endif
#ifndef DPAR_WIDE_TAIL_KF
#define DPAR_WIDE_TAIL_KF 8
#endif
constexpr int kWideTailQ = DPAR_WIDE_TAIL_Q;
constexpr int kWideTailKF = DPAR_WIDE_TAIL_KF;
constexpr uint64_t kWideTailChunk = 64ull * kWideTailQ * kWideWaves;

// Bytes of dynamic LDS a WIDE work item needs with `nslots` slots per
// wavefront (lane_bytes 16).
size_t wide_lds_bytes(size_t lane_bytes, int nslots);

// Bytes of dynamic LDS a SUB work item needs with `ns` slots per wavefront
// (lane_bytes: 16 on the vector path and for matrices, else 4).
size_t sub_lds_bytes(size_t lane_bytes, int ns);

// Broadcast pass of the split executor: copies bytes [0, nbytes) of y_0 into
// y_1 .. y_{p-1} (16-byte lanes when vec16, else 4-byte lanes), one
// workgroup per (row, 256-lane tile), y_0 taken in spans of at most
// span_bytes (every row of a span, then the next span).  rows_lines: every
// output row starts on a 128-byte line (else the 16-byte lanes of each row
// are shifted to its own 4 KB boundaries).  fastdiv_tiles: each
// workgroup finds its row and tile by multiplication instead of division
// (plan.hpp bcast_tile).
hipError_t broadcast(const Tables& tab, int p, uint64_t nbytes, bool vec16,
                     bool rows_lines, uint64_t span_bytes, bool fastdiv_tiles,
                     hipStream_t stream);

// Bytes of dynamic LDS a workgroup needs.
size_t lds_bytes(Path path, Kind kind, int waves, int nslots);

// The reduction of a single rank: bytes (a multiple of 4) from src to dst,
// both 4-byte aligned and not overlapping, one 16-byte lane per thread (the
// last up to 3 dwords one per thread), 256 threads per workgroup.
hipError_t copy_row(uint64_t src, uint64_t dst, uint64_t bytes,
                    hipStream_t stream);

// ------------------------------------------------------------ fixed scratch
// The allocation-free entry point keeps its device tables (opcodes, level
// table, subtree plan, pointer tables) in one statically sized device array
// per GPU, so that it never allocates.
constexpr size_t kFixedScratchBytes = 1u << 20;  // 1 MiB per device
constexpr int kFixedMaxRanks = 32768;            // p the layout admits

// Device address of this GPU's fixed scratch array (the current device).
// Call once per device with that device current; the address differs per
// device.
hipError_t fixed_scratch_address(void** out);

// Copies nbytes from host memory to device address dst (8-byte aligned)
// through kernel arguments of small copy launches on `stream`: nothing is
// allocated and the host buffer may be reused as soon as this returns.  At
// most 7 bytes past dst + nbytes are written (zeros), up to the next 8-byte
// boundary.
hipError_t stage_by_args(void* dst, const void* src, size_t nbytes,
                         hipStream_t stream);

}  // namespace dpar
