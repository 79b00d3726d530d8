/*
 * dpar.h -- doubly-pipelined, dual-root reduction-to-all on one MI355X.
 *
 * C ABI of libdpar.so.  p virtual ranks each hold a vector x_i of m elements
 * in device memory; one call computes y = x_0 (.) x_1 (.) ... (.) x_{p-1}
 * element-wise for an associative, not necessarily commutative operator (.)
 * and writes y into every rank's output buffer y_i (Traeff 2021, Section 1:
 * the reduction-to-all problem).  The operator applications follow exactly
 * the association of Algorithm 1 on two post-order numbered binary trees with
 * dual roots (Section 1.1), so floating-point results are bit-identical to a
 * serial evaluation in that order, for every block count, executor and run.
 *
 * Conventions for every function below:
 *   - Return 0 (DPAR_SUCCESS) or a negative dpar_status_t; no exception or
 *     signal crosses the ABI.  dpar_last_error() gives a text for the last
 *     failure on the calling thread's most recent call.
 *   - Device work is enqueued on the caller's stream and is asynchronous with
 *     respect to the host.
 *   - Nothing is written to any output on an argument error.
 * The header is C99 and C++; like every HIP host program built without
 * hipcc, a C or C++ consumer defines __HIP_PLATFORM_AMD__ for HIP's runtime
 * header (e.g. gcc -D__HIP_PLATFORM_AMD__ -I/opt/rocm/include ... -ldpar).
 */
#ifndef DPAR_H
#define DPAR_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DPAR_SUCCESS = 0,
    DPAR_ERR_INVALID_ARG = -1, /* null array or entry, p < 1, b < 0, b > m, bad rank */
    DPAR_ERR_UNSUPPORTED = -2, /* dtype/op pair, or a size beyond the index range */
    DPAR_ERR_ALIAS = -3,       /* outputs overlap, or partially overlap an input */
    DPAR_ERR_NOMEM = -4,       /* library scratch could not be allocated */
    DPAR_ERR_HIP = -5,         /* HIP runtime or launch error (text in dpar_last_error) */
    DPAR_ERR_TIMEOUT = -6      /* a grid-barrier wait gave up (see dpar_check_status) */
} dpar_status_t;

/* Element types.  A DPAR_U32_MAT2X2 element is a 2x2 matrix of uint32 stored
 * row-major as [a00, a01, a10, a11] (16 bytes). */
typedef enum {
    DPAR_INT32 = 0,
    DPAR_FLOAT32 = 1,
    DPAR_U32_MAT2X2 = 2
} dpar_dtype_t;

/* Operators (Section 1: associative, possibly non-commutative).  Valid
 * pairs: INT32 x {SUM, MAX}, FLOAT32 x {SUM}, U32_MAT2X2 x {MATMUL}.
 *   INT32 SUM   two's-complement addition wrapping modulo 2^32;
 *   INT32 MAX   signed maximum;
 *   FLOAT32 SUM IEEE binary32 addition, round to nearest even, subnormals kept;
 *   MATMUL      C = A.B with every entry mod 2^32 (A is the left operand). */
typedef enum {
    DPAR_SUM = 0,
    DPAR_MAX = 1,
    DPAR_MATMUL = 2
} dpar_op_t;

/* Which trees carry the reduction.  The association of every operator
 * application follows the chosen tree(s), so fp32 results differ between
 * DUAL_ROOT and the one-tree algorithms; SINGLE_TREE and REDUCE_BCAST give
 * identical results (the same tree) and differ only in their round structure
 * (visible with the ROUNDS executors).
 *   DUAL_ROOT     two post-order trees whose roots exchange (Section 1.1,
 *                 Algorithm 1): y = S(root A) (.) S(root B).
 *   SINGLE_TREE   one heap-shaped post-order tree over all p ranks, root
 *                 p - 1, doubly pipelined (the one-tree variant Section 1.2
 *                 compares with): y = S(p - 1).
 *   REDUCE_BCAST  the same tree, a pipelined reduction to the root followed
 *                 by a pipelined broadcast (Section 2's User-Allreduce1). */
typedef enum {
    DPAR_ALG_DUAL_ROOT = 0,
    DPAR_ALG_SINGLE_TREE = 1,
    DPAR_ALG_REDUCE_BCAST = 2
} dpar_alg_t;

/* How the b pipeline rounds are sequenced on the device (Algorithm 1's round
 * loop).  All give bit-identical results.  In the first three, each chunk's
 * y is written to all p outputs right after its up-phase, so reads of later
 * rounds and writes of earlier ones overlap (the paper's double pipelining):
 *   LAUNCH_PER_ROUND  one kernel launch per round j = 0 .. b-1;
 *   GRID_BARRIER      one persistent (co-resident) launch, a device-wide
 *                     barrier after each round;
 *   TICKET            one persistent launch; workgroups claim (round, chunk)
 *                     work items from atomic counters in increasing round
 *                     order, no barrier, several rounds in flight.
 *   SPLIT             the up-phase of every round runs first, one workgroup
 *                     per chunk handed out by the hardware in round order,
 *                     writing each chunk's y only to y_0; a second pass then
 *                     streams y_0 into the other p - 1 outputs.  HBM reads
 *                     and writes share one bus, so separating the two
 *                     directions avoids read/write turnarounds.
 *   AUTO              SPLIT; one launch of every work item in round order
 *                     with the fused write-out instead for calls moving at
 *                     most 40 MB (2 p m times the element size) unless they
 *                     run in level work items with p >= 1024, for calls
 *                     that run in level work items below that, for calls
 *                     that
 *                     run in post-order work items on rows of at most
 *                     3.5 MB (p <= 16), 2.5 MB (p <= 48), 1.5 MB (p <= 64),
 *                     1 MB (p <= 96) or 512 KB,
 *                     for calls that run in subtree work items (p >= 256
 *                     and at most two such items per CU, at least one per
 *                     four CUs; from p = 4096 on, calls of three or four
 *                     per CU run them split), and for calls that run in
 *                     wide work items
 *                     with p <= 36 and at most one such item (16 KB of
 *                     columns) per CU, with p <= 20 and at most two, or
 *                     with p <= 8.
 * The last two run the algorithm's whole round structure, down-phase
 * included (dpar_schedule_rounds gives the number of rounds R):
 *   ROUNDS            one launch per round r = 0 .. R-1.  Round r runs the
 *                     up-step of block r (r < b) for all ranks and writes
 *                     y[r] to the root(s) only; then every rank at depth
 *                     d >= 1 receives block r - d (DUAL_ROOT, SINGLE_TREE:
 *                     Section 1.1's "receive Y[j - d_i] from the parent") or
 *                     block r - d - b + 1 (REDUCE_BCAST: the broadcast after
 *                     the reduction), copied from its parent's output, which
 *                     received it in round r - 1.  Rank i's block j thus
 *                     becomes final in round j + d_i (REDUCE_BCAST: j for
 *                     the root, b + j + d_i - 1 otherwise).
 *   ROUNDS_BARRIER    the same rounds in one persistent (co-resident) launch
 *                     with a device-wide barrier between rounds.
 * These two read each rank's block from its parent's output, so their HBM
 * traffic is about 1.5 times the others'.
 * Every wait at a device-wide barrier is bounded (DPAR_SPIN_LIMIT polls).  A
 * wait that gives up ends the waiting of the rest of that call (its later
 * barriers pass at once), sets a device-wide report flag that
 * dpar_check_status returns as DPAR_ERR_TIMEOUT, and leaves the outputs of a
 * ROUNDS_BARRIER call undefined; a GRID_BARRIER call's outputs are still
 * complete, since its work items are independent and the barrier only
 * orders the rounds.  Each call of these two executors starts from barrier
 * words of its own, zeroed before its launch, so a wait that gave up never
 * affects another call.
 * GRID_BARRIER and ROUNDS_BARRIER need every workgroup of their grid resident
 * at once (a cooperative launch sized to that): do not run them while other
 * work occupies the GPU, e.g. on a concurrent stream.  The other executors
 * may run concurrently with anything, including other dpar calls. */
typedef enum {
    DPAR_EXEC_AUTO = 0,
    DPAR_EXEC_LAUNCH_PER_ROUND = 1,
    DPAR_EXEC_GRID_BARRIER = 2,
    DPAR_EXEC_TICKET = 3,
    DPAR_EXEC_SPLIT = 4,
    DPAR_EXEC_ROUNDS = 5,
    DPAR_EXEC_ROUNDS_BARRIER = 6
} dpar_exec_t;

/* Options of dpar_allreduce_opt.  round_begin / round_end select the rounds
 * [round_begin, round_end) of a ROUNDS or ROUNDS_BARRIER run (round_end = -1:
 * to the last round); successive calls that cover [0, R) in order, on the
 * same stream with the same arguments, give the same outputs as one call.
 * Other executors need round_begin = 0 and round_end = -1. */
typedef struct {
    dpar_alg_t alg;
    dpar_exec_t exec;
    int round_begin;
    int round_end;
} dpar_options_t;

/* One rank's place in the two trees (Section 1.1).  -1 means "none". */
typedef struct {
    int parent;
    int child0;     /* first child: rank-1 whenever the rank has a child */
    int child1;     /* second child (the i'' of Section 1.1) */
    int depth;      /* d_i: 0 at the roots */
    int subtree_lo; /* the rank's subtree is [subtree_lo, rank] */
    int dual;       /* the other root, for the two roots only */
} dpar_node_t;

/* Block decomposition chosen for a call (Section 1.1: b successive blocks of
 * roughly m/b elements).  A wavefront lane owns one quantum of `quantum`
 * elements: 4 (16 bytes) for INT32/FLOAT32 when every block holds at least
 * one quantum (m / 4 >= b), else 1; a matrix is one quantum.  Calls with
 * m mod 4 != 0 that move at most 24 MB (2 p m times the element size) also
 * take one element per lane: one launch instead of a second one for the
 * trailing elements.  Blocks are cut
 * at multiples of `granularity` elements (lines of 8 quanta, 128 bytes, when
 * m allows b such lines, else one quantum): with
 * L = ceil(nquanta * quantum / granularity) lines, block j holds lines
 *     [floor(j*L/b), floor((j+1)*L/b)),
 * clipped at nquanta quanta, and the last block also holds the tail_elems
 * elements that do not fill a quantum.  Inside a round a block is cut at
 * line boundaries into chunks_per_block chunks of at most 64 quanta, one
 * lane per quantum.  With granularity 1 this is the canonical partition
 * [floor(j*m/b), floor((j+1)*m/b)). */
typedef struct {
    int b;                  /* number of blocks / rounds */
    int granularity;        /* elements per line: 32, 8, 4 or 1 */
    int quantum;            /* elements per lane: 4 or 1 */
    size_t nquanta;         /* whole quanta */
    size_t tail_elems;      /* elements after the last whole quantum */
    int chunks_per_block;
    int height;             /* H: largest depth over both trees */
    int waves_per_chunk;    /* wavefronts that cooperate on one chunk */
} dpar_schedule_t;

/* Reduction-to-all (Section 1; Algorithm 1).
 *   x, y    HOST arrays of p DEVICE pointers; x[i] and y[i] each address
 *           m elements of dtype (m*16 bytes for DPAR_U32_MAT2X2).  Pointers
 *           must be aligned to 4 bytes.  Rows that start on 16-byte
 *           boundaries are read and written fastest (each 16-byte lane then
 *           stays within one cache line); other rows take the same path.
 *           The library copies both arrays before
 *           returning; the caller owns and may free them at once.  The
 *           buffers must stay valid, and x unmodified, until the stream work
 *           completes.  The copy goes to a device table once per distinct
 *           pair of arrays (the last 8 pairs are kept): a call whose arrays
 *           match a kept pair enqueues its kernels and nothing else.  A
 *           replaced pair's table is recycled only after the device has
 *           gone idle, and every 32 replacements the library waits for that
 *           (hipDeviceSynchronize) in the call that needs a table.
 *   p       number of virtual ranks, >= 1.
 *   m       elements per rank; m == 0 is a successful no-op.
 *   b       number of pipeline blocks, 1 <= b <= m; b == 0 chooses
 *           ceil(sqrt(m log2 p)) (dpar_block_rule with alpha = beta = 0).
 *   stream  HIP stream (0 = the null stream).
 * Aliasing: output buffers must not overlap each other.  An output buffer may
 * coincide exactly with an input buffer (in place, e.g. y[i] == x[i] like
 * the paper's Y array); any partial overlap between an output and an input
 * returns DPAR_ERR_ALIAS.  Inputs may overlap each other.
 * Result: for every i, y[i][k] = S(root A)[k] (.) S(root B)[k], with
 * S(r) = S(child1) (.) (S(child0) (.) x_r[k]) (Algorithm 1's two "t (.) Y"
 * steps and the dual-root step).  p == 1 copies x_0 to y_0. */
int dpar_allreduce(const void* const* x, void* const* y, int p, size_t m,
                   dpar_dtype_t dtype, dpar_op_t op, int b, hipStream_t stream);

/* dpar_allreduce for callers that cannot allocate memory (code that must not
 * call hipMalloc, e.g. tight serving loops or harnesses that forbid it): the
 * same computation, arguments, results and errors as dpar_allreduce, with
 * no device or pinned host allocation in the call.  The library's device
 * tables (opcodes, level table, subtree plan, the pointer tables) live in a
 * fixed 1 MiB device array per GPU, held until the process ends; they are
 * written by small copy kernels whose data travels in kernel arguments,
 * only when p or the pointer arrays differ from the previous call of this
 * entry point on the device.  Limits and caveats:
 *   - p <= 32768 (DPAR_ERR_UNSUPPORTED beyond);
 *   - every call on a GPU shares that GPU's array: calls of this entry
 *     point that overlap on one GPU (e.g. on two streams without
 *     synchronisation between them) race and give undefined results;
 *   - it cannot be recorded into a HIP graph (DPAR_ERR_UNSUPPORTED under
 *     stream capture);
 *   - the host-side planner still uses ordinary heap memory when p changes.
 * The other entry points are unaffected and may be mixed with it. */
int dpar_allreduce_noalloc(const void* const* x, void* const* y, int p,
                           size_t m, dpar_dtype_t dtype, dpar_op_t op, int b,
                           hipStream_t stream);

/* Same as dpar_allreduce with an explicit round executor. */
int dpar_allreduce_ex(const void* const* x, void* const* y, int p, size_t m,
                      dpar_dtype_t dtype, dpar_op_t op, int b,
                      dpar_exec_t exec, hipStream_t stream);

/* dpar_allreduce with an explicit algorithm, executor and round range.
 * opt == NULL means {DUAL_ROOT, AUTO, 0, -1}.  The ROUNDS executors process
 * m % 4 trailing elements like the rest (no separate tail pass); when m is
 * not a multiple of 4 they use one element per lane. */
int dpar_allreduce_opt(const void* const* x, void* const* y, int p, size_t m,
                       dpar_dtype_t dtype, dpar_op_t op, int b,
                       const dpar_options_t* opt, hipStream_t stream);

/* Graph capture.  A call may be recorded into a HIP graph (stream capture)
 * with every executor except GRID_BARRIER and ROUNDS_BARRIER (refused with
 * DPAR_ERR_UNSUPPORTED).  Under capture a call only enqueues kernels, so an
 * eager call with the same p, algorithm and pointer arrays must come first
 * (it builds the device tables and stages the pointers; otherwise
 * DPAR_ERR_UNSUPPORTED).  If that eager call ran on another stream and its
 * copy of the pointer table may not have run yet, the capturing call waits
 * for it on the host (synchronise first to avoid the wait; a capture mode
 * that forbids it makes the call fail with DPAR_ERR_HIP and leaves the
 * capture to the runtime).  The staged pointer table is then held for the
 * graph: it is never restaged, and dpar_finalize, which frees it, must wait
 * until no graph that captured a call is replayed again.  A replay computes
 * from the buffers' contents at replay time.  Replays of one graph, and a
 * replay and a TICKET call, must not run concurrently. */

/* Tree tables of the library's host-side tree builder (Section 1.1: two
 * post-order numbered, heap-shaped complete binary trees; tree A holds ranks
 * [0, ceil(p/2)), tree B the rest; roots ceil(p/2)-1 and p-1 are duals).
 * Fills *out for 0 <= rank < p.  No device work. */
int dpar_tree_info(int p, int rank, dpar_node_t* out);

/* The same for an algorithm's tree(s): DUAL_ROOT as dpar_tree_info; the
 * one-tree algorithms give one heap-shaped post-order tree over [0, p) with
 * root p - 1 and no dual.  No device work. */
int dpar_tree_info_alg(int p, dpar_alg_t alg, int rank, dpar_node_t* out);

/* Rounds R of the ROUNDS executors' schedule with b blocks: b + H for
 * DUAL_ROOT and SINGLE_TREE, 2b + H - 1 for REDUCE_BCAST (b when p == 1),
 * H = the largest depth of the algorithm's tree(s).  No device work. */
int dpar_schedule_rounds(int p, int b, dpar_alg_t alg);

/* Block-count rule (Section 1.2).  With alpha > 0 and beta > 0 it returns
 * clamp(round(sqrt((4h - 6) beta m / (3 alpha))), 1, m) with h = log2(p + 2)
 * (the pipelining optimum of (4h - 3 + 3(b - 1))(alpha + beta m / b));
 * otherwise clamp(ceil(sqrt(m log2 p)), 1, m).  Returns 0 for m == 0 and a
 * negative status for p < 1. */
int dpar_block_rule(int p, size_t m, double alpha, double beta);

/* Number of rounds in which a rank performs a non-empty exchange under
 * Algorithm 1 with b blocks, void exchanges skipped (Sections 1.1, 1.3):
 * b + d_i for a leaf, b + d_i + 1 for a non-leaf, b for a root without
 * children, 0 for p == 1.  rank == -1 gives the overall count b + H.
 * No device work. */
int dpar_rounds(int p, int b, int rank);

/* The decomposition dpar_allreduce would use for these arguments (with any
 * executor but ROUNDS / ROUNDS_BARRIER, which take one element per lane
 * whenever m is not a multiple of 4).  `aligned` is ignored: the decomposition
 * does not depend on the pointers' alignment.  b == 0 applies the rule.  No
 * device work. */
int dpar_schedule_info(int p, size_t m, dpar_dtype_t dtype, int b, int aligned,
                       dpar_schedule_t* out);

/* Element range [*start, *end) of block j of a schedule.  No device work. */
int dpar_block_bounds(const dpar_schedule_t* s, size_t m, int j, size_t* start,
                      size_t* end);

/* Waits for the stream, then reports a grid-barrier wait that gave up in an
 * earlier GRID_BARRIER or ROUNDS_BARRIER call on this device since the last
 * report (DPAR_ERR_TIMEOUT, returned once: the flag is cleared), or a pending
 * HIP error. */
int dpar_check_status(hipStream_t stream);

/* Profiling aid: records `ev` on the call's stream between the up-phase and
 * the broadcast pass of the calling thread's next reduction call, if that
 * call runs the SPLIT executor, so that each pass can be timed with HIP
 * events.  The next reduction call consumes the setting whatever it runs (a
 * call that does not run SPLIT, or fails, drops it without touching `ev`);
 * NULL clears it.  It never changes what a call computes.  No device work. */
int dpar_set_phase_event(hipEvent_t ev);

/* Text of the calling thread's last error ("" if none). */
const char* dpar_last_error(void);

/* Tuning and test knobs, read from the environment at every call; none of
 * them changes what a call computes:
 *   DPAR_UNIT=seq|level|sub|wide
 *                           force the post-order, level, subtree or wide
 *                           post-order work item (wide: 16-byte lanes and
 *                           the one-launch executors and p < 1024 only,
 *                           else post-order; by default it runs one-launch
 *                           calls with at least 3/4 of a 16 KB column chunk
 *                           per CU, 7/8 with p <= 16, unless the split
 *                           up-phase caps its
 *                           post-order items' residency)
 *   DPAR_WIDE_TAIL=0|1      wide work items: the columns past the last
 *                           whole round of one item per CU in tail items
 *                           (one quantum per lane, shorter chains) unless
 *                           they fill more than 7/8 of a round (default 1;
 *                           0: full items only)
 *   DPAR_WIDE_ROUND=n       wide work items per round for that cut
 *                           (default: the CU count; set, it applies to
 *                           every wide call, also the fused calls of at
 *                           most 20 ranks that otherwise take full items
 *                           only; tests)
 *   DPAR_LEVEL_LOG2T=k      level work items of 2^k quanta (at most what
 *                           fits in LDS)
 *   DPAR_SUB_DEEP=0|1       subtree work items with 8 or 16 loads in flight
 *                           per wavefront (default 16 from p = 1024 on when
 *                           the call has at most one item per CU)
 *   DPAR_WAVES=1|2          wavefronts per post-order work item (default
 *                           1 for p <= 48, else 2)
 *   DPAR_TICKET_BATCH=k     work items claimed per ticket (TICKET)
 *   DPAR_SPLIT_UP=ticket    SPLIT's up-phase on the ticketed persistent
 *                           kernel instead of one launch (comparison)
 *   DPAR_FUSE_BELOW_KB=n    AUTO's single-launch threshold (default 40960)
 *   DPAR_GROUP_BLOCKS=0     one-launch executors (SPLIT, TICKET, AUTO):
 *                           one work item per block even when blocks are
 *                           shorter than half a chunk (default 1: groups of
 *                           consecutive whole blocks)
 *   DPAR_SCALAR=1           one element per lane and the canonical
 *                           element partition for INT32/FLOAT32 (tests)
 *   DPAR_BCAST_SPAN_KB=n    SPLIT's broadcast pass: y_0 streamed out in
 *                           spans of at most n KB (at least 8 tiles of 256
 *                           lanes), each to every output row before the
 *                           next (default 16384)
 *   DPAR_SEQ_WG_PER_CU=n    SPLIT's post-order up-phase at p >= 256 with
 *                           at least 64 work items per CU: workgroups
 *                           resident per CU (default 4; 0 = as many as
 *                           fit); set, it applies to every SPLIT call with
 *                           post-order work items
 *   DPAR_XCD_RUNS=0|1       SPLIT's up-phase: each XCD takes a contiguous
 *                           run of work items (default 1 only when some
 *                           input row is off a 128-byte line)
 *   DPAR_BCAST_FASTDIV=0|1  SPLIT's broadcast pass: workgroups find their
 *                           row and tile by multiplication (1; default for
 *                           passes writing at most 2 GB) or by division (0)
 *   DPAR_SPIN_LIMIT=n       grid-barrier watchdog, in polls (default 2^26)
 *   DPAR_LOG=1              print each call's plan on stderr: p, m, dtype,
 *                           operator, algorithm, tree height H, b, lane
 *                           width, decomposition, executor, work-item kind,
 *                           work items */

/* Frees every library-owned device and pinned host buffer (device tables,
 * counters, staging).  The library re-creates them lazily on the next call.
 * The caller must make sure no enqueued call is still running. */
int dpar_finalize(void);

#ifdef __cplusplus
}
#endif

#endif /* DPAR_H */
