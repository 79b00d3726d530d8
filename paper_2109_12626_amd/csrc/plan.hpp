// Host-side plan: the two trees, the per-rank round program and the block
// decomposition (Traeff 2021, Sections 1.1 and 1.2).  Pure C++, no HIP.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

// Helpers that the HIP kernels call as well are compiled for both sides.
#if defined(__HIPCC__)
#define DPAR_HOST_DEVICE __host__ __device__
#else
#define DPAR_HOST_DEVICE
#endif

namespace dpar {

// Per-rank opcode consumed by the device round program.  One rank's step in
// a round (Algorithm 1): Y <- x_i; if it has a first child, Y <- t (.) Y with
// t = the first child's block; if it has a second child, again with the
// second child's block; then the block goes up (to the parent, or to the
// dual root).  On the device the value going up either stays in a register
// ("current") or waits in a per-depth LDS slot until its parent runs.
enum : uint32_t {
  OP_DEPTH_MASK = 0x3f,   // d_i
  OP_C0 = 1u << 6,        // has child0: v = current (.) v
  OP_C1 = 1u << 7,        // has child1: v = slot[d+1] (.) v
  OP_SAVE = 1u << 8,      // result waits in slot[d] (else it becomes current)
};

// Which trees carry the reduction (Sections 1.1, 1.2 and 2).
enum class Alg : int {
  DUAL_ROOT = 0,     // two trees, roots exchange (Algorithm 1)
  SINGLE_TREE = 1,   // one doubly-pipelined tree over all ranks
  REDUCE_BCAST = 2,  // one tree: pipelined reduce, then pipelined broadcast
};

struct Tree {
  int p = 0;
  int n_a = 0;            // tree A = [0, n_a), tree B = [n_a, p)
  int root_a = -1, root_b = -1;
  int height = 0;         // largest depth over both trees
  // slot of a rank's waiting value = depth - slot_shift (see make_ops)
  int slot_shift = 0;
  std::vector<int> parent, child0, child1, depth, lo, dual;
};

// Heap-shaped complete binary trees, post-order numbered (Section 1.1).
Tree build_tree(int p);

// One heap-shaped post-order tree over all p ranks, root p - 1 (the
// single-tree variants of Sections 1.2 and 2).
Tree build_single_tree(int p);

// The single tree in the two-part form the device round program runs: part
// A = the root's second-child subtree [0, lo(child0)), part B = the
// first-child subtree plus the root, which keeps only its first child.  Then
// y = S(A) (.) S(B) = S(child1) (.) (S(child0) (.) x_root), the single tree's
// value.  Depths stay the real ones (the root's level comes after its
// children's); slot_shift = 1 puts part A's root in slot 0.  For p <= 2 the
// single tree and the dual-root trees give the same product and the
// dual-root form is returned.
Tree kernel_single_tree(int p);

// Opcodes for ranks 0..p-1 (uint32 each).
std::vector<uint32_t> make_ops(const Tree& t);

// Plan of the subtree work item: every tree (the two trees, or the two parts
// of one tree) is cut at `s` levels below its root; each subtree rooted
// there is a "part" that one wavefront walks in post-order (a contiguous
// rank range), and one wavefront per tree then walks the spine (the nodes
// above the parts) with the parts' values, in the same post-order.  Layout
// (uint32):
//   [0] nparts  [1] spine entries of tree A  [2] of tree B  [3] NS = slots
//   per wavefront; then per part: lo, hi (its root), base (slot depth of its
//   root); then kSubSpineRanks spine ranks of tree A and of tree B (the ranks
//   whose own blocks the spine walk needs, padded with a valid rank); then
//   the spine entries of A and of B, two words each: code (0x80000000 |
//   part, or the index of the rank in the tree's spine ranks) and opcode (a
//   part's root opcode without its child bits: the part's value already
//   contains its children).
constexpr int kSubParts = 8;        // wavefronts per subtree work item
constexpr int kSubSpineRanks = 4;   // spine ranks per tree at most
bool make_sub(const Tree& t, const std::vector<uint32_t>& ops, int s,
              std::vector<uint32_t>* out);

// Per-rank down-phase entries for the round-structured executor:
// parent << 8 | depth, parent 0xFFFFFF for a root.  Needs p < 2^24, depth
// < 256.
std::vector<uint32_t> make_down(const Tree& t);

// Non-root ranks ordered by depth for the round-structured down-step: H + 2
// offsets (entry d = index of the first rank at depth d; entries 0 and 1 are
// 0), then the ranks of depth 1, depth 2, ... in ascending order.  The ranks
// that receive a block in one round have consecutive depths, so they are one
// index range of this table.
std::vector<uint32_t> make_depth_order(const Tree& t);

// Rounds of the round-structured device schedule (b + H, or 2b + H - 1 for
// REDUCE_BCAST with H > 0).
int device_rounds(const Tree& real, Alg alg, int b);

// Ranks in level order for level-synchronous evaluation: deepest level
// first, ranks ascending within a level; entry = rank << 16 | code with code
// 0xFFFF for a leaf, 0xFFFE for a rank whose only child is rank - 1, else the
// second child's rank (the first is rank - 1).  The p entries are followed by
// H + 2 level boundaries.  Needs p <= 65534.
std::vector<uint32_t> make_levels(const Tree& t);

// Rounds with a non-empty exchange for one rank (rank == -1: overall).
int rank_rounds(const Tree& t, int b, int rank);

// Block-count rule of Section 1.2 (see dpar_block_rule).
long long block_rule(int p, size_t m, double alpha, double beta);

// Block decomposition (Section 1.1: b successive blocks of roughly m/b
// elements).  A lane owns one "quantum" of g elements (16 bytes on the
// vector path); blocks are cut at "line" boundaries of lq quanta (128 bytes
// on the vector path) so that neighbouring blocks and chunks never share a
// cache line.  Block j = lines [floor(j NL / b), floor((j+1) NL / b)); the
// last line and the tail (elements after g*Q) belong to the last block.
struct Schedule {
  int b = 0;
  int g = 1;                // elements per quantum
  int lq = 1;               // quanta per line
  uint64_t Q = 0;           // whole quanta
  uint64_t NL = 0;          // lines = ceil(Q / lq)
  uint64_t tail = 0;        // elements after g*Q (vector path only)
  int C = 1;                // chunks per block (each <= 64 quanta)
  uint64_t units() const { return (uint64_t)b * (uint64_t)C; }
};

// The decomposition for (m, b) with g elements per quantum and lq quanta per
// line.  Needs 1 <= b <= ceil(m / g / lq) lines.
Schedule make_schedule(uint64_t m, int b, int g, int lq);

// Quanta [qs, qe) of block j.
void block_quanta(const Schedule& s, int j, uint64_t* qs, uint64_t* qe);

// Consecutive whole blocks per work item for executors that issue every
// round's work items from one launch: 1 when a block fills at least half a
// chunk (64 quanta), else the largest G <= b with G NL / b <= 64 / lq lines,
// so that any G consecutive blocks fit one chunk (s.C is then 1).
int block_group(const Schedule& s);

// Quanta [*qs, *qe) of work item t of a post-order or subtree run: item t
// belongs to group g = t / C, which holds the whole blocks [g grp,
// min(g grp + grp, b)), i.e. the lines [floor(g grp NL / b),
// floor(min(g grp + grp, b) NL / b)); the group's lines are cut into C
// chunks at line boundaries and item t is chunk t mod C, clipped at Q
// quanta.  Items in increasing t cover increasing, disjoint quantum ranges.
DPAR_HOST_DEVICE inline void item_quanta(uint64_t NL, uint64_t b, uint64_t C,
                                         uint64_t grp, uint64_t lq,
                                         uint64_t Q, uint64_t t,
                                         uint64_t* qs, uint64_t* qe) {
  const uint64_t g = t / C, c = t % C;
  const uint64_t j0 = g * grp;
  const uint64_t j1 = j0 + grp < b ? j0 + grp : b;
  const uint64_t ls = NL * j0 / b, le = NL * j1 / b;
  const uint64_t nl = le - ls;
  const uint64_t cls = ls + c * nl / C, cle = ls + (c + 1) * nl / C;
  *qs = cls * lq < Q ? cls * lq : Q;
  *qe = cle * lq < Q ? cle * lq : Q;
}

// Work item of workgroup w in a launch of n workgroups when each XCD takes a
// contiguous run of the items: workgroup w runs on XCD k = w mod 8, which
// takes items [k q + min(k, r), (k + 1) q + min(k + 1, r)) in order
// (n = 8 q + r).  A bijection of [0, n).  Used for the up-phase when some
// input row is off a 128-byte line: neighbouring work items then share
// the cache line at their common edge, and on one XCD that line is fetched
// from HBM once (p = 1152, m = 2^22: 3.19 -> 3.05 ms; on aligned rows,
// where no line is shared, it is 0.6% slower, so it is not used there).
DPAR_HOST_DEVICE inline uint64_t xcd_run_index(uint32_t w, uint32_t n) {
  const uint32_t k = w & 7u, j = w >> 3, q = n >> 3, r = n & 7u;
  return (uint64_t)k * q + (k < r ? k : r) + j;
}

// Grid of the split executor's broadcast pass (y_0 -> y_1 .. y_{p-1}): one
// workgroup per (output row, tile of 256 lanes).  The n lanes of y_0 are cut
// into nspan spans of ts tiles each (equal widths; the last span may end in
// tiles past y_0's end, which do nothing); every row of one span is written
// before the next span starts.  Apart from small y_0, ts is a multiple of 8,
// so that workgroup w, which runs on XCD w mod 8, always finds the same
// eighth of the span in its XCD's L2 (with 4095 tiles in a row instead of
// 4096 every XCD would cycle through all of a 16 MB y_0 and the pass would
// take half as long again).
struct BcastGrid {
  uint64_t n = 0;       // lanes of y_0
  uint64_t ts = 1;      // tiles per span
  uint64_t nspan = 0;   // spans
  uint64_t rows = 0;    // output rows p - 1
  uint64_t total = 0;   // workgroups nspan * rows * ts
  uint64_t m_ts = 0;    // fastdiv_magic(ts)
  uint64_t m_span = 0;  // fastdiv_magic(rows * ts)
  uint64_t fast = 0;    // 1: the pass runs bcast_tile<true> (needs
                        // total < 2^32; the host decides, see broadcast())
};

// Division of a 32-bit n by a fixed divisor d without a divide (Lemire,
// Kaser and Kurz, "Faster remainder by direct computation", 2019): with
// M = floor((2^64 - 1) / d) + 1, floor(n / d) is the high 64 bits of the
// 96-bit product M n, exactly, for every n < 2^32 and 1 < d < 2^32.  d = 1
// is kept apart (M would wrap to 0).
DPAR_HOST_DEVICE inline uint64_t fastdiv_magic(uint64_t d) {
  return d > 1 ? ~0ull / d + 1 : 0;
}
DPAR_HOST_DEVICE inline uint32_t fastdiv(uint32_t n, uint64_t M, uint64_t d) {
  if (d == 1) return n;
  // high 64 bits of M n from 32-bit halves, without overflow
  const uint64_t lo = (M & 0xFFFFFFFFull) * n;
  const uint64_t hi = (M >> 32) * n + (lo >> 32);
  return (uint32_t)(hi >> 32);
}

// Spans of at most max(span_bytes, 8 tiles) bytes, as few as that allows;
// ts is a multiple of 8 unless y_0 has at most kBcastNoPadBytes (then it
// stays whole in every XCD's L2 and is not padded).
constexpr uint64_t kBcastNoPadBytes = 2u << 20;
BcastGrid bcast_grid(uint64_t nbytes, uint64_t lane_bytes, int p,
                     uint64_t span_bytes);

// Output row (1 .. p-1) and tile of workgroup w < g.total: span
// w / (rows ts), in it row 1 + (w / ts) mod rows and tile w mod ts.
// FAST (grids of fewer than 2^32 workgroups, g.fast set): the divisions are
// multiplications (fastdiv).
template <bool FAST>
DPAR_HOST_DEVICE inline void bcast_tile(const BcastGrid& g, uint64_t w,
                                        uint64_t* row, uint64_t* tile) {
  const uint64_t per_span = g.rows * g.ts;
  if (FAST) {
    const uint32_t w32 = (uint32_t)w;
    const uint32_t span = fastdiv(w32, g.m_span, per_span);
    const uint32_t r = w32 - span * (uint32_t)per_span;
    const uint32_t q = fastdiv(r, g.m_ts, g.ts);
    *row = 1 + (uint64_t)q;
    *tile = (uint64_t)span * g.ts + (r - q * (uint32_t)g.ts);
    return;
  }
  const uint64_t span = w / per_span;
  const uint64_t r = w - span * per_span;
  *row = 1 + r / g.ts;
  *tile = span * g.ts + r % g.ts;
}

// Row split of the broadcast for output rows that do not all start on
// 16-byte boundaries: a row of ndw dwords (a multiple of 4: the pass copies
// whole 16-byte lanes of y_0) at byte address dst (4-byte aligned) is
// written as h leading dwords, up to the row's first 4 KB boundary, then
// nbody 16-byte quanta [h + 4 l, h + 4 l + 4) for l < nbody, which start on
// that boundary, so that every workgroup's 4 KB tile is whole cache lines
// of one page, and then the ndw - h - 4 nbody (at most 3) trailing dwords.
DPAR_HOST_DEVICE inline void bcast_row_split(uint64_t dst, uint64_t ndw,
                                             uint64_t* h, uint64_t* nbody) {
  const uint64_t lead = ((4096 - (dst & 4095)) & 4095) >> 2;
  *h = lead < ndw ? lead : ndw;
  *nbody = (ndw - *h) >> 2;
}

}  // namespace dpar
