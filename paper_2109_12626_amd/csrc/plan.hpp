// Host-side plan: the two trees, the per-rank round program and the block
// decomposition (Traeff 2021, Sections 1.1 and 1.2).  Pure C++, no HIP.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

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

struct Tree {
  int p = 0;
  int n_a = 0;            // tree A = [0, n_a), tree B = [n_a, p)
  int root_a = -1, root_b = -1;
  int height = 0;         // largest depth over both trees
  std::vector<int> parent, child0, child1, depth, lo, dual;
};

// Heap-shaped complete binary trees, post-order numbered (Section 1.1).
Tree build_tree(int p);

// Opcodes for ranks 0..p-1 (uint32 each).
std::vector<uint32_t> make_ops(const Tree& t);

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

}  // namespace dpar
