// Host-side plan: trees, opcodes, round counts, block rule, decomposition.
#include "plan.hpp"

#include <algorithm>
#include <cmath>
#include <utility>

namespace dpar {

namespace {

// One heap-shaped complete tree on n nodes (heap index h has children 2h and
// 2h+1), numbered in post-order starting at `first`.  Iterative walk: a node
// is numbered when it is popped the second time.
void add_heap_tree(Tree& t, int first, int n) {
  if (n <= 0) return;
  std::vector<int> rank_of(n + 1, -1);
  std::vector<std::pair<int, bool>> st;
  st.reserve(64);
  st.push_back({1, false});
  int next = first;
  while (!st.empty()) {
    auto [h, expanded] = st.back();
    st.pop_back();
    if (expanded) {
      rank_of[h] = next++;
      continue;
    }
    st.push_back({h, true});
    if (2 * h + 1 <= n) st.push_back({2 * h + 1, false});
    if (2 * h <= n) st.push_back({2 * h, false});
  }
  for (int h = 1; h <= n; ++h) {
    const int r = rank_of[h];
    const int left = 2 * h, right = 2 * h + 1;
    t.parent[r] = h > 1 ? rank_of[h / 2] : -1;
    if (right <= n) {            // two children: the right one is r - 1
      t.child0[r] = rank_of[right];
      t.child1[r] = rank_of[left];
    } else if (left <= n) {      // single child, also r - 1
      t.child0[r] = rank_of[left];
      t.child1[r] = -1;
    } else {
      t.child0[r] = t.child1[r] = -1;
    }
    int d = 0;
    for (int x = h; x > 1; x >>= 1) ++d;
    t.depth[r] = d;
    int leftmost = h;
    while (2 * leftmost <= n) leftmost *= 2;
    t.lo[r] = rank_of[leftmost];
  }
}

}  // namespace

Tree build_tree(int p) {
  Tree t;
  t.p = p;
  t.n_a = (p + 1) / 2;
  t.parent.assign(p, -1);
  t.child0.assign(p, -1);
  t.child1.assign(p, -1);
  t.depth.assign(p, 0);
  t.lo.assign(p, 0);
  t.dual.assign(p, -1);
  add_heap_tree(t, 0, t.n_a);
  add_heap_tree(t, t.n_a, p - t.n_a);
  t.root_a = t.n_a - 1;
  t.root_b = p > 1 ? p - 1 : -1;
  if (t.root_b >= 0) {
    t.dual[t.root_a] = t.root_b;
    t.dual[t.root_b] = t.root_a;
  }
  t.height = 0;
  for (int d : t.depth) t.height = std::max(t.height, d);
  return t;
}

Tree build_single_tree(int p) {
  Tree t;
  t.p = p;
  t.n_a = p;
  t.parent.assign(p, -1);
  t.child0.assign(p, -1);
  t.child1.assign(p, -1);
  t.depth.assign(p, 0);
  t.lo.assign(p, 0);
  t.dual.assign(p, -1);
  add_heap_tree(t, 0, p);
  t.root_a = p - 1;
  t.root_b = -1;
  t.height = 0;
  for (int d : t.depth) t.height = std::max(t.height, d);
  return t;
}

Tree kernel_single_tree(int p) {
  if (p <= 2) return build_tree(p);
  Tree t = build_single_tree(p);
  const int r = p - 1, c0 = t.child0[r], c1 = t.child1[r];
  t.n_a = t.lo[c0];              // part A = [0, lo(c0)), its root is c1
  t.root_a = c1;
  t.root_b = r;
  t.parent[c1] = -1;
  t.child1[r] = -1;              // the root keeps only its first child
  t.dual[c1] = r;
  t.dual[r] = c1;
  t.slot_shift = 1;
  return t;
}

bool make_sub(const Tree& t, const std::vector<uint32_t>& ops, int s,
              std::vector<uint32_t>* out) {
  if (t.root_a < 0 || t.root_b < 0) return false;
  std::vector<uint32_t> parts;                 // lo, hi, base
  std::vector<uint32_t> ranks[2], entries[2];  // per tree
  int ns = 1;
  for (int tr = 0; tr < 2; ++tr) {
    const int root = tr == 0 ? t.root_a : t.root_b;
    const int d0 = t.depth[root];
    // post-order over the top s levels: the second child's subtree (lower
    // ranks), the first child's, then the node
    std::vector<std::pair<int, bool>> st{{root, false}};
    while (!st.empty()) {
      auto [v, expanded] = st.back();
      st.pop_back();
      const uint32_t slot = ops[v] & OP_DEPTH_MASK;
      if (t.depth[v] - d0 == s) {              // a part: [lo(v), v]
        if ((int)(parts.size() / 3) >= kSubParts) return false;
        // the walk's slots are the relative depths 0 .. top - slot: a node
        // reads slot d + 1 only when it has a second child, so never below
        // the deepest level
        uint32_t top = slot;
        for (int i = t.lo[v]; i <= v; ++i)
          top = std::max<uint32_t>(top, ops[i] & OP_DEPTH_MASK);
        ns = std::max<int>(ns, (int)(top - slot) + 1);
        entries[tr].push_back(0x80000000u | (uint32_t)(parts.size() / 3));
        entries[tr].push_back(ops[v] & ~(uint32_t)(OP_C0 | OP_C1));
        parts.push_back((uint32_t)t.lo[v]);
        parts.push_back((uint32_t)v);
        parts.push_back(slot);
        continue;
      }
      if (expanded) {                          // a spine node
        if ((int)ranks[tr].size() >= kSubSpineRanks) return false;
        entries[tr].push_back((uint32_t)ranks[tr].size());
        entries[tr].push_back(ops[v]);
        ranks[tr].push_back((uint32_t)v);
        ns = std::max<int>(ns, (int)slot + 2);
        continue;
      }
      st.push_back({v, true});
      if (t.child0[v] >= 0) st.push_back({t.child0[v], false});
      if (t.child1[v] >= 0) st.push_back({t.child1[v], false});
    }
  }
  if (parts.empty()) return false;
  out->clear();
  out->push_back((uint32_t)(parts.size() / 3));
  out->push_back((uint32_t)(entries[0].size() / 2));
  out->push_back((uint32_t)(entries[1].size() / 2));
  out->push_back((uint32_t)ns);
  out->insert(out->end(), parts.begin(), parts.end());
  for (int tr = 0; tr < 2; ++tr) {
    std::vector<uint32_t> r = ranks[tr];
    const uint32_t pad = r.empty() ? (uint32_t)(tr == 0 ? t.root_a : t.root_b)
                                   : r[0];
    r.resize(kSubSpineRanks, pad);
    out->insert(out->end(), r.begin(), r.end());
  }
  out->insert(out->end(), entries[0].begin(), entries[0].end());
  out->insert(out->end(), entries[1].begin(), entries[1].end());
  return true;
}

std::vector<uint32_t> make_down(const Tree& t) {
  std::vector<uint32_t> dn(t.p, 0);
  for (int i = 0; i < t.p; ++i) {
    const uint32_t par = t.parent[i] < 0 ? 0xFFFFFFu : (uint32_t)t.parent[i];
    dn[i] = (par << 8) | ((uint32_t)t.depth[i] & 0xFFu);
  }
  return dn;
}

std::vector<uint32_t> make_depth_order(const Tree& t) {
  const int H = t.height;
  std::vector<uint32_t> out(H + 2, 0u);
  for (int d = 1; d <= H; ++d) {
    out[d] = (uint32_t)(out.size() - (H + 2));
    for (int i = 0; i < t.p; ++i)
      if (t.depth[i] == d) out.push_back((uint32_t)i);
  }
  out[H + 1] = (uint32_t)(out.size() - (H + 2));
  return out;
}

int device_rounds(const Tree& real, Alg alg, int b) {
  if (alg == Alg::REDUCE_BCAST)
    return real.height > 0 ? 2 * b + real.height - 1 : b;
  return b + real.height;
}

std::vector<uint32_t> make_ops(const Tree& t) {
  std::vector<uint32_t> ops(t.p, 0);
  for (int i = 0; i < t.p; ++i) {
    // the slot a waiting value uses; only SAVE and second-child reads use it
    const int slot = std::max(0, t.depth[i] - t.slot_shift);
    uint32_t op = (uint32_t)slot & OP_DEPTH_MASK;
    if (t.child0[i] >= 0) op |= OP_C0;
    if (t.child1[i] >= 0) op |= OP_C1;
    const int par = t.parent[i];
    // A second child's value waits for its sibling subtree; root A's value
    // waits for tree B.  Everything else is consumed by the next rank.
    if ((par >= 0 && t.child1[par] == i) || i == t.root_a) op |= OP_SAVE;
    ops[i] = op;
  }
  return ops;
}

std::vector<uint32_t> make_levels(const Tree& t) {
  std::vector<uint32_t> out;
  out.reserve((size_t)t.p + t.height + 2);
  std::vector<uint32_t> bounds;
  for (int d = t.height; d >= 0; --d) {
    bounds.push_back((uint32_t)out.size());
    for (int i = 0; i < t.p; ++i) {
      if (t.depth[i] != d) continue;
      uint32_t code = 0xFFFFu;
      if (t.child1[i] >= 0)
        code = (uint32_t)t.child1[i];
      else if (t.child0[i] >= 0)
        code = 0xFFFEu;
      out.push_back(((uint32_t)i << 16) | code);
    }
  }
  bounds.push_back((uint32_t)out.size());
  out.insert(out.end(), bounds.begin(), bounds.end());
  return out;
}

int rank_rounds(const Tree& t, int b, int rank) {
  if (t.p == 1) return 0;
  if (rank < 0) return b + t.height;
  const bool leaf = t.child0[rank] < 0;
  if (leaf && t.parent[rank] < 0) return b;
  return leaf ? b + t.depth[rank] : b + t.depth[rank] + 1;
}

long long block_rule(int p, size_t m, double alpha, double beta) {
  if (p < 1) return -1;
  if (m == 0) return 0;
  double b;
  if (alpha > 0.0 && beta > 0.0) {
    const double h = std::log2((double)p + 2.0);
    b = std::floor(std::sqrt((4.0 * h - 6.0) * beta * (double)m /
                             (3.0 * alpha)) + 0.5);
  } else {
    if (p == 1) return 1;
    b = std::ceil(std::sqrt((double)m * std::log2((double)p)));
  }
  if (!(b >= 1.0)) b = 1.0;
  if (b > (double)m) b = (double)m;
  if (b > 2147483647.0) b = 2147483647.0;
  return (long long)b;
}

Schedule make_schedule(uint64_t m, int b, int g, int lq) {
  Schedule s;
  s.b = b;
  s.g = g;
  s.lq = lq;
  s.Q = m / (uint64_t)g;
  s.tail = m - s.Q * (uint64_t)g;
  s.NL = (s.Q + (uint64_t)lq - 1) / (uint64_t)lq;
  const uint64_t max_lines = (s.NL + (uint64_t)b - 1) / (uint64_t)b;
  const uint64_t lines_per_chunk = 64 / (uint64_t)lq;
  s.C = (int)std::max<uint64_t>(1, (max_lines + lines_per_chunk - 1) /
                                       lines_per_chunk);
  return s;
}

void block_quanta(const Schedule& s, int j, uint64_t* qs, uint64_t* qe) {
  const unsigned __int128 NL = s.NL;
  const uint64_t ls = (uint64_t)(NL * (unsigned)j / (unsigned)s.b);
  const uint64_t le = (uint64_t)(NL * (unsigned)(j + 1) / (unsigned)s.b);
  *qs = std::min<uint64_t>(ls * (uint64_t)s.lq, s.Q);
  *qe = std::min<uint64_t>(le * (uint64_t)s.lq, s.Q);
}

int block_group(const Schedule& s) {
  const uint64_t L = 64 / (uint64_t)s.lq;  // lines per chunk
  const uint64_t maxl = (s.NL + (uint64_t)s.b - 1) / (uint64_t)s.b;
  if (s.NL == 0 || 2 * maxl > L) return 1;
  const uint64_t g = (uint64_t)s.b * L / s.NL;
  return (int)std::max<uint64_t>(1, std::min<uint64_t>(g, (uint64_t)s.b));
}

BcastGrid bcast_grid(uint64_t nbytes, uint64_t lane_bytes, int p,
                     uint64_t span_bytes) {
  BcastGrid g;
  if (p < 2 || lane_bytes == 0) return g;
  g.n = nbytes / lane_bytes;
  g.rows = (uint64_t)(p - 1);
  const uint64_t tiles = (g.n + 255) / 256;
  if (tiles == 0) return g;
  uint64_t tmax = span_bytes / (256 * lane_bytes);
  tmax = tmax < 8 ? 8 : tmax & ~(uint64_t)7;
  g.nspan = (tiles + tmax - 1) / tmax;
  g.ts = (tiles + g.nspan - 1) / g.nspan;
  // a span of 8k tiles gives every XCD the same tiles for every row; only
  // a y_0 small enough to sit whole in each XCD's L2 goes without padding
  if (g.nspan > 1 || nbytes > kBcastNoPadBytes)
    g.ts = (g.ts + 7) & ~(uint64_t)7;  // still <= tmax
  g.total = g.nspan * g.rows * g.ts;
  g.m_ts = fastdiv_magic(g.ts);
  g.m_span = fastdiv_magic(g.rows * g.ts);
  return g;
}

}  // namespace dpar
