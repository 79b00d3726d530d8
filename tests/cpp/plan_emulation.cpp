// Symbolic replay of the device work items' evaluation order, driven by the
// same host tables the kernels receive (opcodes, level table, subtree plan).
// Test infrastructure: for each p read from stdin it prints, per tree layout,
// the product each work item would form, as a string over x0..x{p-1};
// tests/test_plan_emulation.py compares them with the oracle's trees.
#include <cstdio>
#include <iostream>
#include <string>
#include <vector>

#include "plan.hpp"

using namespace dpar;
using S = std::string;

static S ap(const S& a, const S& b) { return "(" + a + "*" + b + ")"; }
static S x(int i) { return "x" + std::to_string(i); }

// the post-order walk over ranks [r0, r1) with slots my[d - base]
static S walk(const std::vector<uint32_t>& ops, int r0, int r1,
              std::vector<S>& my, int base, S& cur) {
  S last;
  for (int i = r0; i < r1; ++i) {
    S v = x(i);
    const uint32_t op = ops[i];
    const int d = (int)(op & OP_DEPTH_MASK) - base;
    if (op & OP_C0) v = ap(cur, v);
    if (op & OP_C1) v = ap(my.at(d + 1), v);
    if (op & OP_SAVE) my.at(d) = v; else cur = v;
    last = v;
  }
  return last;
}

static S seq(const Tree& t, const std::vector<uint32_t>& ops, int waves) {
  const int ns = t.height + 1;
  if (waves == 1 || t.p < 2) {
    std::vector<S> my(ns);
    S cur;
    walk(ops, 0, t.p, my, 0, cur);
    return t.p >= 2 ? ap(my.at(0), cur) : my.at(0);
  }
  std::vector<S> a(ns), b(ns);
  S ca, cb;
  walk(ops, 0, t.n_a, a, 0, ca);
  walk(ops, t.n_a, t.p, b, 0, cb);
  return ap(a.at(0), cb);
}

static S level(const Tree& t) {
  const std::vector<uint32_t> lv = make_levels(t);
  std::vector<S> s(t.p);
  for (int i = 0; i < t.p; ++i) s[i] = x(i);
  const int nlev = t.height + 1;
  for (int l = 0; l < nlev; ++l) {
    for (uint32_t k = lv[t.p + l]; k < lv[t.p + l + 1]; ++k) {
      const uint32_t e = lv[k];
      const int node = (int)(e >> 16);
      const uint32_t code = e & 0xFFFFu;
      S v = s[node];
      if (code != 0xFFFFu) v = ap(s[node - 1], v);
      if (code < 0xFFFEu) v = ap(s[code], v);
      s[node] = v;
    }
  }
  return t.p >= 2 ? ap(s[t.n_a - 1], s[t.p - 1]) : s[t.n_a - 1];
}

static S sub(const Tree& t, const std::vector<uint32_t>& ops, bool* ok) {
  std::vector<uint32_t> plan;
  *ok = make_sub(t, ops, 2, &plan);
  if (!*ok) return "";
  const int nparts = plan[0], ns = plan[3];
  const uint32_t* parts = plan.data() + 4;
  const uint32_t* sranks = parts + 3 * nparts;
  const uint32_t* spine = sranks + 2 * kSubSpineRanks;
  std::vector<S> pval(nparts);
  for (int w = 0; w < nparts; ++w) {
    std::vector<S> my(ns);
    S cur;
    pval[w] = walk(ops, parts[3 * w], parts[3 * w + 1] + 1, my, parts[3 * w + 2],
                   cur);
  }
  S root[2];
  for (int tr = 0; tr < 2; ++tr) {
    const int n = tr == 0 ? plan[1] : plan[2];
    const uint32_t* e = spine + (tr == 0 ? 0 : 2 * plan[1]);
    std::vector<S> my(ns);
    S cur;
    for (int k = 0; k < n; ++k) {
      const uint32_t code = e[2 * k], op = e[2 * k + 1];
      S v = (code & 0x80000000u)
                ? pval.at(code & 0xFFFFu)
                : x((int)sranks[tr * kSubSpineRanks + code]);
      const int d = (int)(op & OP_DEPTH_MASK);
      if (op & OP_C0) v = ap(cur, v);
      if (op & OP_C1) v = ap(my.at(d + 1), v);
      if (op & OP_SAVE) my.at(d) = v; else cur = v;
    }
    root[tr] = tr == 0 ? my.at(0) : cur;
  }
  return ap(root[0], root[1]);
}

int main() {
  int p;
  while (std::cin >> p) {
    for (int single = 0; single < 2; ++single) {
      const Tree t = single ? kernel_single_tree(p) : build_tree(p);
      const std::vector<uint32_t> ops = make_ops(t);
      bool ok = false;
      const S s = p >= 64 ? sub(t, ops, &ok) : S();
      std::printf("%d %s seq2 %s\n", p, single ? "single" : "dual",
                  seq(t, ops, 2).c_str());
      std::printf("%d %s seq1 %s\n", p, single ? "single" : "dual",
                  seq(t, ops, 1).c_str());
      std::printf("%d %s level %s\n", p, single ? "single" : "dual",
                  level(t).c_str());
      if (ok)
        std::printf("%d %s sub %s\n", p, single ? "single" : "dual",
                    s.c_str());
    }
  }
  return 0;
}
