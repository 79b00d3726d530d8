"""The two post-order numbered binary trees with dual roots (Section 1.1).

Oracle module: test infrastructure only.

The paper organises the p processors into two roughly equally large, rooted,
post-order numbered binary trees that are "as balanced and complete as
possible"; the two roots talk to each other as duals.  Readings taken where
the text leaves room (each listed in the design notes):

* Tree A holds ranks [0, ceil(p/2)), tree B holds [ceil(p/2), p); for odd p
  the lower tree gets the extra rank.
* "As balanced and complete as possible" is read as the heap-shaped complete
  binary tree: heap indices 1..n, the children of h are 2h and 2h+1, every
  level full except the last, which is filled from the left.  Numbering is
  post-order (left subtree, right subtree, node) starting at the tree's first
  rank, so the root is the tree's last rank.
* Section 1.1 names the first child of i as processor i-1 and the second
  child as i''.  With post-order numbering the right heap child is i-1, so
  child0 is the right heap child and child1 the left one; a node with a single
  (left) heap child has only child0, which is then i-1 as well.
* d_i is the depth (root 0): the correctness argument of Section 1.1 chooses
  d_i as the depth and needs children one level below their parent.

A second shape, ``wbal`` (recursive weight-balanced split, lower subtree gets
ceil((n-1)/2)), is provided for experiments only; its pins are the p=9
structure, one hand-derived fp32 value and the size invariants that fix it.

``layout="single"`` builds one heap-shaped post-order tree over all p ranks
instead (root p-1, no dual): the single-tree alternative discussed in
Section 1.2 and the tree of the reduce-then-broadcast comparison of Section 2.
"""

from dataclasses import dataclass, field
from typing import List, Optional


@dataclass
class Trees:
    """Per-rank tree tables; ``None`` means "no such processor"."""

    p: int
    parent: List[Optional[int]] = field(default_factory=list)
    child0: List[Optional[int]] = field(default_factory=list)
    child1: List[Optional[int]] = field(default_factory=list)
    depth: List[int] = field(default_factory=list)
    lo: List[int] = field(default_factory=list)      # first rank of subtree(i)
    dual: List[Optional[int]] = field(default_factory=list)
    roots: List[int] = field(default_factory=list)   # [root A] or [root A, root B]

    @property
    def height(self) -> int:
        """Largest depth over all trees."""
        return max(self.depth) if self.depth else 0

    def is_root(self, i: int) -> bool:
        return self.parent[i] is None


def heap_postorder_tree(n: int, first: int):
    """Heap-shaped complete tree on ``n`` nodes numbered in post-order from
    ``first``.  Returns (parent, child0, child1, depth, lo) as dicts keyed by
    rank, and the root rank."""
    rank_of = {}
    counter = [first]

    def visit(h):
        if h > n:
            return
        visit(2 * h)          # left subtree first (lower ranks)
        visit(2 * h + 1)      # then the right subtree
        rank_of[h] = counter[0]
        counter[0] += 1

    visit(1)
    parent, child0, child1, depth, lo = {}, {}, {}, {}, {}
    for h, r in rank_of.items():
        left, right = 2 * h, 2 * h + 1
        parent[r] = rank_of[h // 2] if h > 1 else None
        if right <= n:
            child0[r] = rank_of[right]
            child1[r] = rank_of[left]
        elif left <= n:
            child0[r] = rank_of[left]
            child1[r] = None
        else:
            child0[r] = None
            child1[r] = None
        depth[r] = h.bit_length() - 1
        leftmost = h
        while 2 * leftmost <= n:
            leftmost *= 2
        lo[r] = rank_of[leftmost]
    return parent, child0, child1, depth, lo, rank_of[1]


def wbal_postorder_tree(n: int, first: int):
    """Experiment only: recursive weight-balanced split, the lower (second
    child) subtree gets ceil((n-1)/2) nodes.  Same return shape as
    ``heap_postorder_tree``."""
    parent, child0, child1, depth, lo = {}, {}, {}, {}, {}

    def build(start, size, d):
        # ranks [start, start+size) form one subtree; its root is the last
        if size == 0:
            return None
        root = start + size - 1
        rest = size - 1
        n_low = (rest + 1) // 2
        n_high = rest - n_low
        low = build(start, n_low, d + 1)
        high = build(start + n_low, n_high, d + 1)
        if high is not None:
            child0[root], child1[root] = high, low
        elif low is not None:
            child0[root], child1[root] = low, None
        else:
            child0[root], child1[root] = None, None
        for c in (low, high):
            if c is not None:
                parent[c] = root
        depth[root] = d
        lo[root] = start
        return root

    root = build(first, n, 0)
    parent[root] = None
    return parent, child0, child1, depth, lo, root


def build_trees(p: int, shape: str = "heap", layout: str = "dual") -> Trees:
    """The trees for p >= 1 virtual ranks.

    ``layout="dual"``: the two trees with dual roots of Section 1.1.
    ``layout="single"``: one tree of the same shape over all p ranks, root
    p-1, no dual -- the one-tree variant that Section 1.2 compares against
    (one doubly-pipelined binary tree) and the tree of the pipelined
    reduce-then-broadcast of Section 2 (User-Allreduce1)."""
    if p < 1:
        raise ValueError("p must be >= 1")
    make = heap_postorder_tree if shape == "heap" else wbal_postorder_tree
    if shape not in ("heap", "wbal"):
        raise ValueError(shape)
    if layout not in ("dual", "single"):
        raise ValueError(layout)
    n_a = (p + 1) // 2 if layout == "dual" else p
    t = Trees(p=p)
    t.parent = [None] * p
    t.child0 = [None] * p
    t.child1 = [None] * p
    t.depth = [0] * p
    t.lo = [0] * p
    t.dual = [None] * p
    for first, n in ((0, n_a), (n_a, p - n_a)):
        if n == 0:
            continue
        par, c0, c1, dep, lo, root = make(n, first)
        for r in range(first, first + n):
            t.parent[r] = par[r]
            t.child0[r] = c0[r]
            t.child1[r] = c1[r]
            t.depth[r] = dep[r]
            t.lo[r] = lo[r]
        t.roots.append(root)
    if len(t.roots) == 2:
        a, b = t.roots
        t.dual[a], t.dual[b] = b, a
    return t
