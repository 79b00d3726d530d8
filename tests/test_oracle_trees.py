"""Pins for the oracle's tree builder (Section 1.1: two post-order numbered,
as balanced and complete as possible binary trees with dual roots; first
child i-1, second child i''; d_i is the depth).

The expected structures below are derived by hand from those definitions
(heap-shaped complete trees, post-order numbering, tree A = the lower
ceil(p/2) ranks); the invariants are the properties Section 1.1 states.
"""

import math

import pytest

from oracle import build_trees

N = None


def _table(t):
    return [(t.parent[i], t.child0[i], t.child1[i], t.depth[i], t.lo[i],
             t.dual[i]) for i in range(t.p)]


def test_p7_structure():
    # Tree A = ranks 0..3 (heap indices 4,2,3,1 in post-order), tree B =
    # ranks 4..6 (heap 2,3,1).  Root 3: right heap child = rank 2 = i-1 is
    # child0, left heap child rank 1 is child1; rank 1 has the single child 0.
    expected = [
        # parent child0 child1 depth lo dual
        (1, N, N, 2, 0, N),
        (3, 0, N, 1, 0, N),
        (3, N, N, 1, 2, N),
        (N, 2, 1, 0, 0, 6),
        (6, N, N, 1, 4, N),
        (6, N, N, 1, 5, N),
        (N, 5, 4, 0, 4, 3),
    ]
    t = build_trees(7)
    assert _table(t) == expected
    assert t.roots == [3, 6]
    assert t.height == 2


def test_p9_heap_structure():
    # Tree A = ranks 0..4: heap 4,5 -> ranks 0,1; heap 2 -> 2; heap 3 -> 3;
    # root heap 1 -> 4.  Tree B = ranks 5..8: heap 4 -> 5, 2 -> 6, 3 -> 7,
    # 1 -> 8; rank 6 has the single child 5.
    t = build_trees(9)
    assert (t.child0[4], t.child1[4]) == (3, 2)
    assert (t.child0[2], t.child1[2]) == (1, 0)
    assert t.child0[3] is None and t.depth[3] == 1
    assert t.depth[0] == t.depth[1] == 2
    assert (t.child0[8], t.child1[8]) == (7, 6)
    assert (t.child0[6], t.child1[6]) == (5, None)
    assert t.depth[5] == 2 and t.child0[7] is None and t.depth[7] == 1
    assert t.roots == [4, 8] and t.dual[4] == 8 and t.dual[8] == 4


def test_p9_wbal_structure_experiment_only():
    # The weight-balanced alternative: root 4 gets child0 3, child1 1;
    # 3 -> 2 and 1 -> 0 are single-child chains.
    t = build_trees(9, shape="wbal")
    assert (t.child0[4], t.child1[4]) == (3, 1)
    assert (t.child0[3], t.child1[3]) == (2, None)
    assert (t.child0[1], t.child1[1]) == (0, None)


def test_small_p():
    t1 = build_trees(1)
    assert t1.roots == [0] and t1.parent == [None] and t1.dual == [None]
    t2 = build_trees(2)
    assert t2.roots == [0, 1] and t2.dual == [1, 0] and t2.height == 0
    t3 = build_trees(3)
    assert t3.roots == [1, 2] and t3.child0[1] == 0 and t3.child0[2] is None


def _postorder_walk(t, r, out):
    # second child's subtree, first child's subtree, node
    if t.child1[r] is not None:
        _postorder_walk(t, t.child1[r], out)
    if t.child0[r] is not None:
        _postorder_walk(t, t.child0[r], out)
    out.append(r)


@pytest.mark.parametrize("p", list(range(1, 130)) + [255, 256, 511, 576,
                                                      1000, 1151, 1152, 2000])
def test_invariants(p):
    t = build_trees(p)
    n_a = (p + 1) // 2
    # sizes and roots: the last rank of each tree
    assert t.roots[0] == n_a - 1
    if p > 1:
        assert t.roots[1] == p - 1
    for tree_id, (first, n) in enumerate(((0, n_a), (n_a, p - n_a))):
        if n == 0:
            continue
        root = first + n - 1
        walk = []
        _postorder_walk(t, root, walk)
        # post-order numbering: visiting the tree in post-order yields the
        # tree's ranks in increasing order
        assert walk == list(range(first, first + n))
        # heap completeness: full levels, last one partly filled
        H = int(math.floor(math.log2(n)))
        per_level = [0] * (H + 1)
        for r in range(first, first + n):
            per_level[t.depth[r]] += 1
        assert all(per_level[d] == 2 ** d for d in range(H))
        assert 1 <= per_level[H] <= 2 ** H
        # the last level is filled from the left: leaves appear in post-order
        # from left to right, so every depth-H node precedes every leaf one
        # level up
        deep = [r for r in range(first, first + n) if t.depth[r] == H]
        upper_leaves = [r for r in range(first, first + n)
                        if t.depth[r] == H - 1 and t.child0[r] is None]
        if upper_leaves:
            assert max(deep) < min(upper_leaves)
    for i in range(p):
        c0, c1 = t.child0[i], t.child1[i]
        if c0 is not None:
            assert c0 == i - 1                                 # first child
            assert t.depth[c0] == t.depth[i] + 1
            assert t.parent[c0] == i
        if c1 is not None:
            assert c0 is not None
            assert t.depth[c1] == t.depth[i] + 1
            assert t.parent[c1] == i
            # contiguity: subtree(i) = [lo(c1)..c1] u [c1+1..i-1] u {i}
            assert t.lo[c0] == c1 + 1
            assert t.lo[i] == t.lo[c1]
        elif c0 is not None:
            assert t.lo[i] == t.lo[c0]
        else:
            assert t.lo[i] == i
        if t.parent[i] is not None:
            par = t.parent[i]
            assert t.lo[par] <= t.lo[i] <= i < par


@pytest.mark.parametrize("h", [2, 3, 4, 5, 6, 7])
def test_perfect_trees_for_p_2h_minus_2(h):
    # Section 1.2 assumes p = 2^h - 2: two perfect trees of height h - 2
    p = 2 ** h - 2
    t = build_trees(p)
    leaves = [i for i in range(p) if t.child0[i] is None]
    assert len(leaves) == 2 ** (h - 1)
    assert all(t.depth[i] == h - 2 for i in leaves)
    assert t.height == h - 2


def test_left_filled_last_level():
    # heap shape: at p = 1152 each tree has 576 nodes: 511 in full levels
    # 0..8 and 65 at depth 9, all inside the leftmost (lowest-rank) part
    t = build_trees(1152)
    deep = [i for i in range(576) if t.depth[i] == 9]
    assert len(deep) == 65
    assert t.height == 9
    # the depth-9 leaves are the first ones met in post-order
    first_shallow_leaf = min(i for i in range(576)
                             if t.child0[i] is None and t.depth[i] == 8)
    assert max(deep) < first_shallow_leaf
    # statistics: leaves, one-child and two-child nodes
    kinds = [(t.child0[i] is not None) + (t.child1[i] is not None)
             for i in range(1152)]
    assert kinds.count(0) == 576 and kinds.count(1) == 2 \
        and kinds.count(2) == 574


def _max_stack(t):
    """Largest number of partial values alive at once between the steps of
    a post-order stack machine (each step replaces its children's values by
    S(i)); tree A's root value stays alive while tree B is evaluated, until
    the dual step."""
    best = live = 0
    for r in t.roots:
        # iterative post-order over the tree of root r
        order, st = [], [(r, False)]
        while st:
            v, done = st.pop()
            if done:
                order.append(v)
                continue
            st.append((v, True))
            for c in (t.child0[v], t.child1[v]):
                if c is not None:
                    st.append((c, False))
        for v in order:
            nch = sum(c is not None for c in (t.child0[v], t.child1[v]))
            live += 1 - nch              # children's values -> S(v)
            best = max(best, live)
    return best


@pytest.mark.parametrize("p,leaves,one,two,H,stack", [
    (36, 18, 2, 16, 4, 5), (64, 32, 2, 30, 5, 6), (1152, 576, 2, 574, 9, 10)])
def test_tree_statistics(p, leaves, one, two, H, stack):
    t = build_trees(p)
    nch = [sum(c is not None for c in (t.child0[i], t.child1[i]))
           for i in range(p)]
    assert (nch.count(0), nch.count(1), nch.count(2)) == (leaves, one, two)
    assert t.height == H
    assert _max_stack(t) == stack


def test_depth2_subtree_sizes_of_576():
    """The four depth-2 subtrees of a 576-rank heap tree, in rank order: the
    last level is filled from the left, so the first one is the largest."""
    t = build_trees(1152)
    roots = sorted(i for i in range(576) if t.depth[i] == 2)
    assert [r - t.lo[r] + 1 for r in roots] == [192, 127, 127, 127]


def _subtree_size(t, i):
    return i - t.lo[i] + 1


@pytest.mark.parametrize("p", list(range(1, 258)) + [300, 511, 576, 1000,
                                                      1151, 1152, 1999, 2000])
@pytest.mark.parametrize("layout", ["dual", "single"])
def test_wbal_invariants(p, layout):
    """The weight-balanced shape (the alternative reading of "as balanced
    and complete as possible", kept for experiments), pinned by the
    properties that define it, which together fix the tree: every subtree is
    a contiguous post-order rank range [lo_i, i] ending at its root; of the
    s - 1 ranks below a root of an s-rank subtree, the lower ceil((s-1)/2)
    form the second child's subtree, the rest the first child's (i - 1); a
    two-rank subtree has one child; depth grows by one per level; the height
    of an n-rank tree is floor(log2 n)."""
    t = build_trees(p, shape="wbal", layout=layout)
    n_a = (p + 1) // 2 if layout == "dual" else p
    spans = [(0, n_a), (n_a, p - n_a)]
    for first, n in spans:
        if n == 0:
            continue
        root = first + n - 1
        assert t.parent[root] is None and t.depth[root] == 0
        assert t.lo[root] == first
        walk = []
        _postorder_walk(t, root, walk)
        assert walk == list(range(first, first + n))
        assert max(t.depth[first:first + n]) == int(math.floor(math.log2(n)))
    assert t.roots == [root for root in
                       [f + n - 1 for f, n in spans if n > 0]]
    for i in range(p):
        s = _subtree_size(t, i)
        c0, c1 = t.child0[i], t.child1[i]
        below = s - 1
        low, high = (below + 1) // 2, below // 2
        if below == 0:
            assert c0 is None and c1 is None
            continue
        assert c0 == i - 1 and t.parent[c0] == i
        assert t.depth[c0] == t.depth[i] + 1
        if high == 0:          # one rank below: a single (first) child
            assert c1 is None and _subtree_size(t, c0) == 1
            continue
        assert c1 is not None and t.parent[c1] == i
        assert t.depth[c1] == t.depth[i] + 1
        assert t.lo[i] == t.lo[c1]
        assert _subtree_size(t, c1) == low          # second child: lower part
        assert _subtree_size(t, c0) == high
        assert t.lo[c0] == c1 + 1


def test_wbal_p1152_differs_from_heap():
    """At p = 1152 the two readings give different trees (576 = 2^9 + 64:
    the heap's left-filled last level is unbalanced by weight)."""
    h = build_trees(1152)
    w = build_trees(1152, shape="wbal")
    assert h.child1[575] != w.child1[575]
    assert [_subtree_size(w, w.child1[575]), _subtree_size(w, 574)] == \
        [288, 287]
    assert [_subtree_size(h, h.child1[575]), _subtree_size(h, 574)] == \
        [320, 255]
