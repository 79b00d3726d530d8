"""Pins for the oracle's one-tree variants and its per-round records
(Section 1.1's correctness induction, Section 1.2's single-tree remark,
Section 2's reduce-then-broadcast comparison).  CPU only."""

import math
import os

import numpy as np
import pytest

from oracle import allreduce_ltr, allreduce_tree, build_trees, simulate
from oracle.reduce_bcast import simulate_reduce_bcast

SIZES = list(range(1, 131)) + [255, 256, 257, 511, 1000, 1152]
SIM_P = [1, 2, 3, 5, 6, 7, 14, 30, 36, 64, 100]
SIM_B = [1, 2, 4, 7]


def _subtree(t, i):
    out, stack = [], [i]
    while stack:
        v = stack.pop()
        out.append(v)
        stack.extend(c for c in (t.child0[v], t.child1[v]) if c is not None)
    return sorted(out)


@pytest.mark.parametrize("p", SIZES)
def test_single_tree_structure(p):
    t = build_trees(p, layout="single")
    assert t.roots == [p - 1]
    assert all(d is None for d in t.dual)
    H = p.bit_length() - 1                      # floor(log2 p)
    assert t.height == H
    per_depth = [0] * (H + 1)
    for i in range(p):
        per_depth[t.depth[i]] += 1
        for c in (t.child0[i], t.child1[i]):
            if c is not None:
                assert t.parent[c] == i and t.depth[c] == t.depth[i] + 1
        if t.child1[i] is not None:
            assert t.child0[i] is not None
        if t.child0[i] is not None:
            assert t.child0[i] == i - 1         # Section 1.1: first child i-1
        sub = _subtree(t, i)                    # post-order contiguity
        assert sub == list(range(t.lo[i], i + 1))
    # heap shape: every level full except the last
    assert per_depth[:H] == [2 ** d for d in range(H)]
    assert 0 < per_depth[H] <= 2 ** H


@pytest.mark.parametrize("p", range(1, 41))
def test_single_tree_exact_ops_equal_left_to_right(p):
    """Brute force with Python integers: for exactly associative operators
    every association gives the plain product of Section 1."""
    rng = np.random.default_rng(7000 + p)
    xi = rng.integers(-2 ** 31, 2 ** 31, size=(p, 5), dtype=np.int64)
    t = build_trees(p, layout="single")
    got = allreduce_tree(xi.astype(np.int32), "int32", "sum", trees=t)
    want = [sum(int(v) for v in xi[:, k]) % 2 ** 32 for k in range(5)]
    assert [int(v) % 2 ** 32 for v in got] == want
    mats = rng.integers(0, 2 ** 32, size=(p, 3, 4), dtype=np.uint64)
    gotm = allreduce_tree(mats.astype(np.uint32), "u32mat2x2", "matmul",
                          trees=t)
    for k in range(3):
        acc = [1, 0, 0, 1]
        for i in range(p):
            a, b_ = acc, [int(v) for v in mats[i, k]]
            acc = [(a[0] * b_[0] + a[1] * b_[2]) % 2 ** 32,
                   (a[0] * b_[1] + a[1] * b_[3]) % 2 ** 32,
                   (a[2] * b_[0] + a[3] * b_[2]) % 2 ** 32,
                   (a[2] * b_[1] + a[3] * b_[3]) % 2 ** 32]
        assert [int(v) for v in gotm[k]] == acc


GOLDEN = os.path.join(os.path.dirname(__file__), "golden",
                      "fp32_single_tree_examples.txt")


def _examples():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, xs, single, dual, ltr = (c.strip() for c in line.split("|"))
            rows.append((name, [float(v) for v in xs.split()], float(single),
                         float(dual), float(ltr)))
    return rows


@pytest.mark.parametrize("name,xs,single,dual,ltr", _examples())
def test_single_tree_fp32_worked_examples(name, xs, single, dual, ltr):
    x = np.array(xs, dtype=np.float32).reshape(len(xs), 1)
    p = len(xs)
    assert allreduce_tree(x, "float32", "sum",
                          trees=build_trees(p, layout="single"))[0] == single
    assert allreduce_tree(x, "float32", "sum")[0] == dual
    assert allreduce_ltr(x, "float32", "sum")[0] == ltr
    # both one-tree schedules deliver the same value to every rank
    rows, _ = simulate(x, "float32", "sum", 1,
                       trees=build_trees(p, layout="single"))
    assert all(r[0] == single for r in rows)
    rows, _ = simulate_reduce_bcast(x, "float32", "sum", 1)
    assert all(r[0] == single for r in rows)


def _fp32_input(p, m, seed):
    rng = np.random.default_rng(seed)
    # wide exponent range so that the association shows in the low bits
    return (rng.standard_normal((p, m)) *
            np.exp2(rng.integers(-8, 9, size=(p, m)))).astype(np.float32)


@pytest.mark.parametrize("p", SIM_P)
@pytest.mark.parametrize("b", SIM_B)
def test_algorithm1_final_rounds_dual_root(p, b):
    """Section 1.1's induction: before round j a depth-d rank holds y blocks
    up to j-1-d, and in round j it receives block j-d; the roots finish
    block j in round j."""
    m = 13
    x = _fp32_input(p, m, 100 * p + b)
    rows, tr = simulate(x, "float32", "sum", b)
    t = build_trees(p)
    y = allreduce_tree(x, "float32", "sum")
    for i in range(p):
        assert np.array_equal(rows[i], y)
        assert tr.final_round[i] == {j: j + t.depth[i] for j in range(b)}


@pytest.mark.parametrize("p", SIM_P)
@pytest.mark.parametrize("b", SIM_B)
def test_algorithm1_on_one_tree(p, b):
    """Algorithm 1 run on the single tree (no dual exchange): same value as
    the single-tree evaluation on every rank, bit for bit; same round
    structure; b + H rounds."""
    m = 13
    x = _fp32_input(p, m, 200 * p + b)
    t = build_trees(p, layout="single")
    rows, tr = simulate(x, "float32", "sum", b, trees=t)
    y = allreduce_tree(x, "float32", "sum", trees=t)
    for i in range(p):
        assert np.array_equal(rows[i], y)
        assert tr.final_round[i] == {j: j + t.depth[i] for j in range(b)}
    if p > 1:
        assert tr.global_rounds() == b + t.height


@pytest.mark.parametrize("p", [7, 14, 30, 36, 64])
def test_operator_applications_per_round(p):
    """Section 1.2: with one tree every rank, the root included, applies the
    operator at most twice per round; with dual roots each root with two
    children applies it three times in a full round."""
    b = 6
    x = np.ones((p, 12), dtype=np.int32)
    _, tr1 = simulate(x, "int32", "sum", b,
                      trees=build_trees(p, layout="single"))
    assert max(max(v.values()) for v in tr1.ops_per_round.values()) == 2
    t2 = build_trees(p)
    _, tr2 = simulate(x, "int32", "sum", b, trees=t2)
    for r in t2.roots:
        if t2.child1[r] is not None:
            assert max(tr2.ops_per_round[r].values()) == 3
    for i in range(p):
        if i not in t2.roots:
            assert max(tr2.ops_per_round[i].values(), default=0) <= 2


@pytest.mark.parametrize("p", SIM_P)
@pytest.mark.parametrize("b", SIM_B)
def test_reduce_then_broadcast(p, b):
    """The pipelined reduce-then-broadcast on one tree: the single tree's
    value on every rank, the root's block j final in round j, a depth-d rank's
    in round b + j + d - 1; 2b + H - 1 rounds; every non-root sends each of
    the b partial blocks up once and every rank forwards each final block
    once per child."""
    m = 13
    x = _fp32_input(p, m, 300 * p + b)
    t = build_trees(p, layout="single")
    rows, tr = simulate_reduce_bcast(x, "float32", "sum", b)
    y = allreduce_tree(x, "float32", "sum", trees=t)
    for i in range(p):
        assert np.array_equal(rows[i], y)
        want = {j: (j if t.parent[i] is None else b + j + t.depth[i] - 1)
                for j in range(b)}
        assert tr.final_round[i] == want
        nch = sum(c is not None for c in (t.child0[i], t.child1[i]))
        up = 0 if t.parent[i] is None else b
        assert tr.messages.get(i, 0) == up + nch * b
        assert max(tr.ops_per_round.get(i, {0: 0}).values()) <= 2
    assert tr.global_rounds() == (2 * b + t.height - 1 if p > 1 else b)


def test_one_tree_and_dual_root_differ_in_fp32():
    """The association differs, so fp32 results differ for some input (the
    golden examples show one by hand; here on random data at p = 36)."""
    x = _fp32_input(36, 4096, 5)
    a = allreduce_tree(x, "float32", "sum")
    s = allreduce_tree(x, "float32", "sum", trees=build_trees(36,
                                                               layout="single"))
    assert not np.array_equal(a, s)
    # both within the recursive-summation bound of the exact sum
    exact = x.astype(np.float64).sum(axis=0)
    bound = (36 * 2.0 ** -24) * np.abs(x.astype(np.float64)).sum(axis=0)
    for v in (a, s):
        assert np.all(np.abs(v.astype(np.float64) - exact) <= bound)
    assert math.isfinite(float(bound.max()))


@pytest.mark.parametrize("p", [2, 3, 7, 12, 36])
def test_one_tree_schedules_keep_operand_order(p):
    """The 2x2 matrix product does not commute: both one-tree simulations
    must deliver the plain left-to-right product x_0 x_1 ... x_{p-1}."""
    rng = np.random.default_rng(400 + p)
    x = rng.integers(0, 2 ** 32, size=(p, 9, 4), dtype=np.uint64).astype(
        np.uint32)
    want = allreduce_ltr(x, "u32mat2x2", "matmul")
    rows, _ = simulate(x, "u32mat2x2", "matmul", 3,
                       trees=build_trees(p, layout="single"))
    assert all(np.array_equal(r, want) for r in rows)
    rows, _ = simulate_reduce_bcast(x, "u32mat2x2", "matmul", 3)
    assert all(np.array_equal(r, want) for r in rows)
