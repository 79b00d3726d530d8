"""Pins for the plain C oracle (Section 1 problem statement; Section 1.1
trees; Algorithm 1's association), a second oracle written independently
of the numpy one: a stack walk over the ranks in post-order, with the trees
numbered by subtree sizes instead of a recursive traversal.

Each expected value is fixed by something other than the oracle: the
hand-derived worked examples under tests/golden/, hand listings of the
trees, tree invariants, closed forms and brute force in Python integers.
Copies of the C oracle built with a planted mistake must fail them.  The
two oracles must then agree bit for bit on the workloads' shapes.
"""

import math
import os

import numpy as np
import pytest

import synth
from oracle import allreduce_tree, build_trees
from oracle import c_oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
T24 = float(2 ** 24)


def _none(v):
    return -1 if v is None else v


def _golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([c.strip() for c in line.split("|")])
    return rows


def f32col(values):
    return np.array(values, dtype=np.float32).reshape(len(values), 1)


def _wrap32(v):
    v &= 0xFFFFFFFF
    return v - (1 << 32) if v >= 1 << 31 else v


def _py_matmul(a, b):
    M = 1 << 32
    return [(a[0] * b[0] + a[1] * b[2]) % M, (a[0] * b[1] + a[1] * b[3]) % M,
            (a[2] * b[0] + a[3] * b[2]) % M, (a[2] * b[1] + a[3] * b[3]) % M]


def _py_ltr_matmul(x):
    out = np.empty((x.shape[1], 4), dtype=np.uint32)
    for k in range(x.shape[1]):
        acc = [int(v) for v in x[0, k]]
        for i in range(1, x.shape[0]):
            acc = _py_matmul(acc, [int(v) for v in x[i, k]])
        out[k] = acc
    return out


# ---------------------------------------------------------------- the trees

def test_trees_p7_and_p9_hand_listings():
    # p = 7: tree A = ranks 0..3 (heap of 4: root 3, children 2 (right,
    # first) and 1 (left, second), 1 has the single child 0); tree B = ranks
    # 4..6 (root 6 with children 5 and 4).
    par, c0, c1, d, roots = c_oracle.trees(7)
    assert list(par) == [1, 3, 3, -1, 6, 6, -1]
    assert list(c0) == [-1, 0, -1, 2, -1, -1, 5]
    assert list(c1) == [-1, -1, -1, 1, -1, -1, 4]
    assert list(d) == [2, 1, 1, 0, 1, 1, 0]
    assert list(roots) == [3, 6]
    # p = 9: tree A = ranks 0..4, heap of 5: the left subtree (heap 2 with
    # children 4 and 5) takes ranks 0..2, the right leaf (heap 3) rank 3,
    # the root rank 4; tree B = ranks 5..8, shaped as tree A of p = 7.
    par, c0, c1, d, roots = c_oracle.trees(9)
    assert list(par) == [2, 2, 4, 4, -1, 6, 8, 8, -1]
    assert list(c0) == [-1, -1, 1, -1, 3, -1, 5, -1, 7]
    assert list(c1) == [-1, -1, 0, -1, 2, -1, -1, -1, 6]
    assert list(d) == [2, 2, 1, 1, 0, 2, 1, 1, 0]
    assert list(roots) == [4, 8]


def _check_invariants(p, layout):
    par, c0, c1, d, roots = c_oracle.trees(p, layout)
    n_a = (p + 1) // 2 if layout == "dual" else p
    assert roots[0] == n_a - 1
    assert roots[1] == (p - 1 if n_a < p else -1)
    size = [1] * p
    lo = list(range(p))
    for i in range(p):                       # post-order: children first
        if c0[i] >= 0:
            assert c0[i] == i - 1
            assert par[c0[i]] == i and d[c0[i]] == d[i] + 1
            size[i] += size[c0[i]]
            lo[i] = lo[c0[i]]
        if c1[i] >= 0:
            assert c0[i] >= 0 and c1[i] < lo[c0[i]]
            assert par[c1[i]] == i and d[c1[i]] == d[i] + 1
            assert c1[i] == lo[c0[i]] - 1        # subtrees adjacent
            size[i] += size[c1[i]]
            lo[i] = lo[c1[i]]
        assert lo[i] == i - size[i] + 1          # contiguous ranks
    for r, first, n in ((roots[0], 0, n_a), (roots[1], n_a, p - n_a)):
        if n == 0:
            continue
        assert par[r] == -1 and lo[r] == first and size[r] == n
        # heap completeness: every level above the last is full, so the
        # height is floor(log2 n) and exactly n - 2^H + 1 nodes sit at depth H
        H = int(math.floor(math.log2(n)))
        depths = [d[i] for i in range(first, first + n)]
        assert max(depths) == H
        assert depths.count(H) == n - 2 ** H + 1
        for k in range(H):
            assert depths.count(k) == 2 ** k
        # the last level is filled from the left: the deepest nodes are the
        # first ranks of every subtree that holds one (lower ranks deeper)
        if n > 1:
            assert d[first] == H


@pytest.mark.parametrize("p", list(range(1, 130)) + [255, 256, 511, 576, 1000,
                                                     1151, 1152, 2000, 4608,
                                                     32768, 100003])
def test_tree_invariants(p):
    _check_invariants(p, "dual")
    _check_invariants(p, "single")


@pytest.mark.parametrize("p", [1, 2, 7, 9, 36, 64, 1152, 2000])
def test_trees_agree_with_the_numpy_oracle(p):
    for layout in ("dual", "single"):
        par, c0, c1, d, roots = c_oracle.trees(p, layout)
        t = build_trees(p, layout=layout)
        assert list(par) == [_none(v) for v in t.parent]
        assert list(c0) == [_none(v) for v in t.child0]
        assert list(c1) == [_none(v) for v in t.child1]
        assert list(d) == t.depth
        assert [r for r in roots if r >= 0] == t.roots


# ------------------------------------------------------ fp32 worked examples

@pytest.mark.parametrize("row", [r for r in _golden("fp32_worked_examples.txt")
                                 if r[1] == "heap"], ids=lambda r: r[0])
def test_fp32_worked_examples(row):
    _, _, xs, tree_v, _ = row
    x = f32col([float(v) for v in xs.split()])
    assert c_oracle.allreduce(x, "float32", "sum")[0] == float(tree_v)


@pytest.mark.parametrize("row", _golden("fp32_single_tree_examples.txt"),
                         ids=lambda r: r[0])
def test_fp32_single_tree_worked_examples(row):
    _, xs, single, dual, _ = row
    x = f32col([float(v) for v in xs.split()])
    assert c_oracle.allreduce(x, "float32", "sum", layout="single")[0] == \
        float(single)
    assert c_oracle.allreduce(x, "float32", "sum")[0] == float(dual)


def test_fp32_uses_binary32_rounding_not_wider():
    # exactly 2 in real arithmetic; binary32 drops the 1 added to 2^24
    x = f32col([1, T24, 1, -T24, 0, 0, 0])
    assert c_oracle.allreduce(x, "float32", "sum")[0] == 1.0


def test_integer_valued_fp32_is_exact():
    p, m = 7, 1000
    x = synth.generate("uniform_int", 2110, p, m, lo=-1000, hi=1000)
    got = c_oracle.allreduce(x.astype(np.float32), "float32", "sum")
    assert np.array_equal(got.astype(np.int64), x.astype(np.int64).sum(0))


# ------------------------------------------------------------ brute force

@pytest.mark.parametrize("p", [1, 2, 3, 4, 5, 7, 8, 9, 16, 17, 36, 64])
def test_int32_sum_and_max_brute_force(p):
    m = 6
    x = synth.generate("uniform_int", 1000 + p, p, m, lo=-2 ** 31,
                       hi=2 ** 31 - 1)
    s = c_oracle.allreduce(x, "int32", "sum")
    mx = c_oracle.allreduce(x, "int32", "max")
    for k in range(m):
        col = [int(x[i, k]) for i in range(p)]
        assert int(s[k]) == _wrap32(sum(col))
        assert int(mx[k]) == max(col)


@pytest.mark.parametrize("p", [1, 2, 3, 5, 6, 7, 9, 14, 30, 36, 64])
@pytest.mark.parametrize("dist", ["uniform_u32_mat", "odd_det_u32_mat"])
@pytest.mark.parametrize("layout", ["dual", "single"])
def test_matmul_brute_force_left_to_right(p, dist, layout):
    x = synth.generate(dist, 3000 + p, p, 5)
    got = c_oracle.allreduce(x, "u32mat2x2", "matmul", layout=layout)
    assert np.array_equal(got, _py_ltr_matmul(x))


def test_closed_forms():
    for p in (1, 2, 7, 36, 1152):
        ranks = np.repeat(np.arange(p, dtype=np.int32)[:, None], 4, axis=1)
        assert (c_oracle.allreduce(ranks, "int32", "sum")
                == p * (p - 1) // 2).all()
        ones = np.ones((p, 3), dtype=np.float32)
        assert (c_oracle.allreduce(ones, "float32", "sum") == p).all()
        mx = np.zeros((p, 5), dtype=np.int32)
        for k in range(5):
            mx[k % p, k] = 1000
        assert (c_oracle.allreduce(mx, "int32", "max") == 1000).all()
    x = np.full((5, 2), 2 ** 31 - 1, dtype=np.int32)
    assert int(c_oracle.allreduce(x, "int32", "sum")[0]) == \
        _wrap32(5 * (2 ** 31 - 1))


# ------------------------------------------------------- planted mistakes

def _pins_hold(lib):
    """True when every pin below holds for C oracle build ``lib``."""
    ex1 = f32col([1, T24, 1, -T24, 0, 0, 0])           # y = 1
    ex3 = f32col([-T24, 0, T24, 1, 0, 0, 0])           # y = 0
    if c_oracle.allreduce(ex1, "float32", "sum", lib=lib)[0] != 1.0:
        return False
    if c_oracle.allreduce(ex3, "float32", "sum", lib=lib)[0] != 0.0:
        return False
    for p in (7, 9, 30):
        x = synth.generate("odd_det_u32_mat", 3000 + p, p, 5)
        got = c_oracle.allreduce(x, "u32mat2x2", "matmul", lib=lib)
        if not np.array_equal(got, _py_ltr_matmul(x)):
            return False
    return True


def test_pins_hold_for_the_oracle():
    assert _pins_hold(c_oracle.load())


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_planted_mistakes_are_caught(k):
    # 1: second child before the first; 2: child's value on the right;
    # 3: the roots combined the other way round; 4: the children combined
    # with each other before x_i
    assert not _pins_hold(c_oracle.mutant(k))


# --------------------------------------------- threads, broadcast, errors

@pytest.mark.parametrize("m", [1, 5, 7, 1000, 4097])
def test_result_independent_of_threads(m):
    x = synth.generate("normal_f32", 77, 37, m)
    ref = c_oracle.allreduce(x, "float32", "sum", threads=1)
    for t in (2, 3, 8, 9):
        got = c_oracle.allreduce(x, "float32", "sum", threads=t)
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_broadcast_writes_every_row():
    x = synth.generate("odd_det_u32_mat", 5, 9, 17)
    out = np.zeros_like(x)
    c_oracle.allreduce_all(x, "u32mat2x2", "matmul", out, threads=4)
    y = c_oracle.allreduce(x, "u32mat2x2", "matmul")
    assert all(np.array_equal(out[i], y) for i in range(9))


def test_argument_errors_and_empty_rows():
    lib = c_oracle.load()
    x = np.zeros((3, 4), np.int32)
    y = np.zeros(4, np.int32)
    rows = c_oracle._ptrs([x[i] for i in range(3)])
    assert lib.dpo_allreduce(0, 2, rows, 0, 4, y.ctypes.data, 1) == -1
    assert lib.dpo_allreduce(9, 2, rows, 3, 4, y.ctypes.data, 1) == -1
    assert lib.dpo_allreduce(0, 3, rows, 3, 4, y.ctypes.data, 1) == -1
    assert lib.dpo_allreduce(0, 2, rows, 3, 4, y.ctypes.data, 0) == -1
    assert lib.dpo_allreduce(0, 2, rows, 3, 4, None, 1) == -1
    assert lib.dpo_allreduce(0, 2, rows, 3, 0, y.ctypes.data, 1) == 0
    assert lib.dpo_trees(0, 2, *([y.ctypes.data] * 5)) == -1


# ------------------------------------------- agreement with the numpy oracle

@pytest.mark.parametrize("p,dist,dtype,op,m", [
    (7, "uniform_int", "int32", "sum", 1000),
    (36, "uniform_int", "int32", "max", 4096),
    (64, "uniform_u32_mat", "u32mat2x2", "matmul", 512),
    (1152, "normal_f32", "float32", "sum", 4096),
    (1152, "uniform_int", "int32", "sum", 1024),
    (300, "normal_f32", "float32", "sum", 333),
])
def test_agrees_with_the_numpy_oracle(p, dist, dtype, op, m):
    kw = {"lo": -2 ** 20, "hi": 2 ** 20} if dist == "uniform_int" else {}
    x = synth.generate(dist, 2109 + p, p, m, **kw)
    for layout in ("dual", "single"):
        want = allreduce_tree(x, dtype, op,
                              trees=build_trees(p, layout=layout))
        got = c_oracle.allreduce(x, dtype, op, layout=layout, threads=4)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
