"""Pins for the oracle's reduction result (Section 1 problem statement;
Algorithm 1's association; Section 1.1's subtree products).

Each expected value is fixed by something other than the oracle: a
hand-derived worked example (derivation in the comment), a closed form,
brute force in plain Python integers, or the error bound of recursive
floating-point summation.  Several tests plant a mistake in a copy of the
oracle's evaluation and check that the pins notice it.
"""

import math
import os
from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle import (allreduce_all, allreduce_ltr, allreduce_tree, build_trees,
                    combine)

T24 = float(2 ** 24)


def f32col(values):
    return np.array(values, dtype=np.float32).reshape(len(values), 1)


# ------------------------------------------------------ fp32 worked examples

GOLDEN = os.path.join(os.path.dirname(__file__), "golden",
                      "fp32_worked_examples.txt")


def _worked_examples():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, shape, xs, tree_v, ltr_v = (c.strip() for c in line.split("|"))
            rows.append((name, shape, [float(v) for v in xs.split()],
                         float(tree_v), float(ltr_v)))
    return rows


@pytest.mark.parametrize("name,shape,xs,tree_v,ltr_v", _worked_examples())
def test_fp32_worked_examples(name, shape, xs, tree_v, ltr_v):
    x = f32col(xs)
    trees = build_trees(len(xs), shape=shape)
    assert allreduce_tree(x, "float32", "sum", trees=trees)[0] == tree_v
    assert allreduce_ltr(x, "float32", "sum")[0] == ltr_v


def _mutant_tree(x, dtype, op, mutation):
    """A copy of the oracle's evaluation with one planted mistake."""
    t = build_trees(len(x))

    def S(i):
        v = x[i].copy()
        c0, c1 = t.child0[i], t.child1[i]
        if mutation == "child1_first":
            for c in (c1, c0):
                if c is not None:
                    v = combine(dtype, op, S(c), v)
        elif mutation == "children_first":
            if c0 is not None and c1 is not None:
                v = combine(dtype, op, combine(dtype, op, S(c1), S(c0)), v)
            elif c0 is not None:
                v = combine(dtype, op, S(c0), v)
        elif mutation == "operand_swap":
            for c in (c0, c1):
                if c is not None:
                    v = combine(dtype, op, v, S(c))
        return v
    a, b = (S(r) for r in t.roots)
    if mutation == "root_swap":
        return combine(dtype, op, b, a)
    return combine(dtype, op, a, b)


def test_planted_association_mistakes_are_caught():
    ex1 = f32col([1, T24, 1, -T24, 0, 0, 0])
    ex3 = f32col([-T24, 0, T24, 1, 0, 0, 0])
    assert _mutant_tree(ex1, "float32", "sum", "children_first")[0] != 1.0
    assert _mutant_tree(ex3, "float32", "sum", "child1_first")[0] != 0.0
    # operand and root order only show with a non-commutative operator
    x = synth.generate("odd_det_u32_mat", 7, 7, 16)
    ref = _py_ltr_matmul(x)
    for mutation in ("operand_swap", "root_swap", "child1_first"):
        got = _mutant_tree(x, "u32mat2x2", "matmul", mutation)
        assert not np.array_equal(got, ref), mutation


# ------------------------------------------------ brute force in Python ints

def _py_matmul(a, b):
    M = 1 << 32
    return [(a[0] * b[0] + a[1] * b[2]) % M, (a[0] * b[1] + a[1] * b[3]) % M,
            (a[2] * b[0] + a[3] * b[2]) % M, (a[2] * b[1] + a[3] * b[3]) % M]


def _py_ltr_matmul(x):
    p, m = x.shape[0], x.shape[1]
    out = np.empty((m, 4), dtype=np.uint32)
    for k in range(m):
        acc = [int(v) for v in x[0, k]]
        for i in range(1, p):
            acc = _py_matmul(acc, [int(v) for v in x[i, k]])
        out[k] = acc
    return out


def _wrap32(v):
    v &= 0xFFFFFFFF
    return v - (1 << 32) if v >= 1 << 31 else v


@pytest.mark.parametrize("p", [1, 2, 3, 4, 5, 7, 8, 9, 16, 17, 36, 64])
def test_int32_sum_and_max_brute_force(p):
    m = 6
    x = synth.generate("uniform_int", 1000 + p, p, m, lo=-2 ** 31,
                       hi=2 ** 31 - 1)
    s = allreduce_tree(x, "int32", "sum")
    mx = allreduce_tree(x, "int32", "max")
    for k in range(m):
        col = [int(x[i, k]) for i in range(p)]
        assert int(s[k]) == _wrap32(sum(col))
        assert int(mx[k]) == max(col)


@pytest.mark.parametrize("p", [1, 2, 3, 5, 6, 7, 9, 14, 30, 36, 64])
@pytest.mark.parametrize("dist", ["uniform_u32_mat", "odd_det_u32_mat"])
def test_matmul_brute_force_left_to_right(p, dist):
    x = synth.generate(dist, 3000 + p, p, 5)
    got = allreduce_tree(x, "u32mat2x2", "matmul")
    assert np.array_equal(got, _py_ltr_matmul(x))


def test_matmul_is_order_sensitive_on_odd_determinant_inputs():
    # the odd-determinant set makes any swap of two ranks visible
    p = 12
    x = synth.generate("odd_det_u32_mat", 11, p, 32)
    ref = allreduce_tree(x, "u32mat2x2", "matmul")
    for a, b in ((0, 1), (3, 9), (5, 6), (10, 11)):
        y = x.copy()
        y[[a, b]] = y[[b, a]]
        assert not np.array_equal(allreduce_tree(y, "u32mat2x2", "matmul"),
                                  ref)


def test_closed_forms():
    for p in (1, 2, 7, 36, 1152):
        ranks = np.repeat(np.arange(p, dtype=np.int32)[:, None], 4, axis=1)
        assert (allreduce_tree(ranks, "int32", "sum")
                == p * (p - 1) // 2).all()
        ones = np.ones((p, 3), dtype=np.int32)
        assert (allreduce_tree(ones, "int32", "sum") == p).all()
        fones = np.ones((p, 3), dtype=np.float32)
        assert (allreduce_tree(fones, "float32", "sum") == p).all()
        # max with one distinguished rank per column
        mx = np.zeros((p, 5), dtype=np.int32)
        for k in range(5):
            mx[k % p, k] = 1000
        assert (allreduce_tree(mx, "int32", "max") == 1000).all()


def test_int32_wraps():
    x = np.full((5, 2), 2 ** 31 - 1, dtype=np.int32)
    got = allreduce_tree(x, "int32", "sum")
    assert int(got[0]) == _wrap32(5 * (2 ** 31 - 1))


def test_integer_valued_fp32_is_exact():
    # |partial sums| < 2^24 makes every order exact: y equals the integer sum
    p, m = 7, 1000
    x = synth.generate("uniform_int", 2110, p, m, lo=-1000, hi=1000)
    got = allreduce_tree(x.astype(np.float32), "float32", "sum")
    assert np.array_equal(got.astype(np.int64), x.astype(np.int64).sum(0))


@pytest.mark.parametrize("p", [36, 1152])
def test_fp32_error_bound(p):
    # Recursive summation bound: |yhat - y| <= gamma_L * sum |x_i| where L is
    # the most additions any input passes through.  In the tree a value gains
    # at most two additions per level (x_i then the second child) plus the
    # root exchange, so L <= 2 (H + 1) + 1.
    m = 64
    x = synth.generate("normal_f32", 2113, p, m)
    got = allreduce_tree(x, "float32", "sum")
    H = build_trees(p).height
    L = 2 * (H + 1) + 1
    u = 2.0 ** -24
    gamma = L * u / (1 - L * u)
    for k in range(m):
        exact = math.fsum(float(v) for v in x[:, k])
        bound = gamma * math.fsum(abs(float(v)) for v in x[:, k])
        assert abs(float(got[k]) - exact) <= bound


def test_fp32_uses_binary32_rounding_not_wider():
    # a wider accumulator would keep the 1: here the tree must drop it
    x = f32col([1, T24, 1, -T24, 0, 0, 0])
    exact = Fraction(1) + Fraction(2 ** 24) + 1 - 2 ** 24
    assert exact == 2
    assert allreduce_tree(x, "float32", "sum")[0] == 1.0


def test_broadcast_gives_p_identical_copies():
    x = synth.generate("normal_f32", 5, 9, 17)
    out = allreduce_all(x, "float32", "sum")
    y = allreduce_tree(x, "float32", "sum")
    assert out.shape == (9, 17)
    assert all(np.array_equal(out[i], y) for i in range(9))
