"""The reduction-to-all result (Section 1; Algorithm 1).

Oracle module: test infrastructure only.

Problem (Section 1): each of p ranks holds x_i of m elements; every rank must
receive y = x_0 (.) x_1 (.) ... (.) x_{p-1}, element-wise.

For exactly associative operators (int32 SUM/MAX, the 2x2 matrix product) the
method reaches exactly the plain left-to-right product, ``allreduce_ltr``.
For fp32 SUM the association is part of the result, so ``allreduce_tree``
follows Algorithm 1's steps: a non-leaf i first combines the block received
from its first child into its own block, Y <- t (.) Y, then the block from its
second child, Y <- t (.) Y again, so the subtree value is

    S(i) = S(child1) (.) ( S(child0) (.) x_i ),

and the roots exchange their tree values; the lower-numbered root computes
Y (.) t and the higher one t (.) Y, both equal to y = S(root A) (.) S(root B).
Section 1.1 gives the same product over the post-order subtree ranges.

Everything is evaluated on whole column vectors (columns are independent);
there is no blocking, no fusion and no reordering of the operator
applications.
"""

import numpy as np

from .ops import combine
from .trees import build_trees


def _as_rows(x):
    if isinstance(x, (list, tuple)):
        return list(x)
    return [x[i] for i in range(x.shape[0])]


def allreduce_tree(x, dtype: str, op: str, trees=None):
    """y in Algorithm 1's association.  ``x`` is [p, m] (or [p, m, 4] for
    matrices) or a list of p vectors.  Returns one vector y."""
    rows = _as_rows(x)
    p = len(rows)
    t = trees if trees is not None else build_trees(p)

    def subtree(i):
        y = rows[i].copy()                       # Y <- x_i
        if t.child0[i] is not None:              # first child
            y = combine(dtype, op, subtree(t.child0[i]), y)
        if t.child1[i] is not None:              # second child
            y = combine(dtype, op, subtree(t.child1[i]), y)
        return y

    values = [subtree(r) for r in t.roots]
    if len(values) == 1:
        return values[0]
    return combine(dtype, op, values[0], values[1])   # root A on the left


def allreduce_ltr(x, dtype: str, op: str):
    """The plain definition, (((x_0 (.) x_1) (.) x_2) ...) (.) x_{p-1}."""
    rows = _as_rows(x)
    y = rows[0].copy()
    for r in rows[1:]:
        y = combine(dtype, op, y, r)
    return y


def allreduce_all(x, dtype: str, op: str, out=None):
    """What every rank ends with: p copies of y (the broadcast half of the
    reduction-to-all).  ``out`` may be a preallocated [p, ...] array."""
    rows = _as_rows(x)
    y = allreduce_tree(rows, dtype, op)
    if out is None:
        out = np.empty((len(rows),) + y.shape, dtype=y.dtype)
    for i in range(len(rows)):
        out[i] = y
    return out
