"""The allocation-free entry point, dpar_allreduce_noalloc (for callers that
cannot allocate device memory), against
dpar_allreduce through the C ABI: the same inputs give bit-identical outputs
(both equal the oracle's), on calls in a row whose sizes and pointer arrays
change, and on repeated calls whose pointer arrays stay (the fixed scratch
keeps its tables and is not restaged).
"""

import numpy as np
import pytest
import torch

import oracle
import synth

from tests._gpu import (assert_all_ranks_equal, from_dev, need_gpu,
                        poisoned_like, to_dev)

pytestmark = pytest.mark.gpu


def _both(x, dtype, op, b):
    """One dpar_allreduce and one dpar_allreduce_noalloc call on the same
    device input (separate outputs); returns both outputs as numpy."""
    from paper_2109_12626_amd import dpar
    p, m = x.shape[0], x.shape[1]
    xd = to_dev(x)
    y_ref = poisoned_like(xd)
    y_fix = poisoned_like(xd)
    s = torch.cuda.current_stream()
    dpar.dpar_allreduce(dpar.rows(xd), dpar.rows(y_ref), p, m, dtype, op, b, s)
    dpar.dpar_allreduce_noalloc(dpar.rows(xd), dpar.rows(y_fix), p, m, dtype,
                                op, b, s)
    dpar.dpar_check_status(s)
    return from_dev(y_ref, x), from_dev(y_fix, x)


def _check(x, dtype, op, b, what):
    ref, fix = _both(x, dtype, op, b)
    assert np.array_equal(np.ascontiguousarray(ref).view(np.uint32),
                          np.ascontiguousarray(fix).view(np.uint32)), what
    assert_all_ranks_equal(fix, oracle.allreduce_tree(x, dtype, op), what)


def test_two_calls_second_smaller():
    """p = 1152, m = 2^16 fp32 (subtree work items: opcode table, subtree
    plan and 18 KB of pointers in the fixed scratch), then p = 36,
    m = 5003 int32 (a smaller layout; one element per lane, the level
    table): each equal to dpar_allreduce's output."""
    need_gpu()
    x1 = synth.generate("normal_f32", 2301, 1152, 1 << 16)
    _check(x1, "float32", "sum", 0, "p=1152 m=2^16 fp32")
    x2 = synth.generate("uniform_int", 2302, 36, 5003, lo=-1 << 20,
                        hi=1 << 20)
    _check(x2, "int32", "sum", 0, "p=36 m=5003 int32")


def test_same_pointers_new_contents():
    """The second call reuses the staged tables and pointers; it must read
    the buffers' new contents."""
    need_gpu()
    from paper_2109_12626_amd import dpar
    p, m = 64, 1 << 14
    xa = synth.generate("uniform_int", 2303, p, m, lo=0, hi=1 << 16)
    xb = synth.generate("uniform_int", 2304, p, m, lo=0, hi=1 << 16)
    xd = to_dev(xa)
    yd = poisoned_like(xd)
    xs, ys = dpar.pointers(dpar.rows(xd)), dpar.pointers(dpar.rows(yd))
    s = torch.cuda.current_stream()
    for x in (xa, xb, xa):
        xd.copy_(to_dev(x))
        yd.fill_(-1)
        dpar.dpar_allreduce_noalloc(xs, ys, p, m, "int32", "max", 0, s)
        dpar.dpar_check_status(s)
        assert_all_ranks_equal(from_dev(yd, x),
                               oracle.allreduce_tree(x, "int32", "max"),
                               "reused pointers")


@pytest.mark.parametrize("p,m,dtype,op", [
    (1, 1000, "int32", "sum"),
    (2, 4099, "float32", "sum"),
    (7, 1000, "int32", "sum"),
    (64, 4096, "u32mat2x2", "matmul"),
    (300, 20000, "float32", "sum"),
    (2304, 1 << 12, "int32", "max"),
    (36, 1 << 20, "int32", "sum"),          # wide items, one fused launch
    (64, 1 << 18, "u32mat2x2", "matmul"),   # wide items, split
    (40, 4096 * 264 + 100, "int32", "sum"),  # full and tail wide items, split
])
def test_sizes_and_types(p, m, dtype, op):
    need_gpu()
    if dtype == "u32mat2x2":
        x = synth.generate("odd_det_u32_mat", 2305 + p, p, m)
    elif dtype == "float32":
        x = synth.generate("normal_f32", 2305 + p, p, m)
    else:
        x = synth.generate("uniform_int", 2305 + p, p, m, lo=-1000, hi=1000)
    _check(x, dtype, op, 0, f"p={p} m={m} {dtype}")


def _random_case(k):
    r = np.random.default_rng(9900 + k)
    p = int(r.choice([1, 2, 3, 7, 36, 64, 255, 300, 1152, 2304, 5000]))
    dtype, op, dist = [("int32", "sum", "uniform_int"),
                       ("int32", "max", "uniform_int"),
                       ("float32", "sum", "normal_f32"),
                       ("u32mat2x2", "matmul", "odd_det_u32_mat")][
                           int(r.integers(4))]
    words = 4 if dtype == "u32mat2x2" else 1
    m = int(r.integers(1, max(2, min(70000, (1 << 22) // (p * words)))))
    b = int(r.choice([0, 1, int(r.integers(1, m + 1))]))
    return p, m, dtype, op, dist, min(b, m)


@pytest.mark.parametrize("k", range(40))
def test_random_calls(k):
    """Seeded random calls of both entry points in a row (p = 1 .. 5000,
    every operator, the rule's b, b = 1 or a random b): bit-identical
    outputs, equal to the oracle; consecutive cases change p, m and the
    pointer arrays, so the fixed scratch is restaged every time."""
    need_gpu()
    p, m, dtype, op, dist, b = _random_case(k)
    kw = {"lo": -1000, "hi": 1000} if dist == "uniform_int" else {}
    x = synth.generate(dist, 2400 + k, p, m, **kw)
    _check(x, dtype, op, b, f"k={k} p={p} m={m} {dtype} {op} b={b}")


def test_largest_p_and_the_limit():
    """p = 32768 fits the fixed scratch; one more rank is refused before any
    device work."""
    need_gpu()
    from paper_2109_12626_amd import dpar
    x = synth.generate("uniform_int", 2306, 32768, 64, lo=-1000, hi=1000)
    _check(x, "int32", "sum", 0, "p=32768")
    xd = torch.zeros((32769, 4), dtype=torch.int32, device="cuda")
    yd = torch.zeros_like(xd)
    with pytest.raises(dpar.DparError) as ei:
        dpar.dpar_allreduce_noalloc(dpar.rows(xd), dpar.rows(yd), 32769, 4,
                                    "int32", "sum", 0,
                                    torch.cuda.current_stream())
    assert ei.value.code == dpar.DPAR_ERR_UNSUPPORTED
    assert bool((yd == 0).all())
