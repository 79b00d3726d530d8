"""Seeded random combinations of every call parameter, each checked bit for
bit against the oracle: p, m, b (or the rule), dtype and operator, tree
layout, executor, work-item kind, 16-byte or only 4-byte alignment, in-place
or separate outputs, one tensor or separate allocations."""

import numpy as np
import pytest
import torch

import oracle
import synth
from tests._gpu import (POISON, _Env, assert_all_ranks_equal, env_unit, lib,
                        need_gpu)

pytestmark = pytest.mark.gpu

PAIRS = [("int32", "sum", "uniform_int"), ("int32", "max", "uniform_int"),
         ("float32", "sum", "normal_f32"),
         ("u32mat2x2", "matmul", "uniform_u32_mat")]
EXECS = ["auto", "split", "ticket", "launch", "barrier", "rounds",
         "rounds_barrier"]
ALGS = ["dual", "single", "reduce_bcast"]
UNITS = [None, "seq", "level", "sub"]


def _case(k):
    r = np.random.default_rng(9000 + k)
    p = int(r.choice([1, 2, 3, 5, 7, 16, 33, 64, 100, 257, 300]))
    m = int(r.integers(1, 4000))
    b = int(r.choice([0, 1, 2, 3, int(r.integers(1, m + 1))]))
    b = min(b, m)
    dtype, op, dist = PAIRS[int(r.integers(len(PAIRS)))]
    return dict(p=p, m=m, b=b, dtype=dtype, op=op, dist=dist,
                alg=ALGS[int(r.integers(3))],
                exec=EXECS[int(r.integers(len(EXECS)))],
                unit=UNITS[int(r.integers(len(UNITS)))],
                misalign=bool(r.integers(2)), inplace=bool(r.integers(4) == 0),
                separate=bool(r.integers(2)), seed=2200 + k)


@pytest.mark.parametrize("k", range(800))
def test_random_combination(k):
    need_gpu()
    _check_case(_case(k))


def _wide_case(k):
    r = np.random.default_rng(9700 + k)
    p = int(r.integers(2, 129))
    dtype, op, dist = PAIRS[int(r.integers(len(PAIRS)))]
    words = 4 if dtype == "u32mat2x2" else 1
    # up to 2^20 words of input: a few wide items (1024 quanta each) with a
    # ragged last one, or less than one
    m = int(r.integers(1, max(2, (1 << 20) // (p * words))))
    b = int(r.choice([0, 1, int(r.integers(1, m + 1))]))
    return dict(p=p, m=m, b=min(b, m), dtype=dtype, op=op, dist=dist,
                alg=ALGS[int(r.integers(3))],
                exec=["auto", "split", "ticket"][int(r.integers(3))],
                unit="wide", misalign=bool(r.integers(2)),
                inplace=bool(r.integers(4) == 0), separate=bool(r.integers(2)),
                seed=2700 + k,
                wide_round=[None, 1, 2, 3, 5][int(r.integers(5))])


@pytest.mark.parametrize("k", range(160))
def test_random_wide_items(k):
    """Seeded random calls with the wide post-order work item forced (the
    one-launch executors; on 4-byte lanes the library keeps the plain
    post-order item): p = 2 .. 128, every operator and tree layout,
    misaligned rows, in place, separate allocations; rounds of 1, 2, 3 or 5
    wide items in most cases (DPAR_WIDE_ROUND), so that the columns past the
    last whole round go to tail items."""
    need_gpu()
    _check_case(_wide_case(k))


def _mid_case(k):
    r = np.random.default_rng(9800 + k)
    p = int(r.choice([2, 5, 8, 12, 16, 20, 24, 36, 48, 64, 96, 130, 200, 288,
                      400, 511, 700, 1100]))
    dtype, op, dist = PAIRS[int(r.integers(len(PAIRS)))]
    words = 4 if dtype == "u32mat2x2" else 1
    # 4 to 32 MB of input: the sizes where AUTO picks between post-order,
    # wide, subtree and level items and between split and one fused launch
    mmax = max(2, (1 << 23) // (p * words))
    m = int(r.integers(max(1, mmax // 8), mmax))
    return dict(p=p, m=m, b=0, dtype=dtype, op=op, dist=dist,
                alg=ALGS[int(r.integers(3))], exec="auto", unit=None,
                misalign=bool(r.integers(4) == 0),
                inplace=bool(r.integers(6) == 0),
                separate=bool(r.integers(3) == 0), seed=2800 + k)


@pytest.mark.parametrize("k", range(160))
def test_random_auto_mid_size(k):
    """Seeded random calls of 4 to 32 MB under AUTO with the rule's b
    (p = 2 .. 1100, every operator and tree layout, misaligned rows, in
    place, separate allocations): whatever work item and executor the
    library picks, bit for bit against the oracle."""
    need_gpu()
    _check_case(_mid_case(k))


def _check_case(c):
    dpar = lib()
    p, m = c["p"], c["m"]
    kw = {"lo": -50, "hi": 50} if c["dist"] == "uniform_int" else {}
    x = synth.generate(c["dist"], c["seed"], p, m, **kw)
    trees = oracle.build_trees(p) if c["alg"] == "dual" else \
        oracle.build_trees(p, layout="single")
    want = oracle.allreduce_tree(x, c["dtype"], c["op"], trees=trees)
    words = 4 if c["dtype"] == "u32mat2x2" else 1     # int32 words/element
    row = m * words + 1                                 # spare word per row
    off = 1 if c["misalign"] else 0                     # 4-byte offset
    xi = np.ascontiguousarray(x).view(np.int32).reshape(p, m * words)

    def alloc():
        if c["separate"]:
            bufs = [torch.full((row + 4,), POISON, dtype=torch.int32,
                               device="cuda") for _ in range(p)]
            return bufs, [t.data_ptr() + 4 * off for t in bufs]
        t = torch.full((p, row + 4), POISON, dtype=torch.int32, device="cuda")
        return [t], [t.data_ptr() + 4 * (i * (row + 4) + off)
                     for i in range(p)]

    xb, xs = alloc()
    for i in range(p):
        src = torch.from_numpy(xi[i].copy()).cuda()
        if c["separate"]:
            xb[i][off:off + m * words] = src
        else:
            xb[0][i, off:off + m * words] = src
    if c["inplace"]:
        yb, ys = xb, xs
    else:
        yb, ys = alloc()
    torch.cuda.synchronize()
    s = torch.cuda.current_stream()
    with env_unit(c["unit"]), _Env("DPAR_WIDE_ROUND", c.get("wide_round")):
        dpar.dpar_allreduce_opt(xs, ys, p, m, c["dtype"], c["op"], c["b"],
                                c["alg"], c["exec"], 0, -1, s)
    dpar.dpar_check_status(s)
    rows = []
    for i in range(p):
        t = (yb[i] if c["separate"] else yb[0][i]).cpu().numpy()
        rows.append(t[off:off + m * words])
        # nothing written outside the m elements of each row
        assert np.all(t[:off] == POISON) and \
            np.all(t[off + m * words:] == POISON), (str(c), i)
    got = np.stack(rows).view(x.dtype).reshape(x.shape)
    assert_all_ranks_equal(got, want, str(c))


def _large_case(k):
    r = np.random.default_rng(9500 + k)
    p = int(r.integers(257, 5001))
    dtype, op, dist = PAIRS[int(r.integers(len(PAIRS)))]
    words = 4 if dtype == "u32mat2x2" else 1
    # at most 2^22 words of input, so that each case stays small
    m = int(r.integers(1, max(2, min(20000, (1 << 22) // (p * words)))))
    b = int(r.choice([0, 1, 2, int(r.integers(1, m + 1))]))
    return dict(p=p, m=m, b=min(b, m), dtype=dtype, op=op, dist=dist,
                alg=ALGS[int(r.integers(3))],
                exec=["auto", "split", "ticket", "launch"][int(r.integers(4))],
                unit=UNITS[int(r.integers(len(UNITS)))], seed=2600 + k)


@pytest.mark.parametrize("k", range(100))
def test_random_large_p(k):
    """Seeded random calls at p = 257 .. 5000 (deeper trees, the subtree
    and level work items and their chunk choices): bit for bit against the
    oracle, with the library's own choices and with forced work items."""
    need_gpu()
    dpar = lib()
    c = _large_case(k)
    p, m = c["p"], c["m"]
    kw = {"lo": -50, "hi": 50} if c["dist"] == "uniform_int" else {}
    x = synth.generate(c["dist"], c["seed"], p, m, **kw)
    trees = oracle.build_trees(p) if c["alg"] == "dual" else \
        oracle.build_trees(p, layout="single")
    want = oracle.allreduce_tree(x, c["dtype"], c["op"], trees=trees)
    a = np.ascontiguousarray(x)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    xd = torch.from_numpy(a).cuda()
    yd = torch.full_like(xd, POISON)
    s = torch.cuda.current_stream()
    with env_unit(c["unit"]):
        dpar.dpar_allreduce_opt(dpar.rows(xd), dpar.rows(yd), p, m,
                                c["dtype"], c["op"], c["b"], c["alg"],
                                c["exec"], 0, -1, s)
    dpar.dpar_check_status(s)
    got = yd.cpu().numpy().view(x.dtype).reshape(x.shape)
    assert_all_ranks_equal(got, want, str(c))
