"""GPU parity for the one-tree algorithms (Section 1.2's single doubly-
pipelined tree, Section 2's reduce-then-broadcast) and for the
round-structured executors, whose per-round state is checked against the
round in which the oracle's simulations make every block of every rank
final (Section 1.1's induction).  Expected values come from the oracle only.
"""

import numpy as np
import pytest
import torch

import oracle
import synth
from tests._gpu import (POISON, assert_all_ranks_equal, env_group_blocks,
                        env_unit, env_waves, from_dev, lib, need_gpu, to_dev)

pytestmark = pytest.mark.gpu

ALGS = ["dual", "single", "reduce_bcast"]
EXECS = ["split", "ticket", "launch", "barrier", "rounds", "rounds_barrier"]


def _trees(alg, p):
    return oracle.build_trees(p) if alg == "dual" else \
        oracle.build_trees(p, layout="single")


def _want(x, dtype, op, alg):
    return oracle.allreduce_tree(x, dtype, op, trees=_trees(alg, x.shape[0]))


def _run(x, dtype, op, b, alg, exec, y=None, xs=None, ys=None, r0=0, r1=-1):
    dpar = lib()
    p, m = x.shape[0], x.shape[1]
    xd = to_dev(x) if xs is None else None
    if y is None:
        y = torch.empty_like(xd)
        y.view(torch.int32).fill_(POISON)
    s = torch.cuda.current_stream()
    dpar.dpar_allreduce_opt(dpar.rows(xd) if xs is None else xs,
                            dpar.rows(y) if ys is None else ys, p, m, dtype,
                            op, b, alg, exec, r0, r1, s)
    dpar.dpar_check_status(s)
    return y


def _input(dist, seed, p, m, **kw):
    return synth.generate(dist, seed, p, m, **kw)


@pytest.mark.parametrize("alg", ALGS)
@pytest.mark.parametrize("exec", EXECS)
@pytest.mark.parametrize("unit", ["seq1", "seq2", "level"])
@pytest.mark.parametrize("b", [1, 8, 64])
def test_fp32_every_alg_and_executor(alg, exec, unit, b):
    """seq1 / seq2: the post-order item with one wavefront for both trees
    (the default at p = 36) or one per tree."""
    need_gpu()
    x = _input("normal_f32", 2120, 36, 4099)
    want = _want(x, "float32", "sum", alg)
    waves = {"seq1": 1, "seq2": 2}.get(unit)
    with env_unit("seq" if waves else unit), env_waves(waves):
        out = from_dev(_run(x, "float32", "sum", b, alg, exec), x)
    assert_all_ranks_equal(out, want, f"{alg}/{exec}/{unit}/b={b}")


@pytest.mark.parametrize("alg", ALGS)
@pytest.mark.parametrize("exec", EXECS)
def test_matrix_product_keeps_rank_order(alg, exec):
    need_gpu()
    x = _input("uniform_u32_mat", 2121, 64, 1 << 10)
    want = oracle.allreduce_ltr(x, "u32mat2x2", "matmul")
    out = from_dev(_run(x, "u32mat2x2", "matmul", 32, alg, exec), x)
    assert_all_ranks_equal(out, want, f"{alg}/{exec}")


@pytest.mark.parametrize("alg", ALGS)
@pytest.mark.parametrize("exec", ["split", "rounds", "rounds_barrier"])
@pytest.mark.parametrize("p", [1, 2, 3, 4, 5, 7, 129])
def test_small_and_odd_p(alg, exec, p):
    need_gpu()
    x = _input("normal_f32", 2122 + p, p, 1001)
    want = _want(x, "float32", "sum", alg)
    out = from_dev(_run(x, "float32", "sum", 3, alg, exec), x)
    assert_all_ranks_equal(out, want, f"{alg}/{exec}/p={p}")


@pytest.mark.parametrize("alg", ALGS)
@pytest.mark.parametrize("exec", ["rounds", "rounds_barrier"])
@pytest.mark.parametrize("dtype,op", [("int32", "max"), ("int32", "sum")])
def test_rounds_in_place(alg, exec, dtype, op):
    need_gpu()
    x = _input("uniform_int", 2123, 36, 5000, lo=-1000, hi=1000)
    want = _want(x, dtype, op, alg)
    xd = to_dev(x)
    dpar = lib()
    s = torch.cuda.current_stream()
    dpar.dpar_allreduce_opt(dpar.rows(xd), dpar.rows(xd), 36, 5000, dtype, op,
                            16, alg, exec, 0, -1, s)
    dpar.dpar_check_status(s)
    assert_all_ranks_equal(from_dev(xd, x), want, f"in place {alg}/{exec}")


# ---------------------------------------------------------- round structure

def _final_rounds(x, b, alg):
    """Oracle: round in which block j of rank i becomes final."""
    t = _trees(alg, x.shape[0])
    if alg == "reduce_bcast":
        _, tr = oracle.simulate_reduce_bcast(x, "int32", "sum", b, trees=t)
    else:
        _, tr = oracle.simulate(x, "int32", "sum", b, trees=t)
    return tr.final_round


def _unaligned_rows(t, m):
    """Row addresses 4 bytes into each row of a [p, m + 1] int32 tensor:
    not 16-byte aligned.  With m not a multiple of 4 the round-structured
    executors take one element per lane and the canonical block partition
    [floor(j m / b), floor((j + 1) m / b))."""
    return [a + 4 for a in lib().rows(t)]


@pytest.mark.parametrize("alg", ALGS)
@pytest.mark.parametrize("exec", ["rounds", "rounds_barrier"])
@pytest.mark.parametrize("p,b", [(7, 4), (36, 9), (100, 3)])
def test_state_after_every_round_prefix(alg, exec, p, b):
    """After rounds [0, R') every rank holds exactly the blocks the oracle's
    simulation makes final by round R' - 1, the rest still poisoned; running
    the remaining rounds [R', R) then completes every output."""
    need_gpu()
    dpar = lib()
    m = 257
    x = _input("uniform_int", 2124, p, m, lo=-1000, hi=1000)
    want = oracle.allreduce_tree(x, "int32", "sum", trees=_trees(alg, p))
    final = _final_rounds(x, b, alg)
    R = dpar.dpar_schedule_rounds(p, b, alg)
    assert R == 1 + max(max(v.values()) for v in final.values())
    xpad = np.zeros((p, m + 1), dtype=np.int32)
    xpad[:, 1:] = x
    xd = to_dev(xpad)
    xs = _unaligned_rows(xd, m)
    bounds = [oracle.block_bounds(m, b, j) for j in range(b)]
    s = torch.cuda.current_stream()
    for cut in sorted({0, 1, 2, b // 2, b, b + 1, R - 1, R}):
        if not 0 <= cut <= R:
            continue
        yd = torch.full((p, m + 1), POISON, dtype=torch.int32, device="cuda")
        ys = _unaligned_rows(yd, m)
        dpar.dpar_allreduce_opt(xs, ys, p, m, "int32", "sum", b, alg, exec,
                                0, cut, s)
        dpar.dpar_check_status(s)
        got = yd.cpu().numpy()[:, 1:]
        for i in range(p):
            for j, (lo, hi) in enumerate(bounds):
                if final[i][j] < cut:
                    assert np.array_equal(got[i, lo:hi], want[lo:hi]), \
                        (cut, i, j, "should be final")
                else:
                    assert np.all(got[i, lo:hi] == POISON), \
                        (cut, i, j, "should be untouched")
        dpar.dpar_allreduce_opt(xs, ys, p, m, "int32", "sum", b, alg, exec,
                                cut, -1, s)
        dpar.dpar_check_status(s)
        got = yd.cpu().numpy()[:, 1:]
        assert_all_ranks_equal(got, want, f"{alg}/{exec} cut {cut}")


@pytest.mark.parametrize("alg", ALGS)
def test_rounds_large_p_level_unit(alg):
    """p = 1152 at a reduced m: the level work item in the round-structured
    executor (few chunks per round), every element checked."""
    need_gpu()
    x = _input("normal_f32", 2125, 1152, 1 << 12)
    want = _want(x, "float32", "sum", alg)
    for unit in ("level", "seq"):
        with env_unit(unit):
            out = from_dev(_run(x, "float32", "sum", 16, alg, "rounds"), x)
        assert_all_ranks_equal(out, want, f"{alg}/rounds/{unit}")


@pytest.mark.parametrize("alg", ALGS)
@pytest.mark.parametrize("exec", ["rounds", "rounds_barrier", "barrier"])
@pytest.mark.parametrize("b", [1, 2, 8])
def test_round_executors_large_blocks(alg, exec, b):
    """Blocks of up to 2^20 elements: thousands of work items per round and
    a persistent grid filling every CU, with rounds in which only the
    down-step has work."""
    need_gpu()
    x = _input("uniform_int", 2126, 36, 1 << 20, lo=-(1 << 20), hi=1 << 20)
    want = _want(x, "int32", "sum", alg)
    out = from_dev(_run(x, "int32", "sum", b, alg, exec), x)
    assert_all_ranks_equal(out, want, f"{alg}/{exec}/b={b}")


@pytest.mark.parametrize("alg", ALGS)
@pytest.mark.parametrize("exec", EXECS)
@pytest.mark.parametrize("p", [64, 100, 300, 1152])
def test_subtree_unit(alg, exec, p):
    """The subtree work item (trees cut into subtrees, one wavefront each,
    then the spines): bit-exact fp32 for every algorithm and executor."""
    need_gpu()
    x = _input("normal_f32", 2127 + p, p, 2053)
    want = _want(x, "float32", "sum", alg)
    for b in (1, 5):
        with env_unit("sub"):
            out = from_dev(_run(x, "float32", "sum", b, alg, exec), x)
        assert_all_ranks_equal(out, want, f"sub {alg}/{exec}/p={p}/b={b}")


@pytest.mark.parametrize("dtype,op,dist", [("int32", "max", "uniform_int"),
                                           ("u32mat2x2", "matmul",
                                            "uniform_u32_mat")])
def test_subtree_unit_other_operators(dtype, op, dist):
    need_gpu()
    kw = {"lo": -99, "hi": 99} if dist == "uniform_int" else {}
    x = _input(dist, 2128, 200, 999, **kw)
    want = oracle.allreduce_ltr(x, dtype, op)
    for exec in ("split", "ticket", "rounds"):
        with env_unit("sub"):
            out = from_dev(_run(x, dtype, op, 3, "dual", exec), x)
        assert_all_ranks_equal(out, want, f"sub {dtype}/{exec}")


@pytest.mark.parametrize("m", [(1 << 16) + 1, (1 << 16) + 3])
def test_subtree_unit_chosen_with_a_tail(m):
    """p = 1152, one block: the library picks subtree work items for the
    chunked part; the m mod 4 trailing elements go through a separate
    post-order pass with its own LDS slots."""
    need_gpu()
    x = _input("normal_f32", 2129, 1152, m)
    want = _want(x, "float32", "sum", "dual")
    with env_unit(None):
        for exec in ("split", "ticket"):
            out = from_dev(_run(x, "float32", "sum", 1, "dual", exec), x)
            assert_all_ranks_equal(out, want, f"auto unit {exec} m={m}")


@pytest.mark.parametrize("p,m", [(2304, 1 << 14), (4608, 1 << 14),
                                 (4608, (1 << 13) + 3), (1152, 1 << 14)])
def test_unit_rule_at_large_p(p, m):
    """The library's own work-item choice where a level plan would need
    more than two items per CU (p = 2304 and 4608: subtree items) and where
    it would not (p = 1152: level items), for the block rule and b = 1."""
    need_gpu()
    x = _input("normal_f32", 2131 + p, p, m)
    want = _want(x, "float32", "sum", "dual")
    with env_unit(None):
        for b in (1, 0):
            for exec in ("auto", "split", "ticket"):
                out = from_dev(_run(x, "float32", "sum", b, "dual", exec), x)
                assert_all_ranks_equal(out, want, f"{exec}/p={p}/m={m}/b={b}")


@pytest.mark.parametrize("k", [None, 1, 3, 8, 64])
@pytest.mark.parametrize("p,m,b", [(36, 70001, 7), (64, 20483, 1),
                                   (300, 9001, 13)])
def test_ticket_batches(k, p, m, b):
    """The ticket executor with several work items per claim, including
    batch counts that do not divide the number of items: every item is
    evaluated exactly once whatever the batch."""
    need_gpu()
    from tests._gpu import _Env
    x = _input("normal_f32", 2133 + p, p, m)
    want = _want(x, "float32", "sum", "dual")
    with _Env("DPAR_TICKET_BATCH", k):
        out = from_dev(_run(x, "float32", "sum", b, "dual", "ticket"), x)
    assert_all_ranks_equal(out, want, f"ticket k={k} p={p} m={m} b={b}")


@pytest.mark.parametrize("p,m,b", [(288, 875, 1), (1152, 16, 13),
                                   (300, 4099, 3), (97, 2501, 2)])
def test_level_chunk_sizes(p, m, b):
    """Level work items of every chunk size from 1 to 64 quanta (forced),
    the library's own choice included: bit-identical fp32 results."""
    need_gpu()
    from tests._gpu import _Env
    x = _input("normal_f32", 2135 + p, p, m)
    want = _want(x, "float32", "sum", "dual")
    with env_unit("level"):
        for lg in (None, 0, 1, 2, 3, 4, 5, 6):
            with _Env("DPAR_LEVEL_LOG2T", lg):
                for exec in ("auto", "ticket", "launch"):
                    out = from_dev(_run(x, "float32", "sum", b, "dual", exec),
                                   x)
                    assert_all_ranks_equal(out, want,
                                           f"lg={lg} {exec} p={p} m={m}")


@pytest.mark.parametrize("deep", [0, 1])
@pytest.mark.parametrize("p,m,b", [(1152, 16387, 1), (2304, 8192, 3),
                                   (300, 5001, 2), (4099, 4096, 1)])
def test_subtree_unit_load_depths(deep, p, m, b):
    """Subtree work items with 8 and with 16 loads in flight per wavefront
    (forced either way), including a ragged m: bit-identical fp32."""
    need_gpu()
    from tests._gpu import _Env
    x = _input("normal_f32", 2137 + p, p, m)
    want = _want(x, "float32", "sum", "dual")
    with env_unit("sub"), _Env("DPAR_SUB_DEEP", deep):
        for exec in ("split", "ticket", "auto"):
            out = from_dev(_run(x, "float32", "sum", b, "dual", exec), x)
            assert_all_ranks_equal(out, want, f"deep={deep} {exec} p={p}")


_LARGE_P = {}


@pytest.mark.parametrize("p,m", [(2049, 257), (4099, 130), (16384, 64),
                                 (16384, 67), (100003, 37)])
@pytest.mark.parametrize("exec", ["auto", "split", "ticket", "launch",
                                  "rounds"])
@pytest.mark.parametrize("alg", ["dual", "single"])
def test_large_p(p, m, exec, alg):
    """Deeper trees (H up to 15): the LDS slot count, the level table (up to
    p = 65534; at 16384 ranks the level item no longer fits in LDS and the
    library falls back to the post-order item, for the elements after the
    last 16-byte quantum as well; past 65534 ranks there is no level table)
    and the subtree plan."""
    need_gpu()
    key = (p, m, alg)
    if key not in _LARGE_P:    # inputs and oracle results shared by executors
        x = _input("normal_f32", 2160 + p % 97, p, m)
        _LARGE_P[key] = (x, _want(x, "float32", "sum", alg))
    x, want = _LARGE_P[key]
    for b in (1, 3):
        out = from_dev(_run(x, "float32", "sum", b, alg, exec), x)
        assert_all_ranks_equal(out, want, f"{alg}/{exec}/p={p}/b={b}")


@pytest.mark.parametrize("exec", ["auto", "split", "ticket"])
@pytest.mark.parametrize("unit", [None, "seq", "level", "sub"])
@pytest.mark.parametrize("p,m,b", [(1152, 1 << 16, 817), (300, 4099, 1000),
                                   (36, 1 << 10, 103), (7, 16, 13),
                                   (64, 1 << 12, 1024), (129, 5003, 5003)])
def test_grouped_short_blocks(exec, unit, p, m, b):
    """Blocks shorter than half a chunk: the one-launch executors give each
    work item several consecutive whole blocks.  Bit-exact for every work
    item kind, with grouping off (DPAR_GROUP_BLOCKS=0) as well."""
    need_gpu()
    x = _input("normal_f32", 2170 + p, p, m)
    want = _want(x, "float32", "sum", "dual")
    for grouped in (True, False):
        with env_unit(unit), env_group_blocks(grouped):
            out = from_dev(_run(x, "float32", "sum", b, "dual", exec), x)
        assert_all_ranks_equal(out, want,
                               f"{exec}/{unit}/p={p}/m={m}/b={b}/g={grouped}")


@pytest.mark.parametrize("exec", ["split", "ticket"])
def test_grouped_short_blocks_matrix_product(exec):
    need_gpu()
    x = _input("uniform_u32_mat", 2177, 64, 1000)
    want = oracle.allreduce_ltr(x, "u32mat2x2", "matmul")
    out = from_dev(_run(x, "u32mat2x2", "matmul", 300, "dual", exec), x)
    assert_all_ranks_equal(out, want, f"matmul grouped {exec}")


@pytest.mark.parametrize("exec", ["launch", "barrier"])
def test_per_round_executors_take_subtree_items_for_mid_rounds(exec, capfd):
    """p = 256, m = 2^18, b = 2: each round holds 512 full chunks (two per
    CU), so launch per round and the grid barrier run subtree work items
    (the library's choice, shown by DPAR_LOG), bit-exact in fp32."""
    from tests._gpu import _Env
    need_gpu()
    p, m, b = 256, 1 << 18, 2
    x = _input("normal_f32", 2190, p, m)
    want = _want(x, "float32", "sum", "dual")
    with env_unit(None), _Env("DPAR_LOG", 1):
        out = from_dev(_run(x, "float32", "sum", b, "dual", exec), x)
    err = capfd.readouterr().err
    assert "unit=subtree" in err, err[-400:]
    assert_all_ranks_equal(out, want, f"{exec} subtree rounds")


@pytest.mark.parametrize("m,unit", [(1 << 17, "subtree"),
                                    ((1 << 17) + 256, "postorder")])
def test_subtree_item_boundary_two_per_cu(m, unit, capfd):
    """The library's own choice at the boundary of two subtree items per CU
    (256 CUs): p = 1152, m = 2^17 is 512 whole chunks of 64 quanta
    (subtree items, one fused launch); 256 more columns make 513 chunks
    (post-order items, split).  Both at the rule's b, bit-exact in fp32,
    every rank's output."""
    from tests._gpu import _Env
    need_gpu()
    x = _input("normal_f32", 2191, 1152, m)
    want = _want(x, "float32", "sum", "dual")
    with env_unit(None), _Env("DPAR_LOG", 1):
        out = from_dev(_run(x, "float32", "sum", 0, "dual", "auto"), x)
    err = capfd.readouterr().err
    assert f"unit={unit}" in err, err[-400:]
    assert_all_ranks_equal(out, want, f"boundary m={m}")


@pytest.mark.parametrize("alg", ALGS)
@pytest.mark.parametrize("exec", ["auto", "split", "ticket"])
@pytest.mark.parametrize("p", [2, 3, 7, 36, 64, 100, 128])
def test_wide_unit(alg, exec, p, capfd):
    """The wide post-order work item (4 quanta per lane, 4 wavefronts on
    neighbouring columns, each walking both trees): bit-exact fp32 for every
    algorithm and one-launch executor.  m = 4 (3 * 1024 + 300): three whole
    wide items and a ragged fourth (one full wavefront, one partial, two
    without columns).  (Trailing elements: test_wide_unit_choice.)"""
    from tests._gpu import _Env
    need_gpu()
    m = 4 * (3 * 1024 + 300)
    x = _input("normal_f32", 2200 + p, p, m)
    want = _want(x, "float32", "sum", alg)
    for b in (1, 0):
        with env_unit("wide"), _Env("DPAR_LOG", 1):
            out = from_dev(_run(x, "float32", "sum", b, alg, exec), x)
        err = capfd.readouterr().err
        assert "unit=wide " in err, err[-400:]
        assert_all_ranks_equal(out, want, f"wide {alg}/{exec}/p={p}/b={b}")


@pytest.mark.parametrize("dtype,op,dist", [("int32", "max", "uniform_int"),
                                           ("int32", "sum", "uniform_int"),
                                           ("u32mat2x2", "matmul",
                                            "uniform_u32_mat")])
def test_wide_unit_other_operators(dtype, op, dist):
    """Matrices keep the rank order (left-to-right product) through the
    wide item's slots and dual-root combine."""
    need_gpu()
    kw = {"lo": -99, "hi": 99} if dist == "uniform_int" else {}
    x = _input(dist, 2201, 45, 5000, **kw)
    want = oracle.allreduce_ltr(x, dtype, op)
    for exec in ("auto", "split", "ticket"):
        with env_unit("wide"):
            out = from_dev(_run(x, dtype, op, 3, "dual", exec), x)
        assert_all_ranks_equal(out, want, f"wide {dtype}/{exec}")


@pytest.mark.parametrize("exec", ["auto", "split", "ticket"])
@pytest.mark.parametrize("p", [2, 37, 300])
def test_wide_tail_items(exec, p, capfd):
    """Columns past the last whole round of full wide items go to tail items
    (one quantum per lane, 8 visits in flight).  Rounds forced to 4 items
    (DPAR_WIDE_ROUND): m = 4 (5 * 1024 + 300) is 4 full items, then 1324
    quanta in five whole tail items and a ragged sixth (44 quanta, part of
    one wavefront).  Bit-exact fp32 for both trees and for one tree, every
    rank's output."""
    from tests._gpu import _Env
    need_gpu()
    m = 4 * (5 * 1024 + 300)
    x = _input("normal_f32", 2207 + p, p, m)
    for alg in ("dual", "single"):
        want = _want(x, "float32", "sum", alg)
        with env_unit("wide"), _Env("DPAR_LOG", 1), _Env("DPAR_WIDE_ROUND", 4):
            out = from_dev(_run(x, "float32", "sum", 0, alg, exec), x)
        err = capfd.readouterr().err
        assert "unit=wide " in err and " full_items=4" in err, err[-400:]
        assert " items=10" in err, err[-400:]
        assert_all_ranks_equal(out, want, f"wide tail {alg}/{exec}/p={p}")


@pytest.mark.parametrize("dtype,op,dist", [("int32", "max", "uniform_int"),
                                           ("u32mat2x2", "matmul",
                                            "uniform_u32_mat")])
def test_wide_tail_items_other_operators(dtype, op, dist, capfd):
    """Tail items keep the rank order of the matrix product: p = 45,
    m = 5000 (5000 quanta of 16 bytes for the matrices) in rounds of 2
    items: 4 full items, then 904 quanta in 4 tail items (three whole, one
    of 136 quanta)."""
    from tests._gpu import _Env
    need_gpu()
    kw = {"lo": -99, "hi": 99} if dist == "uniform_int" else {}
    x = _input(dist, 2208, 45, 5000 if dtype == "u32mat2x2" else 20000, **kw)
    want = oracle.allreduce_ltr(x, dtype, op)
    for exec in ("auto", "split", "ticket"):
        with env_unit("wide"), _Env("DPAR_LOG", 1), _Env("DPAR_WIDE_ROUND", 2):
            out = from_dev(_run(x, dtype, op, 3, "dual", exec), x)
        err = capfd.readouterr().err
        assert " full_items=4" in err and " items=8" in err, err[-400:]
        assert_all_ranks_equal(out, want, f"wide tail {dtype}/{exec}")


@pytest.mark.parametrize("p,n,unit,full", [
    (36, 264, "wide", 256),        # two fit per CU by LDS; rounds of 256
    (36, 519, "wide", 512),        # a short tail after two rounds
    (36, 504, "wide", 504),        # over 7/8 of a round: no tail items
    (128, 264, "wide", 256),
    (128, 448, "wide", 256),       # 3/4 of a round in tail items
])
def test_wide_tail_choice(p, n, unit, full, capfd):
    """The library's own choice (256 CUs): int32 SUM with rows of n wide
    chunks (16 KB each), split.  Full items in whole rounds of one per CU
    and tail items past them unless those fill more than 7/8 of a round
    (shown by DPAR_LOG); bit-exact against the oracle."""
    from tests._gpu import _Env
    need_gpu()
    m = 4096 * n
    x = _input("uniform_int", 2209, p, m, lo=-1000, hi=1000)
    want = oracle.allreduce_ltr(x, "int32", "sum")
    with env_unit(None), _Env("DPAR_LOG", 1):
        out = from_dev(_run(x, "int32", "sum", 0, "dual", "auto"), x)
    err = capfd.readouterr().err
    assert f"unit={unit} " in err and "exec=split " in err, err[-400:]
    if full is not None:
        assert f" full_items={full}" in err, err[-400:]
    assert_all_ranks_equal(out, want, f"tail choice p={p} n={n}")


F, S = "one_launch_fused", "split"


@pytest.mark.parametrize("p,n", [(12, 401), (20, 480), (8, 300)])
def test_fused_wide_calls_of_few_ranks_take_full_items(p, n, capfd):
    """A fused launch of at most two wide items per CU with at most 20
    ranks runs full items only (no tail items; DPAR_LOG shows
    full_items = items); bit-exact against the oracle."""
    from tests._gpu import _Env
    need_gpu()
    m = 4096 * n + 4
    x = _input("uniform_int", 2211, p, m, lo=-1000, hi=1000)
    want = oracle.allreduce_ltr(x, "int32", "sum")
    with env_unit(None), _Env("DPAR_LOG", 1):
        out = from_dev(_run(x, "int32", "sum", 0, "dual", "auto"), x)
    err = capfd.readouterr().err
    assert "unit=wide " in err and f"exec={F} " in err, err[-400:]
    assert f" items={n + 1} full_items={n + 1}" in err, err[-400:]
    assert_all_ranks_equal(out, want, f"fused full items p={p} n={n}")


@pytest.mark.parametrize("p,m,b,dtype,unit,ex", [
    (36, 1 << 20, 0, "int32", "wide", F),         # 256 wide items
    (36, (1 << 20) + 3, 0, "int32", "wide", F),   # and 3 trailing elements
    (36, 1 << 21, 0, "int32", "wide", S),         # two items per CU
    (8, 1 << 22, 0, "int32", "wide", F),          # four per CU, 8 ranks
    (9, 1 << 22, 0, "int32", "wide", S),
    (36, 4 * (255 * 1024), 0, "int32", "wide", F),  # 3/4 of an item per CU
    (36, 4 * (191 * 1024), 0, "int32", "postorder", S),  # fewer: post-order
    (128, 4 * (192 * 1024), 0, "int32", "wide", S),
    (128, 4 * (191 * 1024), 0, "int32", "postorder", S),
    # post-order items on short rows in one fused launch: rows of at most
    # 3.5 MB up to 16 ranks, 2.5 MB up to 48, 1.5 MB up to 64, 1 MB up to
    # 96, 512 KB beyond
    (48, 5 << 17, 0, "int32", "postorder", F),
    (48, (5 << 17) + 4, 0, "int32", "postorder", S),
    (16, 4 * (192 * 1024), 0, "int32", "postorder", F),  # 7/8 with p <= 16
    (16, 4 * (224 * 1024), 0, "int32", "wide", F),
    (64, 3 << 17, 0, "int32", "postorder", F),
    (64, (3 << 17) + 4, 0, "int32", "postorder", S),
    (96, 1 << 18, 0, "int32", "postorder", F),
    (96, (1 << 18) + 4, 0, "int32", "postorder", S),
    (97, 1 << 18, 0, "int32", "postorder", S),
    (37, 1 << 20, 0, "int32", "wide", S),
    (48, 1 << 20, 0, "int32", "wide", S),
    (16, 4 * (384 * 1024), 0, "int32", "wide", F),  # two per CU, 20 ranks
    (20, 4 * (448 * 1024), 0, "int32", "wide", F),
    (21, 4 * (448 * 1024), 0, "int32", "wide", S),
    (16, 4 * (520 * 1024), 0, "int32", "wide", S),  # more than two per CU
    (8, 4 * (520 * 1024), 0, "int32", "wide", F),
    (128, 1 << 20, 0, "int32", "wide", S),
    (300, 1 << 20, 0, "int32", "wide", S),
    (64, 1 << 18, 0, "u32mat2x2", "wide", S),     # the 64-rank matrix product
    # more ranks, short rows: post-order items fused on rows of at most
    # 512 KB
    (200, 1 << 17, 0, "int32", "postorder", F),
    (200, (1 << 17) + 4, 0, "int32", "postorder", S),
    # level items fused below 512 ranks, split from 1024 on and from 512
    # on with at least one item per CU; subtree items instead of more level
    # items than CUs
    (511, 16384, 0, "int32", "level", F),
    (400, 12288, 0, "int32", "level", F),
    (400, 16384, 0, "int32", "subtree", F),
    (700, 8192, 0, "int32", "level", S),
    (1152, 4096, 0, "int32", "level", S),
    (1152, 1024, 0, "int32", "level", S),
    (2304, 1024, 0, "int32", "level", S),
    # subtree items fused from a quarter of an item per CU on
    (1152, 16384, 0, "int32", "subtree", F),
    (4608, 12288, 0, "int32", "subtree", S),
    # from 2048 ranks on level items up to four per CU, then subtree items
    (2304, 4096, 0, "int32", "level", S),
    (2304, 8192, 0, "int32", "subtree", S),
    # from 4096 ranks on subtree items up to four per CU, split beyond two
    (4096, 196608, 0, "int32", "subtree", S),
])
def test_wide_unit_choice(p, m, b, dtype, unit, ex, capfd):
    """The library's own choice under AUTO (256 CUs): wide items where their
    slots fit in LDS, at least 3/4 of a wide item per CU (7/8 up to 16
    ranks) and no residency
    cap for post-order items, post-order items otherwise; wide items of at
    most 36 ranks and one item per CU, of at most 20 ranks and two per CU,
    or of at most 8 ranks, in one fused launch, else split; post-order items
    in one fused launch on short rows; level items fused with few ranks and
    split with many (shown by DPAR_LOG); bit-exact against the oracle."""
    from tests._gpu import _Env
    need_gpu()
    if dtype == "u32mat2x2":
        x = _input("uniform_u32_mat", 2202, p, m)
        op = "matmul"
    else:
        x = _input("uniform_int", 2203, p, m, lo=-1000, hi=1000)
        op = "sum"
    want = oracle.allreduce_ltr(x, dtype, op)
    with env_unit(None), _Env("DPAR_LOG", 1):
        out = from_dev(_run(x, dtype, op, b, "dual", "auto"), x)
    err = capfd.readouterr().err
    assert f"unit={unit} " in err, err[-400:]
    assert f"exec={ex} " in err, err[-400:]
    assert_all_ranks_equal(out, want, f"choice p={p} m={m} b={b}")


def test_wide_unit_needs_its_slots_in_lds(capfd):
    """p = 1024: the four wavefronts' depth slots (10 per wavefront, 16 KB
    each) exceed the LDS a workgroup may use, so a forced wide item falls
    back to the post-order item, bit-exact."""
    from tests._gpu import _Env
    need_gpu()
    x = _input("normal_f32", 2205, 1024, 8192)
    want = _want(x, "float32", "sum", "dual")
    for exec in ("split", "auto"):
        with env_unit("wide"), _Env("DPAR_LOG", 1):
            out = from_dev(_run(x, "float32", "sum", 1, "dual", exec), x)
        err = capfd.readouterr().err
        assert "unit=wide " not in err, err[-400:]
        assert_all_ranks_equal(out, want, f"p=1024 wide fallback {exec}")


def test_wide_unit_not_under_the_residency_cap(capfd):
    """p = 256, m = 2^22 int32 (rows of 16 MB), the rule's b = 5793: the
    split up-phase has 17379 post-order items, more than 64 per CU, and
    runs them under its residency cap rather than taking wide items (shown
    by DPAR_LOG).  Every output row equals row 0 (checked on the device),
    row 0 equals the oracle."""
    from tests._gpu import _Env
    need_gpu()
    p, m = 256, 1 << 22
    x = _input("uniform_int", 2206, p, m, lo=-1000, hi=1000)
    want = oracle.allreduce_ltr(x, "int32", "sum")
    xd = to_dev(x)
    del x
    y = torch.empty_like(xd)
    y.view(torch.int32).fill_(POISON)
    dpar = lib()
    st = torch.cuda.current_stream()
    with env_unit(None), _Env("DPAR_LOG", 1):
        dpar.dpar_allreduce_opt(dpar.rows(xd), dpar.rows(y), p, m, "int32",
                                "sum", 0, "dual", "auto", 0, -1, st)
        dpar.dpar_check_status(st)
    err = capfd.readouterr().err
    assert "unit=postorder " in err, err[-400:]
    assert bool((y == y[0:1]).all().item()), "rows differ"
    np.testing.assert_array_equal(y[0].cpu().numpy(), want)


@pytest.mark.parametrize("exec", ["auto", "split", "ticket"])
def test_wide_unit_on_misaligned_rows(exec, capfd):
    """The library's own choice on rows 4 bytes past a 16-byte boundary, one
    row per separate allocation (16-byte lanes at 4-byte aligned addresses;
    the broadcast then shifts each output row to its own 4 KB boundary):
    p = 40, m = 2^20 + 5 (5 trailing elements), wide items, bit-exact."""
    from tests._gpu import _Env
    need_gpu()
    dpar = lib()
    p, m = 40, (1 << 20) + 5
    x = _input("normal_f32", 2207, p, m)
    want = _want(x, "float32", "sum", "dual")
    xb = [torch.empty(m + 8, dtype=torch.float32, device="cuda")
          for _ in range(p)]
    yb = [torch.full((m + 8,), float("nan"), dtype=torch.float32,
                     device="cuda") for _ in range(p)]
    for i in range(p):
        xb[i][1:1 + m] = torch.from_numpy(np.ascontiguousarray(x[i])).cuda()
    xs = [t.data_ptr() + 4 for t in xb]
    ys = [t.data_ptr() + 4 for t in yb]
    s = torch.cuda.current_stream()
    with env_unit(None), _Env("DPAR_LOG", 1):
        dpar.dpar_allreduce_opt(xs, ys, p, m, "float32", "sum", 0, "dual",
                                exec, 0, -1, s)
        dpar.dpar_check_status(s)
    err = capfd.readouterr().err
    assert "unit=wide " in err, err[-400:]
    got = np.stack([t[1:1 + m].cpu().numpy() for t in yb])
    assert_all_ranks_equal(got, want, f"wide misaligned {exec}")
    for t in yb:  # nothing written outside the m elements
        assert bool(torch.isnan(t[0]).item())
        assert bool(torch.isnan(t[1 + m:]).all().item())
