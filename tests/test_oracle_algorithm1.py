"""Pins that tie the oracle's closed-form tree evaluation to a literal
round-by-round simulation of Algorithm 1 (Section 1.1), and the simulation
to the paper's counts.

The simulation and the tree evaluation are two independent formulations:
one moves blocks between ranks in rounds with telephone-model exchanges, the
other evaluates subtree products recursively.  Agreement is bit-exact,
including fp32.
"""

import numpy as np
import pytest

import synth
from oracle import (DeadlockError, allreduce_tree, block_bounds, build_trees,
                    simulate)

PS = [1, 2, 3, 5, 6, 7, 14, 30, 36, 64, 100]
BS = [1, 2, 4, 7]


@pytest.mark.parametrize("p", PS)
@pytest.mark.parametrize("b", BS)
def test_simulation_equals_tree_evaluation_fp32(p, b):
    m = 23
    x = synth.generate("normal_f32", 40 + p, p, m)
    Y, _ = simulate(x, "float32", "sum", b)
    y = allreduce_tree(x, "float32", "sum")
    for i in range(p):
        assert np.array_equal(Y[i], y), i


@pytest.mark.parametrize("p", [2, 3, 7, 9, 36])
def test_simulation_equals_tree_evaluation_matmul(p):
    x = synth.generate("odd_det_u32_mat", 50 + p, p, 9)
    Y, _ = simulate(x, "u32mat2x2", "matmul", 3)
    y = allreduce_tree(x, "u32mat2x2", "matmul")
    for i in range(p):
        assert np.array_equal(Y[i], y), i


@pytest.mark.parametrize("p", PS)
@pytest.mark.parametrize("b", BS)
def test_round_spans(p, b):
    # Each rank works in b + d_i rounds (Section 1.1); counting the rounds in
    # which a rank performs a non-empty exchange gives b + d_i for leaves,
    # one more for a non-leaf (its last round only sends Y[b-1] down), b for
    # a root without children, and b + H overall.
    x = np.zeros((p, 2 * b + 1), dtype=np.int32)
    _, tr = simulate(x, "int32", "sum", b)
    t = build_trees(p)
    for i in range(p):
        leaf = t.child0[i] is None
        if p == 1:
            want = 0
        elif leaf and t.parent[i] is None:
            want = b
        elif leaf:
            want = b + t.depth[i]
        else:
            want = b + t.depth[i] + 1
        assert tr.span(i) == want, (i, tr.active_rounds.get(i))
    assert tr.global_rounds() == (0 if p == 1 else b + t.height)


def test_p7_b4_schedule_table():
    # Hand-derived for p = 7, b = 4: rank 1 (depth 1, child 0) in round 2
    # exchanges with child 0 (sends Y[0], receives Y[2]) and then with its
    # parent (sends Y[2], receives Y[1]); in round 5 it only sends Y[3] down.
    x = np.zeros((7, 8), dtype=np.int32)
    _, tr = simulate(x, "int32", "sum", 4)
    assert tr.active_rounds[1] == [0, 1, 2, 3, 4, 5]
    assert tr.steps_per_round[1][2] == 2 and tr.steps_per_round[1][5] == 1
    assert tr.active_rounds[0] == [0, 1, 2, 3, 4, 5]
    assert tr.active_rounds[2] == [0, 1, 2, 3, 4]
    assert tr.active_rounds[3] == [0, 1, 2, 3, 4]
    assert tr.global_rounds() == 6


def test_leaf_rounds_have_holes_when_b_below_depth():
    # p = 7, b = 1: the depth-2 leaf sends Y[0] in round 0, is idle in
    # round 1 and receives y's only block in round 2.
    x = np.zeros((7, 3), dtype=np.int32)
    _, tr = simulate(x, "int32", "sum", 1)
    assert tr.active_rounds[0] == [0, 2]


@pytest.mark.parametrize("p", [7, 36, 100])
def test_step_and_operator_counts_per_round(p):
    # at most three exchanges per round; at most two (.) per round for a
    # non-root and three for a root (Sections 1.1 and 1.2)
    b = 5
    x = np.zeros((p, 11), dtype=np.int32)
    _, tr = simulate(x, "int32", "sum", b)
    t = build_trees(p)
    for i in range(p):
        assert max(tr.steps_per_round[i].values()) <= 3
        cap = 3 if t.parent[i] is None else 2
        assert max(tr.ops_per_round[i].values()) <= cap
    # a root with two children applies (.) three times in a full round
    assert tr.ops_per_round[t.roots[0]][1] == 3


@pytest.mark.parametrize("p", [3, 7, 36])
def test_literal_loop_bound_deadlocks(p):
    # Running j = 0 .. b + d_i literally, a leaf's last round has no partner
    x = np.zeros((p, 8), dtype=np.int32)
    with pytest.raises(DeadlockError) as e:
        simulate(x, "int32", "sum", 4, skip_void=False)
    t = build_trees(p)
    deepest = max(range(p), key=lambda i: t.depth[i])
    assert deepest in e.value.blocked


def test_failed_rank_blocks_its_neighbours():
    # a rank that stops leaves its parent waiting in the up-phase and its
    # children waiting for result blocks
    p, b = 15, 4
    t = build_trees(p)
    victim = next(i for i in range(p)
                  if t.parent[i] is not None and t.child0[i] is not None)
    x = np.zeros((p, 8), dtype=np.int32)
    with pytest.raises(DeadlockError) as e:
        simulate(x, "int32", "sum", b, fail=(victim, 1))
    blocked = e.value.blocked
    assert t.parent[victim] in blocked
    assert t.child0[victim] in blocked
    assert victim not in blocked


def test_result_does_not_depend_on_blocking():
    p, m = 30, 37
    x = synth.generate("normal_f32", 77, p, m)
    outs = [simulate(x, "float32", "sum", b)[0][0] for b in (1, 3, 8, 37)]
    assert all(np.array_equal(o, outs[0]) for o in outs)


def test_block_bounds():
    for m in (1, 7, 1000, 4097):
        for b in (1, 2, 3, 7, m):
            if b > m:
                continue
            sizes = [block_bounds(m, b, j)[1] - block_bounds(m, b, j)[0]
                     for j in range(b)]
            assert sum(sizes) == m
            assert max(sizes) - min(sizes) <= 1
            assert min(sizes) >= 1
            assert block_bounds(m, b, -1) is None
            assert block_bounds(m, b, b) is None


def test_p7_b4_rank1_exchanges():
    """Rank 1 (depth 1, one child: rank 0, parent: rank 3) at b = 4, from
    Algorithm 1's steps: in round j it exchanges with child0 (sends
    Y[j - 2], receives Y[j]) and then with its parent (sends Y[j], receives
    Y[j - 1]); blocks outside [0, 4) are virtual.  Round 2 is therefore
    (child: send 0, receive 2), (parent: send 2, receive 1), and round 5
    only sends Y[3] to the child."""
    x = np.zeros((7, 8), dtype=np.int32)
    _, tr = simulate(x, "int32", "sum", 4)
    log = tr.exchange_log[1]
    by_round = {}
    for (j, kind, partner, sj, rj) in log:
        by_round.setdefault(j, []).append((kind, partner, sj, rj))
    assert by_round[2] == [("child", 0, 0, 2), ("parent", 3, 2, 1)]
    assert by_round[5] == [("child", 0, 3, None)]
    assert by_round[0] == [("child", 0, None, 0), ("parent", 3, 0, None)]
    assert sorted(by_round) == [0, 1, 2, 3, 4, 5]
