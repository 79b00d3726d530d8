"""Rendezvous simulation of the pipelined reduce-then-broadcast (Section 2).

Oracle module: test infrastructure only.

Section 2 compares the dual-root algorithm with User-Allreduce1: a pipelined
reduction to the root of ONE binary tree followed by a pipelined broadcast
from that root, both with the same b blocks.  Section 1.2 prices it at
2(2h + 2(b - 1)) steps.  The paper gives no code for it; this module states
the plain reading used here, on the single post-order tree of
``build_trees(p, layout="single")``, with one-directional messages:

Reduction, rounds j = 0 .. b-1 (global round j):
  receive the partial block j from child0, Y[j] <- t (.) Y[j]; the same with
  child1; a non-root then sends Y[j] to its parent.  The root's Y[j] is final.

Broadcast, rounds k = 0 .. b + H - 2 (global round b + k), as in the
down-going half of Algorithm 1:
  send Y[k - d_i] to child0 and to child1 (the block received one round
  earlier; the root sends block k), then, for a non-root, receive block
  k - (d_i - 1) from the parent.

Blocks outside [0, b) are not sent.  So a rank at depth d >= 1 receives the
final block j in global round b + j + d - 1 and the call takes 2b + H - 1
rounds (b for p = 1).  A scheduler pairs the k-th message from A to B with
the k-th receive posted by B for A and checks that both name the same phase,
round and block.  The association of every product is the single tree's
S(i) = S(child1) (.) (S(child0) (.) x_i).
"""

from collections import deque
from dataclasses import dataclass, field
from typing import Dict, List

from .algorithm1 import DeadlockError, ProtocolError
from .blocks import block_bounds
from .ops import combine
from .trees import build_trees


@dataclass
class Msg:
    partner: int
    send: bool           # True: this rank sends; False: it receives
    phase: str           # "reduce" or "bcast"
    round: int           # global round
    block: int
    payload: object = None


@dataclass
class RBTrace:
    """``final_round[i][j]``: global round in which rank i's block j took its
    final value.  ``ops_per_round[i][r]``: operator applications of rank i in
    global round r.  ``messages[i]``: messages rank i sent."""
    final_round: Dict[int, Dict[int, int]] = field(default_factory=dict)
    ops_per_round: Dict[int, Dict[int, int]] = field(default_factory=dict)
    messages: Dict[int, int] = field(default_factory=dict)
    rounds_used: List[int] = field(default_factory=list)

    def global_rounds(self) -> int:
        return (max(self.rounds_used) + 1) if self.rounds_used else 0


def simulate_reduce_bcast(x, dtype: str, op: str, b: int, trees=None):
    """Run the reduce-then-broadcast for all ranks.  Returns (Y, trace)."""
    rows = [x[i].copy() for i in range(len(x))]
    p = len(rows)
    m = rows[0].shape[0]
    t = trees if trees is not None else build_trees(p, layout="single")
    if len(t.roots) != 1:
        raise ValueError("reduce-then-broadcast runs on one tree")
    if not (0 < b <= max(m, 1)):
        raise ValueError("need 0 < b <= m")
    H = t.height
    trace = RBTrace()

    def blk(j):
        return block_bounds(m, b, j)

    def used(r):
        trace.rounds_used.append(r)

    def program(i):
        Y = rows[i]
        d = t.depth[i]
        children = [c for c in (t.child0[i], t.child1[i]) if c is not None]
        par = t.parent[i]
        for j in range(b):                                  # reduction
            bb = blk(j)
            for c in children:
                got = yield Msg(c, False, "reduce", j, j)
                Y[bb[0]:bb[1]] = combine(dtype, op, got, Y[bb[0]:bb[1]])
                o = trace.ops_per_round.setdefault(i, {})
                o[j] = o.get(j, 0) + 1
                used(j)
            if par is None:
                trace.final_round.setdefault(i, {})[j] = j
                used(j)
            else:
                yield Msg(par, True, "reduce", j, j, Y[bb[0]:bb[1]].copy())
                trace.messages[i] = trace.messages.get(i, 0) + 1
                used(j)
        for k in range(b + H - 1 if H > 0 else 0):          # broadcast
            r = b + k
            s_j = k - d
            if 0 <= s_j < b:
                bb = blk(s_j)
                for c in children:
                    yield Msg(c, True, "bcast", r, s_j, Y[bb[0]:bb[1]].copy())
                    trace.messages[i] = trace.messages.get(i, 0) + 1
                    used(r)
            r_j = k - (d - 1)
            if par is not None and 0 <= r_j < b:
                got = yield Msg(par, False, "bcast", r, r_j)
                bb = blk(r_j)
                Y[bb[0]:bb[1]] = got
                trace.final_round.setdefault(i, {})[r_j] = r
                used(r)

    gens = {i: program(i) for i in range(p)}
    pending: Dict[int, Msg] = {}

    def advance(i, value):
        try:
            pending[i] = gens[i].send(value)
        except StopIteration:
            pending.pop(i, None)

    for i in range(p):
        advance(i, None)
    ready = deque(range(p))
    while ready:
        i = ready.popleft()
        a = pending.get(i)
        if a is None:
            continue
        o = pending.get(a.partner)
        if o is None or o.partner != i or o.send == a.send:
            continue
        if (a.phase, a.round, a.block) != (o.phase, o.round, o.block):
            raise ProtocolError(
                f"ranks {i} and {a.partner} disagree: {a.phase}@{a.round} "
                f"block {a.block} vs {o.phase}@{o.round} block {o.block}")
        snd = a if a.send else o
        s_rank = i if a.send else a.partner
        r_rank = a.partner if a.send else i
        advance(s_rank, None)
        advance(r_rank, snd.payload)
        ready.append(i)
        ready.append(a.partner)

    if pending:
        raise DeadlockError({i: (r.partner, r.phase, r.round)
                             for i, r in pending.items()})
    return rows, trace
