"""Literal rendezvous simulation of Algorithm 1 (Section 1.1).

Oracle module: test infrastructure only.

Every virtual rank runs the per-processor program of Algorithm 1 as a Python
generator on its own pipelining array Y (initialised to x_i) and a temporary
t.  Each communication step is a telephone-model bidirectional exchange: the
rank yields (partner, kind, round, block it sends) and is resumed with the
block the partner sent.  A scheduler pairs the k-th exchange of A with B with
the k-th exchange of B with A (the order MPI's Sendrecv matching would
impose) and checks that both sides are in the same round and agree on the
kind of step.  Nothing is reordered: a rank only advances when its partner
is ready.

Per round j = 0 .. b + d_i the program is:

1. with child0: send Y[j - (d_i + 1)], receive t, then Y[j] <- t (.) Y[j];
2. with child1: the same;
3. a root exchanges Y[j] with its dual and combines, the lower-numbered root
   as Y[j] (.) t and the higher one as t (.) Y[j]; any other rank sends Y[j]
   to its parent and receives Y[j - d_i] from it.

Blocks outside [0, b) are the paper's zero-element virtual blocks.  With
``skip_void=True`` an exchange in which both the sent and the received block
are virtual is not performed (Section 1.3: the implementation sends and
receives zero-element blocks and stops after the last non-empty block from
the parent, so such exchanges carry nothing).  With ``skip_void=False`` the
loop bound is taken literally and every exchange is attempted; the scheduler
then reports the deadlock this causes.

``fail=(rank, round)`` stops one rank at the start of that round, to show
which ranks the blocking exchanges leave stuck.
"""

from collections import deque
from dataclasses import dataclass, field
from typing import Dict, List, Optional

from .blocks import block_bounds
from .ops import combine
from .trees import build_trees


class DeadlockError(RuntimeError):
    """Raised when no pending exchange can be paired.  ``blocked`` maps each
    stuck rank to (partner, kind, round)."""

    def __init__(self, blocked):
        self.blocked = blocked
        super().__init__(f"deadlock: {len(blocked)} ranks blocked: "
                         f"{sorted(blocked.items())[:8]}")


class ProtocolError(RuntimeError):
    pass


@dataclass
class _Req:
    partner: int
    kind: str            # "child", "parent" or "dual" (the step's role)
    round: int
    send_j: int          # index of the block sent (may be virtual)
    recv_j: int          # index of the block expected back
    payload: object      # array or None for a virtual block


@dataclass
class Trace:
    """What the simulation recorded, per rank.  ``final_round[i][k]`` is the
    round in which block k of rank i took its final value y[k]: for a
    non-root the round of the parent exchange that delivered it, for a root
    the round in which it finished Y[k] (after the dual exchange, if any)."""
    active_rounds: Dict[int, List[int]] = field(default_factory=dict)
    exchanges: Dict[int, int] = field(default_factory=dict)
    ops_per_round: Dict[int, Dict[int, int]] = field(default_factory=dict)
    steps_per_round: Dict[int, Dict[int, int]] = field(default_factory=dict)
    final_round: Dict[int, Dict[int, int]] = field(default_factory=dict)
    # per rank, every exchange in order: (round, kind, partner, block sent,
    # block received), a block index None where it is virtual
    exchange_log: Dict[int, List[tuple]] = field(default_factory=dict)

    def span(self, i: int) -> int:
        r = self.active_rounds.get(i, [])
        return (r[-1] - r[0] + 1) if r else 0

    def global_rounds(self) -> int:
        last = [r[-1] for r in self.active_rounds.values() if r]
        return (max(last) + 1) if last else 0


def simulate(x, dtype: str, op: str, b: int, trees=None,
             skip_void: bool = True, fail=None):
    """Run Algorithm 1 for all ranks.  Returns (Y, trace) where Y[i] is rank
    i's final array."""
    rows = [x[i].copy() for i in range(len(x))]
    p = len(rows)
    m = rows[0].shape[0]
    t = trees if trees is not None else build_trees(p)
    if not (0 < b <= max(m, 1)):
        raise ValueError("need 0 < b <= m")
    trace = Trace()

    def blk(j):
        return block_bounds(m, b, j)

    def note(i, j, ops, steps):
        ar = trace.active_rounds.setdefault(i, [])
        if not ar or ar[-1] != j:
            ar.append(j)
        trace.exchanges[i] = trace.exchanges.get(i, 0) + steps
        o = trace.ops_per_round.setdefault(i, {})
        o[j] = o.get(j, 0) + ops
        s = trace.steps_per_round.setdefault(i, {})
        s[j] = s.get(j, 0) + steps

    def take(Y, j):
        bb = blk(j)
        return None if bb is None else Y[bb[0]:bb[1]].copy()

    def log(i, j, kind, partner, s_j, r_j):
        trace.exchange_log.setdefault(i, []).append(
            (j, kind, partner, s_j if blk(s_j) is not None else None,
             r_j if blk(r_j) is not None else None))

    def program(i):
        Y = rows[i]                                    # Y <- x_i
        d = t.depth[i]
        for j in range(0, b + d + 1):
            if fail is not None and fail == (i, j):
                return
            for c in (t.child0[i], t.child1[i]):
                if c is None:
                    continue
                s_j, r_j = j - (d + 1), j
                if skip_void and blk(s_j) is None and blk(r_j) is None:
                    continue
                got = yield _Req(c, "child", j, s_j, r_j, take(Y, s_j))
                log(i, j, "child", c, s_j, r_j)
                bb = blk(r_j)
                ops = 0
                if bb is not None:
                    Y[bb[0]:bb[1]] = combine(dtype, op, got, Y[bb[0]:bb[1]])
                    ops = 1
                note(i, j, ops, 1)
            if t.parent[i] is None:
                q = t.dual[i]
                if q is None:
                    # a root without a dual has Y[j] complete now
                    if blk(j) is not None:
                        trace.final_round.setdefault(i, {})[j] = j
                    continue
                if skip_void and blk(j) is None:
                    continue
                got = yield _Req(q, "dual", j, j, j, take(Y, j))
                log(i, j, "dual", q, j, j)
                bb = blk(j)
                ops = 0
                if bb is not None:
                    mine = Y[bb[0]:bb[1]]
                    Y[bb[0]:bb[1]] = (combine(dtype, op, mine, got) if i < q
                                      else combine(dtype, op, got, mine))
                    ops = 1
                    trace.final_round.setdefault(i, {})[j] = j
                note(i, j, ops, 1)
            else:
                s_j, r_j = j, j - d
                if skip_void and blk(s_j) is None and blk(r_j) is None:
                    continue
                got = yield _Req(t.parent[i], "parent", j, s_j, r_j,
                                take(Y, s_j))
                log(i, j, "parent", t.parent[i], s_j, r_j)
                bb = blk(r_j)
                if bb is not None:
                    Y[bb[0]:bb[1]] = got
                    trace.final_round.setdefault(i, {})[r_j] = j
                note(i, j, 0, 1)

    gens = {i: program(i) for i in range(p)}
    pending: Dict[int, Optional[_Req]] = {}

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
        req = pending.get(i)
        if req is None:
            continue
        other = pending.get(req.partner)
        if other is None or other.partner != i:
            continue
        pair = {req.kind, other.kind}
        if req.round != other.round or pair not in ({"child", "parent"},
                                                     {"dual"}):
            raise ProtocolError(
                f"ranks {i} and {req.partner} disagree: {req.kind}@{req.round}"
                f" vs {other.kind}@{other.round}")
        if req.send_j != other.recv_j or other.send_j != req.recv_j:
            raise ProtocolError(
                f"ranks {i} and {req.partner} exchange mismatched blocks in "
                f"round {req.round}")
        q = req.partner
        a, bpay = req.payload, other.payload
        advance(i, bpay)
        advance(q, a)
        ready.append(i)
        ready.append(q)

    if pending:
        raise DeadlockError({i: (r.partner, r.kind, r.round)
                             for i, r in pending.items()})
    return rows, trace

