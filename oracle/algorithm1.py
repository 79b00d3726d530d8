"""Round-by-round simulation of the doubly-pipelined dual-root schedule
(Section 1.1), stated per tree edge.

Oracle module: test infrastructure only.

What Section 1.1 defines, restated as traffic on the edges of the trees:

* Rank i keeps an array Y of the b blocks, starting as x_i.  Its depth is
  d_i (roots 0, children one deeper than their parent).
* In round j every tree edge (parent q, child c) carries one bidirectional
  exchange.  Upwards goes the child's block j, which by then holds the
  product over the child's whole subtree for that block; the parent folds it
  into its own block j from the left (first child's block first, then the
  second child's), so that S(q) = S(c1) (.) (S(c0) (.) x_q).  Downwards goes
  the parent's block j - d_c, which holds the final result y for that block:
  it reached the parent one round earlier.  The child stores it.
* In round j the two roots exchange block j, once both hold their tree's
  product for it, and both end with y[j] = S(root A) (.) S(root B) (the
  lower-numbered root computes mine (.) received, the other received (.)
  mine).
* Blocks outside [0, b) are empty: an exchange that would move only empty
  blocks carries nothing (Section 1.3 sends and receives zero-element blocks
  and stops after the last real one), and is skipped with
  ``skip_void=True``.

A rank takes its exchanges of a round in the order first child, second
child, then parent (or dual), and its exchanges with a partner are
rendezvous: the simulation processes a round edge by edge from the deepest
edges up, then the root pair, so every block sent up is complete when it
leaves, and every block sent down was made final in an earlier round (this
is checked).  An exchange happens when both ends reach it; a rank whose
partner never takes part (it has stopped, or is itself stuck) waits forever
and takes no further step, and the run ends in a DeadlockError naming every
waiting rank.

``skip_void=False`` has every rank attempt an exchange on each of its edges
in every round j = 0 .. b + d_i, empty or not, as a loop bound of b + d_i
rounds taken literally would: a deepest leaf then attempts round b + d_i
with a parent whose rounds ended one earlier, and waits forever.
``fail=(rank, round)`` stops one rank at the start of that round.

The result is a round-by-round schedule, independent of the recursive
evaluation in ``reduce.allreduce_tree``; the tests compare the two bit for
bit.
"""

from dataclasses import dataclass, field
from typing import Dict, List

from .blocks import block_bounds
from .ops import combine
from .trees import build_trees


class DeadlockError(RuntimeError):
    """Raised when some rank waits for an exchange its partner never takes
    part in.  ``blocked`` maps each waiting rank to (partner, kind, round)."""

    def __init__(self, blocked):
        self.blocked = blocked
        super().__init__(f"deadlock: {len(blocked)} ranks blocked: "
                         f"{sorted(blocked.items())[:8]}")


class ProtocolError(RuntimeError):
    """The schedule would move a block that is not ready."""


@dataclass
class Trace:
    """What the simulation recorded, per rank.  ``final_round[i][k]`` is the
    round in which block k of rank i took its final value y[k]: for a
    non-root the round in which it came down from the parent, for a root the
    round in which it finished Y[k] (after the dual exchange, if any)."""
    active_rounds: Dict[int, List[int]] = field(default_factory=dict)
    exchanges: Dict[int, int] = field(default_factory=dict)
    ops_per_round: Dict[int, Dict[int, int]] = field(default_factory=dict)
    steps_per_round: Dict[int, Dict[int, int]] = field(default_factory=dict)
    final_round: Dict[int, Dict[int, int]] = field(default_factory=dict)
    # per rank, every exchange in the order the rank takes them: (round,
    # kind, partner, block sent, block received), None for an empty block
    exchange_log: Dict[int, List[tuple]] = field(default_factory=dict)

    def span(self, i: int) -> int:
        r = self.active_rounds.get(i, [])
        return (r[-1] - r[0] + 1) if r else 0

    def global_rounds(self) -> int:
        last = [r[-1] for r in self.active_rounds.values() if r]
        return (max(last) + 1) if last else 0


def simulate(x, dtype: str, op: str, b: int, trees=None,
             skip_void: bool = True, fail=None):
    """Run the schedule for all ranks.  Returns (Y, trace) where Y[i] is rank
    i's final array."""
    Y = [x[i].copy() for i in range(len(x))]
    p = len(Y)
    m = Y[0].shape[0]
    t = trees if trees is not None else build_trees(p)
    if not (0 < b <= max(m, 1)):
        raise ValueError("need 0 < b <= m")
    trace = Trace()
    H = t.height
    by_depth = [[] for _ in range(H + 1)]
    for i in range(p):
        by_depth[t.depth[i]].append(i)

    def blk(j):
        return block_bounds(m, b, j)

    def real(j):
        return blk(j) is not None

    def last_round(i):
        # the rounds a rank's loop runs through: j = 0 .. b + d_i
        return b + t.depth[i]

    # how far each rank got: ranks that stopped or wait forever take no
    # further step
    stopped = set()
    blocked = {}
    # blocks of Y[i] that hold their final value, with the round they did
    final = {i: {} for i in range(p)}
    # log entries with the rank's own step order inside a round
    steps = {i: [] for i in range(p)}

    def note(i, j, step, kind, partner, sent, recv, ops):
        steps[i].append((j, step, kind, partner,
                         sent if real(sent) else None,
                         recv if real(recv) else None))
        ar = trace.active_rounds.setdefault(i, [])
        if not ar or ar[-1] != j:
            ar.append(j)
        trace.exchanges[i] = trace.exchanges.get(i, 0) + 1
        o = trace.ops_per_round.setdefault(i, {})
        o[j] = o.get(j, 0) + ops
        s = trace.steps_per_round.setdefault(i, {})
        s[j] = s.get(j, 0) + 1

    def can_step(i, j):
        return i not in stopped and i not in blocked

    def attempts(i, j, void):
        """Does rank i take part in this round's exchange on an edge?"""
        if j > last_round(i):
            return False
        return not (skip_void and void)

    def rendezvous(a, b_, j, kind_a, kind_b, void):
        """Both ends of an edge in round j: True if the exchange happens;
        otherwise an end that waits for it is marked blocked."""
        wa = attempts(a, j, void) and can_step(a, j)
        wb = attempts(b_, j, void) and can_step(b_, j)
        if wa and wb:
            return True
        if wa and attempts(a, j, void):
            blocked[a] = (b_, kind_a, j)
        if wb and attempts(b_, j, void):
            blocked[b_] = (a, kind_b, j)
        return False

    rounds = b + H + 1
    for j in range(rounds):
        if fail is not None and fail[1] == j:
            stopped.add(fail[0])
        # child-to-parent and parent-to-child traffic, deepest edges first;
        # at each parent the first child's edge before the second child's
        for d in range(H, 0, -1):
            for q in by_depth[d - 1]:
                for step, c in ((0, t.child0[q]), (1, t.child1[q])):
                    if c is None:
                        continue
                    up, down = j, j - t.depth[c]
                    void = not real(up) and not real(down)
                    if not rendezvous(c, q, j, "parent", "child", void):
                        continue
                    ops = 0
                    if real(up):
                        s, e = blk(up)
                        Y[q][s:e] = combine(dtype, op, Y[c][s:e], Y[q][s:e])
                        ops = 1
                    if real(down):
                        if final[q].get(down, j) >= j:
                            raise ProtocolError(
                                f"round {j}: rank {q} sends block {down} to "
                                f"rank {c} before it is final")
                        s, e = blk(down)
                        Y[c][s:e] = Y[q][s:e]
                        final[c][down] = j
                    note(q, j, step, "child", c, down, up, ops)
                    note(c, j, 2, "parent", q, up, down, 0)
        # the roots: block j is now their tree's product
        if len(t.roots) == 2:
            ra, rb = t.roots
            void = not real(j)
            if rendezvous(ra, rb, j, "dual", "dual", void):
                ops = 0
                if real(j):
                    s, e = blk(j)
                    ta, tb = Y[ra][s:e].copy(), Y[rb][s:e].copy()
                    Y[ra][s:e] = combine(dtype, op, ta, tb)   # mine (.) got
                    Y[rb][s:e] = combine(dtype, op, ta, tb)   # got (.) mine
                    final[ra][j] = final[rb][j] = j
                    ops = 1
                note(ra, j, 2, "dual", rb, j, j, ops)
                note(rb, j, 2, "dual", ra, j, j, ops)
        else:
            r = t.roots[0]
            if real(j) and can_step(r, j):
                final[r][j] = j

    if blocked:
        raise DeadlockError(blocked)
    for i in range(p):
        for (j, _, kind, partner, sent, recv) in sorted(
                steps[i], key=lambda e: (e[0], e[1])):
            trace.exchange_log.setdefault(i, []).append(
                (j, kind, partner, sent, recv))
        if final[i]:
            trace.final_round[i] = dict(final[i])
    return Y, trace
