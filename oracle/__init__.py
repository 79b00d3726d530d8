"""CPU oracle for the doubly-pipelined, dual-root reduction-to-all (Traeff 2021).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
link this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library in ``paper_2109_12626_amd/`` and imports nothing from it.

It is a plain, slow, obviously correct restatement of what the method
computes (numpy, one array operation per rank, vectorised only over the
independent columns):

* ``trees``       -- the two post-order numbered, heap-shaped complete binary
                     trees and their dual roots (Section 1.1).
* ``ops``         -- the element operators: int32 SUM (two's-complement wrap),
                     int32 MAX, fp32 SUM (IEEE binary32, round to nearest even)
                     and the non-commutative 2x2 uint32 matrix product mod 2^32.
* ``reduce``      -- the result y every rank receives, evaluated in the exact
                     association the trees impose (Algorithm 1, lines for the
                     two children and the dual root), plus the plain
                     left-to-right definition of Section 1 for exact operators.
* ``algorithm1``  -- a literal round-by-round rendezvous simulation of
                     Algorithm 1 with blocking, virtual empty blocks and the
                     telephone-model exchanges, used to pin the tree
                     evaluation, the round counts and the round in which
                     every rank's every block becomes final.  On one tree
                     (``build_trees(p, layout="single")``) it is the
                     single doubly-pipelined tree of Section 1.2.
* ``reduce_bcast`` -- a rendezvous simulation of the pipelined reduction to
                     the root of one tree followed by the pipelined
                     broadcast (Section 2's User-Allreduce1).
* ``blocks``      -- the block partition and the block-count rule of
                     Section 1.2.
* ``c_oracle``    -- a second evaluation of y in plain C (``c/``), written
                     independently of ``reduce``: the trees numbered from
                     subtree sizes and a stack walk over the ranks in
                     post-order, on host threads over column ranges
                     (imported on its own: ``from oracle import c_oracle``).

Parity status: every function here is pinned by ``tests/test_oracle_*.py``
(hand-derived worked examples, closed forms, brute force, the error bound of
recursive summation and the independent Algorithm-1 simulation; the C
oracle by ``tests/test_oracle_c.py``, planted mistakes included).  The
``wbal`` tree shape (an experiment only) is pinned by its p=9 structure, a
hand-derived fp32 value and the invariants that fix it for every p up to 257
and larger sizes up to 2000.
"""

from .trees import Trees, build_trees, heap_postorder_tree
from .ops import DTYPES, OPS, combine, valid_pair, element_shape, numpy_dtype
from .reduce import allreduce_tree, allreduce_ltr, allreduce_all
from .algorithm1 import simulate, DeadlockError
from .reduce_bcast import simulate_reduce_bcast
from .blocks import block_bounds, block_rule_lit, block_rule_cal, log2_height

__all__ = [
    "Trees", "build_trees", "heap_postorder_tree",
    "DTYPES", "OPS", "combine", "valid_pair", "element_shape", "numpy_dtype",
    "allreduce_tree", "allreduce_ltr", "allreduce_all",
    "simulate", "DeadlockError", "simulate_reduce_bcast",
    "block_bounds", "block_rule_lit", "block_rule_cal", "log2_height",
]
