"""Pipeline blocks and the block-count rule (Sections 1.1 and 1.2).

Oracle module: test infrastructure only.

* Blocks (Section 1.1): the m elements are split into b successive blocks,
  0 < b <= m, of roughly m/b elements; block j is read here as the
  canonical range [floor(j m / b), floor((j+1) m / b)).  Blocks with j < 0 or
  j >= b are the paper's virtual empty blocks (returned as None).
* Rule (Section 1.2): for p = 2^h - 2 the time with b blocks is
  (4h - 3 + 3(b - 1)) (alpha + beta m / b); balancing the terms gives
  b* = sqrt((4h - 6) beta m / (3 alpha)) and the O(log p + sqrt(m log p))
  term.  Two readings are provided:
    - ``block_rule_lit(p, m)``  = clamp(ceil(sqrt(m log2 p)), 1, m): the
      sqrt(m log p) growth with the system constants dropped;
    - ``block_rule_cal(p, m, alpha, beta)`` = clamp(round(b*), 1, m) with the
      real-valued h = log2(p + 2).
  Both return 0 for m = 0 (nothing to split).
"""

import math


def block_bounds(m: int, b: int, j: int):
    """Element range [start, end) of block j, or None for a virtual block."""
    if not (0 < b):
        raise ValueError("b must be positive")
    if j < 0 or j >= b:
        return None
    return (j * m) // b, ((j + 1) * m) // b


def log2_height(p: int) -> float:
    """h with p = 2^h - 2, extended to every p >= 1."""
    return math.log2(p + 2)


def block_rule_lit(p: int, m: int) -> int:
    if m == 0:
        return 0
    if p <= 1:
        return 1
    b = math.ceil(math.sqrt(m * math.log2(p)))
    return max(1, min(m, b))


def block_rule_cal(p: int, m: int, alpha: float, beta: float) -> int:
    if m == 0:
        return 0
    if not (alpha > 0 and beta > 0):
        raise ValueError("alpha and beta must be positive")
    h = log2_height(p)
    b = math.sqrt((4 * h - 6) * beta * m / (3 * alpha))
    return max(1, min(m, int(math.floor(b + 0.5))))
