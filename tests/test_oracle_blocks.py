"""Pins for the block-count rule (Section 1.2).

The time with b blocks for p = 2^h - 2 is (4h - 3 + 3(b - 1))(a + B m / b);
balancing its increasing and decreasing terms gives
b* = sqrt((4h - 6) B m / (3 a)), and the best time
(4h - 6) a + 2 sqrt(3 (4h - 6) a B m) + 3 B m.
"""

import math

import pytest

from oracle import block_rule_cal, block_rule_lit


def test_literal_rule_values_for_the_workloads():
    # ceil(sqrt(m log2 p)): p=36, m=2^20 -> sqrt(5421035.1) = 2328.3
    assert block_rule_lit(36, 1 << 20) == 2329
    assert block_rule_lit(1152, 1 << 22) == 6532
    assert [block_rule_lit(1152, 1 << k) for k in (4, 10, 16, 22)] == \
        [13, 103, 817, 6532]
    assert block_rule_lit(1, 100) == 1
    assert block_rule_lit(7, 0) == 0
    assert block_rule_lit(1 << 20, 3) == 3          # clamped to m


def test_literal_rule_exact_square():
    # p = 4, m = 8: m log2 p = 16, sqrt = 4 exactly
    assert block_rule_lit(4, 8) == 4


@pytest.mark.parametrize("h", [3, 4, 6, 11])
@pytest.mark.parametrize("m", [1000, 1 << 20])
def test_calibrated_rule_reduces_for_p_2h_minus_2(h, m):
    p = 2 ** h - 2
    want = math.sqrt((4 * h - 6) * m / 3)
    got = block_rule_cal(p, m, 1.0, 1.0)
    assert got == max(1, min(m, int(math.floor(want + 0.5))))


def test_calibrated_rule_minimises_the_model():
    # the integer b it returns is within one of the minimiser of T(b)
    h, m, a, B = 8, 1 << 22, 5e-6, 1.5e-9
    p = 2 ** h - 2

    def T(b):
        return (4 * h - 3 + 3 * (b - 1)) * (a + B * m / b)
    best = min(range(1, 5000), key=T)
    assert abs(block_rule_cal(p, m, a, B) - best) <= 1
    bstar = math.sqrt((4 * h - 6) * B * m / (3 * a))
    tstar = (4 * h - 6) * a + 2 * math.sqrt(3 * (4 * h - 6) * a * B * m) \
        + 3 * B * m
    assert T(bstar) == pytest.approx(tstar, rel=1e-12)
