"""The five workloads, as data: shapes, value distributions, seeds and the
block counts each is run with.  Seeds are 2109 + workload number.

``b`` entries are integers or the string "rule" (the sqrt(m log2 p) block
count, computed by whichever side consumes the workload).
"""

from dataclasses import dataclass, field
from typing import Dict, List, Tuple, Union


@dataclass(frozen=True)
class Workload:
    name: str
    p: int
    m: int
    dtype: str              # "int32" | "float32" | "u32mat2x2"
    ops: Tuple[str, ...]
    dist: str
    dist_kw: Dict = field(default_factory=dict, hash=False, compare=False)
    seed: int = 0
    bs: Tuple[Union[int, str], ...] = (1,)
    note: str = ""


P7_SMALL = Workload(
    name="p7_m1000_int32_sum", p=7, m=1000, dtype="int32", ops=("sum",),
    dist="uniform_int", dist_kw={"lo": -1000, "hi": 1000}, seed=2110,
    bs=(4,), note="two trees of 4 and 3 ranks, blocks of 250")

P36_INT = Workload(
    name="p36_m2^20_int32_sum", p=36, m=1 << 20, dtype="int32", ops=("sum",),
    dist="uniform_int", dist_kw={"lo": -(1 << 20), "hi": 1 << 20}, seed=2111,
    bs=(1, 8, 64, "rule"))

P64_MAT = Workload(
    name="p64_m2^18_u32mat2x2_matmul", p=64, m=1 << 18, dtype="u32mat2x2",
    ops=("matmul",), dist="uniform_u32_mat", seed=2112, bs=(32,),
    note="non-commutative: checks the rank order")

P1152_F32 = Workload(
    name="p1152_m2^22_fp32_sum", p=1152, m=1 << 22, dtype="float32",
    ops=("sum",), dist="normal_f32", seed=2113, bs=("rule",),
    note="36x32 rank layout; headline bandwidth workload")

P1152_SWEEP = [
    Workload(
        name=f"p1152_m2^{k}_int32_maxsum", p=1152, m=1 << k, dtype="int32",
        ops=("max", "sum"), dist="uniform_int",
        dist_kw={"lo": 0, "hi": (1 << 16) - 1}, seed=2114, bs=(1, "rule"),
        note="latency-bound to bandwidth-bound crossover")
    for k in (4, 10, 16, 22)
]

ALL: List[Workload] = [P7_SMALL, P36_INT, P64_MAT, P1152_F32] + P1152_SWEEP


def elem_bytes(dtype: str) -> int:
    return 16 if dtype == "u32mat2x2" else 4
