"""The C ABI on the CPU: the library loads, exports every function the header
declares, and its host-side plan (trees, round counts, block rule, block
decomposition) agrees with the independently written oracle.  Argument
checks run before any device work, so their error codes are testable here.
"""

import math
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
from paper_2109_12626_amd import dpar

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dpar.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dpar_[a-z_]+)\s*\(", text)))


def test_plain_c_program_uses_the_abi(tmp_path):
    """tests/cpp/c_consumer.c, compiled as C99 with gcc against the header
    and linked to libdpar.so, calls the entry points that need no device and
    gets the documented results (the boundary is a C ABI, not only a Python
    one).  HIP's host headers need __HIP_PLATFORM_AMD__ outside hipcc."""
    import shutil
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    libdir = os.path.dirname(dpar.LIB_PATH)
    exe = tmp_path / "c_consumer"
    subprocess.run([gcc, "-std=c99", "-Wall", "-Werror",
                    "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                    "-I", os.path.join(rocm, "include"),
                    os.path.join(ROOT, "tests", "cpp", "c_consumer.c"),
                    "-L", libdir, "-ldpar", f"-Wl,-rpath,{libdir}",
                    "-o", str(exe)], check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True)
    lines = res.stdout.split("\n")
    assert res.returncode == 0, res.stdout + res.stderr
    assert not [ln for ln in lines if ln.startswith("FAIL")]
    assert sum(ln.startswith("ok ") for ln in lines) == 12


def test_library_exports_every_declared_function():
    names = _declared()
    assert "dpar_allreduce" in names and len(names) >= 9
    out = subprocess.run(["nm", "-D", "--defined-only", dpar.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r" T (dpar_\w+)", out))
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    L = dpar.lib()
    for n in names:
        assert hasattr(L, n)


@pytest.mark.parametrize("p", list(range(1, 70)) + [127, 128, 576, 1151, 1152,
                                                     4097])
def test_tree_info_matches_oracle(p):
    t = oracle.build_trees(p)
    none = lambda v: -1 if v is None else v  # noqa: E731
    for i in range(p):
        got = dpar.dpar_tree_info(p, i)
        assert got == {"parent": none(t.parent[i]), "child0": none(t.child0[i]),
                       "child1": none(t.child1[i]), "depth": t.depth[i],
                       "subtree_lo": t.lo[i], "dual": none(t.dual[i])}, i


@pytest.mark.parametrize("p", [1, 2, 3, 5, 7, 9, 14, 36, 64, 100])
@pytest.mark.parametrize("b", [1, 2, 4, 7])
def test_round_counts_match_simulation(p, b):
    x = np.zeros((p, 2 * b + 2), dtype=np.int32)
    _, tr = oracle.simulate(x, "int32", "sum", b)
    for i in range(p):
        assert dpar.dpar_rounds(p, b, i) == tr.span(i), i
    assert dpar.dpar_rounds(p, b, -1) == tr.global_rounds()


def test_block_rule_matches_oracle():
    for p in (1, 2, 7, 36, 64, 1152, 4095):
        for m in (0, 1, 2, 16, 1000, 1024, 1 << 16, 1 << 20, 1 << 22,
                  12345678):
            assert dpar.dpar_block_rule(p, m) == oracle.block_rule_lit(p, m)
            if m:
                assert dpar.dpar_block_rule(p, m, 3e-6, 1e-9) == \
                    oracle.block_rule_cal(p, m, 3e-6, 1e-9)
    assert dpar.dpar_block_rule(1152, 1 << 22) == 6532


@pytest.mark.parametrize("m,b,dtype,aligned", [
    (1000, 4, "int32", True), (1 << 20, 2329, "int32", True),
    (1 << 22, 6532, "float32", True), (1 << 18, 32, "u32mat2x2", True),
    (1003, 7, "float32", True), (16, 13, "int32", True), (5, 5, "int32", True),
    (1000, 4, "float32", False), (12345, 17, "u32mat2x2", False),
    (1 << 16, 817, "int32", True)])
def test_block_decomposition(m, b, dtype, aligned):
    s = dpar.dpar_schedule_info(36, m, dtype, b, aligned)
    assert s.b == b
    # 16-byte lanes whenever every block holds a whole quantum, whatever the
    # alignment (the flag is ignored), unless trailing elements remain and
    # the call moves at most 24 MB; a matrix is one quantum
    small_tail = m % 4 != 0 and 2 * 36 * m * 4 <= 24 << 20
    vec4 = dtype != "u32mat2x2" and m // 4 >= b and not small_tail
    assert s.quantum == (4 if vec4 else 1)
    vec = vec4 or dtype == "u32mat2x2"
    other = dpar.dpar_schedule_info(36, m, dtype, b, not aligned)
    assert [getattr(other, f) for f, _ in other._fields_] == \
        [getattr(s, f) for f, _ in s._fields_]
    lines = -(-(s.nquanta * s.quantum) // (8 * s.quantum))
    want_g = s.quantum * (8 if vec and lines >= b else 1)
    assert s.granularity == want_g
    assert s.nquanta * s.quantum + s.tail_elems == m
    bounds = [dpar.dpar_block_bounds(s, m, j) for j in range(b)]
    assert bounds[0][0] == 0 and bounds[-1][1] == m
    for (s0, e0), (s1, _) in zip(bounds, bounds[1:]):
        assert e0 == s1
        assert s1 % s.granularity == 0          # cut at line boundaries
    sizes = [e - s_ for s_, e in bounds]
    sizes[-1] -= s.tail_elems
    assert min(sizes) >= 1
    # every block but the last is a whole number of lines; sizes differ by at
    # most one line (the last may also lose part of its final line)
    assert max(sizes[:-1] or [0]) - min(sizes[:-1] or [0]) <= s.granularity
    assert abs(sizes[0] - m / b) <= 2 * s.granularity
    # chunks: at most 64 quanta each
    per_block = -(-max(sizes) // s.quantum)
    assert -(-per_block // s.chunks_per_block) <= 64 + 8


@pytest.mark.parametrize("p,m,quantum", [
    (288, 8750, 1), (288, 21250, 4), (288, 21252, 4), (1152, 2125, 1),
    (1152, 8750, 4), (1152, 2124, 4), (7, 1 << 18 | 1, 1), (2, 1572863, 1),
    (2, 1572867, 4)])
def test_small_calls_with_trailing_elements_take_one_element_per_lane(
        p, m, quantum):
    # m mod 4 != 0 and at most 24 MB moved: one launch, one element per lane
    s = dpar.dpar_schedule_info(p, m, "int32", 1, True)
    assert s.quantum == quantum
    assert s.tail_elems == (m % 4 if quantum == 4 else 0)


@pytest.mark.parametrize("m,b", [(20, 7), (27, 7), (1000, 251), (5, 5)])
def test_scalar_path_matches_canonical_partition(m, b):
    # blocks shorter than one quantum of 4 elements: one element per lane
    # and Section 1.1's partition into b blocks of roughly m / b elements
    s = dpar.dpar_schedule_info(9, m, "float32", b, aligned=True)
    assert s.quantum == 1 and s.granularity == 1
    for j in range(b):
        assert dpar.dpar_block_bounds(s, m, j) == oracle.block_bounds(m, b, j)


# ------------------------------------------------------------ argument errors

A = 1 << 30  # fake, never dereferenced: every case fails before device work


def _err(fn, *args, **kw):
    with pytest.raises(dpar.DparError) as e:
        fn(*args, **kw)
    return e.value.code


def test_argument_errors():
    xs = [A + i * 4096 for i in range(4)]
    ys = [A + (1 << 20) + i * 4096 for i in range(4)]
    ok = (xs, ys, 4, 1000, "int32", "sum", 4)
    f = dpar.dpar_allreduce
    assert _err(f, xs, ys, 0, 1000, "int32", "sum", 4) == dpar.DPAR_ERR_INVALID_ARG
    assert _err(f, xs, ys, 4, 1000, "int32", "sum", -1) == dpar.DPAR_ERR_INVALID_ARG
    assert _err(f, xs, ys, 4, 1000, "int32", "sum", 1001) == \
        dpar.DPAR_ERR_INVALID_ARG
    assert _err(f, xs, ys, 4, 1000, "float32", "max", 4) == \
        dpar.DPAR_ERR_UNSUPPORTED
    assert _err(f, xs, ys, 4, 1000, "int32", "matmul", 4) == \
        dpar.DPAR_ERR_UNSUPPORTED
    assert _err(f, xs[:3] + [0], ys, 4, 1000, "int32", "sum", 4) == \
        dpar.DPAR_ERR_INVALID_ARG
    assert _err(f, xs, ys[:3] + [A + 2], 4, 1000, "int32", "sum", 4) == \
        dpar.DPAR_ERR_INVALID_ARG                    # not 4-byte aligned
    assert _err(dpar.dpar_allreduce_ex, *ok, 9) == dpar.DPAR_ERR_INVALID_ARG
    # m = 0 is a successful no-op (nothing is touched)
    assert f(xs, ys, 4, 0, "int32", "sum", 0) == 0


def test_alias_rules():
    f = dpar.dpar_allreduce
    n = 1000 * 4
    xs = [A + i * 8192 for i in range(4)]
    ys = [A + (1 << 20) + i * 8192 for i in range(4)]
    # two outputs overlap
    bad = list(ys)
    bad[2] = ys[1] + 16
    assert _err(f, xs, bad, 4, 1000, "int32", "sum", 4) == dpar.DPAR_ERR_ALIAS
    # an output partially overlaps an input
    bad = list(ys)
    bad[0] = xs[3] + 64
    assert _err(f, xs, bad, 4, 1000, "int32", "sum", 4) == dpar.DPAR_ERR_ALIAS
    assert n < 8192


@pytest.mark.skipif(os.path.exists("/dev/kfd"),
                    reason="would launch on fake addresses with a GPU present")
def test_overlapping_inputs_pass_the_alias_check():
    # inputs that overlap each other are allowed: without a GPU the call gets
    # past every argument check and fails only at the device
    ys = [A + (1 << 20) + i * 8192 for i in range(4)]
    code = _call_code(dpar.dpar_allreduce, [A] * 4, ys, 4, 1000, "int32",
                      "sum", 4)
    assert code == dpar.DPAR_ERR_HIP


def _call_code(fn, *args):
    try:
        fn(*args)
        return 0
    except dpar.DparError as e:
        return e.code


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="a GPU is present")
def test_valid_call_without_gpu_fails_loudly():
    xs = [A + i * 8192 for i in range(4)]
    code = _call_code(dpar.dpar_allreduce, xs, xs, 4, 1000, "int32", "sum", 4)
    assert code == dpar.DPAR_ERR_HIP


def test_info_argument_errors():
    assert _err(dpar.dpar_tree_info, 0, 0) == dpar.DPAR_ERR_INVALID_ARG
    assert _err(dpar.dpar_tree_info, 5, 5) == dpar.DPAR_ERR_INVALID_ARG
    assert _err(dpar.dpar_rounds, 5, 0, 1) == dpar.DPAR_ERR_INVALID_ARG
    assert _err(dpar.dpar_block_rule, 0, 10) == dpar.DPAR_ERR_INVALID_ARG


@pytest.mark.parametrize("p", list(range(1, 40)) + [127, 128, 1151, 1152])
@pytest.mark.parametrize("alg", ["single", "reduce_bcast"])
def test_tree_info_alg_matches_oracle_single_tree(p, alg):
    t = oracle.build_trees(p, layout="single")
    none = lambda v: -1 if v is None else v  # noqa: E731
    for i in range(p):
        got = dpar.dpar_tree_info_alg(p, alg, i)
        assert got == {"parent": none(t.parent[i]), "child0": none(t.child0[i]),
                       "child1": none(t.child1[i]), "depth": t.depth[i],
                       "subtree_lo": t.lo[i], "dual": -1}, i
    assert dpar.dpar_tree_info_alg(p, "dual", p - 1) == \
        dpar.dpar_tree_info(p, p - 1)


@pytest.mark.parametrize("p", [1, 2, 3, 5, 7, 14, 36, 64, 100])
@pytest.mark.parametrize("b", [1, 2, 5])
def test_schedule_rounds_match_simulations(p, b):
    """The device round structure's length equals the rounds the oracle's
    simulations use: Algorithm 1 on the dual-root trees and on one tree,
    and the reduce-then-broadcast."""
    x = np.zeros((p, 2 * b + 2), dtype=np.int32)
    _, tr = oracle.simulate(x, "int32", "sum", b)
    want = tr.global_rounds() if p > 1 else b
    assert dpar.dpar_schedule_rounds(p, b, "dual") == want
    t1 = oracle.build_trees(p, layout="single")
    _, tr = oracle.simulate(x, "int32", "sum", b, trees=t1)
    want = tr.global_rounds() if p > 1 else b
    assert dpar.dpar_schedule_rounds(p, b, "single") == want
    _, tr = oracle.simulate_reduce_bcast(x, "int32", "sum", b)
    assert dpar.dpar_schedule_rounds(p, b, "reduce_bcast") == \
        tr.global_rounds()


def test_option_errors():
    xs = [A + i * 4096 for i in range(4)]
    ys = [A + (1 << 20) + i * 4096 for i in range(4)]
    f = dpar.dpar_allreduce_opt
    args = (xs, ys, 4, 1000, "int32", "sum", 4)
    assert _err(f, *args, alg=7) == dpar.DPAR_ERR_INVALID_ARG
    assert _err(f, *args, exec=7) == dpar.DPAR_ERR_INVALID_ARG
    # a round range needs a round-structured executor
    assert _err(f, *args, exec="split", round_begin=1) == \
        dpar.DPAR_ERR_INVALID_ARG
    assert _err(f, *args, exec="launch", round_end=2) == \
        dpar.DPAR_ERR_INVALID_ARG
    # reversed, negative and too long ranges (R = 4 + 1 here)
    assert dpar.dpar_schedule_rounds(4, 4, "dual") == 5
    assert _err(f, *args, exec="rounds", round_begin=3, round_end=2) == \
        dpar.DPAR_ERR_INVALID_ARG
    assert _err(f, *args, exec="rounds", round_begin=-1) == \
        dpar.DPAR_ERR_INVALID_ARG
    assert _err(f, *args, exec="rounds", round_end=6) == \
        dpar.DPAR_ERR_INVALID_ARG
    # the alias rules hold for every executor
    bad = list(ys)
    bad[2] = ys[1] + 16
    assert _err(f, xs, bad, 4, 1000, "int32", "sum", 4, alg="single",
                exec="rounds") == dpar.DPAR_ERR_ALIAS
    assert _err(dpar.dpar_tree_info_alg, 5, 3, 0) == dpar.DPAR_ERR_INVALID_ARG
    assert _err(dpar.dpar_schedule_rounds, 5, 0, 0) == \
        dpar.DPAR_ERR_INVALID_ARG
    # an empty round range is a successful no-op (no device work)
    assert f(*args, exec="rounds", round_begin=2, round_end=2) == 0


def test_work_item_limit_is_checked_before_narrowing():
    # b = 1 over 2^39 elements would need 2^31 chunks of 64 quanta: refused
    # before any device work, whatever the int width of the chunk count
    xs = [A, A + (1 << 41)]
    ys = [A + (2 << 41), A + (3 << 41)]
    assert _err(dpar.dpar_allreduce_ex, xs, ys, 2, 1 << 39, "int32", "sum", 1,
                "split") == dpar.DPAR_ERR_UNSUPPORTED


def test_noalloc_argument_errors_before_device_work():
    """dpar_allreduce_noalloc checks its arguments like dpar_allreduce, and
    refuses p beyond the ranks its fixed device memory holds, all before
    any device work (so on the CPU too)."""
    f = dpar.dpar_allreduce_noalloc
    xs = [A + i * 4096 for i in range(4)]
    ys = [A + (1 << 20) + i * 4096 for i in range(4)]
    assert _err(f, xs, ys, 0, 1000, "int32", "sum", 4) == \
        dpar.DPAR_ERR_INVALID_ARG
    assert _err(f, xs, ys, 4, 1000, "int32", "sum", 1001) == \
        dpar.DPAR_ERR_INVALID_ARG
    assert _err(f, xs, ys, 4, 1000, "float32", "max", 4) == \
        dpar.DPAR_ERR_UNSUPPORTED
    assert _err(f, xs, [A + 8] + ys[1:], 4, 1000, "int32", "sum", 4) == \
        dpar.DPAR_ERR_ALIAS
    big = 32769
    bx = [A + i * 8192 for i in range(big)]
    by = [A + (1 << 32) + i * 8192 for i in range(big)]
    assert _err(f, bx, by, big, 16, "int32", "sum", 0) == \
        dpar.DPAR_ERR_UNSUPPORTED
    assert "32768" in dpar.dpar_last_error()
    # m = 0 is a successful no-op, as for dpar_allreduce
    assert f(xs, ys, 4, 0, "int32", "sum", 0) == 0


def test_binding_pointer_arrays():
    """rows() and pointers() only marshal addresses: the C arrays they
    build hold exactly the row addresses, whichever route builds them."""
    import ctypes
    import torch
    for shape in ((5, 7), (1, 3), (4, 2, 4), (300, 1)):
        t = torch.zeros(shape, dtype=torch.float32)
        r = dpar.rows(t)
        assert isinstance(r, ctypes.Array) and len(r) == shape[0]
        step = t.stride(0) * t.element_size()
        want = [t.data_ptr() + i * step for i in range(shape[0])]
        assert list(r) == want
        assert dpar.pointers(r) is r                   # reused as it is
        assert list(dpar.pointers(want)) == want       # plain ints
        assert list(dpar.pointers(list(t))) == want    # tensors
        mixed = [want[0]] + list(t)[1:]
        assert list(dpar.pointers(mixed)) == want
    assert len(dpar.rows(torch.zeros(0, 3))) == 0
    assert len(dpar.pointers([])) == 0
    big = [(1 << 63) + 4096 * i for i in range(3)]     # above 2^63
    assert list(dpar.pointers(big)) == big
    with pytest.raises(ValueError):
        dpar.rows(torch.tensor(1.0))
