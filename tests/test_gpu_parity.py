"""GPU parity: the HIP path through the C ABI against the CPU oracle, element
by element, on seeded inputs.  Integer and matrix results must be bit-exact;
fp32 SUM must also be bit-exact, because the kernels apply the additions in
exactly the tree order the oracle follows (Algorithm 1's association).

Small and mid-size cases compare every element of every rank's output (the
full-size workloads are in test_gpu_fullsize.py).
"""

import numpy as np
import pytest
import torch

import oracle
import synth
from synth import configs
from tests._gpu import (POISON, assert_all_ranks_equal, env_bcast_span_kb,
                        env_unit, env_waves, from_dev, need_gpu,
                        poisoned_like, resolve_b, run, to_dev, workload_input)

pytestmark = pytest.mark.gpu

EXECS = ["launch", "barrier", "ticket", "split"]
UNITS = ["seq", "level"]


@pytest.fixture(autouse=True)
def _gpu():
    need_gpu()
    yield
    torch.cuda.synchronize()


def _want(x, dtype, op):
    return oracle.allreduce_tree(x, dtype, op)


# ------------------------------------------------------------ p = 7, m = 1000

@pytest.mark.parametrize("unit", UNITS)
@pytest.mark.parametrize("exec", EXECS)
@pytest.mark.parametrize("b", [4, 1, 2, 7, 249, 250, 251, 1000])
def test_p7_int32_sum_every_executor_and_b(exec, b, unit):
    w = configs.P7_SMALL
    x = workload_input(w)
    with env_unit(unit):
        out = run(x, "int32", "sum", b, exec)
    assert_all_ranks_equal(out, _want(x, "int32", "sum"), f"b={b} {exec}")


@pytest.mark.parametrize("waves", [1, 2])
@pytest.mark.parametrize("dtype,op", [("int32", "sum"), ("int32", "max"),
                                      ("float32", "sum")])
def test_p7_all_ops_both_wave_layouts(waves, dtype, op):
    w = configs.P7_SMALL
    x = workload_input(w)
    if dtype == "float32":
        x = synth.generate("normal_f32", 7, w.p, w.m)
    with env_waves(waves):
        out = run(x, dtype, op, 4)
    assert_all_ranks_equal(out, _want(x, dtype, op))


def test_fp32_worked_examples_on_device():
    # the hand-derived association examples, repeated over 300 columns
    path = "tests/golden/fp32_worked_examples.txt"
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        name, shape, xs, tree_v, _ = (c.strip() for c in line.split("|"))
        if shape != "heap":
            continue
        col = np.array([float(v) for v in xs.split()], dtype=np.float32)
        x = np.repeat(col[:, None], 300, axis=1)
        out = run(x, "float32", "sum", 3)
        assert (out == np.float32(float(tree_v))).all(), name


# ------------------------------------------------------------ edge cases

@pytest.mark.parametrize("unit", UNITS)
@pytest.mark.parametrize("p", [1, 2, 3, 4, 5, 8, 9, 15, 16, 17, 31, 33, 100])
@pytest.mark.parametrize("m", [1, 3, 4, 5, 64, 255, 256, 257, 1027])
def test_small_p_and_m(p, m, unit):
    x = synth.generate("normal_f32", 100 + p, p, m)
    b = min(m, 3)
    with env_unit(unit):
        out = run(x, "float32", "sum", b)
    assert_all_ranks_equal(out, _want(x, "float32", "sum"), f"p={p} m={m}")


@pytest.mark.parametrize("exec", EXECS)
@pytest.mark.parametrize("dtype,op,dist", [
    ("int32", "max", "uniform_int"), ("float32", "sum", "normal_f32"),
    ("u32mat2x2", "matmul", "odd_det_u32_mat")])
def test_level_unit_all_dtypes_and_executors(exec, dtype, op, dist):
    p, m = 300, 1000
    kw = {"lo": -99, "hi": 99} if dist == "uniform_int" else {}
    x = synth.generate(dist, 61, p, m, **kw)
    for b in (1, 7, 40):
        with env_unit("level"):
            out = run(x, dtype, op, b, exec)
        assert_all_ranks_equal(out, _want(x, dtype, op), f"b={b}")


@pytest.mark.parametrize("span_kb", [1, 4, 36, 16384])
@pytest.mark.parametrize("p,m,dtype,op,dist", [
    (9, 40000, "float32", "sum", "normal_f32"),       # 16-byte lanes
    (5, 40001, "int32", "max", "uniform_int"),        # + a scalar tail
    (4, 9999, "u32mat2x2", "matmul", "odd_det_u32_mat"),
    (3, 123457, "float32", "sum", "normal_f32")])
def test_split_broadcast_in_spans(span_kb, p, m, dtype, op, dist):
    """The broadcast pass taken in spans of y_0 (every row of a span, then
    the next span; 8 tiles at least, padded to equal widths): all outputs
    equal the oracle's y, whatever the span."""
    kw = {"lo": -999, "hi": 999} if dist == "uniform_int" else {}
    x = synth.generate(dist, 900 + p, p, m, **kw)
    with env_bcast_span_kb(span_kb):
        out = run(x, dtype, op, 7, "split")
    assert_all_ranks_equal(out, _want(x, dtype, op), f"span {span_kb} KB")


def test_split_broadcast_unaligned_rows_in_spans():
    """Rows only 4-byte aligned (16-byte lanes across cache lines) with
    several spans."""
    p, m = 6, 30001
    x = synth.generate("normal_f32", 77, p, m)
    xd = to_dev(np.pad(x, ((0, 0), (1, 0))))
    yd = poisoned_like(xd)
    from paper_2109_12626_amd import dpar
    xs = [t[1:] for t in xd]
    ys = [t[1:] for t in yd]
    with env_bcast_span_kb(2):
        dpar.dpar_allreduce_ex(xs, ys, p, m, "float32", "sum", 5, "split",
                               torch.cuda.current_stream())
        dpar.dpar_check_status(torch.cuda.current_stream())
    out = yd.cpu().numpy()
    assert_all_ranks_equal(out[:, 1:], _want(x, "float32", "sum"))
    assert (out[:, 0].view(np.int32) == POISON).all()


@pytest.mark.parametrize("exec", ["auto", "split", "ticket", "rounds"])
@pytest.mark.parametrize("m", [1, 2, 3, 15, 21, 87, 2125, 8750, 21250])
def test_paper_counts_at_p288(m, exec):
    """The per-process counts of the paper's Table 2 that leave elements
    after the last 16-byte quantum, at its 288 processes, with its block of
    16000 elements: the trailing elements go through their own pass."""
    p = 288
    b = max(1, -(-m // 16000))
    x = synth.generate("uniform_int", 288 + m, p, m, lo=-1000, hi=1000)
    out = run(x, "int32", "sum", b, exec)
    assert_all_ranks_equal(out, _want(x, "int32", "sum"), f"m={m} {exec}")
    xf = synth.generate("normal_f32", 289 + m, p, m)
    out = run(xf, "float32", "sum", b, exec)
    assert_all_ranks_equal(out, _want(xf, "float32", "sum"), f"m={m} {exec}")


@pytest.mark.parametrize("exec", EXECS)
def test_m_zero_is_a_noop(exec):
    from paper_2109_12626_amd import dpar
    xd = torch.zeros((5, 8), dtype=torch.int32, device="cuda")
    yd = poisoned_like(xd)
    dpar.dpar_allreduce_ex(dpar.rows(xd), dpar.rows(yd), 5, 0, "int32", "sum",
                           0, exec, torch.cuda.current_stream())
    torch.cuda.synchronize()
    assert (yd == POISON).all()


@pytest.mark.parametrize("m,b", [(16, 13), (16, 16), (10, 10), (7, 7),
                                 (1024, 1024), (1003, 300)])
def test_b_large_uses_scalar_lanes(m, b):
    x = synth.generate("uniform_int", 3, 1152, m, lo=0, hi=65535)
    for op in ("sum", "max"):
        out = run(x, "int32", op, b)
        assert_all_ranks_equal(out, _want(x, "int32", op), f"{op} m={m} b={b}")


@pytest.mark.parametrize("offset", [4, 8, 12])
def test_unaligned_pointers(offset):
    # rows start 4/8/12 bytes past a 16-byte boundary: 16-byte lanes that
    # straddle them
    p, m = 37, 1001
    x = synth.generate("normal_f32", 5, p, m)
    big = torch.zeros((p, m + 8), dtype=torch.float32, device="cuda")
    k = offset // 4
    big[:, k:k + m] = torch.from_numpy(x).cuda()
    yb = torch.full((p, m + 8), float("nan"), device="cuda")
    from paper_2109_12626_amd import dpar
    xs = [a + offset for a in dpar.rows(big)]
    ys = [a + offset for a in dpar.rows(yb)]
    dpar.dpar_allreduce(xs, ys, p, m, "float32", "sum", 5,
                        torch.cuda.current_stream())
    dpar.dpar_check_status(torch.cuda.current_stream())
    out = yb[:, k:k + m].cpu().numpy()
    assert_all_ranks_equal(out, _want(x, "float32", "sum"))
    # bytes outside the rows are untouched
    assert torch.isnan(yb[:, :k]).all() and torch.isnan(yb[:, k + m:]).all()


@pytest.mark.parametrize("exec", ["auto", "split", "ticket", "launch",
                                  "barrier", "rounds"])
@pytest.mark.parametrize("dtype,op,dist", [
    ("int32", "max", "uniform_int"), ("float32", "sum", "normal_f32"),
    ("u32mat2x2", "matmul", "odd_det_u32_mat")])
@pytest.mark.parametrize("scalar", [0, 1])
def test_rows_of_every_misalignment(exec, dtype, op, dist, scalar):
    """The rows of one [p, m] tensor with m = 1 mod 4: row i starts 4 i
    bytes (mod 16) past a 16-byte boundary, so the rows straddle cache lines
    in every way at once; with 16-byte lanes and with one element per lane
    (DPAR_SCALAR=1, integer and fp32 only)."""
    p, m = 23, 4097
    kw = {"lo": -99, "hi": 99} if dist == "uniform_int" else {}
    x = synth.generate(dist, 3100 + p, p, m, **kw)
    from tests._gpu import _Env
    with _Env("DPAR_SCALAR", scalar):
        for b in (1, 5, 300):
            out = run(x, dtype, op, b, exec)
            assert_all_ranks_equal(out, _want(x, dtype, op),
                                   f"{exec} b={b} scalar={scalar}")


@pytest.mark.parametrize("span_kb", [4, 16384])
@pytest.mark.parametrize("offset", [4, 8, 12])
@pytest.mark.parametrize("dtype,op,dist", [
    ("int32", "sum", "uniform_int"), ("float32", "sum", "normal_f32"),
    ("u32mat2x2", "matmul", "odd_det_u32_mat")])
def test_split_with_output_rows_off_16_byte_boundaries(span_kb, offset, dtype,
                                                       op, dist):
    """16-byte lanes on rows 4, 8 or 12 bytes past a 16-byte boundary (m a
    multiple of 4, so no trailing elements): the broadcast pass shifts each
    row's stores to the row's own 16-byte boundaries and copies the leading
    and trailing dwords one by one.  Nothing outside the rows is touched."""
    p, m = 9, 6000
    kw = {"lo": -999, "hi": 999} if dist == "uniform_int" else {}
    x = synth.generate(dist, 700 + offset, p, m, **kw)
    words = 4 if dtype == "u32mat2x2" else 1
    k = offset // 4
    xi = np.ascontiguousarray(x).view(np.int32).reshape(p, m * words)
    big = torch.zeros((p, m * words + 8), dtype=torch.int32, device="cuda")
    big[:, k:k + m * words] = torch.from_numpy(xi).cuda()
    yb = torch.full_like(big, POISON)
    from paper_2109_12626_amd import dpar
    xs = [a + offset for a in dpar.rows(big)]
    ys = [a + offset for a in dpar.rows(yb)]
    s = torch.cuda.current_stream()
    with env_bcast_span_kb(span_kb):
        dpar.dpar_allreduce_ex(xs, ys, p, m, dtype, op, 5, "split", s)
    dpar.dpar_check_status(s)
    got = yb.cpu().numpy()
    out = got[:, k:k + m * words].copy().view(x.dtype).reshape(x.shape)
    assert_all_ranks_equal(out, _want(x, dtype, op), f"offset {offset}")
    assert (got[:, :k] == POISON).all() and (got[:, k + m * words:] == POISON).all()


@pytest.mark.parametrize("offset", [16, 48, 112])
@pytest.mark.parametrize("dtype,op,dist", [
    ("int32", "sum", "uniform_int"), ("u32mat2x2", "matmul", "odd_det_u32_mat")])
def test_split_with_rows_off_the_cache_lines(offset, dtype, op, dist):
    """Rows on 16-byte boundaries but 16, 48 or 112 bytes past a 128-byte
    line: the broadcast pass shifts each output row's stores to the row's
    own 4 KB boundary and the up-phase hands each XCD a contiguous run of
    work items.  Nothing outside the rows is touched."""
    p, m = 11, 9000
    kw = {"lo": -999, "hi": 999} if dist == "uniform_int" else {}
    x = synth.generate(dist, 800 + offset, p, m, **kw)
    words = 4 if dtype == "u32mat2x2" else 1
    k = offset // 4
    xi = np.ascontiguousarray(x).view(np.int32).reshape(p, m * words)
    # rows 128-byte aligned in `big` (stride a multiple of 32 words)
    stride = -(-(m * words + k + 32) // 32) * 32
    big = torch.zeros((p, stride), dtype=torch.int32, device="cuda")
    big[:, k:k + m * words] = torch.from_numpy(xi).cuda()
    yb = torch.full_like(big, POISON)
    from paper_2109_12626_amd import dpar
    xs = [a + offset for a in dpar.rows(big)]
    ys = [a + offset for a in dpar.rows(yb)]
    s = torch.cuda.current_stream()
    for b in (1, 7):
        yb.fill_(POISON)
        dpar.dpar_allreduce_ex(xs, ys, p, m, dtype, op, b, "split", s)
        dpar.dpar_check_status(s)
        got = yb.cpu().numpy()
        out = got[:, k:k + m * words].copy().view(x.dtype).reshape(x.shape)
        assert_all_ranks_equal(out, _want(x, dtype, op), f"offset {offset}")
        assert (got[:, :k] == POISON).all()
        assert (got[:, k + m * words:] == POISON).all()


@pytest.mark.parametrize("exec", ["auto", "split"])
def test_rows_16_bytes_apart_from_the_lines(exec):
    """One [36, 2^16 + 4] int32 tensor: row i starts 16 i bytes (mod 128)
    past a 128-byte line, every row on a 16-byte boundary."""
    p, m = 36, (1 << 16) + 4
    x = synth.generate("uniform_int", 4343, p, m, lo=-1000, hi=1000)
    out = run(x, "int32", "sum", 0, exec)
    assert_all_ranks_equal(out, _want(x, "int32", "sum"), exec)


@pytest.mark.parametrize("exec", ["auto", "split"])
def test_large_call_with_rows_of_every_misalignment(exec):
    """One [4, 2^20 + 1] fp32 tensor: its rows start 0, 4, 8 and 12 bytes
    past a 16-byte boundary and the call moves 33.5 MB, so it takes 16-byte
    lanes plus a pass for the trailing element, and the broadcast shifts
    every row's stores to its own boundaries."""
    p, m = 4, (1 << 20) + 1
    x = synth.generate("normal_f32", 4242, p, m)
    out = run(x, "float32", "sum", 0, exec)
    assert_all_ranks_equal(out, _want(x, "float32", "sum"), exec)


def test_in_place():
    p, m = 64, 4099
    x = synth.generate("normal_f32", 9, p, m)
    want = _want(x, "float32", "sum")
    xd = to_dev(x)
    from paper_2109_12626_amd import dpar
    dpar.dpar_allreduce(dpar.rows(xd), dpar.rows(xd), p, m, "float32", "sum",
                        0, torch.cuda.current_stream())
    dpar.dpar_check_status(torch.cuda.current_stream())
    assert_all_ranks_equal(xd.cpu().numpy(), want)


def test_separate_allocations_and_permuted_pointer_order():
    # buffers from separate allocations, handed over in an arbitrary order:
    # the rank order is the order of the pointer array
    p, m = 29, 777
    x = synth.generate("odd_det_u32_mat", 4, p, m)
    perm = np.random.default_rng(0).permutation(p)
    xs_t = [to_dev(x[i]) for i in range(p)]
    ys_t = [poisoned_like(t) for t in xs_t]
    from paper_2109_12626_amd import dpar
    xs = [xs_t[i].data_ptr() for i in perm]
    ys = [ys_t[i].data_ptr() for i in perm]
    dpar.dpar_allreduce(xs, ys, p, m, "u32mat2x2", "matmul", 5,
                        torch.cuda.current_stream())
    dpar.dpar_check_status(torch.cuda.current_stream())
    want = _want(x[perm], "u32mat2x2", "matmul")
    for i in range(p):
        got = from_dev(ys_t[i], x)
        assert np.array_equal(got, want), i


def test_shared_input_buffer():
    # every rank reads the same input buffer (inputs may overlap)
    from paper_2109_12626_amd import dpar
    p, m = 40, 3000
    x = synth.generate("uniform_int", 8, 1, m, lo=-9, hi=9)
    xd = to_dev(x)
    yd = torch.empty((p, m), dtype=torch.int32, device="cuda")
    dpar.dpar_allreduce([xd.data_ptr()] * p, dpar.rows(yd), p, m, "int32",
                        "sum", 6, torch.cuda.current_stream())
    dpar.dpar_check_status(torch.cuda.current_stream())
    want = _want(np.repeat(x, p, axis=0), "int32", "sum")
    assert_all_ranks_equal(yd.cpu().numpy(), want)


def test_int32_wraps_on_device():
    x = np.full((33, 100), 2 ** 31 - 1, dtype=np.int32)
    out = run(x, "int32", "sum", 2)
    assert_all_ranks_equal(out, _want(x, "int32", "sum"))


def test_repeat_runs_are_identical():
    p, m = 300, 1 << 14
    x = synth.generate("normal_f32", 77, p, m)
    outs = [run(x, "float32", "sum", b, e) for b, e in
            ((0, "ticket"), (1, "launch"), (64, "barrier"), (0, "ticket"))]
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])
    assert_all_ranks_equal(outs[0], _want(x, "float32", "sum"))


def test_single_rank_and_two_ranks():
    for p in (1, 2):
        x = synth.generate("odd_det_u32_mat", 12, p, 300)
        out = run(x, "u32mat2x2", "matmul", 7)
        assert_all_ranks_equal(out, _want(x, "u32mat2x2", "matmul"), f"p={p}")


def test_one_library_hip_runtime_loaded():
    # torch's HIP runtime and the library's must be the same object
    import paper_2109_12626_amd  # noqa: F401
    torch.zeros(1, device="cuda")
    maps = open("/proc/self/maps").read()
    libs = {ln.split()[-1] for ln in maps.splitlines()
            if "libamdhip64" in ln}
    assert len(libs) == 1, libs
    assert any("libdpar.so" in ln for ln in maps.splitlines())


# ------------------------------------------------------------ workloads

@pytest.mark.parametrize("b", list(configs.P36_INT.bs))
@pytest.mark.parametrize("exec", EXECS)
def test_p36_int32_sum_full(b, exec):
    w = configs.P36_INT
    x = workload_input(w)
    bb = resolve_b(b, w.p, w.m)
    out = run(x, "int32", "sum", bb, exec)
    assert_all_ranks_equal(out, _want(x, "int32", "sum"), f"b={bb} {exec}")


@pytest.mark.parametrize("dist", ["uniform_u32_mat", "odd_det_u32_mat"])
def test_p64_matmul_full(dist):
    w = configs.P64_MAT
    x = synth.generate(dist, w.seed, w.p, w.m)
    out = run(x, "u32mat2x2", "matmul", w.bs[0])
    assert_all_ranks_equal(out, _want(x, "u32mat2x2", "matmul"))


@pytest.mark.parametrize("w", [w for w in configs.ALL if w.p * w.m <= 1 << 27],
                         ids=lambda w: w.name)
def test_every_workload_against_the_c_oracle(w):
    """Each workload of at most 2^27 elements in its own dtype, operators
    and block counts, default call: every element of every rank against the
    plain C oracle (a second oracle, written independently of the numpy
    one)."""
    from oracle import c_oracle
    x = workload_input(w)
    for op in w.ops:
        want = c_oracle.allreduce(x, w.dtype, op, threads=8)
        for b in w.bs:
            bb = resolve_b(b, w.p, w.m)
            out = run(x, w.dtype, op, bb)
            assert_all_ranks_equal(out, want, f"{w.name} {op} b={bb}")


@pytest.mark.parametrize("unit", UNITS + [None])
@pytest.mark.parametrize("k", [4, 10, 16])
@pytest.mark.parametrize("op", ["max", "sum"])
@pytest.mark.parametrize("b", [1, "rule"])
def test_p1152_int32_sweep_full(k, op, b, unit):
    w = next(v for v in configs.P1152_SWEEP if v.m == 1 << k)
    x = workload_input(w)
    bb = resolve_b(b, w.p, w.m)
    with env_unit(unit):
        out = run(x, "int32", op, bb)
    assert_all_ranks_equal(out, _want(x, "int32", op), f"m=2^{k} b={bb}")


@pytest.mark.parametrize("unit", UNITS)
def test_p1152_fp32_reduced_size_every_element(unit):
    # the headline shape with fewer columns (several chunks and a ragged tail)
    w = configs.P1152_F32
    m = 3 * 4096 + 7
    x = workload_input(w, m=m)
    for exec in EXECS:
        with env_unit(unit):
            out = run(x, "float32", "sum", resolve_b("rule", w.p, m), exec)
        assert_all_ranks_equal(out, _want(x, "float32", "sum"), exec)


def test_plan_log_names_the_plan(capfd):
    """DPAR_LOG=1 prints the plan of each call on stderr (diagnostics only:
    the result is unchanged)."""
    from tests._gpu import _Env
    w = configs.P7_SMALL
    x = workload_input(w)
    with _Env("DPAR_LOG", 1):
        out = run(x, "int32", "sum", 0, "split")
    err = capfd.readouterr().err
    line = next(v for v in err.splitlines() if v.startswith("dpar: "))
    b = oracle.block_rule_lit(w.p, w.m)
    for part in (f"p={w.p}", f"m={w.m}", "int32 sum", "alg=dual_root",
                 "H=2", f"b={b} (rule)", "exec=split", "items="):
        assert part in line, (part, line)
    assert_all_ranks_equal(out, _want(x, "int32", "sum"), "logged call")


def test_phase_event_belongs_to_the_next_call_only():
    """dpar_set_phase_event: recorded between the split executor's two
    passes of the next call; a next call that runs another executor drops
    the setting, so a later split call leaves the event alone."""
    from paper_2109_12626_amd import dpar
    p, m = 64, 1 << 18
    x = synth.generate("uniform_int", 2310, p, m, lo=0, hi=1000)
    xd = to_dev(x)
    yd = poisoned_like(xd)
    xs, ys = dpar.pointers(dpar.rows(xd)), dpar.pointers(dpar.rows(yd))
    s = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    # recorded: start <= mid <= end
    t0, mid, t1 = ev(), ev(), ev()
    mid.record(s)
    t0.record(s)
    dpar.dpar_set_phase_event(mid)
    dpar.dpar_allreduce_ex(xs, ys, p, m, "int32", "sum", 1, "split", s)
    t1.record(s)
    t1.synchronize()
    assert 0 <= t0.elapsed_time(mid) <= t0.elapsed_time(t1)
    # dropped by a ticket call: the split call after it does not record it
    mark, t2 = ev(), ev()
    mark.record(s)
    t0.record(s)
    dpar.dpar_set_phase_event(mark)
    dpar.dpar_allreduce_ex(xs, ys, p, m, "int32", "sum", 1, "ticket", s)
    dpar.dpar_allreduce_ex(xs, ys, p, m, "int32", "sum", 1, "split", s)
    t2.record(s)
    t2.synchronize()
    assert mark.elapsed_time(t0) >= 0          # still the first record
    dpar.dpar_check_status(s)
    assert_all_ranks_equal(from_dev(yd, x), _want(x, "int32", "sum"),
                           "phase event calls")


@pytest.mark.parametrize("shift", [0, 1, 2, 3])
@pytest.mark.parametrize("m", [1, 3, 4, 7, 1023, 1 << 20, (1 << 20) + 5])
def test_one_rank_copies_at_every_alignment(m, shift):
    """p = 1: y_0 = x_0, through the copy kernel (16-byte lanes, the last
    up to 3 elements one per thread) on rows shifted by 0..3 elements off
    16-byte boundaries, with neighbours of the output left untouched; in
    place the call writes nothing."""
    from paper_2109_12626_amd import dpar
    x = synth.generate("uniform_int", 2320 + m % 997, 1, m + 8, lo=-1000, hi=1000)
    xd = to_dev(x)
    yd = torch.full((1, m + 8), POISON, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream()
    xs = [xd.data_ptr() + 4 * ((shift + 1) % 4)]
    ys = [yd.data_ptr() + 4 * shift]
    dpar.dpar_allreduce(xs, ys, 1, m, "int32", "sum", 0, s)
    dpar.dpar_check_status(s)
    got = yd.cpu().numpy()[0]
    src = x[0][(shift + 1) % 4:(shift + 1) % 4 + m]
    assert np.array_equal(got[shift:shift + m], src)
    assert (got[:shift] == POISON).all() and (got[shift + m:] == POISON).all()
    before = xd.clone()
    dpar.dpar_allreduce(xs, xs, 1, m, "int32", "sum", 0, s)
    dpar.dpar_check_status(s)
    assert torch.equal(xd, before)
