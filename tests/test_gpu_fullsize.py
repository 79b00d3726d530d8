"""Full-size workloads at p = 1152, m = 2^22 (19.3 GB in, 19.3 GB out), run
in the launch configuration the benchmark times (block count from the
sqrt(m log2 p) rule, the default split executor), and with every algorithm
and executor at that size.

* fp32 SUM: every one of the 2^22 columns of y_0 is compared bit for bit
  with the CPU oracle's full evaluation in the trees' association (a few
  seconds of numpy per tree layout; the default call also against the plain
  C oracle), and every rank's row with y_0 on the device; the result also
  lies within the recursive summation bound of the exact sum.
* int32 SUM and MAX: every column equals the exact column sum (wrapped) and
  maximum, the plain definition that the exactly associative operators
  reach; sampled columns are also compared with the oracle's evaluation.
"""

import gc

import numpy as np
import pytest
import torch

import oracle
from synth import configs
from tests._gpu import _Env, need_gpu, poisoned_like, to_dev, workload_input

pytestmark = pytest.mark.gpu


def _sample_cols(m, b, rng):
    cols = set(range(64)) | set(range(m - 67, m))
    for j in (1, 2, b // 2, b - 1):
        s, _ = oracle.block_bounds(m, b, j)
        cols |= set(range(max(0, s - 5), min(m, s + 5)))
    cols |= set(rng.choice(m, 2048, replace=False).tolist())
    return np.array(sorted(cols))


def _run_full(w, op):
    from paper_2109_12626_amd import dpar
    x = workload_input(w)
    b = oracle.block_rule_lit(w.p, w.m)
    xd = to_dev(x)
    yd = poisoned_like(xd)
    s = torch.cuda.current_stream()
    dpar.dpar_allreduce(dpar.rows(xd), dpar.rows(yd), w.p, w.m, w.dtype, op,
                        b, s)
    dpar.dpar_check_status(s)
    return x, xd, yd, b


def _check_sampled(x, yd, b, dtype, op, seed, trees=None):
    cols = _sample_cols(x.shape[1], b, np.random.default_rng(seed))
    want = oracle.allreduce_tree(x[:, cols], dtype, op, trees=trees)
    got = yd[:, torch.from_numpy(cols).cuda()].cpu().numpy()
    for i in range(x.shape[0]):
        assert np.array_equal(got[i], want), f"rank {i}"


def _check_rows_identical(yd):
    for i in range(1, yd.shape[0]):
        assert torch.equal(yd[i], yd[0]), f"rank {i} differs from rank 0"


@pytest.fixture(autouse=True)
def _cleanup():
    need_gpu()
    yield
    gc.collect()
    torch.cuda.empty_cache()


def _check_all_columns(yd, want, what=""):
    """y_0 equals the oracle's y in every column, bit for bit (rows 1..p-1
    are compared with y_0 on the device by _check_rows_identical)."""
    got = yd[0].cpu().numpy()
    g = got.view(np.uint32)
    wv = np.ascontiguousarray(want).view(np.uint32)
    bad = np.flatnonzero(g != wv)
    assert bad.size == 0, (
        f"{what}: {bad.size} of {g.size} columns differ from the oracle, "
        f"first at {bad[0]}: got {got[bad[0]]!r} want {want[bad[0]]!r}")


@pytest.fixture(scope="module")
def fp32_full():
    """The headline input on the host and the device, and the oracle's full
    y for each tree layout (computed once, on first use)."""
    need_gpu()
    w = configs.P1152_F32
    x = workload_input(w)
    xd = to_dev(x)
    wants = {}

    def want(layout):
        if layout not in wants:
            trees = (oracle.build_trees(w.p) if layout == "dual" else
                     oracle.build_trees(w.p, layout="single"))
            wants[layout] = oracle.allreduce_tree(x, w.dtype, "sum",
                                                  trees=trees)
        return wants[layout]

    yield w, x, xd, want
    del xd
    gc.collect()
    torch.cuda.empty_cache()


def test_p1152_fp32_sum_full_size(fp32_full):
    """The benchmark's call (default executor, the rule's b = 6532): all
    4,194,304 columns against the oracle, all 1152 rows identical."""
    from paper_2109_12626_amd import dpar
    w, x, xd, want = fp32_full
    b = oracle.block_rule_lit(w.p, w.m)
    yd = poisoned_like(xd)
    s = torch.cuda.current_stream()
    dpar.dpar_allreduce(dpar.rows(xd), dpar.rows(yd), w.p, w.m, w.dtype,
                        "sum", b, s)
    dpar.dpar_check_status(s)
    _check_all_columns(yd, want("dual"), "default call")
    _check_rows_identical(yd)
    # every column within the recursive-summation bound of the exact sum:
    # at most 2 (H + 1) + 1 additions on any input's path, H = 9
    L = 2 * (9 + 1) + 1
    u = 2.0 ** -24
    gamma = L * u / (1 - L * u)
    y0 = yd[0].double()
    step = 1 << 18
    for c in range(0, w.m, step):
        blk = xd[:, c:c + step].double()
        exact = blk.sum(0)
        mag = blk.abs().sum(0)
        err = (y0[c:c + step] - exact).abs()
        # fp64 summation of 1152 terms is exact to ~1e-13 relative, far
        # below the fp32 bound
        assert bool((err <= gamma * mag + 1e-30).all()), f"columns from {c}"
    del yd, y0


def test_p1152_fp32_sum_against_the_c_oracle(fp32_full):
    """The benchmark's call once more, every column of y_0 against the plain
    C oracle (a second oracle, written independently of the numpy one) on
    the host's cores, and every row against y_0."""
    import os
    from oracle import c_oracle
    from paper_2109_12626_amd import dpar
    w, x, xd, _ = fp32_full
    b = oracle.block_rule_lit(w.p, w.m)
    yd = poisoned_like(xd)
    s = torch.cuda.current_stream()
    dpar.dpar_allreduce(dpar.rows(xd), dpar.rows(yd), w.p, w.m, w.dtype,
                        "sum", b, s)
    dpar.dpar_check_status(s)
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    want = c_oracle.allreduce(x, w.dtype, "sum", threads=threads)
    _check_all_columns(yd, want, "default call, C oracle")
    _check_rows_identical(yd)
    del yd


@pytest.mark.parametrize("op", ["sum", "max"])
def test_p1152_int32_full_size(op):
    w = next(v for v in configs.P1152_SWEEP if v.m == 1 << 22)
    x, xd, yd, b = _run_full(w, op)
    _check_sampled(x, yd, b, "int32", op, 2)
    _check_rows_identical(yd)
    step = 1 << 18
    y0 = yd[0]
    for c in range(0, w.m, step):
        blk = xd[:, c:c + step]
        if op == "sum":
            want = blk.to(torch.int64).sum(0)
            want = ((want + 2 ** 31) % 2 ** 32 - 2 ** 31).to(torch.int32)
        else:
            want = blk.max(0).values
        assert torch.equal(y0[c:c + step], want), f"columns from {c}"


@pytest.mark.parametrize("alg", ["dual", "single", "reduce_bcast"])
@pytest.mark.parametrize("exec", ["split", "ticket", "launch", "barrier",
                                  "rounds", "rounds_barrier"])
def test_p1152_fp32_every_alg_and_executor(fp32_full, alg, exec):
    """The headline shape through every algorithm and executor at the rule's
    b: every column bit-exact against the oracle's tree(s), every rank's row
    identical to rank 0's."""
    from paper_2109_12626_amd import dpar
    w, x, xd, want = fp32_full
    b = oracle.block_rule_lit(w.p, w.m)
    yd = poisoned_like(xd)
    s = torch.cuda.current_stream()
    dpar.dpar_allreduce_opt(dpar.rows(xd), dpar.rows(yd), w.p, w.m, w.dtype,
                            "sum", b, alg, exec, 0, -1, s)
    dpar.dpar_check_status(s)
    _check_all_columns(yd, want("dual" if alg == "dual" else "single"),
                       f"{alg}/{exec}")
    _check_rows_identical(yd)
    del yd


@pytest.mark.parametrize("exec,b", [("auto", 0), ("ticket", 0), ("rounds", 0),
                                    ("auto", 1), ("launch", 1)])
def test_rows_beyond_32_bit_offsets(exec, b):
    """p = 3 rows of 2^31 + 4099 int32 (8.6 GB each, 52 GB in and out): every
    byte offset past 2^32 goes through 64-bit address arithmetic.  The rows
    (not 16-byte aligned) are taken one element per lane (DPAR_SCALAR=1), so
    one launch of all work items (split) or of one round's chunks (b = 1)
    would need more than 2^32 threads and goes out in pieces; then once
    more with 16-byte lanes on the misaligned rows.  Checked against the
    exact wrapped column sum, computed on the device in int64, for every
    element (a property that holds at any size)."""
    from paper_2109_12626_amd import dpar
    need_gpu()
    p, m = 3, (1 << 31) + 4099
    g = torch.Generator(device="cuda").manual_seed(2170)
    xd = torch.randint(-(1 << 30), 1 << 30, (p, m), dtype=torch.int32,
                       device="cuda", generator=g)
    step = 1 << 28
    wants = []
    for c in range(0, m, step):
        want = xd[:, c:c + step].to(torch.int64).sum(0)
        wants.append(((want + 2 ** 31) % 2 ** 32 - 2 ** 31).to(torch.int32))
    s = torch.cuda.current_stream()
    for scalar in (1, 0):
        yd = poisoned_like(xd)
        with _Env("DPAR_SCALAR", scalar):
            dpar.dpar_allreduce_opt(dpar.rows(xd), dpar.rows(yd), p, m,
                                    "int32", "sum", b, "dual", exec, 0, -1, s)
        dpar.dpar_check_status(s)
        for k, c in enumerate(range(0, m, step)):
            for i in range(p):
                assert torch.equal(yd[i, c:c + step], wants[k]), \
                    (exec, scalar, i, c)
        del yd
    del xd
