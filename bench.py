"""Benchmark: effective reduction-to-all bandwidth on one MI355X.

Workload: p = 1152 virtual ranks (the 36 x 32 layout), m = 2^22 fp32 values
per rank drawn N(0, 1) from a seeded generator, operator SUM, block count b
from the sqrt(m log2 p) rule (b = 6532), the library's default executor
(the up-phase of every round, one workgroup per work item in round order,
then the broadcast pass).  One step = one
dpar_allreduce call: the tree-order reduction of all p vectors and the write
of y to all p output buffers, inputs and outputs resident in HBM.

Metric: effective GB/s = (p*m*4 bytes read + p*m*4 bytes written) / time,
and its fraction of the 8 TB/s HBM peak.

Prints ONE JSON line.  Extra lines go to stderr.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
  python bench.py --calib-copy      # a plain 4 GiB device copy, for the
                                    # rocprofv3 FETCH/WRITE calibration
  python bench.py --sweep OUT.jsonl # every workload, executor, block count
  python bench.py --table2          # the paper's Table 2 counts at p = 288
  python bench.py --copy-compare    # calls beside a device copy of their bytes
  python bench.py --copy-ceiling    # interleaved read+write rates, headline size
  python bench.py --fixed-cost      # fixed vs per-byte cost per phase, mid sizes
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

P, M, ELEM = 1152, 1 << 22, 4
SEED = 2113
WORKLOAD = "p1152_m2^22_fp32_sum"
HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_p1152_m2^22_fp32_sum.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2109_12626_amd", "csrc", "kernels.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_sha():
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic_per_launch(phase):
    """HBM bytes per launch of the phase's kernel from committed rocprofv3
    counter runs (FETCH_SIZE, WRITE_SIZE in KiB per dispatch), each scaled by
    what the same counter reads for a plain device copy of known size; None
    when the kernel source changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_sha") != kernel_sha() or phase not in t.get("kernels", {}):
        return None
    k = t["kernels"][phase]
    fetch = k["fetch_kib_per_dispatch"] * 1024 * t["fetch_scale"]
    write = k["write_kib_per_dispatch"] * 1024 * t["write_scale"]
    return int(fetch + write)


def host_cores():
    """Cores the oracle may use: the process's CPU affinity, at most 16 (one
    GPU's share of the host cores of an 8-GPU node)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _oracle_pass(rows, out, threads):
    """One pass of the numpy oracle over the whole workload: the tree-order
    reduction of all rows and the copy of y into every output row.  With
    threads > 1 the columns are cut into that many contiguous ranges, each
    evaluated by the unchanged oracle on its own thread (numpy releases the
    GIL inside its array operations)."""
    import oracle
    if threads == 1:
        oracle.allreduce_all(rows, "float32", "sum", out=out)
        return
    from concurrent.futures import ThreadPoolExecutor
    m = rows[0].shape[0]
    cuts = [m * k // threads for k in range(threads + 1)]

    def part(k):
        c0, c1 = cuts[k], cuts[k + 1]
        oracle.allreduce_all([r[c0:c1] for r in rows], "float32", "sum",
                             out=out[:, c0:c1])

    with ThreadPoolExecutor(max_workers=threads) as pool:
        list(pool.map(part, range(threads)))


def _c_oracle_pass(rows, out, threads):
    """One pass of the C oracle over the whole workload (the same reduction
    and copy-out; its own threads over contiguous column ranges)."""
    from oracle import c_oracle
    c_oracle.allreduce_all(rows, "float32", "sum", out, threads=threads)


def _time_legs(one_pass, rows, out):
    """Each pass repeated until at least 10 s have passed (at most 8
    passes), on one thread and on the host's cores: {threads: (GB/s, runs,
    seconds, seconds per run)}."""
    legs = {}
    for threads in (1, host_cores()):
        if threads in legs:
            continue
        runs, t0 = 0, time.perf_counter()
        while True:
            one_pass(rows, out, threads)
            runs += 1
            dt = time.perf_counter() - t0
            if dt >= 10.0 or runs >= 8:
                break
        per_run = dt / runs
        legs[threads] = (2.0 * P * M * ELEM / per_run / 1e9, runs, dt,
                         per_run)
    return legs


def _leg_record(legs, what):
    n = max(legs)
    gbs, runs, dt, per_run = legs[n]
    g1, runs1, dt1, per1 = legs[1]
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": n,
            "kind": "oracle",
            "sample": f"{what}: the whole workload (p={P}, m={M}), tree-order "
                      f"reduce + copy to {P} outputs, columns split over {n} "
                      f"threads, {runs} runs in {dt:.1f} s, {per_run:.2f} s "
                      f"per run",
            "single_thread": {"value": round(g1, 4), "unit": "GB/s",
                              "cores": 1,
                              "sample": f"{runs1} runs in {dt1:.1f} s, "
                                        f"{per1:.2f} s per run"}}


def cpu_baseline(x_host, b, check):
    """The CPU oracles, as they stand, on the whole workload: tree-order
    reduce of all 1152 ranks over all 2^22 columns plus the copy of y into
    1152 outputs, once on one thread, once with the columns split over the
    host's cores.  The plain C oracle's legs are the baseline; the numpy
    oracle's are reported beside them.  ``check(out, who)`` is called on
    each oracle's output (the full-column check of the GPU result)."""
    import numpy as np
    out = np.empty((P, M), dtype=np.float32)
    out.fill(0.0)               # first touch of the pages, outside the timing
    rows = [x_host[i] for i in range(P)]
    base = _leg_record(_time_legs(_c_oracle_pass, rows, out), "C oracle")
    check(out, "C oracle")
    out.fill(0.0)
    base["numpy_oracle"] = _leg_record(_time_legs(_oracle_pass, rows, out),
                                       "numpy oracle")
    check(out, "numpy oracle")
    return base


def calib_copy():
    import torch
    n = 1 << 30  # 4 GiB of fp32
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calib_copy_bytes": n * 4, "dispatches": 3}))


# Per-process counts of the paper's Table 2 (Section 2): int32 elements.
TABLE2_COUNTS = [0, 1, 2, 8, 15, 21, 25, 87, 150, 212, 250, 875, 1500, 2125,
                 2500, 8750, 15000, 21250, 25000, 87500, 150000, 212500,
                 250000, 875000, 1500000, 2125000, 2500000, 4597152, 6694304,
                 8388608]


def table2():
    """The paper's only experiment, replayed on one GPU: p = 288 virtual
    ranks (its 36 nodes x 8 processes), int32 SUM, the per-process counts of
    its Table 2 and its fixed block of 16000 elements (b = ceil(count /
    16000)).  Columns: the doubly-pipelined dual-root algorithm with the
    default executor and with the round-structured executor (the paper's
    b + H rounds, down-phase included), and the single-tree pipelined
    reduce-then-broadcast (User-Allreduce1) with the same two executors.
    Each entry: minimum and median of the per-call GPU time (HIP events on
    the call's stream) over back-to-back calls after warm-up; the paper
    takes the minimum over repetitions too."""
    import numpy as np
    import torch

    from paper_2109_12626_amd import dpar
    p, blk = 288, 16000
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    g = torch.Generator(device=dev)
    g.manual_seed(2109)
    variants = [("dual", "auto"), ("dual", "rounds"),
                ("reduce_bcast", "auto"), ("reduce_bcast", "rounds")]
    out = []
    for count in TABLE2_COUNTS:
        b = max(1, -(-count // blk))
        # each rank's input and output in an allocation of its own, as each
        # of the paper's processes has its own buffers (a p x count array
        # would leave most rows off the 128-byte lines for odd counts)
        x = y = None
        torch.cuda.empty_cache()
        x = [torch.randint(-1000, 1001, (max(count, 1),), dtype=torch.int32,
                           device=dev, generator=g) for _ in range(p)]
        y = [torch.empty_like(t) for t in x]
        xs, ys = dpar.pointers(x), dpar.pointers(y)
        ref = None
        rec = {"count": count, "b": b}
        for alg, ex in variants:
            def call():
                dpar.dpar_allreduce_opt(xs, ys, p, count, "int32", "sum", b,
                                        alg, ex, 0, -1, stream)
            reps = 20 if count <= 250000 else 8
            for _ in range(3):
                call()
            dpar.dpar_check_status(stream)
            ts = []
            for _ in range(reps):
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                call()
                e1.record(stream)
                e1.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e3)
            dpar.dpar_check_status(stream)
            if count:
                # every algorithm and executor gives the same int32 result
                got = torch.stack([t[:count:max(1, count // 4096)]
                                   for t in y])
                assert bool((got == got[0]).all()), (count, alg, ex)
                if ref is None:
                    ref = got[0]
                assert torch.equal(ref, got[0]), (count, alg, ex)
            rec[f"{alg}/{ex}"] = {"us_min": round(min(ts), 2),
                                  "us_median": round(float(np.median(ts)), 2)}
        out.append(rec)
        log(json.dumps(rec))
    print(json.dumps({"table2_p": p, "block": blk, "rows": out}))


COPY_COMPARE = [  # p, m, dtype, op
    (36, 1 << 20, "int32", "sum"),
    (64, 1 << 18, "u32mat2x2", "matmul"),
    (1152, 1 << 16, "int32", "sum"),
    (1152, 1 << 16, "int32", "max"),
    (1152, 1 << 18, "float32", "sum"),
    (1152, 1 << 22, "float32", "sum"),
]


def copy_compare():
    """The library's call (default executor, b from the sqrt(m log2 p)
    rule) beside a plain device copy of the same bytes (torch's copy_ of the
    [p, m] input into the [p, m] output: p*m*e read, p*m*e written, as the
    call moves).  Both back to back on warm caches, the minimum and median of
    20 timed calls after 3 untimed ones."""
    import numpy as np
    import torch

    from paper_2109_12626_amd import dpar
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    g = torch.Generator(device=dev)
    g.manual_seed(2109)
    out = []

    def timed(fn):
        for _ in range(3):
            fn()
        ts = []
        for _ in range(20):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return min(ts), float(np.median(ts))

    for p, m, dt, op in COPY_COMPARE:
        words = m * (4 if dt == "u32mat2x2" else 1)
        if dt == "float32":
            x = torch.randn(p, words, device=dev, generator=g)
        else:
            x = torch.randint(-2 ** 31, 2 ** 31 - 1, (p, words),
                              dtype=torch.int32, device=dev, generator=g)
        y = torch.empty_like(x)
        xs, ys = dpar.pointers(dpar.rows(x)), dpar.pointers(dpar.rows(y))
        b = dpar.dpar_block_rule(p, m)
        nbytes = 2 * x.numel() * 4

        def call():
            dpar.dpar_allreduce(xs, ys, p, m, dt, op, b, stream)
        lib_t = timed(call)
        dpar.dpar_check_status(stream)
        assert bool((y[:, :4096] == y[0, :4096]).all()), (p, m, dt, op)
        copy_t = timed(lambda: y.copy_(x))
        rec = {"p": p, "m": m, "dtype": dt, "op": op, "b": b,
               "bytes": nbytes,
               "call_ms": [round(lib_t[0], 4), round(lib_t[1], 4)],
               "copy_ms": [round(copy_t[0], 4), round(copy_t[1], 4)],
               "call_GBs": round(nbytes / lib_t[0] / 1e6, 1),
               "copy_GBs": round(nbytes / copy_t[0] / 1e6, 1)}
        out.append(rec)
        log(json.dumps(rec))
        del x, y
        torch.cuda.empty_cache()
    print(json.dumps({"copy_compare": out}))


def copy_ceiling():
    """Interleaved read+write HBM traffic at the headline size, 19.33 GB read
    and 19.33 GB written per call, each entry the minimum and median of 8
    timed calls after 2 untimed ones (HIP events on the call's stream, warm):
      - the library at p = 1 (its copy kernel: one 16-byte load and one
        streaming store per thread, 256 threads per workgroup, the broadcast
        pass's shape) copying one row of p*m floats;
      - torch's copy_ of the same bytes (the runtime's copy kernel);
      - the headline call with the executors that interleave the two
        directions in one launch (ticket; one fused launch of every work
        item) and with the split executor, whose phases run one direction
        each (their times with the phase event)."""
    import numpy as np
    import torch

    from paper_2109_12626_amd import dpar
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    n = P * M
    nbytes = 2 * n * ELEM
    out = {}

    def timed(fn, phase=False):
        for _ in range(2):
            fn()
        ts, ups = [], []
        for _ in range(8):
            e0, e1, e2 = [torch.cuda.Event(enable_timing=True)
                          for _ in range(3)]
            e1.record(stream)
            e0.record(stream)
            if phase:
                dpar.dpar_set_phase_event(e1)
            fn()
            e2.record(stream)
            e2.synchronize()
            ts.append(e0.elapsed_time(e2))
            if phase:
                ups.append(e0.elapsed_time(e1))
        rec = {"ms_min": round(min(ts), 4),
               "ms_median": round(float(np.median(ts)), 4),
               "GB/s": round(nbytes / min(ts) / 1e6, 1)}
        if phase:
            up = min(ups)
            rec["up_ms"] = round(up, 4)
            rec["up_read_GB/s"] = round((n + M) * ELEM / up / 1e6, 1)
            bc = float(np.median([t - u for t, u in zip(ts, ups)]))
            rec["broadcast_ms_median"] = round(bc, 4)
        return rec

    x = torch.randn(P, M, device=dev)
    y = torch.empty_like(x)
    xs, ys = dpar.pointers(dpar.rows(x)), dpar.pointers(dpar.rows(y))
    flat_x, flat_y = x.view(-1), y.view(-1)
    out["library_copy_p1"] = timed(lambda: dpar.dpar_allreduce(
        [flat_x.data_ptr()], [flat_y.data_ptr()], 1, n, "float32", "sum", 1,
        stream))
    assert torch.equal(flat_y[:: 1 << 20], flat_x[:: 1 << 20])
    out["torch_copy_"] = timed(lambda: flat_y.copy_(flat_x))
    b = dpar.dpar_block_rule(P, M)
    call = lambda ex: (lambda: dpar.dpar_allreduce_ex(  # noqa: E731
        xs, ys, P, M, "float32", "sum", b, ex, stream))
    out["call_ticket"] = timed(call("ticket"))
    os.environ["DPAR_FUSE_BELOW_KB"] = str(1 << 30)
    out["call_one_fused_launch"] = timed(call("auto"))
    os.environ.pop("DPAR_FUSE_BELOW_KB")
    out["call_split"] = timed(call("split"), phase=True)
    dpar.dpar_check_status(stream)
    for k, v in out.items():
        log(k, json.dumps(v))
    print(json.dumps({"copy_ceiling_bytes_per_call": nbytes, "rates": out}))


FIXED_COST = [  # name, p, m, dtype, op
    ("p36_int32_sum", 36, 1 << 20, "int32", "sum"),
    ("p64_u32mat2x2_matmul", 64, 1 << 18, "u32mat2x2", "matmul"),
    ("p1152_int32_sum", 1152, 1 << 16, "int32", "sum"),
]


def fixed_cost():
    """Where the mid-size workloads' time goes: each is run with the split
    executor at 1/4 .. 8 times its m (same p, dtype, operator, b from the
    sqrt(m log2 p) rule), cold caches (a 512 MiB write between calls), and
    each phase's minimum time t over 10 calls is fitted as t = a + B / r
    (least squares over the six sizes; B the phase's algorithmic bytes):
    a is what the phase costs whatever it moves (launch, filling the GPU
    with workgroups, draining the last ones), r the rate at which it moves
    bytes once running.  Also the AUTO executor's whole call."""
    import numpy as np
    import torch

    from paper_2109_12626_amd import dpar
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    flush = torch.empty(1 << 27, dtype=torch.float32, device=dev)
    out = []
    for name, p, m0, dt, op in FIXED_COST:
        esz = 16 if dt == "u32mat2x2" else 4
        pts = []
        for f in (0.25, 0.5, 1, 2, 4, 8):
            m = int(m0 * f)
            x = torch.randint(0, 1 << 16, (p, m * esz // 4), dtype=torch.int32,
                              device=dev)
            y = torch.empty_like(x)
            xs, ys = dpar.pointers(dpar.rows(x)), dpar.pointers(dpar.rows(y))
            b = dpar.dpar_block_rule(p, m)
            rec = {"m": m, "b": b}
            for ex in ("split", "auto"):
                fn = lambda: dpar.dpar_allreduce_ex(  # noqa: E731
                    xs, ys, p, m, dt, op, b, ex, stream)
                fn()
                ups, tots = [], []
                for it in range(12):
                    flush.fill_(float(it))
                    e0, e1, e2 = [torch.cuda.Event(enable_timing=True)
                                  for _ in range(3)]
                    e1.record(stream)
                    e0.record(stream)
                    if ex == "split":
                        dpar.dpar_set_phase_event(e1)
                    fn()
                    e2.record(stream)
                    e2.synchronize()
                    if it >= 2:
                        tots.append(e0.elapsed_time(e2))
                        ups.append(e0.elapsed_time(e1))
                if ex == "split":
                    rec["up_ms"] = min(ups)
                    rec["bcast_ms"] = min(t - u for t, u in zip(tots, ups))
                    rec["split_ms"] = min(tots)
                else:
                    rec["auto_ms"] = min(tots)
            dpar.dpar_check_status(stream)
            rec["up_bytes"] = (p + 1) * m * esz
            rec["bcast_bytes"] = (p - 1) * m * esz
            rec["call_bytes"] = 2 * p * m * esz
            pts.append(rec)
            del x, y
            torch.cuda.empty_cache()

        def fit(tkey, bkey):
            B = np.array([r[bkey] for r in pts], dtype=float)
            t = np.array([r[tkey] for r in pts], dtype=float) * 1e-3
            A = np.stack([np.ones_like(B), B], axis=1)
            (a, inv_r), *_ = np.linalg.lstsq(A, t, rcond=None)
            return {"fixed_us": round(a * 1e6, 2),
                    "rate_TB/s": round(1.0 / inv_r / 1e12, 3)}
        own = next(r for r in pts if r["m"] == m0)
        res = {"workload": name, "p": p, "m": m0, "dtype": dt, "op": op,
               "up": fit("up_ms", "up_bytes"),
               "broadcast": fit("bcast_ms", "bcast_bytes"),
               "split_call": fit("split_ms", "call_bytes"),
               "auto_call": fit("auto_ms", "call_bytes"),
               "at_own_m": {k: round(own[k], 4) for k in
                            ("up_ms", "bcast_ms", "split_ms", "auto_ms")},
               "points": [{k: (round(v, 4) if isinstance(v, float) else v)
                           for k, v in r.items()} for r in pts]}
        out.append(res)
        log(json.dumps({k: v for k, v in res.items() if k != "points"}))
    print(json.dumps({"fixed_cost": out}))


# AUTO's choice audited against the forced alternatives, int32 SUM: (1) p
# ranks, rows of n chunks of 16 KB (m = 4096 n), post-order or wide items;
# (2) many ranks, short rows, post-order, subtree or level items.
def _forced(unit, fused):
    env = {"DPAR_UNIT": unit}
    if fused:
        env["DPAR_FUSE_BELOW_KB"] = str(1 << 30)
    return env, "auto" if fused else "split"


AUDIT_GRIDS = [
    ("rows of 16 KB chunks",
     (8, 12, 16, 20, 24, 32, 36, 40, 48, 64, 96, 128, 200, 288, 511, 700,
      1152),
     [4096 * n for n in (32, 64, 96, 128, 160, 192, 224, 256, 320, 401, 512,
                         640)],
     {"auto": ({}, "auto"),
      "postorder_split": _forced("seq", False),
      "postorder_fused": _forced("seq", True),
      "wide_split": _forced("wide", False),
      "wide_fused": _forced("wide", True)}),
    ("many ranks, short rows",
     (256, 400, 511, 700, 1152, 2304, 4608),
     [256, 1024, 4096, 8192, 16384, 32768, 65536, 131072, 262144],
     {"auto": ({}, "auto"),
      "postorder_split": _forced("seq", False),
      "postorder_fused": _forced("seq", True),
      "subtree_split": _forced("sub", False),
      "subtree_fused": _forced("sub", True),
      "level_split": _forced("level", False),
      "level_fused": _forced("level", True)}),
]


def auto_audit():
    """AUTO's executor and work-item choice beside the forced alternatives
    (the work items of each grid, split or one fused launch; a forced item
    that does not fit falls back as the library does), int32 SUM over the
    grids of AUDIT_GRIDS, minimum of 8 calls (two passes over the modes of
    4 each), in two regimes: back-to-back
    calls, and calls each after a 512 MB write that flushes the caches.
    Prints one JSON line per case and a summary per grid and regime: how far
    AUTO is from the best of the forced modes and itself."""
    import torch

    from paper_2109_12626_amd import dpar
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    flush = torch.empty(1 << 27, dtype=torch.float32, device=dev)
    keys = ("DPAR_UNIT", "DPAR_FUSE_BELOW_KB")
    saved = {k: os.environ.get(k) for k in keys}
    grids = []
    for (title, ps, ms, modes), flushed in (
            (g, f) for f in (False, True) for g in AUDIT_GRIDS):
        rows = []
        for p, m in ((p, m) for p in ps for m in ms):
            if 2 * p * m * 4 > 24e9:
                continue
            x = torch.randint(-1000, 1000, (p, m), dtype=torch.int32,
                              device=dev)
            y = torch.empty_like(x)
            xs, ys = dpar.pointers(dpar.rows(x)), dpar.pointers(dpar.rows(y))
            rec = {"p": p, "m": m, "flushed": flushed}
            # two passes over the modes, the minimum of both: no mode is
            # only measured first, right after the inputs were written
            ts = {name: [] for name in modes}
            for _ in range(2):
                for name, (env, ex) in modes.items():
                    for k in keys:
                        os.environ.pop(k, None)
                    os.environ.update(env)
                    fn = lambda: dpar.dpar_allreduce_ex(  # noqa: E731
                        xs, ys, p, m, "int32", "sum", 0, ex, stream)
                    fn()
                    dpar.dpar_check_status(stream)
                    for it in range(4):
                        if flushed:
                            flush.fill_(float(it))
                        e0 = torch.cuda.Event(enable_timing=True)
                        e1 = torch.cuda.Event(enable_timing=True)
                        e0.record(stream)
                        fn()
                        e1.record(stream)
                        e1.synchronize()
                        ts[name].append(e0.elapsed_time(e1) * 1e3)
            for name in modes:
                rec[name + "_us"] = round(min(ts[name]), 1)
            best = min(modes, key=lambda k: rec[k + "_us"])
            rec["best"] = best
            rec["auto_over_best_pct"] = round(
                (rec["auto_us"] / rec[best + "_us"] - 1) * 100, 1)
            rows.append(rec)
            log(json.dumps(rec))
            del x, y
            torch.cuda.empty_cache()
        over = sorted(r["auto_over_best_pct"] for r in rows)
        grids.append({"grid": title, "flushed": flushed,
                      "modes": list(modes), "cases": rows,
                      "auto_over_best_pct": {
                          "mean": round(sum(over) / len(over), 2),
                          "median": over[len(over) // 2],
                          "max": over[-1],
                          "over_3": sum(v > 3 for v in over),
                          "over_6": sum(v > 6 for v in over)}})
    for k, v in saved.items():
        if v is None:
            os.environ.pop(k, None)
        else:
            os.environ[k] = v
    print(json.dumps({"auto_audit": grids}))


def sweep(out_path, only=(), execs=("split", "ticket", "launch", "barrier"),
          algs=("dual",)):
    """Every workload x executor x block count, cold caches (a 512 MiB
    scratch write between calls), min and median of several calls.  Writes
    JSON lines to out_path and a table to stderr."""
    import numpy as np
    import torch

    import synth
    from synth import configs
    from paper_2109_12626_amd import dpar

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    scratch = torch.empty(1 << 27, dtype=torch.float32, device=dev)
    out = open(out_path, "w")

    def timed(fn, reps):
        ts = []
        for _ in range(reps):
            scratch.fill_(1.0)                      # evict L2 and MALL
            a = torch.cuda.Event(enable_timing=True)
            z = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            z.record(stream)
            z.synchronize()
            ts.append(a.elapsed_time(z))
        return min(ts), float(np.median(ts))

    def alpha_beta(xs, ys, w, op):
        # per-round executor cost (launch per round) and per-column cost
        f = lambda b: (lambda: dpar.dpar_allreduce_ex(  # noqa: E731
            xs, ys, w.p, w.m, w.dtype, op, b, "launch", stream))
        t1 = timed(f(1), 3)[0]
        bb = min(256, w.m)
        tb = timed(f(bb), 3)[0]
        alpha = max((tb - t1) / max(bb - 1, 1), 1e-4) * 1e-3   # s per round
        beta = t1 * 1e-3 / w.m                                   # s per column
        return alpha, beta

    for w in configs.ALL:
        if only and not any(o in w.name for o in only):
            continue
        x = synth.generate(w.dist, w.seed, w.p, w.m, **w.dist_kw)
        xd = torch.from_numpy(x.view(np.int32) if x.dtype == np.uint32
                              else x).to(dev)
        yd = torch.empty_like(xd)
        xs, ys = dpar.pointers(dpar.rows(xd)), dpar.pointers(dpar.rows(yd))
        nbytes = 2.0 * w.p * w.m * (16 if w.dtype == "u32mat2x2" else 4)
        for op in w.ops:
            alpha, beta = alpha_beta(xs, ys, w, op)
            bcal = dpar.dpar_block_rule(w.p, w.m, alpha, beta)
            blist = []
            for b in list(w.bs) + [1, "cal"]:
                bb = (dpar.dpar_block_rule(w.p, w.m) if b == "rule" else
                      bcal if b == "cal" else b)
                tag = b if isinstance(b, str) else "given"
                if bb not in [v for v, _ in blist]:
                    blist.append((bb, tag))
            for bb, tag in blist:
              for alg in algs:
                for ex in execs:
                    slow = ex in ("launch", "barrier", "rounds",
                                  "rounds_barrier") and bb > 512
                    reps = 2 if slow else 7
                    fn = lambda: dpar.dpar_allreduce_opt(  # noqa: E731
                        xs, ys, w.p, w.m, w.dtype, op, bb, alg, ex, 0, -1,
                        stream)
                    fn()
                    dpar.dpar_check_status(stream)
                    tmin, tmed = timed(fn, reps)
                    rec = {"workload": w.name, "op": op, "b": bb, "b_kind": tag,
                           "alg": alg, "exec": ex, "ms_min": round(tmin, 4),
                           "ms_median": round(tmed, 4),
                           "GB/s": round(nbytes / (tmin * 1e-3) / 1e9, 2),
                           "pct_peak": round(100 * nbytes / (tmin * 1e-3) / 1e9
                                             / HBM_PEAK_GBS, 2),
                           "alpha_us": round(alpha * 1e6, 3),
                           "beta_ns": round(beta * 1e9, 4)}
                    out.write(json.dumps(rec) + "\n")
                    out.flush()
                    log(f"{w.name:34s} {op:4s} b={bb:<6d} ({tag:5s}) "
                        f"{alg:12s} {ex:14s} "
                        f"min {tmin:9.4f} ms  med {tmed:9.4f} ms  "
                        f"{rec['GB/s']:9.1f} GB/s  {rec['pct_peak']:5.1f}%")
        del xd, yd, x
        torch.cuda.empty_cache()
    out.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy", action="store_true")
    ap.add_argument("--table2", action="store_true",
                    help="the paper's Table 2 counts at p = 288")
    ap.add_argument("--copy-compare", action="store_true",
                    help="calls beside a plain device copy of their bytes")
    ap.add_argument("--copy-ceiling", action="store_true",
                    help="interleaved read+write rates at the headline size")
    ap.add_argument("--fixed-cost", action="store_true",
                    help="fixed and per-byte cost of each phase, mid sizes")
    ap.add_argument("--auto-audit", action="store_true",
                    help="AUTO's choice beside forced work items and "
                         "executors, int32 SUM over a grid of p and m")
    ap.add_argument("--sweep", metavar="OUT_JSONL",
                    help="measure every workload, executor and block count")
    ap.add_argument("--only", default="",
                    help="with --sweep: comma-separated workload-name parts")
    ap.add_argument("--sweep-execs", default="split,ticket,launch,barrier",
                    help="with --sweep: comma-separated executors")
    ap.add_argument("--sweep-algs", default="dual",
                    help="with --sweep: comma-separated algorithms")
    ap.add_argument("--alg", default="dual",
                    choices=["dual", "single", "reduce_bcast"],
                    help="trees: dual roots (the paper's algorithm), one "
                         "tree, or one tree with reduce then broadcast")
    ap.add_argument("--workload", default=WORKLOAD,
                    help="time another workload (name from synth.configs) "
                         "with the same protocol; the default is the headline")
    ap.add_argument("--op", default=None, help="with --workload")
    ap.add_argument("--b", type=int, default=None,
                    help="block count (default: the sqrt(m log2 p) rule)")
    ap.add_argument("--exec", default="auto",
                    choices=["auto", "launch", "barrier", "ticket", "split",
                             "rounds", "rounds_barrier"])
    args = ap.parse_args()

    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only; the p virtual ranks "
              "all live in one GPU's HBM (use --gpus 1)", file=sys.stderr)
        sys.exit(2)
    if args.calib_copy:
        calib_copy()
        return
    if args.table2:
        table2()
        return
    if args.copy_compare:
        copy_compare()
        return
    if args.copy_ceiling:
        copy_ceiling()
        return
    if args.fixed_cost:
        fixed_cost()
        return
    if args.auto_audit:
        auto_audit()
        return
    if args.sweep:
        sweep(args.sweep, [v for v in args.only.split(",") if v],
              [v for v in args.sweep_execs.split(",") if v],
              [v for v in args.sweep_algs.split(",") if v])
        return

    import numpy as np
    import torch

    import synth
    from paper_2109_12626_amd import dpar

    from synth import configs
    w = next(v for v in configs.ALL if v.name == args.workload)
    op = args.op or w.ops[0]
    p_, m_, esz = w.p, w.m, (16 if w.dtype == "u32mat2x2" else 4)
    headline = (w.name == WORKLOAD and op == "sum" and args.b is None
                and args.alg == "dual")
    dev = torch.device("cuda:0")
    t0 = time.perf_counter()
    x_host = synth.generate(w.dist, w.seed, p_, m_, **w.dist_kw)
    log(f"inputs generated in {time.perf_counter() - t0:.1f} s")
    xd = torch.from_numpy(x_host.view(np.int32) if x_host.dtype == np.uint32
                          else x_host).to(dev)
    yd = torch.empty_like(xd)
    torch.cuda.synchronize()
    xs, ys = dpar.pointers(dpar.rows(xd)), dpar.pointers(dpar.rows(yd))
    b = args.b if args.b is not None else dpar.dpar_block_rule(p_, m_)
    stream = torch.cuda.current_stream(dev)

    def step():
        dpar.dpar_allreduce_opt(xs, ys, p_, m_, w.dtype, op, b, args.alg,
                                args.exec, 0, -1, stream)

    for _ in range(args.warmup):
        step()
    dpar.dpar_check_status(stream)
    # poison the outputs so that the checks after the timed region see what
    # the timed calls wrote, not what the warm-up calls left
    yd.view(torch.int32).fill_(-0x21524111)   # 0xDEADBEEF
    torch.cuda.synchronize()

    split = args.exec in ("auto", "split")
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    starts = [ev() for _ in range(args.steps)]
    mids = [ev() for _ in range(args.steps)]
    ends = [ev() for _ in range(args.steps)]
    for e in mids:          # create the events before handing them over
        e.record(stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        starts[k].record(stream)
        if split:
            dpar.dpar_set_phase_event(mids[k])
        step()
        ends[k].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dpar.dpar_check_status(stream)
    call_ms = [s_.elapsed_time(e) for s_, e in zip(starts, ends)]
    avg_ms = sum(call_ms) / len(call_ms)
    ms_per_step = wall * 1e3 / args.steps
    nbytes = 2.0 * p_ * m_ * esz
    value = nbytes / (ms_per_step * 1e-3) / 1e9

    def rate(nb, ms):
        return round(nb / (ms * 1e-3) / 1e9, 2)

    srt = sorted(call_ms)
    med_ms = (srt[(len(srt) - 1) // 2] + srt[len(srt) // 2]) / 2
    phases = {"call": {"avg_ms": round(avg_ms, 4),
                       "min_ms": round(srt[0], 4),
                       "median_ms": round(med_ms, 4),
                       "algorithmic_bytes": int(nbytes),
                       "GB/s": rate(nbytes, avg_ms)}}
    if split:
        up_ms = sum(s_.elapsed_time(m) for s_, m in zip(starts, mids)) / args.steps
        bc_ms = sum(m.elapsed_time(e) for m, e in zip(mids, ends)) / args.steps
        up_bytes = p_ * m_ * esz + m_ * esz          # read all x, write y_0
        bc_bytes = (p_ - 1) * m_ * esz               # write y_1 .. y_{p-1}
        phases["up"] = {"kernel": "k_round (up-phase of every round, y into y_0)",
                        "avg_ms": round(up_ms, 4), "algorithmic_bytes": up_bytes,
                        "GB/s": rate(up_bytes, up_ms)}
        phases["broadcast"] = {"kernel": "k_bcast (y_0 to the other ranks)",
                               "avg_ms": round(bc_ms, 4),
                               "algorithmic_bytes": bc_bytes,
                               "GB/s": rate(bc_bytes, bc_ms)}
        dom = max(("up", "broadcast"), key=lambda k: phases[k]["avg_ms"])
    else:
        phases["fused"] = {"kernel": "k_ticket/k_round/k_barrier (fused)",
                           "avg_ms": round(avg_ms, 4),
                           "algorithmic_bytes": int(nbytes),
                           "GB/s": rate(nbytes, avg_ms)}
        dom = "fused"
    dk = phases[dom]
    log(f"b={b} exec={args.exec}: wall {ms_per_step:.3f} ms/step, call avg "
        f"{avg_ms:.3f} ms (min {min(call_ms):.3f}), {value:.1f} GB/s = "
        f"{value / HBM_PEAK_GBS:.1%} of peak; phases {json.dumps(phases)}")

    # checks outside the timed region: every output row equals y_0, and
    # y_0 matches the oracle (sampled columns here; every column below when
    # the oracle's full output is at hand)
    import oracle
    for i in range(1, p_):
        if not torch.equal(yd[i], yd[0]):
            log(f"bench: output row {i} differs from row 0")
            sys.exit(1)
    cols = np.unique(np.array([0, 1, 2, 3, 1000, m_ // 2, m_ - 1]) % m_)
    trees = (oracle.build_trees(p_) if args.alg == "dual" else
             oracle.build_trees(p_, layout="single"))
    want = oracle.allreduce_tree(x_host[:, cols], w.dtype, op, trees=trees)
    got = yd[0, torch.from_numpy(cols).to(dev)].cpu().numpy()
    if x_host.dtype == np.uint32:
        got = got.view(np.uint32)
    if not np.array_equal(got, want):
        log("bench: spot check against the oracle FAILED")
        sys.exit(1)

    cpu = None
    if headline and not args.no_cpu_baseline:
        y0 = yd[0].cpu().numpy()

        def check(full, who):
            for r in (0, p_ // 2, p_ - 1):
                if not np.array_equal(full[r].view(np.uint32),
                                      full[0].view(np.uint32)):
                    log(f"bench: the {who}'s output rows differ")
                    sys.exit(1)
            bad = np.flatnonzero(y0.view(np.uint32) != full[0].view(np.uint32))
            if bad.size:
                log(f"bench: {bad.size} of {m_} columns differ from the "
                    f"{who}, first at {bad[0]}")
                sys.exit(1)

        cpu = cpu_baseline(x_host, b, check)
        cpu["checked"] = (f"all {m_} columns of y_0 equal the C oracle's y "
                          "and the numpy oracle's y")
        npo = cpu["numpy_oracle"]
        log(f"cpu oracle (C): {cpu['value']} GB/s on {cpu['cores']} threads, "
            f"{cpu['single_thread']['value']} GB/s on one; numpy oracle: "
            f"{npo['value']} GB/s on {npo['cores']} threads, "
            f"{npo['single_thread']['value']} GB/s on one; {cpu['checked']}")

    line = {
        "metric": "effective allreduce GB/s and % of HBM peak at p=1152, "
                  "m=2^22 fp32 SUM, 1 GPU",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "pct_of_hbm_peak": round(100.0 * value / HBM_PEAK_GBS, 2),
        "config": {"workload": w.name, "p": p_, "m": m_, "op": op,
                   "b": b, "block_rule": ("ceil(sqrt(m log2 p))"
                                          if args.b is None else "given"),
                   "executor": "split" if args.exec == "auto" else args.exec,
                   "algorithm": args.alg,
                   "bytes_per_step": int(nbytes)},
        "roofline": {"bound": "hbm", "kernel": dk["kernel"],
                     "achieved": dk["GB/s"], "peak": HBM_PEAK_GBS,
                     "unit": "GB/s",
                     "frac": round(dk["GB/s"] / HBM_PEAK_GBS, 4),
                     "traffic": traffic_per_launch(dom) if headline else None,
                     "per_launch_bytes": dk["algorithmic_bytes"],
                     "avg_launch_ms": dk["avg_ms"]},
        "phases": phases,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
