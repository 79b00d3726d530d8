"""Benchmark: effective reduction-to-all bandwidth on one MI355X.

Workload: p = 1152 virtual ranks (the 36 x 32 layout), m = 2^22 fp32 values
per rank drawn N(0, 1) from a seeded generator, operator SUM, block count b
from the sqrt(m log2 p) rule (b = 6532), the library's default executor
(ticketed up-phase in round order, then the broadcast pass).  One step = one
dpar_allreduce call: the tree-order reduction of all p vectors and the write
of y to all p output buffers, inputs and outputs resident in HBM.

Metric: effective GB/s = (p*m*4 bytes read + p*m*4 bytes written) / time,
and its fraction of the 8 TB/s HBM peak.

Prints ONE JSON line.  Extra lines go to stderr.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
  python bench.py --calib-copy      # a plain 4 GiB device copy, for the
                                    # rocprofv3 FETCH/WRITE calibration
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


def traffic_per_launch():
    """HBM bytes per launch from committed rocprofv3 counter runs, scaled by
    the same counters on a plain copy of known size; None when the kernel
    source changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_sha") != kernel_sha():
        return None
    fetch = t["fetch_kib_per_dispatch"] * 1024 * t["fetch_scale"]
    write = t["write_kib_per_dispatch"] * 1024 * t["write_scale"]
    return fetch + write


def cpu_baseline(x_host, b):
    """The CPU oracle, as it stands, on a bounded sample: all 1152 ranks,
    the first 2^20 of the 2^22 columns, tree-order reduce plus the copy of y
    into 1152 outputs.  numpy runs it on one thread."""
    import numpy as np
    import oracle
    cols = 1 << 20
    xs = x_host[:, :cols]
    out = np.empty((P, cols), dtype=np.float32)
    t0 = time.perf_counter()
    oracle.allreduce_all([xs[i] for i in range(P)], "float32", "sum", out=out)
    dt = time.perf_counter() - t0
    gbs = 2.0 * P * cols * ELEM / dt / 1e9
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"p={P}, first {cols} of {M} columns (1/4 of the "
                      f"workload), tree-order reduce + copy to {P} outputs, "
                      f"{dt:.2f} s"}


def calib_copy():
    import torch
    n = 1 << 30  # 4 GiB of fp32
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calib_copy_bytes": n * 4, "dispatches": 3}))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy", action="store_true")
    ap.add_argument("--exec", default="auto",
                    choices=["auto", "launch", "barrier", "ticket", "split"])
    args = ap.parse_args()

    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only; the p virtual ranks "
              "all live in one GPU's HBM (use --gpus 1)", file=sys.stderr)
        sys.exit(2)
    if args.calib_copy:
        calib_copy()
        return

    import numpy as np
    import torch

    import synth
    from paper_2109_12626_amd import dpar

    dev = torch.device("cuda:0")
    t0 = time.perf_counter()
    x_host = synth.generate("normal_f32", SEED, P, M)
    log(f"inputs generated in {time.perf_counter() - t0:.1f} s")
    xd = torch.from_numpy(x_host).to(dev)
    yd = torch.empty_like(xd)
    torch.cuda.synchronize()
    xs, ys = dpar.rows(xd), dpar.rows(yd)
    b = dpar.dpar_block_rule(P, M)
    stream = torch.cuda.current_stream(dev)

    def step():
        dpar.dpar_allreduce_ex(xs, ys, P, M, "float32", "sum", b, args.exec,
                               stream)

    for _ in range(args.warmup):
        step()
    dpar.dpar_check_status(stream)

    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        starts[k].record(stream)
        step()
        ends[k].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dpar.dpar_check_status(stream)
    per_launch_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    avg_ms = sum(per_launch_ms) / len(per_launch_ms)
    ms_per_step = wall * 1e3 / args.steps

    nbytes = 2.0 * P * M * ELEM
    value = nbytes / (ms_per_step * 1e-3) / 1e9
    achieved = nbytes / (avg_ms * 1e-3) / 1e9
    log(f"b={b} exec={args.exec}: wall {ms_per_step:.3f} ms/step, event "
        f"avg {avg_ms:.3f} ms (min {min(per_launch_ms):.3f}), "
        f"{value:.1f} GB/s = {value / HBM_PEAK_GBS:.1%} of peak")

    # spot check: a few columns against the oracle (outside the timed region)
    import oracle
    cols = np.array([0, 1, 2, 3, 1000, M // 2, M - 1])
    want = oracle.allreduce_tree(x_host[:, cols], "float32", "sum")
    got = yd[:, torch.from_numpy(cols).to(dev)].cpu().numpy()
    if not all(np.array_equal(got[i], want) for i in range(P)):
        log("bench: spot check against the oracle FAILED")
        sys.exit(1)

    cpu = None if args.no_cpu_baseline else cpu_baseline(x_host, b)
    if cpu:
        log(f"cpu oracle: {cpu['value']} GB/s ({cpu['sample']})")

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
        "config": {"workload": WORKLOAD, "p": P, "m": M, "op": "sum",
                   "b": b, "block_rule": "ceil(sqrt(m log2 p))",
                   "executor": "split" if args.exec == "auto" else args.exec,
                   "bytes_per_step": int(nbytes)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic_per_launch()},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
