"""Calls in flight on two streams at once, and from two host threads: each
call has its own counter slot and staged pointer table, so results must not
mix.  The persistent grid-barrier executors are left out: they need every
workgroup of their grid resident at once and are not meant to share the GPU
with other work."""

import threading

import numpy as np
import pytest
import torch

import oracle
import synth
from tests._gpu import POISON, assert_all_ranks_equal, lib, need_gpu, to_dev

pytestmark = pytest.mark.gpu

EXECS = ["split", "ticket", "launch", "rounds"]


def _case(seed, p, m):
    x = synth.generate("normal_f32", seed, p, m)
    return x, oracle.allreduce_tree(x, "float32", "sum")


def _poisoned(xd):
    y = torch.empty_like(xd)
    y.view(torch.int32).fill_(POISON)
    return y


@pytest.mark.parametrize("e1", EXECS)
@pytest.mark.parametrize("e2", EXECS)
def test_two_streams_interleaved(e1, e2):
    need_gpu()
    dpar = lib()
    (x1, w1), (x2, w2) = _case(2130, 36, 50001), _case(2131, 100, 20011)
    x1d, x2d = to_dev(x1), to_dev(x2)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    torch.cuda.synchronize()
    for it in range(3):
        y1, y2 = _poisoned(x1d), _poisoned(x2d)
        torch.cuda.synchronize()
        dpar.dpar_allreduce_opt(dpar.rows(x1d), dpar.rows(y1), 36, 50001,
                                "float32", "sum", 5 + it, "dual", e1, 0, -1, s1)
        dpar.dpar_allreduce_opt(dpar.rows(x2d), dpar.rows(y2), 100, 20011,
                                "float32", "sum", 7 + it, "dual", e2, 0, -1, s2)
        outs.append((y1, y2))
    torch.cuda.synchronize()
    dpar.dpar_check_status(s1)
    dpar.dpar_check_status(s2)
    for y1, y2 in outs:
        assert_all_ranks_equal(y1.cpu().numpy(), w1, f"stream 1 {e1}")
        assert_all_ranks_equal(y2.cpu().numpy(), w2, f"stream 2 {e2}")


def test_two_host_threads():
    need_gpu()
    dpar = lib()
    cases = [_case(2132 + k, 20 + 17 * k, 30000 + 7 * k) for k in range(2)]
    devs = [to_dev(x) for x, _ in cases]
    errors = []

    def work(k):
        try:
            s = torch.cuda.Stream()
            x, want = cases[k]
            p, m = x.shape
            with torch.cuda.stream(s):
                for it in range(4):
                    y = _poisoned(devs[k])
                    dpar.dpar_allreduce_opt(
                        dpar.rows(devs[k]), dpar.rows(y), p, m, "float32",
                        "sum", 3 + it, "dual", EXECS[(k + it) % len(EXECS)],
                        0, -1, s)
                    s.synchronize()
                    got = y.cpu().numpy()
                    for i in range(p):
                        if not np.array_equal(got[i], want):
                            errors.append((k, it, i))
                            break
        except Exception as e:  # noqa: BLE001 - reported below
            errors.append((k, repr(e)))

    ts = [threading.Thread(target=work, args=(k,)) for k in range(2)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert not errors, errors


def test_pointer_set_staged_on_a_busy_stream_used_on_another():
    """A call on stream B with the pointer arrays that a call on stream A has
    just staged: A is still busy, so A's copy of the table has not run, and
    B's kernels must wait for it."""
    need_gpu()
    dpar = lib()
    p, m = 300, 40000
    busy = torch.zeros(64 << 20, dtype=torch.float32, device="cuda")
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    for it in range(3):
        x, want = _case(2140 + it, p, m)
        xd = to_dev(x)
        y = _poisoned(xd)
        torch.cuda.synchronize()
        xs, ys = dpar.rows(xd), dpar.rows(y)
        with torch.cuda.stream(sa):
            for _ in range(30):
                busy.add_(1.0)
        for s in (sa, sb):
            dpar.dpar_allreduce_opt(xs, ys, p, m, "float32", "sum", 0,
                                    "dual", "auto", 0, -1, s)
        sb.synchronize()
        got_b = y.cpu().numpy()       # B's call is done, A's may not be
        torch.cuda.synchronize()
        dpar.dpar_check_status(sa)
        assert_all_ranks_equal(got_b, want, f"stream B, round {it}")
        assert_all_ranks_equal(y.cpu().numpy(), want, f"both, round {it}")


def test_many_pointer_sets_on_two_streams():
    """More distinct pointer sets than the library keeps staged plus the
    tables it retires before recycling them, alternating between two
    streams without synchronisation, twice over: every output equals the
    oracle (a call reading a recycled table too early would write another
    set's result, or read another set's inputs)."""
    need_gpu()
    dpar = lib()
    p, m, n = 40, 3001, 50
    cases = [_case(2200 + k, p, m) for k in range(n)]
    xds = [to_dev(x) for x, _ in cases]
    ys = [_poisoned(xd) for xd in xds]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for rnd, order in enumerate((range(n), reversed(range(n)))):
        for y in ys:
            y.view(torch.int32).fill_(POISON)
        torch.cuda.synchronize()
        for k in order:
            s = s1 if k % 2 == 0 else s2
            dpar.dpar_allreduce_opt(dpar.rows(xds[k]), dpar.rows(ys[k]), p, m,
                                    "float32", "sum", 0, "dual", "auto", 0,
                                    -1, s)
        torch.cuda.synchronize()
        dpar.dpar_check_status(s1)
        for k in range(n):
            assert_all_ranks_equal(ys[k].cpu().numpy(), cases[k][1],
                                   f"round {rnd}, set {k}")


@pytest.mark.parametrize("k", range(16))
def test_random_calls_on_two_streams(k):
    """Seeded random pairs of calls interleaved on two streams, three rounds
    with fresh outputs (new pointer sets, staged on either stream), then
    one pointer set used on both streams in turn without synchronisation:
    every output equals the oracle."""
    need_gpu()
    dpar = lib()
    r = np.random.default_rng(9990 + k)
    cases = []
    for j in range(2):
        p = int(r.choice([2, 7, 36, 130, 300, 1152]))
        m = int(r.integers(1, max(2, min(1 << 17, (1 << 21) // p))))
        ex = EXECS[int(r.integers(len(EXECS)))]
        x, want = _case(2500 + 2 * k + j, p, m)
        cases.append((p, m, ex, to_dev(x), want))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = []
    torch.cuda.synchronize()
    for rnd in range(3):
        for j, (p, m, ex, xd, want) in enumerate(cases):
            y = _poisoned(xd)
            torch.cuda.synchronize()
            dpar.dpar_allreduce_opt(dpar.rows(xd), dpar.rows(y), p, m,
                                    "float32", "sum", 0, "dual", ex, 0, -1,
                                    streams[(j + rnd) % 2])
            outs.append((y, want, f"round {rnd} case {j} p={p} m={m} {ex}"))
    p, m, ex, xd, want = cases[0]
    y = _poisoned(xd)
    torch.cuda.synchronize()
    xs, ys = dpar.rows(xd), dpar.rows(y)
    for s in streams:
        dpar.dpar_allreduce_opt(xs, ys, p, m, "float32", "sum", 0, "dual",
                                ex, 0, -1, s)
    outs.append((y, want, f"shared set p={p} m={m} {ex}"))
    torch.cuda.synchronize()
    for s in streams:
        dpar.dpar_check_status(s)
    for y, want, what in outs:
        assert_all_ranks_equal(y.cpu().numpy(), want, what)
