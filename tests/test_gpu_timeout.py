"""The DPAR_ERR_TIMEOUT contract of the cooperative executors (Algorithm 1's
round loop, whose per-round synchronisation the device-wide barrier stands
in for).

The give-up is forced from the host: DPAR_SPIN_LIMIT=0 makes every barrier
wait give up after its first poll, so every kernel still exits normally; no
wait is left unbounded.  Checked: the report comes once and is then cleared;
a GRID_BARRIER call's outputs stay complete; and later calls, including the
one that reuses the timed-out call's counter slot (64 calls later), run
their own barriers again and match the oracle.
"""

import pytest
import torch

import oracle
from synth import configs

from _gpu import (_Env, assert_all_ranks_equal, from_dev, lib, need_gpu,
                  poisoned_like, to_dev, workload_input)

pytestmark = pytest.mark.gpu

SLOTS = 64  # the library's counter slots in rotation


def _setup(p, m, seed_cfg=configs.P36_INT):
    need_gpu()
    x = workload_input(seed_cfg, m=m, p=p)
    want = oracle.allreduce_tree(x, seed_cfg.dtype, "sum")
    xd = to_dev(x)
    yd = poisoned_like(xd)
    dpar = lib()
    return dpar, x, want, xd, yd, dpar.rows(xd), dpar.rows(yd)


def _call(dpar, xs, ys, p, m, b, exec, stream):
    dpar.dpar_allreduce_opt(xs, ys, p, m, "int32", "sum", b, "dual", exec, 0,
                            -1, stream)


def test_grid_barrier_timeout_reported_once_outputs_complete():
    # 512 work items per round: hundreds of workgroups, whose arrivals at a
    # barrier spread far beyond one poll
    p, m, b = 64, 1 << 20, 8
    dpar, x, want, xd, yd, xs, ys = _setup(p, m)
    s = torch.cuda.current_stream()
    dpar.dpar_check_status(s)            # start from a cleared report flag
    with _Env("DPAR_SPIN_LIMIT", 0):
        _call(dpar, xs, ys, p, m, b, "barrier", s)
        with pytest.raises(dpar.DparError) as ei:
            dpar.dpar_check_status(s)
    assert ei.value.code == dpar.DPAR_ERR_TIMEOUT
    assert "spin limit" in str(ei.value)
    # the report is given once
    assert dpar.dpar_check_status(s) == 0
    # the barrier only orders independent work items: outputs complete
    assert_all_ranks_equal(from_dev(yd, x), want, "after a timed-out call")
    # the next call waits at its own barriers again
    yd.fill_(-1)
    with _Env("DPAR_SPIN_LIMIT", 1 << 20):
        _call(dpar, xs, ys, p, m, b, "barrier", s)
        assert dpar.dpar_check_status(s) == 0
    assert_all_ranks_equal(from_dev(yd, x), want, "call after the timeout")


def test_rounds_barrier_after_timeout_every_slot_clean():
    """A timed-out ROUNDS_BARRIER call leaves its barrier words out of step;
    the calls after it, through a full rotation of the counter slots, start
    from zeroed words and match the oracle with no further timeout."""
    p, m, b = 36, 1 << 16, 8
    dpar, x, want, xd, yd, xs, ys = _setup(p, m)
    s = torch.cuda.current_stream()
    dpar.dpar_check_status(s)
    with _Env("DPAR_SPIN_LIMIT", 0):
        _call(dpar, xs, ys, p, m, b, "rounds_barrier", s)
        with pytest.raises(dpar.DparError) as ei:
            dpar.dpar_check_status(s)
    assert ei.value.code == dpar.DPAR_ERR_TIMEOUT
    assert dpar.dpar_check_status(s) == 0
    # (that call's outputs are undefined: not compared)
    with _Env("DPAR_SPIN_LIMIT", 1 << 20):
        for k in range(SLOTS + 2):
            yd.fill_(-1)
            _call(dpar, xs, ys, p, m, b, "rounds_barrier", s)
            assert dpar.dpar_check_status(s) == 0, k
            assert_all_ranks_equal(from_dev(yd, x), want, f"call {k}")


def test_timeout_in_one_call_does_not_skip_waits_of_a_later_one():
    """After a give-up, a later GRID_BARRIER call on another stream waits at
    its own barriers: the give-up word belongs to the call that set it, so
    the later call neither reports a timeout nor loses its outputs."""
    p, m, b = 64, 1 << 20, 4
    dpar, x, want, xd, yd, xs, ys = _setup(p, m)
    s1 = torch.cuda.current_stream()
    s2 = torch.cuda.Stream()
    dpar.dpar_check_status(s1)
    with _Env("DPAR_SPIN_LIMIT", 0):
        _call(dpar, xs, ys, p, m, b, "barrier", s1)
    with pytest.raises(dpar.DparError) as ei:
        dpar.dpar_check_status(s1)
    assert ei.value.code == dpar.DPAR_ERR_TIMEOUT
    yd2 = poisoned_like(xd)
    ys2 = dpar.rows(yd2)
    s2.wait_stream(s1)
    with _Env("DPAR_SPIN_LIMIT", 1 << 20):
        _call(dpar, xs, ys2, p, m, b, "barrier", s2)
        assert dpar.dpar_check_status(s2) == 0
    assert_all_ranks_equal(from_dev(yd2, x), want, "second stream")
