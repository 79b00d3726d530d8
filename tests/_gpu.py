"""Helpers for the GPU parity tests: upload seeded inputs, run the library
through the C ABI, read the outputs back.  The expected values always come
from the CPU oracle."""

import os

import numpy as np
import pytest
import torch

import oracle
import synth

NP_TO_TORCH = {np.int32: torch.int32, np.float32: torch.float32,
               np.uint32: torch.int32}
POISON = -0x21524111  # 0xDEADBEEF as int32


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def lib():
    from paper_2109_12626_amd import dpar
    return dpar


def to_dev(x):
    """numpy [p, m](, 4) -> torch device tensor with the same bytes."""
    a = np.ascontiguousarray(x)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(a).to("cuda")


def from_dev(t, like):
    a = t.cpu().numpy()
    if like.dtype == np.uint32:
        a = a.view(np.uint32)
    return a


def poisoned_like(xd):
    y = torch.empty_like(xd)
    y.view(torch.int32).fill_(POISON)
    return y


def run(x, dtype, op, b, exec="auto", y=None, x_ptrs=None, y_ptrs=None,
        m=None, stream=None):
    """One call on device copies of x; returns the outputs as numpy."""
    dpar = lib()
    p = x.shape[0]
    m = x.shape[1] if m is None else m
    xd = to_dev(x)
    yd = poisoned_like(xd) if y is None else y
    xs = dpar.rows(xd) if x_ptrs is None else x_ptrs(xd)
    ys = dpar.rows(yd) if y_ptrs is None else y_ptrs(yd)
    s = torch.cuda.current_stream() if stream is None else stream
    dpar.dpar_allreduce_ex(xs, ys, p, m, dtype, op, b, exec, s)
    dpar.dpar_check_status(s)
    return from_dev(yd, x)


def assert_all_ranks_equal(out, want, what=""):
    """Every rank's output equals want bit for bit (for fp32 that includes
    the sign of zero)."""
    o = np.ascontiguousarray(out).view(np.uint32)
    w = np.ascontiguousarray(want).view(np.uint32)
    assert o.shape[1:] == w.shape, (what, o.shape, w.shape)
    eq = (o == w[None]).reshape(o.shape[0], -1).all(axis=1)
    if eq.all():
        return
    i = int(np.argmin(eq))
    bad = np.argwhere(o[i] != w)
    raise AssertionError(
        f"{what} rank {i}: {len(bad)} elements differ, first at "
        f"{bad[0].tolist()}: got {out[i][tuple(bad[0])]} want "
        f"{want[tuple(bad[0])]}")


def workload_input(w, m=None, p=None):
    return synth.generate(w.dist, w.seed, w.p if p is None else p,
                          w.m if m is None else m, **w.dist_kw)


def rule(p, m):
    return oracle.block_rule_lit(p, m)


def resolve_b(b, p, m):
    return rule(p, m) if b == "rule" else b


def gib(nbytes):
    return nbytes / 2 ** 30


class _Env:
    """Context manager setting one library knob (environment variable)."""

    def __init__(self, name, value):
        self.name, self.value = name, value

    def __enter__(self):
        self.old = os.environ.get(self.name)
        if self.value is None:
            os.environ.pop(self.name, None)
        else:
            os.environ[self.name] = str(self.value)

    def __exit__(self, *a):
        if self.old is None:
            os.environ.pop(self.name, None)
        else:
            os.environ[self.name] = self.old


def env_waves(n):
    """Wavefronts per chunk of the post-order (SEQ) work item: 1 or 2."""
    return _Env("DPAR_WAVES", n)


def env_unit(u):
    """Work-item evaluation: "seq", "level" or None (the library chooses)."""
    return _Env("DPAR_UNIT", u)


def env_group_blocks(on):
    """Grouping of short blocks in the one-launch executors: 1 or 0."""
    return _Env("DPAR_GROUP_BLOCKS", 1 if on else 0)


def env_bcast_span_kb(kb):
    """Span of y_0 (KB) per pass of the split executor's broadcast."""
    return _Env("DPAR_BCAST_SPAN_KB", kb)
