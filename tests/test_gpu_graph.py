"""Calls recorded into a HIP graph (torch.cuda.graph stream capture) and
replayed: every replay, with eager work and synchronisation in between and
new input contents each time, must equal the oracle's result for those
contents."""

import numpy as np
import pytest
import torch

import oracle
import synth
from tests._gpu import POISON, lib, need_gpu, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("alg", ["dual", "single", "reduce_bcast"])
@pytest.mark.parametrize("exec", ["auto", "split", "ticket", "launch", "rounds"])
@pytest.mark.parametrize("p,m,b", [(7, 1000, 4), (36, 65539, 8),
                                   (300, 4096, 3)])
def test_captured_call_replays(alg, exec, p, m, b):
    need_gpu()
    _replays(alg, exec, p, m, b)


@pytest.mark.parametrize("exec", ["auto", "split", "ticket"])
def test_captured_wide_items_replay(exec):
    """p = 36, m = 2^20, the rule's b: wide work items (one fused launch
    under AUTO, split, ticket) recorded into a graph and replayed."""
    need_gpu()
    _replays("dual", exec, 36, 1 << 20, 0)


@pytest.mark.parametrize("k", range(24))
def test_random_captured_calls(k):
    """Seeded random captures (p = 1 .. 1500, m up to 2^18, every tree
    layout, the executors a graph may hold, the rule's b or a random one),
    each replayed with new inputs and eager work between the replays."""
    need_gpu()
    r = np.random.default_rng(9950 + k)
    p = int(r.choice([1, 2, 5, 36, 64, 130, 288, 700, 1152, 1500]))
    m = int(r.integers(1, max(2, min(1 << 18, (1 << 22) // p))))
    b = int(r.choice([0, 1, int(r.integers(1, m + 1))]))
    alg = ["dual", "single", "reduce_bcast"][int(r.integers(3))]
    exec = ["auto", "split", "ticket", "launch", "rounds"][int(r.integers(5))]
    _replays(alg, exec, p, m, min(b, m))


def _replays(alg, exec, p, m, b):
    dpar = lib()
    trees = oracle.build_trees(p) if alg == "dual" else \
        oracle.build_trees(p, layout="single")
    inputs = [synth.generate("normal_f32", 2140 + k, p, m) for k in range(4)]
    xd = to_dev(inputs[0])
    yd = torch.empty_like(xd)
    xs, ys = dpar.pointers(dpar.rows(xd)), dpar.pointers(dpar.rows(yd))
    # the eager call that builds the tables and stages the pointers
    dpar.dpar_allreduce_opt(xs, ys, p, m, "float32", "sum", b, alg, exec, 0,
                            -1, torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dpar.dpar_allreduce_opt(xs, ys, p, m, "float32", "sum", b, alg, exec,
                                0, -1, torch.cuda.current_stream())
    for k in range(1, 4):
        xd.copy_(torch.from_numpy(inputs[k]).cuda())
        yd.view(torch.int32).fill_(POISON)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        want = oracle.allreduce_tree(inputs[k], "float32", "sum", trees=trees)
        got = yd.cpu().numpy()
        for i in range(p):
            assert np.array_equal(got[i], want), (k, i)
        # eager work on the same buffers between replays
        dpar.dpar_allreduce_opt(xs, ys, p, m, "float32", "sum", b, alg,
                                "split", 0, -1, torch.cuda.current_stream())
        torch.cuda.synchronize()
    del g
    # the captured call's pointer table stays pinned until dpar_finalize;
    # release it, so that the tests do not depend on the allocator handing
    # the same addresses to later tests (8 staging slots)
    torch.cuda.synchronize()
    dpar.dpar_finalize()


# the refused call leaves the graph empty, which torch warns about
@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")
def test_capture_needs_an_eager_call_first():
    need_gpu()
    dpar = lib()
    p, m = 11, 777
    xd = to_dev(synth.generate("normal_f32", 2150, p, m))
    yd = torch.empty_like(xd)
    g = torch.cuda.CUDAGraph()
    with pytest.raises(dpar.DparError) as e:
        with torch.cuda.graph(g):
            dpar.dpar_allreduce_opt(dpar.rows(xd), dpar.rows(yd), p, m,
                                    "float32", "sum", 2, "dual", "split", 0,
                                    -1, torch.cuda.current_stream())
    assert e.value.code == dpar.DPAR_ERR_UNSUPPORTED


# the refused call leaves the graph empty, which torch warns about
@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")
def test_cooperative_executors_refused_under_capture():
    need_gpu()
    dpar = lib()
    p, m = 9, 500
    xd = to_dev(synth.generate("normal_f32", 2151, p, m))
    yd = torch.empty_like(xd)
    xs, ys = dpar.pointers(dpar.rows(xd)), dpar.pointers(dpar.rows(yd))
    dpar.dpar_allreduce_opt(xs, ys, p, m, "float32", "sum", 2, "dual",
                            "barrier", 0, -1, torch.cuda.current_stream())
    torch.cuda.synchronize()
    for ex in ("barrier", "rounds_barrier"):
        g = torch.cuda.CUDAGraph()
        with pytest.raises(dpar.DparError) as e:
            with torch.cuda.graph(g):
                dpar.dpar_allreduce_opt(xs, ys, p, m, "float32", "sum", 2,
                                        "dual", ex, 0, -1,
                                        torch.cuda.current_stream())
        assert e.value.code == dpar.DPAR_ERR_UNSUPPORTED
