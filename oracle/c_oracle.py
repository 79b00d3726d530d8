"""ctypes binding of the plain C oracle (``oracle/c/dpar_oracle.c``).

Oracle module: test infrastructure only.  It builds and loads the C oracle
with gcc; it shares nothing with the HIP library.

The C oracle evaluates the same result as ``reduce.allreduce_tree`` by a
different route: the ranks in post-order with a stack of subtree values
(Section 1.1's trees; Algorithm 1's association), on host threads over
contiguous column ranges.
"""

import ctypes
import os
import subprocess
import tempfile

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "c", "dpar_oracle.c")
LIB = os.path.join(HERE, "c", "libdpar_oracle.so")

KINDS = {("int32", "sum"): 0, ("int32", "max"): 1, ("float32", "sum"): 2,
         ("u32mat2x2", "matmul"): 3}
LAYOUTS = {"dual": 2, "single": 1}
_NP = {"int32": np.int32, "float32": np.float32, "u32mat2x2": np.uint32}

CFLAGS = ["-O2", "-std=c99", "-fPIC", "-shared", "-pthread",
          "-fno-fast-math", "-ffp-contract=off", "-Wall", "-Wextra",
          "-Werror"]


def build(out=None, mutant=0, verbose=False):
    """Compiles the C oracle (or, for tests, a copy with planted mistake
    ``mutant``) to ``out`` (default: next to the source)."""
    lib = out or LIB
    tmp = f"{lib}.tmp{os.getpid()}"   # concurrent builders never share it
    cmd = (["gcc"] + CFLAGS + [f"-DDPO_MUTANT={int(mutant)}",
                               "-I", os.path.dirname(SRC), SRC, "-o", tmp])
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    return lib


def _bind(lib):
    lib.dpo_trees.argtypes = [ctypes.c_int, ctypes.c_int] + \
        [ctypes.c_void_p] * 5
    lib.dpo_trees.restype = ctypes.c_int
    lib.dpo_allreduce.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                  ctypes.c_int, ctypes.c_size_t,
                                  ctypes.c_void_p, ctypes.c_int]
    lib.dpo_allreduce.restype = ctypes.c_int
    lib.dpo_allreduce_all.argtypes = [ctypes.c_int, ctypes.c_int,
                                      ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_int, ctypes.c_size_t,
                                      ctypes.c_int]
    lib.dpo_allreduce_all.restype = ctypes.c_int
    return lib


_LIB = None


def load(path=None):
    """The C oracle, built first when the shared library is not there."""
    global _LIB
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _LIB is None:
        if not os.path.exists(LIB) or (os.path.getmtime(LIB)
                                       < os.path.getmtime(SRC)):
            build()
        _LIB = _bind(ctypes.CDLL(LIB))
    return _LIB


def mutant(k):
    """A copy of the C oracle with planted mistake k (see the source)."""
    d = tempfile.mkdtemp(prefix="dpo_mutant_")
    return load(build(os.path.join(d, f"libdpo_m{k}.so"), mutant=k))


def trees(p, layout="dual", lib=None):
    """(parent, child0, child1, depth, roots) as int32 arrays, -1 = none."""
    lib = lib or load()
    arrs = [np.empty(p, np.int32) for _ in range(4)]
    roots = np.empty(2, np.int32)
    rc = lib.dpo_trees(p, LAYOUTS[layout],
                       *[a.ctypes.data for a in arrs], roots.ctypes.data)
    if rc:
        raise ValueError(f"dpo_trees({p}) returned {rc}")
    return arrs + [roots]


def _rows(x):
    rows = list(x) if isinstance(x, (list, tuple)) else [x[i] for i in
                                                         range(x.shape[0])]
    for r in rows:
        if not r.flags.c_contiguous:
            raise ValueError("rows must be C-contiguous")
    return rows


def _ptrs(rows):
    return (ctypes.c_void_p * len(rows))(*[r.ctypes.data for r in rows])


def allreduce(x, dtype, op, layout="dual", threads=1, lib=None):
    """y for rows ``x`` ([p, m] or [p, m, 4], or a list of rows)."""
    lib = lib or load()
    rows = _rows(x)
    p = len(rows)
    m = rows[0].shape[0]
    y = np.empty(rows[0].shape, dtype=_NP[dtype])
    for r in rows:
        if r.dtype != y.dtype or r.shape != y.shape:
            raise ValueError("rows must share the operator's dtype and shape")
    rc = lib.dpo_allreduce(KINDS[(dtype, op)], LAYOUTS[layout], _ptrs(rows),
                           p, m, y.ctypes.data, threads)
    if rc:
        raise RuntimeError(f"dpo_allreduce returned {rc}")
    return y


def allreduce_all(x, dtype, op, out, layout="dual", threads=1, lib=None):
    """Writes y into every row of ``out`` (p rows, same shape as x's)."""
    lib = lib or load()
    rows = _rows(x)
    outs = _rows(out)
    p = len(rows)
    if len(outs) != p:
        raise ValueError("one output row per rank")
    for r in rows + outs:
        if r.dtype != _NP[dtype] or r.shape != rows[0].shape:
            raise ValueError("rows must share the operator's dtype and shape")
    rc = lib.dpo_allreduce_all(KINDS[(dtype, op)], LAYOUTS[layout],
                               _ptrs(rows), _ptrs(outs), p,
                               rows[0].shape[0], threads)
    if rc:
        raise RuntimeError(f"dpo_allreduce_all returned {rc}")
    return out
