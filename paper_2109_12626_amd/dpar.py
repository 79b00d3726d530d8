"""Python binding of libdpar.so (include/dpar.h).

Argument marshalling only: every step of the reduction runs in the library's
HIP kernels.  The functions keep the C names.  torch is imported first so that
the library binds to the HIP runtime torch already loaded (one runtime per
process); torch serves only for device memory and streams.
"""

import ctypes
import os

import numpy as np

import torch  # noqa: F401  (must precede loading libdpar: one HIP runtime)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("DPAR_LIB_PATH") or os.path.join(_HERE, "libdpar.so")

DPAR_SUCCESS = 0
DPAR_ERR_INVALID_ARG = -1
DPAR_ERR_UNSUPPORTED = -2
DPAR_ERR_ALIAS = -3
DPAR_ERR_NOMEM = -4
DPAR_ERR_HIP = -5
DPAR_ERR_TIMEOUT = -6

DPAR_INT32, DPAR_FLOAT32, DPAR_U32_MAT2X2 = 0, 1, 2
DPAR_SUM, DPAR_MAX, DPAR_MATMUL = 0, 1, 2
DPAR_EXEC_AUTO, DPAR_EXEC_LAUNCH_PER_ROUND, DPAR_EXEC_GRID_BARRIER, \
    DPAR_EXEC_TICKET, DPAR_EXEC_SPLIT, DPAR_EXEC_ROUNDS, \
    DPAR_EXEC_ROUNDS_BARRIER = 0, 1, 2, 3, 4, 5, 6
DPAR_ALG_DUAL_ROOT, DPAR_ALG_SINGLE_TREE, DPAR_ALG_REDUCE_BCAST = 0, 1, 2

DTYPES = {"int32": DPAR_INT32, "float32": DPAR_FLOAT32,
          "u32mat2x2": DPAR_U32_MAT2X2}
OPS = {"sum": DPAR_SUM, "max": DPAR_MAX, "matmul": DPAR_MATMUL}
EXECS = {"auto": DPAR_EXEC_AUTO, "launch": DPAR_EXEC_LAUNCH_PER_ROUND,
         "barrier": DPAR_EXEC_GRID_BARRIER, "ticket": DPAR_EXEC_TICKET,
         "split": DPAR_EXEC_SPLIT, "rounds": DPAR_EXEC_ROUNDS,
         "rounds_barrier": DPAR_EXEC_ROUNDS_BARRIER}
ALGS = {"dual": DPAR_ALG_DUAL_ROOT, "single": DPAR_ALG_SINGLE_TREE,
        "reduce_bcast": DPAR_ALG_REDUCE_BCAST}


class DparError(RuntimeError):
    def __init__(self, code, msg):
        self.code = code
        super().__init__(f"dpar error {code}: {msg}")


class dpar_node_t(ctypes.Structure):
    _fields_ = [("parent", ctypes.c_int), ("child0", ctypes.c_int),
                ("child1", ctypes.c_int), ("depth", ctypes.c_int),
                ("subtree_lo", ctypes.c_int), ("dual", ctypes.c_int)]


class dpar_options_t(ctypes.Structure):
    _fields_ = [("alg", ctypes.c_int), ("exec", ctypes.c_int),
                ("round_begin", ctypes.c_int), ("round_end", ctypes.c_int)]


class dpar_schedule_t(ctypes.Structure):
    _fields_ = [("b", ctypes.c_int), ("granularity", ctypes.c_int),
                ("quantum", ctypes.c_int),
                ("nquanta", ctypes.c_size_t), ("tail_elems", ctypes.c_size_t),
                ("chunks_per_block", ctypes.c_int), ("height", ctypes.c_int),
                ("waves_per_chunk", ctypes.c_int)]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with "
            "`python -c 'import __graft_entry__ as g; g.build()'`")
    L = ctypes.CDLL(LIB_PATH)
    vp, sz, i = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
    L.dpar_allreduce.argtypes = [vp, vp, i, sz, i, i, i, vp]
    L.dpar_allreduce_ex.argtypes = [vp, vp, i, sz, i, i, i, i, vp]
    L.dpar_allreduce_noalloc.argtypes = [vp, vp, i, sz, i, i, i, vp]
    L.dpar_allreduce_opt.argtypes = [vp, vp, i, sz, i, i, i,
                                     ctypes.POINTER(dpar_options_t), vp]
    L.dpar_tree_info.argtypes = [i, i, ctypes.POINTER(dpar_node_t)]
    L.dpar_tree_info_alg.argtypes = [i, i, i, ctypes.POINTER(dpar_node_t)]
    L.dpar_schedule_rounds.argtypes = [i, i, i]
    L.dpar_block_rule.argtypes = [i, sz, ctypes.c_double, ctypes.c_double]
    L.dpar_rounds.argtypes = [i, i, i]
    L.dpar_schedule_info.argtypes = [i, sz, i, i, i,
                                     ctypes.POINTER(dpar_schedule_t)]
    L.dpar_block_bounds.argtypes = [ctypes.POINTER(dpar_schedule_t), sz, i,
                                    ctypes.POINTER(sz), ctypes.POINTER(sz)]
    L.dpar_check_status.argtypes = [vp]
    L.dpar_set_phase_event.argtypes = [vp]
    L.dpar_last_error.restype = ctypes.c_char_p
    L.dpar_last_error.argtypes = []
    L.dpar_finalize.argtypes = []
    for name in ("dpar_allreduce", "dpar_allreduce_ex", "dpar_allreduce_opt",
                 "dpar_allreduce_noalloc",
                 "dpar_tree_info", "dpar_tree_info_alg",
                 "dpar_schedule_rounds", "dpar_block_rule", "dpar_rounds",
                 "dpar_schedule_info", "dpar_block_bounds",
                 "dpar_check_status", "dpar_finalize",
                 "dpar_set_phase_event"):
        getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _check(rc):
    if rc < 0:
        raise DparError(rc, lib().dpar_last_error().decode())
    return rc


def _addr(v):
    if isinstance(v, torch.Tensor):
        return v.data_ptr()
    return int(v)


def _array_of(addrs):
    """A C array of void* viewing a uint64 numpy array (kept alive by it)."""
    if addrs.size == 0:
        return (ctypes.c_void_p * 0)()
    return (ctypes.c_void_p * addrs.size).from_buffer(addrs)


def pointers(seq):
    """A reusable C array of device addresses (ints or tensors); passing it
    instead of a list saves the conversion on every call."""
    if isinstance(seq, ctypes.Array):
        return seq
    if all(type(v) is int for v in seq):
        # plain addresses: one conversion in numpy instead of one per entry
        # (p = 1152: about 40 instead of 300 us on the host)
        return _array_of(np.array(seq, dtype=np.uint64))
    return (ctypes.c_void_p * len(seq))(*[_addr(v) for v in seq])


_ptr_array = pointers


def _stream(stream):
    if stream is None:
        return None
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _enum(table, v):
    return table[v] if isinstance(v, str) else int(v)


def rows(t):
    """Device addresses of the rows of a [p, ...] tensor, as a reusable C
    array (indexable and iterable like a list of ints)."""
    if t.dim() < 1:
        raise ValueError("need at least one dimension")
    step = t.stride(0) * t.element_size()
    if step < 0:
        raise ValueError("rows with a negative stride")
    addrs = np.arange(t.shape[0], dtype=np.uint64) * np.uint64(step)
    addrs += np.uint64(t.data_ptr())
    return _array_of(addrs)


def dpar_allreduce(x, y, p, m, dtype, op, b=0, stream=None):
    """x, y: sequences of p device addresses (ints or tensors)."""
    return _check(lib().dpar_allreduce(
        _ptr_array(x), _ptr_array(y), int(p), int(m), _enum(DTYPES, dtype),
        _enum(OPS, op), int(b), _stream(stream)))


def dpar_allreduce_noalloc(x, y, p, m, dtype, op, b=0, stream=None):
    """The allocation-free variant of dpar_allreduce (include/dpar.h)."""
    return _check(lib().dpar_allreduce_noalloc(
        _ptr_array(x), _ptr_array(y), int(p), int(m), _enum(DTYPES, dtype),
        _enum(OPS, op), int(b), _stream(stream)))


def dpar_allreduce_ex(x, y, p, m, dtype, op, b=0, exec="auto", stream=None):
    return _check(lib().dpar_allreduce_ex(
        _ptr_array(x), _ptr_array(y), int(p), int(m), _enum(DTYPES, dtype),
        _enum(OPS, op), int(b), _enum(EXECS, exec), _stream(stream)))


def dpar_allreduce_opt(x, y, p, m, dtype, op, b=0, alg="dual", exec="auto",
                       round_begin=0, round_end=-1, stream=None):
    opt = dpar_options_t(_enum(ALGS, alg), _enum(EXECS, exec),
                         int(round_begin), int(round_end))
    return _check(lib().dpar_allreduce_opt(
        _ptr_array(x), _ptr_array(y), int(p), int(m), _enum(DTYPES, dtype),
        _enum(OPS, op), int(b), ctypes.byref(opt), _stream(stream)))


def dpar_tree_info(p, rank):
    out = dpar_node_t()
    _check(lib().dpar_tree_info(int(p), int(rank), ctypes.byref(out)))
    return {f: getattr(out, f) for f, _ in dpar_node_t._fields_}


def dpar_tree_info_alg(p, alg, rank):
    out = dpar_node_t()
    _check(lib().dpar_tree_info_alg(int(p), _enum(ALGS, alg), int(rank),
                                    ctypes.byref(out)))
    return {f: getattr(out, f) for f, _ in dpar_node_t._fields_}


def dpar_schedule_rounds(p, b, alg="dual"):
    return _check(lib().dpar_schedule_rounds(int(p), int(b), _enum(ALGS, alg)))


def dpar_block_rule(p, m, alpha=0.0, beta=0.0):
    return _check(lib().dpar_block_rule(int(p), int(m), float(alpha),
                                        float(beta)))


def dpar_rounds(p, b, rank=-1):
    return _check(lib().dpar_rounds(int(p), int(b), int(rank)))


def dpar_schedule_info(p, m, dtype, b=0, aligned=True):
    out = dpar_schedule_t()
    _check(lib().dpar_schedule_info(int(p), int(m), _enum(DTYPES, dtype),
                                    int(b), int(bool(aligned)),
                                    ctypes.byref(out)))
    return out


def dpar_block_bounds(sched, m, j):
    s, e = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().dpar_block_bounds(ctypes.byref(sched), int(m), int(j),
                                   ctypes.byref(s), ctypes.byref(e)))
    return s.value, e.value


def dpar_check_status(stream=None):
    return _check(lib().dpar_check_status(_stream(stream)))


def dpar_set_phase_event(event):
    """event: a torch.cuda.Event that has been recorded once (so that it
    exists), a raw hipEvent_t handle, or None."""
    if event is None:
        h = None
    elif isinstance(event, torch.cuda.Event):
        h = ctypes.c_void_p(event.cuda_event)
    else:
        h = ctypes.c_void_p(int(event))
    return _check(lib().dpar_set_phase_event(h))


def dpar_last_error():
    return lib().dpar_last_error().decode()


def dpar_finalize():
    return _check(lib().dpar_finalize())


# ------------------------------------------------------------ convenience

_ELEM = {"int32": 4, "float32": 4, "u32mat2x2": 16}


def allreduce(x, y=None, dtype=None, op="sum", b=0, exec="auto", stream=None,
              alg="dual"):
    """Tensor front end: x is a [p, m] (or [p, m, 4] uint32 for matrices)
    device tensor, or a list of p 1-D tensors; y likewise (default: a new
    [p, ...] tensor).  Returns y.  Only marshals addresses."""
    if isinstance(x, torch.Tensor):
        p = x.shape[0]
        xs = rows(x)
        sample = x[0]
    else:
        p = len(x)
        xs = [t.data_ptr() for t in x]
        sample = x[0]
    if dtype is None:
        dtype = {torch.int32: "int32", torch.float32: "float32",
                 torch.uint32: "u32mat2x2"}[sample.dtype]
    m = sample.numel() * sample.element_size() // _ELEM[dtype]
    if y is None:
        y = torch.empty((p,) + tuple(sample.shape), dtype=sample.dtype,
                        device=sample.device)
    ys = rows(y) if isinstance(y, torch.Tensor) else [t.data_ptr() for t in y]
    if stream is None:
        stream = torch.cuda.current_stream(sample.device)
    dpar_allreduce_opt(xs, ys, p, m, dtype, op, b, alg, exec, 0, -1, stream)
    return y
