"""Element operators (Section 1: an associative, not necessarily commutative
element-wise operator).

Oracle module: test infrastructure only.

Supported (dtype, op) pairs and their exact meaning:

* ``int32 sum``      -- two's-complement addition that wraps modulo 2^32
                        (the paper is silent on overflow; wrapping keeps the
                        operator exactly associative).
* ``int32 max``      -- signed maximum.
* ``float32 sum``    -- IEEE-754 binary32 addition, round to nearest even,
                        subnormals kept; NOT associative, so the order of
                        application is part of the result.
* ``u32mat2x2 matmul`` -- each element is a 2x2 matrix of uint32 stored
                        row-major as [a00, a01, a10, a11]; combine(A, B) is the
                        matrix product A.B with every entry taken mod 2^32.
                        Associative and non-commutative, so it exposes any
                        mistake in the rank order.

``combine(a, b)`` always returns a (.) b with ``a`` the LEFT operand.
Arrays hold one vector per call: shape [m] for the scalar types and [m, 4]
for matrices.
"""

import numpy as np

DTYPES = ("int32", "float32", "u32mat2x2")
OPS = ("sum", "max", "matmul")

_VALID = {("int32", "sum"), ("int32", "max"), ("float32", "sum"),
          ("u32mat2x2", "matmul")}


def valid_pair(dtype: str, op: str) -> bool:
    return (dtype, op) in _VALID


def numpy_dtype(dtype: str):
    return {"int32": np.int32, "float32": np.float32,
            "u32mat2x2": np.uint32}[dtype]


def element_shape(dtype: str):
    """Trailing shape of one element: () for scalars, (4,) for a matrix."""
    return (4,) if dtype == "u32mat2x2" else ()


def element_bytes(dtype: str) -> int:
    return 16 if dtype == "u32mat2x2" else 4


def _matmul_2x2(a, b):
    # uint32 arithmetic in numpy wraps modulo 2^32 element-wise
    a00, a01, a10, a11 = a[..., 0], a[..., 1], a[..., 2], a[..., 3]
    b00, b01, b10, b11 = b[..., 0], b[..., 1], b[..., 2], b[..., 3]
    out = np.empty(np.broadcast_shapes(a.shape, b.shape), dtype=np.uint32)
    out[..., 0] = a00 * b00 + a01 * b10
    out[..., 1] = a00 * b01 + a01 * b11
    out[..., 2] = a10 * b00 + a11 * b10
    out[..., 3] = a10 * b01 + a11 * b11
    return out


def combine(dtype: str, op: str, a, b):
    """a (.) b for whole vectors, ``a`` on the left."""
    if not valid_pair(dtype, op):
        raise ValueError(f"unsupported pair {dtype} {op}")
    if dtype == "int32" and op == "sum":
        s = a.view(np.uint32) + b.view(np.uint32)
        return s.view(np.int32)
    if dtype == "int32" and op == "max":
        return np.maximum(a, b)
    if dtype == "float32":
        assert a.dtype == np.float32 and b.dtype == np.float32
        return np.add(a, b, dtype=np.float32)
    return _matmul_2x2(a, b)
