"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle.

This module holds none of the method's arithmetic: it only turns
(seed, rank, element index) into input values.  Both the CPU oracle and the
HIP library are fed from it; it imports neither.

Generator: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014) in its widely used 64-bit finaliser form
(Vigna's splitmix64: increment 0x9E3779B97F4A7C15, then xor-shift-multiply
with 0xBF58476D1CE4E5B9 and 0x94D049BB133111EB, shifts 30, 27, 31).  It is
used counter-style: the 64-bit word for (seed, rank, k) is the first output of
a SplitMix64 stream whose state is

    key = (seed << 48) ^ (rank << 32) ^ k          (seed, rank < 2^16, k < 2^32)

so any single element can be produced on its own, which lets the oracle
check sampled columns of full-size workloads without the whole input.

Distributions (one 64-bit word per value unless stated):

* ``uniform_int(lo, hi)``  int32 lo + (z mod (hi - lo + 1)).
* ``uniform_u32``          uint32 z >> 32 (matrix entries use k = 4 e + c).
* ``odd_det_u32``          2x2 uint32 matrices with odd determinant
                           (a00, a11 odd, a01 even), i.e. invertible mod 2^32.
* ``normal_f32``           Box-Muller in float64 from the words for k = 2e and
                           k = 2e + 1 (u1 = (top 53 bits + 1) / 2^53 in (0, 1],
                           u2 = top 53 bits / 2^53), cos branch, rounded to
                           float32.  Values come from the host's libm; every
                           consumer in one process reads the same arrays.
"""

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def splitmix64(state):
    """First SplitMix64 output for each uint64 state (array in, array out)."""
    with np.errstate(over="ignore"):
        z = np.asarray(state, dtype=np.uint64) + GAMMA
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        return z ^ (z >> np.uint64(31))


def keys(seed: int, rank, k):
    """State words for ranks (broadcast against) element counters k."""
    if not (0 <= seed < 1 << 16):
        raise ValueError("seed must fit in 16 bits")
    r = np.asarray(rank, dtype=np.uint64)
    kk = np.asarray(k, dtype=np.uint64)
    return (np.uint64(seed) << np.uint64(48)) ^ (r << np.uint64(32)) ^ kk


def words(seed: int, rank, k):
    return splitmix64(keys(seed, rank, k))


# ---------------------------------------------------------------- per value

def uniform_int(seed, rank, cols, lo, hi):
    """int32 uniform in [lo, hi] for element indices ``cols``."""
    span = np.uint64(hi - lo + 1)
    z = words(seed, rank, cols)
    return (np.int64(lo) + (z % span).astype(np.int64)).astype(np.int32)


def uniform_u32_mat(seed, rank, cols):
    """2x2 uint32 matrices, shape [..., 4]."""
    c = np.asarray(cols, dtype=np.uint64)[..., None] * np.uint64(4) \
        + np.arange(4, dtype=np.uint64)
    z = words(seed, np.asarray(rank, dtype=np.uint64)[..., None], c)
    return (z >> np.uint64(32)).astype(np.uint32)


def odd_det_u32_mat(seed, rank, cols):
    a = uniform_u32_mat(seed, rank, cols)
    a[..., 0] |= np.uint32(1)
    a[..., 3] |= np.uint32(1)
    a[..., 1] &= np.uint32(0xFFFFFFFE)
    return a


def normal_f32(seed, rank, cols):
    c = np.asarray(cols, dtype=np.uint64)
    r = np.asarray(rank, dtype=np.uint64)
    z1 = words(seed, r, c * np.uint64(2))
    z2 = words(seed, r, c * np.uint64(2) + np.uint64(1))
    u1 = ((z1 >> np.uint64(11)).astype(np.float64) + 1.0) * (2.0 ** -53)
    u2 = (z2 >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)
    return (np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2)).astype(
        np.float32)


_DIST = {
    "uniform_int": lambda s, r, c, **kw: uniform_int(s, r, c, kw["lo"], kw["hi"]),
    "uniform_u32_mat": lambda s, r, c, **kw: uniform_u32_mat(s, r, c),
    "odd_det_u32_mat": lambda s, r, c, **kw: odd_det_u32_mat(s, r, c),
    "normal_f32": lambda s, r, c, **kw: normal_f32(s, r, c),
}


def sample(dist: str, seed: int, ranks, cols, **kw):
    """Values for every (rank, col) pair: array [len(ranks), len(cols)(, 4)]."""
    r = np.asarray(ranks, dtype=np.int64)[:, None]
    c = np.asarray(cols, dtype=np.int64)[None, :]
    return _DIST[dist](seed, r, c, **kw)


def generate(dist: str, seed: int, p: int, m: int, out=None, threads=None,
             **kw):
    """The full [p, m](, 4) input, one rank row at a time on a thread pool
    (numpy releases the GIL inside its loops)."""
    sample_row = _DIST[dist](seed, np.int64(0), np.arange(1), **kw)
    shape = (p, m) + sample_row.shape[1:]
    if out is None:
        out = np.empty(shape, dtype=sample_row.dtype)
    cols = np.arange(m, dtype=np.int64)

    def row(i):
        out[i] = _DIST[dist](seed, np.int64(i), cols, **kw)

    n = threads or min(16, os.cpu_count() or 1)
    if p * m < (1 << 16) or n == 1:
        for i in range(p):
            row(i)
    else:
        with ThreadPoolExecutor(max_workers=n) as ex:
            list(ex.map(row, range(p)))
    return out
