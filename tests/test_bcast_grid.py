"""Grid of the split executor's broadcast pass (y_0 copied into the other
p - 1 outputs, Section 1.1's delivery of y to every rank): every (output
row, tile of y_0) pair is written by exactly one workgroup, spans stay
within their byte budget (at least 8 tiles), and with several spans the
span width is a multiple of 8 tiles.  CPU only: tests/cpp/bcast_check.cpp
enumerates the library planner's grid."""

import os
import shutil
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2109_12626_amd", "csrc")

MB = 1 << 20


def _cases():
    out = [
        (16 * MB, 16, 1152, 16 * MB),     # the p = 1152, m = 2^22 fp32 pass
        (32 * MB, 16, 1152, 16 * MB),     # m = 2^23: two spans
        (32 * MB, 16, 9, 8 * MB),
        (4 * MB, 16, 64, 16 * MB),        # 2^18 matrices
        (4 * MB - 12, 4, 7, 1 * MB),      # 4-byte lanes, ragged end
        (4000, 16, 7, 4096),              # tiny spans: 8 tiles minimum
        (16, 16, 2, 4096),
        (256 * 16 * 9 + 16, 16, 3, 4096),  # 10 tiles, one span of 8 max
        (1 << 30, 16, 2, 16 * MB),
        (16 * MB - 4096, 16, 1152, 16 * MB),  # 4095 tiles: padded to 4096
        (2 * MB, 16, 5, 16 * MB),         # whole y_0 fits each L2: no padding
        (2 * MB + 16, 16, 5, 16 * MB),
    ]
    rng = np.random.default_rng(2110)
    for _ in range(300):
        lane = int(rng.choice([4, 16]))
        n = int(rng.integers(1, 1 << 16))
        p = int(rng.integers(2, 40))
        span = int(rng.choice([1024, 4096, 65536, 1 << 20, 16 * MB]))
        out.append((n * lane, lane, p, span))
    return out


CASES = _cases()


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = tmp_path_factory.mktemp("bcast") / "bcast_check"
    subprocess.run([gxx, "-O2", "-std=c++17", "-I", CSRC,
                    os.path.join(ROOT, "tests", "cpp", "bcast_check.cpp"),
                    os.path.join(CSRC, "plan.cpp"), "-o", str(exe)],
                   check=True)
    return str(exe)


@pytest.fixture(scope="module")
def grids(checker):
    text = "\n".join(" ".join(map(str, c)) for c in CASES)
    res = subprocess.run([checker], input=text, capture_output=True,
                         text=True, check=True)
    rows = [tuple(map(int, line.split())) for line in res.stdout.splitlines()]
    assert len(rows) == len(CASES)
    return dict(zip(CASES, rows))


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c)))
def test_broadcast_grid_covers_every_output_once(grids, case):
    nbytes, lane, p, span = case
    n, ts, nspan, rows, total, covered, padded, bad = grids[case]
    tiles = -(-n // 256)
    assert n == nbytes // lane and rows == p - 1
    assert bad == 0
    assert covered == rows * tiles            # every pair exactly once
    assert total == nspan * rows * ts == covered + padded
    budget = max(span // (256 * lane), 8)
    assert nspan == -(-tiles // max(budget & ~7, 8))
    assert ts <= max(budget & ~7, 8)
    if nspan > 1 or nbytes > 2 * MB:
        # every XCD (workgroup index mod 8) sees the same tiles in every row
        assert ts % 8 == 0
        assert padded < nspan * 8 * rows      # less than 8 tiles per span
    else:
        assert ts == tiles and padded == 0


def test_headline_pass_is_one_span(grids):
    """At p = 1152, m = 2^22 fp32 (16 MB rows) y_0 goes out as one span of
    4096 tiles; at m = 2^23 as two."""
    assert grids[(16 * MB, 16, 1152, 16 * MB)][1:3] == (4096, 1)
    assert grids[(32 * MB, 16, 1152, 16 * MB)][1:3] == (4096, 2)


# rows of ndw = 4 n dwords (the pass copies the n 16-byte lanes of y_0)
SPLITS = [(base + d, ndw) for base in (0, 1 << 40, 4096 * 7 + 128)
          for d in (0, 4, 8, 12, 132, 4092)
          for ndw in (4, 8, 12, 16, 1020, 1024, 1028, 4096, 4 << 20)]


@pytest.fixture(scope="module")
def splits(checker):
    text = "\n".join(f"split {d} {n}" for d, n in SPLITS)
    res = subprocess.run([checker], input=text, capture_output=True,
                         text=True, check=True)
    rows = [tuple(map(int, line.split())) for line in res.stdout.splitlines()]
    assert len(rows) == len(SPLITS)
    return dict(zip(SPLITS, rows))


@pytest.mark.parametrize("case", SPLITS, ids=lambda c: f"{c[0]}-{c[1]}")
def test_row_split_writes_every_dword_once_with_aligned_stores(splits, case):
    """Rows off 16-byte boundaries are written as leading dwords up to the
    row's first 4 KB boundary, 16-byte stores from there (each workgroup's
    4 KB tile starting on a 4 KB boundary), and at most 3 trailing dwords:
    every dword of the row once, nothing outside."""
    dst, ndw = case
    h, nbody, covered, twice, outside, misaligned = splits[case]
    assert h == min(((4096 - dst % 4096) % 4096) // 4, ndw)
    assert covered == ndw and twice == 0 and outside == 0
    assert misaligned == 0
    assert 0 <= ndw - h - 4 * nbody <= 3
    assert nbody <= ndw // 4          # body lanes inside the row's grid


DIVISORS = [1, 2, 3, 5, 7, 8, 63, 64, 1151, 4096, 4096 * 1151, 65537,
            (1 << 31) - 1, 1 << 31, (1 << 31) + 1, (1 << 32) - 1,
            1000003, 123456789]


def test_fastdiv_is_exact(checker):
    """The broadcast grid's division by multiplication (Lemire, Kaser and
    Kurz 2019) equals integer division for 32-bit dividends: edges, around
    multiples of the divisor, and 200000 pseudo-random points per divisor."""
    text = "\n".join(f"div {d}" for d in DIVISORS)
    res = subprocess.run([checker], input=text, capture_output=True,
                         text=True, check=True)
    assert [int(v) for v in res.stdout.split()] == [0] * len(DIVISORS)
