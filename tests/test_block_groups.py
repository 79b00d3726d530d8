"""Work-item groups of the one-launch executors: when blocks (Section 1.1's
b successive blocks) are shorter than half a chunk, the host hands G
consecutive whole blocks to one work item.  The groups must cover the lines
[0, NL) exactly once, in block order, each within one chunk (64 quanta), and
G must be the largest such count.  CPU only: tests/cpp/group_check.cpp
prints the library planner's choice."""

import os
import shutil
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2109_12626_amd", "csrc")


def _cases():
    out = [(1 << 22, 6532, 4, 8), (1 << 22, 1, 4, 8), (1 << 16, 817, 4, 8),
           (1 << 16, 1, 4, 8), (1 << 10, 103, 4, 1), (16, 13, 1, 1),
           (1000, 4, 4, 8), (1 << 20, 2329, 4, 8), (1 << 18, 32, 1, 8),
           (1 << 16, 2048, 4, 8), (1 << 16, 4096, 4, 1), (4099, 7, 1, 1)]
    rng = np.random.default_rng(2109)
    for _ in range(400):
        g = int(rng.choice([1, 4]))
        m = int(rng.integers(1, 1 << 20))
        q = m // g
        if q == 0:
            continue
        b = int(rng.integers(1, q + 1))
        lq = 8 if (q + 7) // 8 >= b else 1
        out.append((m, b, g, lq))
    return out


CASES = _cases()


@pytest.fixture(scope="module")
def planned(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = tmp_path_factory.mktemp("grp") / "group_check"
    subprocess.run([gxx, "-O1", "-std=c++17", "-I", CSRC,
                    os.path.join(ROOT, "tests", "cpp", "group_check.cpp"),
                    os.path.join(CSRC, "plan.cpp"), "-o", str(exe)],
                   check=True)
    text = "\n".join(" ".join(map(str, c)) for c in CASES)
    res = subprocess.run([str(exe)], input=text, capture_output=True,
                         text=True, check=True)
    rows = [tuple(int(v) for v in line.split())
            for line in res.stdout.splitlines()]
    assert len(rows) == len(CASES)
    return dict(zip(CASES, rows))


def _groups(NL, b, G):
    """Lines of each group: blocks [k G, min(k G + G, b)), block j = lines
    [floor(j NL / b), floor((j + 1) NL / b))."""
    out = []
    for k in range(-(-b // G)):
        j0, j1 = k * G, min(k * G + G, b)
        out.append((NL * j0 // b, NL * j1 // b))
    return out


@pytest.mark.parametrize("case", CASES[:12])
def test_named_cases(planned, case):
    m, b, g, lq = case
    Q, NL, C, G = planned[case]
    want = {(1 << 22, 6532, 4, 8): 1, (1 << 22, 1, 4, 8): 1,
            (1 << 16, 817, 4, 8): 3, (1 << 16, 1, 4, 8): 1,
            (1 << 10, 103, 4, 1): 25, (16, 13, 1, 1): 13}
    if case in want:
        assert G == want[case], (case, G)


def test_groups_cover_the_lines_once_within_a_chunk(planned):
    for case, (Q, NL, C, G) in planned.items():
        m, b, g, lq = case
        L = 64 // lq
        maxl = -(-NL // b)
        assert 1 <= G <= b
        assert (G == 1) == (2 * maxl > L), case
        groups = _groups(NL, b, G)
        assert groups[0][0] == 0 and groups[-1][1] == NL, case
        for (a0, a1), (c0, _) in zip(groups, groups[1:]):
            assert a1 == c0, case                  # contiguous, in order
        if G > 1:
            assert C == 1, case
            for a0, a1 in groups:
                assert 0 < a1 - a0 <= L, case      # one chunk of lines
                assert min(a1 * lq, Q) - a0 * lq <= 64, case
            # the largest such G: G + 1 blocks may exceed a chunk
            assert G == b or (G + 1) * NL > b * L, case
