"""The order in which the split executor's up-phase hands work items to
workgroups when input rows are off 16-byte boundaries: workgroup w runs on
XCD w mod 8, and each XCD takes one contiguous run of the launch's items in
order.  The mapping must be a bijection of [0, n) (every work item of
Section 1.1's blocks evaluated once).  CPU only: tests/cpp/xcd_check.cpp
enumerates the library's mapping."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2109_12626_amd", "csrc")

NS = list(range(1, 200)) + [1023, 1024, 1025, 19596, 65535, 65536, 1 << 20,
                            (1 << 24) - 1]


@pytest.fixture(scope="module")
def checked(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = tmp_path_factory.mktemp("xcd") / "xcd_check"
    subprocess.run([gxx, "-O2", "-std=c++17", "-I", CSRC,
                    os.path.join(ROOT, "tests", "cpp", "xcd_check.cpp"),
                    "-o", str(exe)], check=True)
    res = subprocess.run([str(exe)], input="\n".join(map(str, NS)),
                         capture_output=True, text=True, check=True)
    return dict(line.split(" ", 1) for line in res.stdout.splitlines())


@pytest.mark.parametrize("n", NS)
def test_every_item_once_in_contiguous_runs_per_xcd(checked, n):
    assert checked[str(n)] == "ok"
