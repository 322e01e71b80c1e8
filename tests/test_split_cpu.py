"""Work split of the one-row-block approximator products, checked on the host.

The split (which workgroup streams which k-chunks of which item, and where
each piece of a cut item keeps its partial sums) is shared code between the
host plans and the kernels.  tests/native/split_check.cpp compiles that code
for the host and checks it against brute force over a grid of shapes.
"""
import os
import subprocess

import pytest

from paper_2606_03819_amd import build

HERE = os.path.dirname(os.path.abspath(__file__))


def test_split_invariants(tmp_path):
    hipcc = build.hipcc()
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    exe = tmp_path / "split_check"
    src = os.path.join(HERE, "native", "split_check.cpp")
    inc = os.path.join(os.path.dirname(HERE), "paper_2606_03819_amd", "csrc")
    rocm_inc = os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(hipcc))), "include")
    c = subprocess.run([hipcc, "-O1", "-std=c++17", "-x", "c++", "-D__HIP_PLATFORM_AMD__", "-I", rocm_inc, "-I", inc,
                        src, "-o", str(exe)], capture_output=True, text=True)
    assert c.returncode == 0, c.stderr[-3000:]
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    print(r.stdout)
    assert r.returncode == 0, r.stdout
    assert r.stdout.strip().endswith(" 0 failures")
