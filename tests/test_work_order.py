"""The attention kernel's work-item order on the host (no GPU): every ticket
number of the persistent workgroups' queues stands for one (block row, query
head) item or for padding, and every item is taken exactly once, for each
order, chunk size and a range of shapes (ragged block counts, GQA ratios 1 to
8, chunk sizes that do not divide the rows).  The mapping is plain integer
arithmetic in csrc/work_order.h, compiled here by the host C++ compiler; the
GPU test test_work_orders_give_identical_output checks the same property
through the kernel's outputs."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2509_24745_amd", "csrc")
ROCM_INCLUDE = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")


def test_every_item_taken_exactly_once(tmp_path):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None or not os.path.isdir(os.path.join(ROCM_INCLUDE, "hip")):
        pytest.skip("host C++ compiler or HIP headers not found")
    exe = tmp_path / "work_order_check"
    subprocess.run([cxx, "-std=c++17", "-O2", "-D__HIP_PLATFORM_AMD__", "-I" + ROCM_INCLUDE,
                    "-I" + CSRC, os.path.join(ROOT, "tests", "work_order_check.cpp"), "-o",
                    str(exe)], check=True, timeout=300)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:]
    cases, _, bad = r.stdout.strip().splitlines()[-1].split()[:3]
    assert int(cases) > 3000 and int(bad.rstrip(",")) == 0, r.stdout[-2000:]
