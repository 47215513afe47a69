"""The revolving-door walk used by the enumeration kernel, compiled for the
host with g++: every t-subset of {0..n-1} exactly once, one element in and
one out per step, and the (n, t) walk starts with the whole (b, t) walk for
every b <= n (the enumeration kernel stops each walk early on that basis).
The enumeration plans, compiled with hipcc: every k-subset exactly once."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def test_revolving_door_properties(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = tmp_path / "revdoor_check"
    subprocess.run(["g++", "-O2", "-std=c++17", os.path.join(HERE, "host", "revdoor_check.cpp"),
                    "-o", str(exe)], check=True)
    r = subprocess.run([str(exe)], stdout=subprocess.PIPE, text=True)
    assert r.returncode == 0, r.stdout
    assert "revolving door OK" in r.stdout


def test_enumeration_plans_cover_every_subset_once(tmp_path):
    """The enumeration plans (two or three key ranges; owned parts over one or
    two of them times a walked part) cover every k-subset exactly once, for
    the benchmark's shapes and edge cases; compiled for the host with hipcc
    (the plan header includes the HIP runtime header)."""
    hipcc = shutil.which("hipcc") or ("/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else None)
    if hipcc is None:
        pytest.skip("hipcc not available")
    exe = tmp_path / "plan_check"
    csrc = os.path.join(os.path.dirname(HERE), "paper_2608_25230_amd", "csrc")
    inc = os.path.join(os.path.dirname(HERE), "include")
    subprocess.run([hipcc, "-O2", "-std=c++17", "-I", csrc, "-I", inc, os.path.join(HERE, "host", "plan_check.cpp"),
                    "-o", str(exe)], check=True, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    r = subprocess.run([str(exe)], stdout=subprocess.PIPE, text=True)
    assert r.returncode == 0, r.stdout
    assert "plans OK" in r.stdout

