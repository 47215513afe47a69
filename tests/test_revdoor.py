"""The revolving-door walk used by the enumeration kernel, compiled for the
host with g++: every t-subset of {0..n-1} exactly once, one element in and
one out per step, and the (n, t) walk starts with the whole (b, t) walk for
every b <= n (the enumeration kernel stops each walk early on that basis)."""
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
