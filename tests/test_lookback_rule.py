"""The one-pass geometry build's look-back rule, compiled for the host.

tests/c_client/lookback_sim.cpp runs rows under random schedules with the
same status rules as the kernel (paper_2607_21927_amd/csrc/lookback.h) and
checks that a row that gives up -- or meets a poisoned prefix -- is poisoned,
that every other row keeps its exact offset, and that the stripped total is
negative exactly when some row is poisoned (the give-up is reported, never a
wrong CSR with a success code)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_lookback_rule_simulated_on_cpu(tmp_path):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = tmp_path / "lookback_sim"
    subprocess.run([cxx, "-O2", "-std=c++17", "-Wall", "-Werror",
                    "-I", os.path.join(ROOT, "paper_2607_21927_amd", "csrc"),
                    os.path.join(ROOT, "tests", "c_client", "lookback_sim.cpp"), "-o", str(exe)],
                   check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    print(r.stdout)
    assert r.returncode == 0, r.stdout
    assert r.stdout.strip().endswith("OK")
