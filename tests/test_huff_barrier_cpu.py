"""The entropy decoder's one-launch hand-off protocol (csrc/huff_barrier.h),
run on the host with threads as workgroups: every waiter is released and
sees the serial step's result, launches in a row need no clearing, a waiter
gives up after exactly its spin limit, and the word stays consistent after
give-ups.  No GPU."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2609_09020_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_huff_barrier_protocol_on_host(tmp_path):
    exe = str(tmp_path / "huff_barrier_host")
    subprocess.run(["g++", "-O2", "-std=c++17", "-pthread", "-I", CSRC,
                    os.path.join(HERE, "huff_barrier_host.cpp"), "-o", exe], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().endswith("OK")
    assert "bound: 7 waiters gave up after 1000 polls each (limit 1000)" in r.stdout
