"""The staging copy pool of the host path (``csrc/tt_copy.cpp``), built on its
own with g++ and run on the CPU: concurrent callers, sizes from 0 bytes to 2 MB
around the chunk size, unaligned offsets, workers that fall asleep between
copies, plain copies and the widening copies of 16- and 24-bit IDs into int32.  Every
copy is compared value by value, and the bytes around the destination must
stay untouched.  A second build runs under ThreadSanitizer."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "tests", "native", "copy_pool_stress.cpp"),
       os.path.join(ROOT, "paper_2607_29678_amd", "csrc", "tt_copy.cpp")]


def _build(tmp_path, extra):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not found")
    exe = str(tmp_path / ("stress" + ("_tsan" if extra else "")))
    r = subprocess.run([gxx, "-O2", "-std=c++17", "-pthread", *extra, *SRC, "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def test_copy_pool_stress(tmp_path):
    exe = _build(tmp_path, [])
    r = subprocess.run([exe, "3", "400"], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr


def test_copy_pool_thread_sanitizer(tmp_path):
    exe = _build(tmp_path, ["-fsanitize=thread", "-g"])
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([exe, "2", "60"], capture_output=True, text=True, timeout=240, env=env)
    assert r.returncode == 0 and "WARNING: ThreadSanitizer" not in r.stderr, r.stdout + r.stderr[-4000:]
