"""Host scheduler of expert copies (csrc/expert_sched.h) under a fake copy
engine that delays copies, refuses them when started, or completes them with
an error, built with g++ and run under AddressSanitizer + UndefinedBehavior-
Sanitizer (copies completed by polling) and under ThreadSanitizer (copies
completed by a worker thread).  No GPU: the scheduler and the cache policy
are host code; the GPU runtime drives the same scheduler with its HIP copy
engine.  The checks (tests/host/expert_sched_test.cpp): every needed expert
is held by its slot once the layer runs, a refused or failed prefetch is
invalidated and loaded on demand when used, a refused on-demand copy is an
error of the layer that leaves its slots empty, and delays do not change the
logical hit and miss counts."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "host", "expert_sched_test.cpp")
INC = os.path.join(ROOT, "paper_2502_02040_amd", "csrc")


def _build_and_run(tmp_path, flags, args):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "expert_sched_test")
    r = subprocess.run([gxx, "-std=c++17", "-O1", "-g", *flags, "-I", INC, SRC, "-o", exe], capture_output=True,
                       text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-3000:]
    r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, (r.stdout + r.stderr)[-3000:]
    assert r.stdout.startswith("ok"), r.stdout
    return r.stdout


def test_scheduler_with_fake_copy_engine_asan_ubsan(tmp_path):
    out = _build_and_run(tmp_path, ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"], [])
    assert "polled engine" in out


def test_scheduler_with_threaded_fake_copy_engine_tsan(tmp_path):
    out = _build_and_run(tmp_path, ["-fsanitize=thread"], ["threaded"])
    assert "threaded engine" in out
