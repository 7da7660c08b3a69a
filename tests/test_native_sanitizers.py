"""The host code under AddressSanitizer and UBSan (CPU only): the planner and
the collective scheduler replay every plan shape on exactly-sized host
buffers, the C oracle runs every function the same way, and the engine
proxy's balanced issue runs against simulated engines, and two processes
ping-pong through the cross-process mailbox.  A read or write
outside a documented buffer, or undefined behaviour such as signed overflow,
fails the run.  The oracle's driver shares nothing with the other two."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2609_34334_amd", "csrc")
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer"]


def _run(cmd, tmp_path, exe):
    r = subprocess.run(cmd, capture_output=True, text=True, cwd=tmp_path)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    return r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_planner_and_scheduler_under_sanitizers(tmp_path):
    exe = str(tmp_path / "plan_bounds")
    cmd = ["g++", "-std=c++17", *SAN, "-I/opt/rocm/include", "-D__HIP_PLATFORM_AMD__",
           os.path.join(HERE, "native", "plan_bounds.cpp"), os.path.join(CSRC, "plan.cpp"),
           os.path.join(CSRC, "schedule.cpp"), "-o", exe]
    out = _run(cmd, tmp_path, exe)
    assert "plans replayed: 18432" in out, out


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_bounds")
    cmd = ["gcc", "-std=c11", *SAN, "-fno-fast-math", "-ffp-contract=off",
           os.path.join(HERE, "native", "oracle_bounds.c"), "-o", exe]
    out = _run(cmd, tmp_path, exe)
    assert "oracle cases run: 896" in out, out


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_proxy_balanced_issue_simulation(tmp_path):
    """The SDMA proxy's balanced issue against simulated engines (one at
    half rate, all equal, all work on one engine, a failed issue)."""
    exe = str(tmp_path / "balance_sim")
    cmd = ["g++", "-std=c++17", *SAN, os.path.join(HERE, "native", "balance_sim.cpp"),
           os.path.join(CSRC, "schedule.cpp"), "-o", exe]
    out = _run(cmd, tmp_path, exe)
    assert "balance cases: 133" in out, out


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_mailbox_across_a_fork(tmp_path):
    """The cross-process mailbox between a parent and a forked child."""
    exe = str(tmp_path / "mailbox_check")
    cmd = ["g++", "-std=c++17", *SAN, "-I/opt/rocm/include", "-D__HIP_PLATFORM_AMD__",
           os.path.join(HERE, "native", "mailbox_check.cpp"), os.path.join(CSRC, "mailbox.cpp"),
           "-o", exe]
    out = _run(cmd, tmp_path, exe)
    assert "mailbox cases: 1512" in out, out
