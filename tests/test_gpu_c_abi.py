"""The C ABI from plain C: tests/native/c_abi_check (built by build()) links
libhoccl.so, allocates with hipMalloc and runs every collective without
Python or torch in the process, checking closed forms (also for one ring
hop) and the argument errors."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "c_abi_check")


def test_c_program_drives_the_library():
    assert os.path.exists(EXE), "tests/native/c_abi_check is missing: run __graft_entry__.build()"
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "c abi ok" in r.stdout, (r.returncode, r.stdout, r.stderr[-3000:])
