"""The cross-process mailboxes (hoccl_mailbox_*, host memory only, so on
the CPU): payloads and sequence numbers in one process, wrap-around,
timeouts, argument errors, and a ping-pong with a second process that
exercises both the polling and the sleeping wait."""
import ctypes
import os
import secrets
import subprocess
import sys
import time

import pytest

import paper_2609_34334_amd as hc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def fresh(tag):
    return f"/hoccl-test-{tag}-{os.getpid()}-{secrets.token_hex(4)}"


def test_post_wait_read_and_wrap():
    name = fresh("a")
    box = hc.Mailbox(name, 3, 100)
    try:
        other = hc.Mailbox(name)                 # a second mapping of the same object
        box.post(1, 1, b"hello")
        other.wait(1, 1, 1000)
        assert other.read(1) == b"hello"
        other.wait(1, 0, 0)                      # an older number counts as reached
        box.post(2, 0xFFFFFFFF, b"")
        other.wait(2, 0xFFFFFFFF, 0)
        assert other.read(2) == b""
        box.post(2, 1 << 32, b"x" * 100)         # wraps to 0, which comes after 2^32 - 1
        other.wait(2, 1 << 32, 0)
        assert other.read(2) == b"x" * 100
        other.close()
    finally:
        hc.Mailbox.unlink(name)
        box.close()


def test_timeouts_and_argument_errors():
    name = fresh("b")
    box = hc.Mailbox(name, 2, 64)
    try:
        t0 = time.perf_counter()
        with pytest.raises(hc.HocclError) as e:
            box.wait(0, 1, 20)
        assert e.value.status == hc.ERR_TIMEOUT
        assert 0.015 < time.perf_counter() - t0 < 5.0
        for bad in (lambda: box.post(2, 1, b""), lambda: box.wait(2, 1, 0), lambda: box.read(2),
                    lambda: box.post(0, 1, b"y" * 65)):
            with pytest.raises(hc.HocclError) as e:
                bad()
            assert e.value.status == hc.ERR_INVALID_ARG
        with pytest.raises(hc.HocclError):
            hc.Mailbox(name, 2, 64)              # the name exists
    finally:
        hc.Mailbox.unlink(name)
        box.close()
    with pytest.raises(hc.HocclError):
        hc.Mailbox(name)                         # unlinked: no longer opens
    for bad in ("noslash", "/", "/a/b", "/" + "n" * 300):
        with pytest.raises(hc.HocclError):
            hc.Mailbox(bad, 1, 8)
    L = hc.lib()
    h = ctypes.c_void_p()
    assert L.hoccl_mailbox_create(fresh("c").encode(), 0, 8, ctypes.byref(h)) == hc.ERR_INVALID_ARG
    assert L.hoccl_mailbox_create(fresh("c").encode(), 1, (1 << 20) + 1, ctypes.byref(h)) == hc.ERR_INVALID_ARG


CHILD = r"""
import sys, time
sys.path.insert(0, sys.argv[1])
import paper_2609_34334_amd as hc
box = hc.Mailbox(sys.argv[2])
for k in range(1, int(sys.argv[3]) + 1):
    box.wait(0, k, 10000)
    msg = box.read(0)
    if k % 50 == 0:
        time.sleep(0.002)                        # the parent's next wait sleeps on the futex
    box.post(1, k, msg[::-1])
box.close()
"""


def test_ping_pong_across_processes():
    name = fresh("d")
    box = hc.Mailbox(name, 2, 4096)
    n = 400
    p = subprocess.Popen([sys.executable, "-c", CHILD, ROOT, name, str(n)])
    try:
        for k in range(1, n + 1):
            msg = f"message {k} ".encode() * (k % 7 + 1)
            box.post(0, k, msg)
            if k % 75 == 0:
                time.sleep(0.002)               # the child's wait sleeps on the futex
            box.wait(1, k, 120_000 if k == 1 else 10_000)   # the first reply waits for the child's start
            assert box.read(1) == msg[::-1], k
        assert p.wait(timeout=60) == 0
    finally:
        if p.poll() is None:
            p.kill()
        hc.Mailbox.unlink(name)
        box.close()
