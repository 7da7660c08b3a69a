"""Stream order with the collective held behind a host flag.

The caller's stream first waits (hipStreamWaitValue32) on a flag in coherent
host memory, then gets the collective.  While the flag is unset the stream
must not be done and every output must still hold its canary, on every copy
path and for the reductions; once the host sets the flag the result must
equal the oracle bit for bit.  The caller's stream owns its hardware queue
(CU-masked stream), outputs are read on another such stream, and a timer
thread sets the flag after 5 s in any case, so no wait can outlast the test."""
import ctypes
import threading
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import assert_bitwise, from_dev, to_dev

pytestmark = pytest.mark.gpu

HIP = ctypes.CDLL("libamdhip64.so.7")          # the HIP runtime torch has loaded
V = ctypes.c_void_p
HIP.hipHostMalloc.argtypes = [ctypes.POINTER(V), ctypes.c_size_t, ctypes.c_uint]
HIP.hipStreamWaitValue32.argtypes = [V, V, ctypes.c_uint32, ctypes.c_uint, ctypes.c_uint32]
HIP_HOST_MALLOC_MAPPED, HIP_HOST_MALLOC_COHERENT, WAIT_EQ = 0x2, 0x40000000, 0x1


@pytest.fixture(autouse=True)
def _defaults():
    saved = hc.get_config()
    yield
    hc.set_config(**saved)


_STREAMS = []


def own_queue_streams():
    """Two CU-masked streams (each owns a hardware queue), created once."""
    while len(_STREAMS) < 2:
        h = V()
        mask = (ctypes.c_uint32 * 8)(*([0xFFFFFFFF] * 8))
        assert HIP.hipExtStreamCreateWithCUMask(ctypes.byref(h), 8, mask) == 0
        _STREAMS.append(torch.cuda.ExternalStream(h.value))
    return _STREAMS


_FLAG = None


def flag():
    global _FLAG
    if _FLAG is None:
        p = V()
        assert HIP.hipHostMalloc(ctypes.byref(p), 64,
                                 HIP_HOST_MALLOC_MAPPED | HIP_HOST_MALLOC_COHERENT) == 0
        _FLAG = p.value
    return _FLAG


CANARY = {hc.BF16: 0x7A5A, hc.FP32: 0x7A5A7A5A}


def fill_canary(t, dt):
    t.view(torch.int16 if dt == hc.BF16 else torch.int32).fill_(CANARY[dt])


def gated(run, outs, dt):
    """Run once ungated (library state and workspace exist afterwards, so
    the gated call needs no allocation or device synchronisation), refill
    the outputs with canaries, then enqueue wait(flag == k) and run(s) on an
    own-queue stream, check the gated window, release and synchronise."""
    s, rs = own_queue_streams()
    with torch.cuda.stream(s):
        run(s)
    torch.cuda.synchronize()
    for o in outs:
        fill_canary(o, dt)
    f = flag()
    cell = ctypes.c_uint32.from_address(f)
    cell.value = 0
    k = int(time.time() * 1000) % 1_000_000 + 1
    torch.cuda.synchronize()
    release = threading.Timer(5.0, lambda: setattr(cell, "value", k))
    release.start()
    try:
        assert HIP.hipStreamWaitValue32(V(s.cuda_stream), V(f), k, WAIT_EQ, 0xFFFFFFFF) == 0
        with torch.cuda.stream(s):
            run(s)
        time.sleep(0.05)
        assert not s.query(), "the stream finished while its gate was closed"
        want = np.uint16(CANARY[dt]) if dt == hc.BF16 else np.uint32(CANARY[dt])
        with torch.cuda.stream(rs):
            for o in outs:
                got = from_dev(o, dt).view(want.dtype)
                assert (got == want).all(), "an output changed before the gate opened"
        assert not s.query()
    finally:
        release.cancel()
        cell.value = k
    s.synchronize()
    torch.cuda.synchronize()


@pytest.mark.parametrize("path", ["hip", "engines", "engines_kernel", "kernel"])
def test_copy_collectives_wait_for_the_gate(path):
    if path.startswith("engines") and hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    hc.set_config(copy_path=path.split("_")[0], proxy_handshake=0 if path == "engines_kernel" else -1)
    R, n = 8, 70_001
    x = [W.random_bits(401, r, n, 2) for r in range(R)]
    ref = oracle.allgather_new(x, hc.BF16)
    send = [to_dev(a, hc.BF16) for a in x]
    outs = [torch.empty(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    gated(lambda s: hc.allgather(send, outs, stream=s), outs, hc.BF16)
    for r in range(R):
        assert_bitwise(from_dev(outs[r], hc.BF16), ref[r], f"{path} allgather rank {r}")
    # send/recv: one message (the caller's stream itself on the SDMA path)
    a = to_dev(W.random_bits(402, 0, n, 2), hc.BF16)
    o = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    gated(lambda s: hc.sendrecv([a, a], [o, o], [1, -1], stream=s), [o], hc.BF16)
    assert_bitwise(from_dev(o, hc.BF16), from_dev(a, hc.BF16), f"{path} sendrecv")


@pytest.mark.parametrize("algo", ["ring", "direct"])
def test_reductions_wait_for_the_gate(algo):
    hc.set_config(reduce_algo=algo)
    R, n = 8, 40_003
    x = [W.random_values("bf16", 403, r, R * n) for r in range(R)]
    ref = oracle.reduce_scatter_new(x, hc.BF16)
    send = [to_dev(a, hc.BF16) for a in x]
    outs = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    gated(lambda s: hc.reduce_scatter(send, outs, stream=s), outs, hc.BF16)
    for r in range(R):
        assert_bitwise(from_dev(outs[r], hc.BF16), ref[r], f"{algo} reduce-scatter rank {r}")
    xa = [W.random_values("fp32", 404, r, 50_000) for r in range(4)]
    refa = oracle.allreduce_new(xa, hc.FP32)
    senda = [to_dev(a, hc.FP32) for a in xa]
    outa = [torch.empty(50_000, device="cuda") for _ in range(4)]
    gated(lambda s: hc.allreduce(senda, outa, stream=s), outa, hc.FP32)
    for r in range(4):
        assert_bitwise(from_dev(outa[r], hc.FP32), refa[r], f"{algo} all-reduce rank {r}")


@pytest.mark.parametrize("handshake", [-1, 0])
def test_grouped_allreduce_on_the_engines_waits_for_the_gate(handshake):
    """All-reduce in 4 chunk groups on the engine proxy: each group's gather
    copies run on a library stream that waits for that group's reductions,
    and the caller's stream joins those streams.  Behind a closed gate none
    of it may run, and once the gate opens the result is the oracle's."""
    if hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    hc.set_config(copy_path="engines", allreduce_chunk_groups=4, proxy_handshake=handshake)
    R, n = 8, 1_000_003
    x = [W.random_values("bf16", 408, r, n) for r in range(R)]
    ref = oracle.allreduce_new(x, hc.BF16)
    send = [to_dev(a, hc.BF16) for a in x]
    outs = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    gated(lambda s: hc.allreduce(send, outs, stream=s), outs, hc.BF16)
    assert hc.last_stats()["copy_ops"] > 0
    for r in range(R):
        assert_bitwise(from_dev(outs[r], hc.BF16), ref[r], f"grouped all-reduce rank {r}")


def test_debug_log_names_the_plan(tmp_path):
    """HOCCL_DEBUG=1 logs each executed plan (checked in a child process)."""
    import subprocess
    import sys
    import os
    code = ("import torch, paper_2609_34334_amd as hc; "
            "x = [torch.ones(64, device='cuda') for _ in range(4)]; "
            "hc.allreduce(x); torch.cuda.synchronize()")
    env = dict(os.environ, HOCCL_DEBUG="1")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env,
                       timeout=120)
    assert r.returncode == 0, r.stderr[-2000:]
    assert "hoccl: device 0" in r.stderr and "plan {" in r.stderr, r.stderr[-2000:]


@pytest.mark.parametrize("K,n", [(300, 2048), (24, (1 << 19) + 3)], ids=["4KiB", "1MiB"])
def test_many_engine_operations_in_flight(K, n):
    """Engine-proxy send/recv operations queued behind a closed gate, each
    copying buffer k into buffer k+1: when the gate opens they must run in
    stream order, so every buffer ends up holding buffer 0's bits and none
    keeps its canary.  300 messages of 4 KiB (more than the old pool of 64
    handshake slots) take the ungated form; 24 of just over 1 MiB take the
    form whose copies start on an event the proxy polls, so each message's
    copies must wait for the previous message's handshake."""
    if hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    hc.set_config(copy_path="engines")
    bufs = [torch.full((n,), 0x7A5A, dtype=torch.int16, device="cuda").view(torch.bfloat16)
            for _ in range(K + 1)]
    first = to_dev(W.random_bits(405, 0, n, 2), hc.BF16)
    bufs[0].copy_(first)
    s, _ = own_queue_streams()
    hc.sendrecv([bufs[0], bufs[0]], [bufs[1], bufs[1]], [1, -1], stream=s)   # warm path
    torch.cuda.synchronize()
    bufs[1].view(torch.int16).fill_(0x7A5A)
    torch.cuda.synchronize()
    f = flag()
    cell = ctypes.c_uint32.from_address(f)
    cell.value = 0
    k = int(time.time() * 1000) % 1_000_000 + 1
    release = threading.Timer(5.0, lambda: setattr(cell, "value", k))
    release.start()
    try:
        assert HIP.hipStreamWaitValue32(V(s.cuda_stream), V(f), k, WAIT_EQ, 0xFFFFFFFF) == 0
        with torch.cuda.stream(s):
            for i in range(K):
                hc.sendrecv([bufs[i], bufs[i]], [bufs[i + 1], bufs[i + 1]], [1, -1], stream=s)
        assert not s.query(), "the stream finished while its gate was closed"
    finally:
        release.cancel()
        cell.value = k
    s.synchronize()
    torch.cuda.synchronize()
    want = from_dev(first, hc.BF16)
    for i in (1, K // 2, K):
        assert_bitwise(from_dev(bufs[i], hc.BF16), want, f"buffer {i}")


@pytest.mark.parametrize("case,calls", [("ring_reduce_scatter", 100), ("kernel_sendrecv", 500)])
def test_many_launches_queue_without_stalling_the_host(case, calls):
    """Hundreds of collectives queued behind a closed gate, as a training
    step queues its gradient reductions behind unfinished compute: the
    enqueueing thread must not wait for the GPU.  The HIP runtime stages
    the arguments of every launch that has not started and makes the
    caller wait once about 1 MB of them is pending.  100 ring
    reduce-scatters (700 launches of an 8-rank step) or 500 CU-kernel
    send/recvs fit only with arguments sized to the launch (with a fixed
    2 KiB of slots, some 450 launches fill it).  The timer opens the gate
    after 10 s in any case; the results must equal the oracle bit for bit."""
    s, _ = own_queue_streams()
    R = 8
    if case == "ring_reduce_scatter":
        n = 4096
        x = [W.random_values("bf16", 406, r, R * n) for r in range(R)]
        ref = oracle.reduce_scatter_new(x, hc.BF16)
        send = [to_dev(a, hc.BF16) for a in x]
        outs = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
        run = lambda: hc.reduce_scatter(send, outs, stream=s)
    else:
        hc.set_config(copy_path="kernel")
        n = 2048
        a = to_dev(W.random_bits(407, 0, n, 2), hc.BF16)
        outs = [torch.empty(n, dtype=torch.bfloat16, device="cuda")]
        ref = [from_dev(a, hc.BF16)]
        run = lambda: hc.sendrecv([a, a], [outs[0], outs[0]], [1, -1], stream=s)
    run()                                       # library state and workspace
    torch.cuda.synchronize()
    for o in outs:
        fill_canary(o, hc.BF16)
    torch.cuda.synchronize()
    f = flag()
    cell = ctypes.c_uint32.from_address(f)
    cell.value = 0
    k = int(time.time() * 1000) % 1_000_000 + 1
    fired = []
    release = threading.Timer(10.0, lambda: (fired.append(True), setattr(cell, "value", k)))
    release.start()
    try:
        assert HIP.hipStreamWaitValue32(V(s.cuda_stream), V(f), k, WAIT_EQ, 0xFFFFFFFF) == 0
        t0 = time.perf_counter()
        with torch.cuda.stream(s):
            for _ in range(calls):
                run()
        enqueue_s = time.perf_counter() - t0
        assert enqueue_s < 2.0 and not fired, (
            f"enqueueing {calls} calls took {enqueue_s:.1f} s: the host waited for the GPU")
        assert not s.query(), "the stream ran before the gate opened"
    finally:
        release.cancel()
        cell.value = k
    s.synchronize()
    torch.cuda.synchronize()
    for r in range(len(outs)):
        assert_bitwise(from_dev(outs[r], hc.BF16), ref[r], f"{case} rank {r}")
