"""Zero CUs, shown by occupancy rather than by a trace.

Every CU's wave slots are held by a bounded spin kernel
(tests/native/occupy.hip) on one hardware queue: two rounds of blocks, each
spinning SPIN_MS.  A collective issued on another queue a few milliseconds
into the first round finishes long before that round ends if its copies need
no CU; if they need one, it can only finish once the first round's blocks
exit.  A kernel trace cannot tell the two apart: the HIP runtime's own
device-to-device copies dispatch nothing on the application's queues, yet in
the runtime PyTorch bundles they wait for free CUs.

The copy collectives on the default path (AUTO = the engine proxy with the
host-function handshake) must finish inside the first round; the CU copy
kernel, the positive control, must not.  Every result is also checked bit
for bit.  The spin is bounded by the GPU's real-time counter, so every block
exits whatever else runs."""
import ctypes
import os
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import assert_bitwise, from_dev, to_dev

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
SPIN_MS = 40.0
ISSUE_AT_MS = 5.0
HIP = ctypes.CDLL("libamdhip64.so.7")          # the HIP runtime torch has loaded


@pytest.fixture(autouse=True)
def _defaults():
    saved = hc.get_config()
    yield
    hc.set_config(**saved)


_OCC = {}


def occupy():
    if "lib" not in _OCC:
        path = os.path.join(HERE, "native", "liboccupy.so")
        if not os.path.exists(path):
            import __graft_entry__
            __graft_entry__._build_occupy_helper()
        lib = ctypes.CDLL(path)
        lib.occupy_launch.argtypes = [ctypes.c_int, ctypes.c_uint64, ctypes.c_void_p]
        lib.occupy_launch.restype = ctypes.c_int
        streams = []
        for _ in range(2):                     # each owns a hardware queue
            h = ctypes.c_void_p()
            mask = (ctypes.c_uint32 * 8)(*([0xFFFFFFFF] * 8))
            assert HIP.hipExtStreamCreateWithCUMask(ctypes.byref(h), 8, mask) == 0
            streams.append(torch.cuda.ExternalStream(h.value))
        _OCC.update(lib=lib, streams=streams)
    return _OCC


def finish_time_beside_spin(run):
    """Runs `run(stream)` once unhindered, then again ISSUE_AT_MS into a spin
    that holds every CU slot; returns (milliseconds from the spin's start to
    the collective's end, the first round's end)."""
    o = occupy()
    spin_s, coll_s = o["streams"]
    run(coll_s)                                # library state, warm path
    torch.cuda.synchronize()
    blocks = 4 * torch.cuda.get_device_properties(0).multi_processor_count   # two rounds
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(spin_s)
    assert o["lib"].occupy_launch(blocks, int(SPIN_MS * 1e5), ctypes.c_void_p(spin_s.cuda_stream)) == 0
    time.sleep(ISSUE_AT_MS / 1e3)
    run(coll_s)
    t1.record(coll_s)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1), SPIN_MS


def _copy_workloads():
    R, n = 8, 1 << 20
    shards = [W.random_bits(501, r, n, 2) for r in range(R)]
    ag_ref = oracle.allgather_new(shards, hc.BF16)
    ag_in = [to_dev(a, hc.BF16) for a in shards]
    ag_out = [torch.empty(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    blocks = [W.random_bits(502, r, R * 4096, 2) for r in range(R)]
    a2a_ref = [np.zeros(R * 4096, np.uint16) for _ in range(R)]
    oracle.alltoall(blocks, a2a_ref, 4096, hc.BF16)
    a2a_in = [to_dev(a, hc.BF16) for a in blocks]
    a2a_out = [torch.empty(R * 4096, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    peers = [r + 1 if r + 1 < R else -1 for r in range(R)]
    p2p_ref = [np.zeros(n, np.uint16) for _ in range(R)]
    oracle.sendrecv(shards, p2p_ref, peers, n, hc.BF16)
    p2p_out = [torch.zeros(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    return [
        ("all-gather", lambda s: hc.allgather(ag_in, ag_out, stream=s), ag_out, ag_ref),
        ("all-to-all", lambda s: hc.alltoall(a2a_in, a2a_out, stream=s), a2a_out, a2a_ref),
        ("send/recv", lambda s: hc.sendrecv(ag_in, p2p_out, peers, stream=s), p2p_out, p2p_ref),
    ]


@pytest.mark.parametrize("path", ["auto", "engines"])
def test_copy_collectives_finish_while_every_cu_is_busy(path):
    if hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    hc.set_config(copy_path=path)
    for name, run, outs, ref in _copy_workloads():
        done_ms, round_ms = finish_time_beside_spin(run)
        s = hc.last_stats()
        assert s["copy_path_used"] == hc.COPY_SDMA and s["cus_used_max"] == 0, (name, s)
        assert done_ms < round_ms - 10, (
            f"{path} {name}: finished {done_ms:.1f} ms after the spin began, not before its "
            f"first round ended ({round_ms:.0f} ms): its copies needed a CU")
        for r in range(len(outs)):
            if name == "send/recv" and r == 0:
                continue                       # rank 0 receives nothing
            assert_bitwise(from_dev(outs[r], hc.BF16), ref[r], f"{path} {name} rank {r}")


def test_cu_copy_kernel_waits_for_the_cus():
    """The positive control: the CU copy kernel cannot run before CU slots free up."""
    hc.set_config(copy_path="kernel")
    name, run, outs, ref = _copy_workloads()[0]
    done_ms, round_ms = finish_time_beside_spin(run)
    assert done_ms >= round_ms - 2, f"the CU copy kernel finished at {done_ms:.1f} ms, inside the spin"
    for r in range(len(outs)):
        assert_bitwise(from_dev(outs[r], hc.BF16), ref[r], f"kernel {name} rank {r}")


def test_graph_replay_on_auto_finishes_while_every_cu_is_busy():
    """A graph captured on AUTO records the engine copies as a host node:
    its replay, too, needs no CU.  The replayed all-gather is bit-exact."""
    if hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    hc.set_config(copy_path="auto")
    name, run, outs, ref = _copy_workloads()[0]
    o = occupy()
    coll_s = o["streams"][1]
    run(coll_s)                                # eager first: library state
    torch.cuda.synchronize()
    assert hc.last_stats()["copy_path_used"] == hc.COPY_SDMA
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=coll_s):
        run(coll_s)
    torch.cuda.synchronize()
    assert hc.last_stats()["copy_path_used"] == hc.COPY_SDMA
    for t in outs:
        t.zero_()
    torch.cuda.synchronize()

    def replay(s):
        with torch.cuda.stream(s):
            g.replay()

    done_ms, round_ms = finish_time_beside_spin(replay)
    assert done_ms < round_ms - 10, (
        f"the replay finished {done_ms:.1f} ms after the spin began: its copies needed a CU")
    for r in range(len(outs)):
        assert_bitwise(from_dev(outs[r], hc.BF16), ref[r], f"replayed {name} rank {r}")
    del g
