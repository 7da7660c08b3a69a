"""Parity under the workloads' own concurrency: the FSDP all-gather, the full
pipeline send/recv schedule (224 messages, all 32 rounds enqueued ahead, each
round into buffers of its own) and the EP all-to-all(v), on the default copy
path (AUTO: the SDMA engine proxy with its host-function handshake), start
together with a loop of bf16 8192^3 GEMMs on another hardware queue behind
one host gate, as the benchmark's interference runs do.  Every output
element is then compared with the oracle.  Also: calls from several host
threads at once, which the library serialises per device."""
import numpy as np
import pytest
import torch

import bench
import oracle
import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import assert_bitwise, from_dev, to_dev

pytestmark = pytest.mark.gpu

_GEMM = []


def gemm():
    if not _GEMM:
        _GEMM.append(bench.make_gemm())
    return _GEMM[0]


def beside_gemm(enqueue, reset, k=8):
    """Run `enqueue(stream)` once outside the gate (the library's first call
    on a device initialises it, which synchronises the device and must not
    wait for a closed gate), `reset()` its outputs to canaries, then enqueue
    it and k GEMMs behind one host gate, open it and synchronise; the gate's
    timer must not have had to open it (otherwise the collectives did not
    start with the GEMMs)."""
    g = gemm()
    gs, cs = g[4], g[5]
    with torch.cuda.stream(cs):
        enqueue(cs)
    torch.cuda.synchronize()
    reset()
    torch.cuda.synchronize()
    gate, open_gate = bench.host_gate()
    try:
        gs.wait_event(gate)
        cs.wait_event(gate)
        with torch.cuda.stream(cs):
            enqueue(cs)
        bench._gemm_run(g, k)
    finally:
        blocked = open_gate()
    torch.cuda.synchronize()
    assert not blocked, "the host was held up while enqueueing: the collectives did not start with the GEMMs"


@pytest.fixture(autouse=True)
def _auto():
    saved = hc.get_config()
    hc.set_config(copy_path="auto", sdma_engines=0)
    yield
    hc.set_config(**saved)


def test_allgather_fsdp_beside_gemm():
    R = 8
    x = W.ag_parameters(R)
    n = x[0].size
    send = [to_dev(a, hc.BF16) for a in x]
    recv = [torch.empty(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    beside_gemm(lambda s: hc.allgather(send, recv, stream=s),
                lambda: [t.view(torch.int16).fill_(0x7A5A) for t in recv])
    assert hc.last_stats()["copy_path_used"] == hc.COPY_SDMA
    ref = oracle.allgather_new(x, hc.BF16)
    for r in range(R):
        assert_bitwise(from_dev(recv[r], hc.BF16), ref[r], f"all-gather beside the GEMM, rank {r}")


def test_pipeline_schedule_beside_gemm():
    """16 microbatches, forward (r -> r+1) then backward (r -> r-1) each:
    32 rounds of 7 concurrent 16 MiB messages, every round into its own
    receive buffers, every message compared with the oracle."""
    R, mbs = 8, 16
    shape_n = 2048 * 4096
    xs = [[W.random_bits(400 + mb, r, shape_n, 2) for r in range(R)] for mb in range(mbs)]
    send = [[to_dev(a, hc.BF16) for a in x] for x in xs]
    fwd = [r + 1 if r + 1 < R else -1 for r in range(R)]
    bwd = [r - 1 for r in range(R)]
    rounds = [(mb, peers) for mb in range(mbs) for peers in (fwd, bwd)]
    recv = [[torch.full((shape_n,), 0x7A5A, dtype=torch.int16, device="cuda").view(torch.bfloat16)
             for _ in range(R)] for _ in rounds]

    def schedule(s):
        for i, (mb, peers) in enumerate(rounds):
            hc.sendrecv(send[mb], recv[i], peers, stream=s)
    beside_gemm(schedule, lambda: [t.view(torch.int16).fill_(0x7A5A) for rr in recv for t in rr])
    for i, (mb, peers) in enumerate(rounds):
        ref = [np.full(shape_n, 0x7A5A, np.uint16) for _ in range(R)]
        oracle.sendrecv(xs[mb], ref, peers, shape_n, hc.BF16)
        for r in range(R):
            assert_bitwise(from_dev(recv[i][r], hc.BF16), ref[r], f"round {i} rank {r}")


def test_alltoallv_ep_beside_gemm():
    R = 8
    send_np, counts, sd, rd, rsz = W.a2a_tokens(R)
    send = [to_dev(a, hc.BF16) for a in send_np]
    recv = [torch.zeros(s, dtype=torch.bfloat16, device="cuda") for s in rsz]

    def many(s):                                 # back to back, the last one checked
        for _ in range(8):
            hc.alltoallv(send, counts, sd, recv, rd, stream=s)
    beside_gemm(many, lambda: [t.zero_() for t in recv])
    ref = [np.zeros(s, np.uint16) for s in rsz]
    oracle.alltoallv(send_np, counts, sd, ref, rd, hc.BF16)
    for r in range(R):
        assert_bitwise(from_dev(recv[r], hc.BF16), ref[r], f"EP all-to-all(v) beside the GEMM, rank {r}")


@pytest.mark.parametrize("path", ["engines", "kernel"])
def test_calls_from_several_host_threads(path):
    """Four host threads call the library at once, each on its own stream
    with its own buffers: reduce-scatters, all-gathers and send/recvs in a
    loop.  The library serialises the calls per device; every result must
    match the oracle."""
    import threading
    R, n, loops = 4, 20_011, 12
    x = [W.random_values("bf16", 1200, r, R * n) for r in range(R)]
    rs_ref = oracle.reduce_scatter_new(x, hc.BF16)
    g = [W.random_bits(1201, r, n, 2) for r in range(R)]
    ag_ref = oracle.allgather_new(g, hc.BF16)
    errors, results = [], {}

    def worker(k):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                send = [to_dev(a, hc.BF16) for a in x]
                shards = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
                gs = [to_dev(a, hc.BF16) for a in g]
                full = [torch.empty(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
                moved = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
                for _ in range(loops):
                    hc.reduce_scatter(send, shards, stream=s)
                    hc.allgather(gs, full, stream=s)
                    hc.sendrecv(gs, moved, [(r + k + 1) % R for r in range(R)], stream=s)
                s.synchronize()
                results[k] = ([from_dev(t, hc.BF16) for t in shards], [from_dev(t, hc.BF16) for t in full],
                              [from_dev(t, hc.BF16) for t in moved])
        except Exception as e:          # reported by the main thread
            errors.append(repr(e))

    with hc.config(copy_path=path):
        hc.reduce_scatter([to_dev(a, hc.BF16) for a in x])     # initialise on this thread first
        torch.cuda.synchronize()
        threads = [threading.Thread(target=worker, args=(k,)) for k in range(4)]
        for t in threads:
            t.start()
        for t in threads:
            t.join(timeout=120)
        assert not any(t.is_alive() for t in threads), "a thread did not finish"
    assert not errors, errors
    for k in range(4):
        shards, full, moved = results[k]
        for r in range(R):
            assert_bitwise(shards[r], rs_ref[r], f"thread {k} reduce-scatter rank {r}")
            assert_bitwise(full[r], ag_ref[r], f"thread {k} all-gather rank {r}")
            assert_bitwise(moved[(r + k + 1) % R], g[r], f"thread {k} send/recv from rank {r}")
