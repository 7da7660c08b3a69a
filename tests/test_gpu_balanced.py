"""Parity of the SDMA proxy's balanced issue, where the copies are cut into
pieces as the engines take them: on all 16 engines right after a 2 GiB
free (one engine then runs at about half rate while the driver releases
the memory, so the finish-time gate moves the last pieces to the others),
with 64 KiB minimum pieces (many cuts, sizes that are no multiple of
4 KiB), and against issuing every copy at once.  Every output element is
compared with the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import assert_bitwise, from_dev, to_dev

pytestmark = pytest.mark.gpu

SIZE_MAX = (1 << 64) - 1
R = 8


@pytest.fixture(autouse=True)
def _engines():
    if hc.sdma_engine_count() == 0:
        pytest.skip("no SDMA engine can be driven directly")
    saved = hc.get_config()
    yield
    hc.set_config(**saved)


def free_2gib():
    """Allocate and release 2 GiB of device memory: the window in which one
    engine is slowed starts."""
    F = [torch.empty(64 << 20, dtype=torch.uint8, device="cuda") for _ in range(32)]
    torch.cuda.synchronize()
    del F
    torch.cuda.empty_cache()


@pytest.mark.parametrize("slice_bytes", [0, 4 << 20, SIZE_MAX])
def test_allgather_16_engines_after_free(slice_bytes):
    n = (16 << 20) // 4                      # 16 MiB shards: 64 copies of 16 MiB
    x = [W.random_bits(700, r, n, 4).view(np.int32) for r in range(R)]
    send = [to_dev(a, hc.INT32) for a in x]
    recv = [torch.full((R * n,), -7, dtype=torch.int32, device="cuda") for _ in range(R)]
    hc.set_config(copy_path="engines", sdma_engines=16, proxy_slice_bytes=slice_bytes)
    free_2gib()
    hc.allgather(send, recv)
    torch.cuda.synchronize()
    assert hc.last_stats()["copy_path_used"] == hc.COPY_SDMA
    ref = oracle.allgather_new(x, hc.INT32)
    for r in range(R):
        assert_bitwise(from_dev(recv[r], hc.INT32), ref[r], f"all-gather rank {r}")


def test_alltoall_16_engines_after_free():
    n = (8 << 20) // 4                       # 8 MiB blocks
    x = [W.random_bits(701, r, R * n, 4).view(np.int32) for r in range(R)]
    send = [to_dev(a, hc.INT32) for a in x]
    recv = [torch.full((R * n,), -7, dtype=torch.int32, device="cuda") for _ in range(R)]
    hc.set_config(copy_path="engines", sdma_engines=16, proxy_slice_bytes=4 << 20)
    free_2gib()
    hc.alltoall(send, recv)
    torch.cuda.synchronize()
    ref = [np.zeros(R * n, np.int32) for _ in range(R)]
    oracle.alltoall(x, ref, n, hc.INT32)
    for r in range(R):
        assert_bitwise(from_dev(recv[r], hc.INT32), ref[r], f"all-to-all rank {r}")


@pytest.mark.parametrize("engines", [4, 16])
def test_sendrecv_small_pieces_odd_sizes(engines):
    """Messages of 3 MiB plus 1237 elements around the ring, cut into 64 KiB
    pieces: the last piece of every message is no multiple of 4 KiB."""
    n = (3 << 20) // 2 + 1237
    x = [W.random_bits(702, r, n, 2) for r in range(R)]
    peers = [(r + 1) % R for r in range(R)]
    send = [to_dev(a, hc.BF16) for a in x]
    recv = [torch.full((n,), 0x7A5A, dtype=torch.int16, device="cuda").view(torch.bfloat16) for _ in range(R)]
    hc.set_config(copy_path="engines", sdma_engines=engines, proxy_slice_bytes=64 << 10)
    hc.sendrecv(send, recv, peers)
    torch.cuda.synchronize()
    ref = [np.full(n, 0x7A5A, np.uint16) for _ in range(R)]
    oracle.sendrecv(x, ref, peers, n, hc.BF16)
    for r in range(R):
        assert_bitwise(from_dev(recv[r], hc.BF16), ref[r], f"send/recv rank {r}")


@pytest.mark.parametrize("engines,slice_bytes", [(0, 64 << 10), (0, 0), (0, SIZE_MAX), (16, 0)])
def test_alltoallv_ep_balanced_and_static(engines, slice_bytes):
    send_np, counts, sd, rd, rsz = W.a2a_tokens(R)
    send = [to_dev(a, hc.BF16) for a in send_np]
    recv = [torch.zeros(s, dtype=torch.bfloat16, device="cuda") for s in rsz]
    hc.set_config(copy_path="engines", sdma_engines=engines, proxy_slice_bytes=slice_bytes)
    hc.alltoallv(send, counts, sd, recv, rd)
    torch.cuda.synchronize()
    ref = [np.zeros(s, np.uint16) for s in rsz]
    oracle.alltoallv(send_np, counts, sd, ref, rd, hc.BF16)
    for r in range(R):
        assert_bitwise(from_dev(recv[r], hc.BF16), ref[r], f"EP all-to-all(v) rank {r}")


def test_slice_bytes_validation():
    for bad in (4096, (64 << 10) + 1, 1000):
        with pytest.raises(hc.HocclError):
            hc.set_config(proxy_slice_bytes=bad)
    hc.set_config(proxy_slice_bytes=64 << 10)
    hc.set_config(proxy_slice_bytes=SIZE_MAX)
    hc.set_config(proxy_slice_bytes=0)


def test_pipeline_schedule_queued_ahead_balanced():
    """The pipeline schedule's 32 rounds (16 microbatches, forward then
    backward, 7 messages of 16 MiB each) enqueued ahead on one stream, on
    16 engines with 4 MiB pieces: every round's copies go out by balanced
    issue as its gate opens, each round into buffers of its own, and every
    message matches the oracle."""
    n = 2048 * 4096
    mbs = 16
    xs = [[W.random_bits(710 + mb, r, n, 2) for r in range(R)] for mb in range(mbs)]
    send = [[to_dev(a, hc.BF16) for a in x] for x in xs]
    fwd = [r + 1 if r + 1 < R else -1 for r in range(R)]
    bwd = [r - 1 for r in range(R)]
    rounds = [(mb, peers) for mb in range(mbs) for peers in (fwd, bwd)]
    recv = [[torch.full((n,), 0x7A5A, dtype=torch.int16, device="cuda").view(torch.bfloat16)
             for _ in range(R)] for _ in rounds]
    hc.set_config(copy_path="engines", sdma_engines=16, proxy_slice_bytes=4 << 20)
    for i, (mb, peers) in enumerate(rounds):
        hc.sendrecv(send[mb], recv[i], peers)
    torch.cuda.synchronize()
    for i, (mb, peers) in enumerate(rounds):
        ref = [np.full(n, 0x7A5A, np.uint16) for _ in range(R)]
        oracle.sendrecv(xs[mb], ref, peers, n, hc.BF16)
        for r in range(R):
            assert_bitwise(from_dev(recv[i][r], hc.BF16), ref[r], f"round {i} rank {r}")
