"""Large copies on the engine proxy, bit for bit against the definitions
the oracle implements (all-gather: the shards concatenated in rank order;
all-to-all: block d of rank s lands at block s of rank d): chains of
dependent 50.3 MB copies, one copy of 16 MiB plus a ragged tail, and an
all-to-all of 64 MiB blocks."""
import pytest
import torch

import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import assert_bitwise, from_dev, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _defaults():
    saved = hc.get_config()
    if hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    yield
    hc.set_config(**saved)


def test_ring_allgather_chains_of_large_copies():
    """The ring all-gather forwards every shard hop by hop: 8 chains of 7
    dependent copies of 50.3 MB (one GPT-6.7B block's shards).  A hop that
    started before the previous one finished would forward stale bytes."""
    hc.set_config(copy_path="engines", allgather_direct=0)
    R = 8
    x = W.ag_parameters(R)
    n = x[0].size
    out = [torch.zeros(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    hc.allgather([to_dev(a, hc.BF16) for a in x], out)
    torch.cuda.synchronize()
    # The oracle's all-gather is the concatenation of the shards in rank
    # order; compared block by block to keep host memory small.
    for r in range(R):
        got = from_dev(out[r], hc.BF16)
        for s in range(R):
            assert_bitwise(got[s * n:(s + 1) * n], x[s], f"rank {r} block {s}")


@pytest.mark.parametrize("extra", [0, 5, 2047])
def test_large_ragged_copy(extra):
    """One message of 16 MiB plus a few bf16 elements, left whole by the
    planner (chunk_bytes larger than the message): one engine copy whose
    length is not a multiple of 4 KiB."""
    hc.set_config(copy_path="engines", chunk_bytes=1 << 30)
    n = (8 << 20) + extra
    a = W.random_bits(631, 0, n, 2)
    src = to_dev(a, hc.BF16)
    dst = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
    hc.sendrecv([src, src], [dst, dst], [1, -1])
    torch.cuda.synchronize()
    assert hc.last_stats()["copy_ops"] == 1
    assert_bitwise(from_dev(dst, hc.BF16), a, f"16 MiB + {extra} elements")


def test_alltoall_of_power_of_two_blocks():
    """All-to-all over R = 8 with 64 MiB blocks (the layout of the size
    sweep's 512 MiB point): every block must land where the definition puts
    it."""
    hc.set_config(copy_path="engines")
    R, blk = 8, 32 << 20                     # bf16 elements: 64 MiB blocks
    send = [torch.empty(R * blk, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    for s in range(R):
        send[s].view(torch.int16).copy_(torch.arange(R * blk, device="cuda", dtype=torch.int32)
                                        .remainder(32749).add(s * 1000).to(torch.int16))
    recv = [torch.empty(R * blk, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    hc.alltoall(send, recv)
    torch.cuda.synchronize()
    for d in range(R):
        for s in range(R):
            got = recv[d][s * blk:(s + 1) * blk].view(torch.int16)
            want = send[s][d * blk:(d + 1) * blk].view(torch.int16)
            assert torch.equal(got, want), (d, s)
