"""One ring hop of one rank (hoccl_ring_hop) against the oracle.

Hops chained in ring order over chunk j -- first (x[j+1] + x[j+2]), middle
hops adding x[j+3] ... x[j-1], last adding x[j] -- must give rank j's block
of the oracle's reduce-scatter bit for bit; R = 2 is a single "only" hop.
The cases cover every dtype, a ragged count, views that start off a 16-byte
boundary (the kernel's scalar head, or a fully scalar segment when the
operands disagree in alignment), the partial updated in place, small
workgroup budgets and the headline chunk: 3,145,728 bf16 elements, one
rank's share of the GPT-6.7B gradient bucket."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import NAME, TORCH, assert_bitwise, from_dev, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _defaults():
    saved = hc.get_config()
    yield
    hc.set_config(**saved)


def placed(a, dt, shift):
    """`a` on the device, starting `shift` elements into its allocation."""
    t = to_dev(np.concatenate([np.zeros(shift, a.dtype), a]), dt)
    return t[shift:]


def chain(blocks, j, in_place, out_shift=0):
    """Rank j's reduced block from the R ranks' blocks j, hop by hop."""
    R = len(blocks)
    if R == 2:
        return hc.ring_hop(blocks[(j + 1) % R], blocks[j], hop="only")
    local = blocks[0]
    acc = torch.float32 if local.dtype == torch.bfloat16 else local.dtype

    def fresh(dtype):
        if not out_shift:
            return None
        return torch.empty(local.numel() + out_shift, dtype=dtype, device="cuda")[out_shift:]

    partial = hc.ring_hop(blocks[(j + 1) % R], blocks[(j + 2) % R], out=fresh(acc), hop="first")
    for k in range(3, R):
        partial = hc.ring_hop(partial, blocks[(j + k) % R], out=partial if in_place else fresh(acc),
                              hop="middle")
    return hc.ring_hop(partial, blocks[j], out=fresh(local.dtype), hop="last")


@pytest.mark.parametrize("layout", ["aligned", "head", "scalar"])
@pytest.mark.parametrize("R", [2, 3, 8])
@pytest.mark.parametrize("dt", [hc.INT32, hc.FP32, hc.BF16], ids=NAME.get)
def test_hops_in_ring_order_equal_the_oracle(dt, R, layout):
    n = 70_001
    x = [W.random_values(NAME[dt], 601 + R, r, R * n) for r in range(R)]
    j = R - 1
    ref = oracle.reduce_scatter_new(x, dt)[j]
    # "head": every operand one element off a 16-byte boundary, so the
    # kernel runs a scalar head and then its vector loop; "scalar": the
    # inputs and outputs disagree in alignment, so no vector loop is legal.
    shift = {"aligned": 0, "head": 1, "scalar": 1}[layout]
    out_shift = {"aligned": 0, "head": 1, "scalar": 3}[layout]
    blocks = [placed(x[r][j * n:(j + 1) * n], dt, shift) for r in range(R)]
    got = chain(blocks, j, in_place=layout == "aligned", out_shift=out_shift)
    torch.cuda.synchronize()
    assert got.dtype == TORCH[dt]
    assert_bitwise(from_dev(got, dt), ref, f"{NAME[dt]} R={R} {layout}")
    s = hc.last_stats()
    assert s["reduce_launches"] == 1 and s["copy_ops"] == 0


@pytest.mark.parametrize("wg", [1, 8, 0])
def test_budgets_give_the_same_bits(wg):
    hc.set_config(workgroups_per_step=wg)
    R, n = 8, 200_003
    x = [W.random_values("bf16", 611, r, R * n) for r in range(R)]
    j = 5
    ref = oracle.reduce_scatter_new(x, hc.BF16)[j]
    blocks = [to_dev(x[r][j * n:(j + 1) * n], hc.BF16) for r in range(R)]
    got = chain(blocks, j, in_place=True)
    torch.cuda.synchronize()
    assert_bitwise(from_dev(got, hc.BF16), ref, f"workgroups {wg}")
    if wg:
        assert hc.last_stats()["workgroups_per_step"] == wg


def test_headline_chunk():
    """Rank 3's hops over its 3,145,728-element block of the headline
    reduce-scatter input (bf16, normal(0, 1e-3))."""
    R, n = 8, 3_145_728
    x = W.rs_gradients(R, R * n)
    j = 3
    ref = oracle.reduce_scatter_new(x, hc.BF16)[j]
    blocks = [to_dev(x[r][j * n:(j + 1) * n], hc.BF16) for r in range(R)]
    got = chain(blocks, j, in_place=True)
    torch.cuda.synchronize()
    assert_bitwise(from_dev(got, hc.BF16), ref, "headline chunk")
    s = hc.last_stats()
    assert s["hbm_bytes_algorithmic"] == n * (4 + 2 + 2)        # the last hop: fp32 + bf16 in, bf16 out


def test_hop_in_a_graph_replays_the_same_bits():
    """A captured middle hop (no allocation, no copies) replays like the
    eager call; the graph is replayed three times with eager work between."""
    n = 100_000
    part = to_dev(W.random_values("fp32", 621, 0, n), hc.FP32)
    loc = to_dev(W.random_values("bf16", 621, 1, n), hc.BF16)
    eager = hc.ring_hop(part, loc, hop="middle")
    out = torch.empty_like(eager)
    s = torch.cuda.Stream()
    hc.ring_hop(part, loc, out=out, hop="middle", stream=s)      # state exists before capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        hc.ring_hop(part, loc, out=out, hop="middle", stream=s)
    for k in range(3):
        out.fill_(float(k + 7))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int32), eager.view(torch.int32)), f"replay {k}"
    del g
