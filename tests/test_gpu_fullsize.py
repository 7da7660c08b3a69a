"""Parity at the benchmark workloads' full sizes, in the launch
configuration bench.py times (the library defaults), against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import assert_bitwise, from_dev, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _defaults():
    saved = hc.get_config()
    yield
    hc.set_config(**saved)


@pytest.mark.parametrize("algo", ["ring", "direct", "fused2", "fused4", "fused7"])
def test_reduce_scatter_gradient_bucket(algo):
    """bf16, R=8, 25,165,824 elements per rank: every output element; the
    ring also with 2, 4 and 7 hops fused per launch."""
    if algo.startswith("fused"):
        hc.set_config(reduce_algo="ring", fused_hops=int(algo[5:]))
    else:
        hc.set_config(reduce_algo=algo)
    R, n_in = 8, 25_165_824
    x = W.rs_gradients(R, n_in)
    ref = oracle.reduce_scatter_new(x, hc.BF16)
    out = hc.reduce_scatter([to_dev(a, hc.BF16) for a in x])
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(out[r], hc.BF16), ref[r], f"{algo} rank {r}")


@pytest.mark.parametrize("path", ["hip", "engines", "kernel"])
@pytest.mark.parametrize("algo", ["ring", "direct"])
def test_allreduce_fp32_R4(path, algo):
    hc.set_config(copy_path=path, reduce_algo=algo)
    x = W.allreduce_fp32(4, 1_048_576)
    ref = oracle.allreduce_new(x, hc.FP32)
    send = [to_dev(a, hc.FP32) for a in x]
    recv = [torch.empty_like(t) for t in send]
    hc.allreduce(send, recv)
    torch.cuda.synchronize()
    for r in range(4):
        assert_bitwise(from_dev(recv[r], hc.FP32), ref[r], f"rank {r}")


@pytest.mark.parametrize("path", ["hip", "engines", "kernel"])
def test_allgather_fsdp_block(path):
    """201,326,592 bf16 parameters over R=8: each rank's output is compared
    with the concatenation of the shards (the oracle's definition)."""
    hc.set_config(copy_path=path)
    R = 8
    x = W.ag_parameters(R)
    n = x[0].size
    out = hc.allgather([to_dev(a, hc.BF16) for a in x])
    torch.cuda.synchronize()
    for r in range(R):
        got = from_dev(out[r], hc.BF16)
        for s in range(R):
            assert np.array_equal(got[s * n:(s + 1) * n], x[s]), (r, s)


@pytest.mark.parametrize("path", ["hip", "engines", "kernel"])
def test_pp_activation_round(path):
    hc.set_config(copy_path=path)
    R = 8
    x = W.p2p_activations(R)
    n = x[0].size
    for peers in ([r + 1 if r + 1 < R else -1 for r in range(R)], [r - 1 for r in range(R)]):
        ref = [np.zeros(n, np.uint16) for _ in range(R)]
        oracle.sendrecv(x, ref, peers, n, hc.BF16)
        recv = [torch.zeros(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
        hc.sendrecv([to_dev(a, hc.BF16) for a in x], recv, peers)
        torch.cuda.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(recv[r], hc.BF16), ref[r], f"{peers} rank {r}")


@pytest.mark.parametrize("path,sched", [("hip", 0), ("engines", 0), ("engines", 1), ("kernel", 2)])
def test_alltoallv_ep_dispatch(path, sched):
    """EP dispatch at full size; also copied stage by stage as the
    collective scheduler decomposes its traffic matrix."""
    hc.set_config(copy_path=path, a2a_schedule=sched)
    R = 8
    send, counts, sd, rd, rsz = W.a2a_tokens(R)
    ref = [np.zeros(s, np.uint16) for s in rsz]
    oracle.alltoallv(send, counts, sd, ref, rd, hc.BF16)
    recv = [torch.zeros(s, dtype=torch.bfloat16, device="cuda") for s in rsz]
    hc.alltoallv([to_dev(a, hc.BF16) for a in send], counts, sd, recv, rd)
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(recv[r], hc.BF16), ref[r], f"rank {r}")
