"""GPU parity at the edges: the largest rank count the ABI allows, and a
reduce-scatter whose per-rank input exceeds 2^32 elements (every byte offset
past 4 GiB), checked on sampled outputs that the oracle recomputes one by
one."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import ES, NAME, assert_bitwise, from_dev, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _defaults():
    saved = hc.get_config()
    yield
    hc.set_config(**saved)


@pytest.mark.parametrize("path", ["auto", "hip", "kernel"])
@pytest.mark.parametrize("algo", ["ring", "direct"])
def test_max_ranks(path, algo):
    R = 64
    hc.set_config(copy_path=path, reduce_algo=algo)
    for dt in (hc.BF16, hc.FP32):
        n = 97
        x = [W.random_values(NAME[dt], 201, r, R * n) for r in range(R)]
        ref = oracle.reduce_scatter_new(x, dt)
        got = hc.reduce_scatter([to_dev(a, dt) for a in x])
        torch.cuda.synchronize()
        for r in range(0, R, 7):
            assert_bitwise(from_dev(got[r], dt), ref[r], f"RS R=64 r={r}")
        x = [W.random_values(NAME[dt], 202, r, 1000) for r in range(R)]
        ref = oracle.allreduce_new(x, dt)
        send = [to_dev(a, dt) for a in x]
        recv = [torch.empty_like(t) for t in send]
        hc.allreduce(send, recv)
        torch.cuda.synchronize()
        for r in range(0, R, 9):
            assert_bitwise(from_dev(recv[r], dt), ref[r], f"AR R=64 r={r}")
    shards = [W.random_bits(203, r, 33, 2) for r in range(R)]
    ref = oracle.allgather_new(shards, hc.BF16)
    got = hc.allgather([to_dev(a, hc.BF16) for a in shards])
    torch.cuda.synchronize()
    for r in (0, 31, 63):
        assert_bitwise(from_dev(got[r], hc.BF16), ref[r], f"AG R=64 r={r}")


@pytest.mark.parametrize("algo", ["ring", "direct"])
def test_reduce_scatter_beyond_4g_elements(algo):
    """R=2, recvcount 2^31 + 11 bf16 elements: each send buffer holds
    2^32 + 22 elements (8 GiB), so offsets pass both 2^31 and 2^32
    elements.  Output element i of rank r is the fold of x[k][r*n + i] over
    the ranks starting at r+1; the oracle recomputes each sample as a
    one-element reduce-scatter of exactly those inputs."""
    hc.set_config(reduce_algo=algo)
    R, n = 2, (1 << 31) + 11
    send = [W.device_normal_bf16(204, r, R * n) for r in range(R)]
    out = hc.reduce_scatter(send)
    torch.cuda.synchronize()
    rng = np.random.default_rng(205)
    idx = sorted(set([0, 1, n - 1, n - 2, (1 << 31) - 1, 1 << 30] +
                     list(rng.integers(0, n, 60))))
    idx_t = torch.tensor(idx, device="cuda", dtype=torch.int64)
    for r in range(R):
        # contributions of every rank to rank r's block at the sampled i
        contrib = [from_dev(send[k][r * n + idx_t], hc.BF16) for k in range(R)]
        got = from_dev(out[r][idx_t], hc.BF16)
        for t, i in enumerate(idx):
            tiny = []
            for k in range(R):
                a = np.zeros(R, np.uint16)
                a[r] = contrib[k][t]
                tiny.append(a)
            ref = oracle.reduce_scatter_new(tiny, hc.BF16)
            assert got[t] == ref[r][0], (algo, r, i, hex(got[t]), hex(ref[r][0]))
    del send, out
    torch.cuda.empty_cache()
