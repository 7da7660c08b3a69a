"""Randomised GPU parity: 160 seeded cases (HOCCL_RANDOM_CASES=N for more),
each drawing a collective, dtype (bytes for a quarter of the copies), rank
count (up to 64), ragged count, misaligned buffer offset, copy path,
reduction algorithm, launch shape, group options, the engine proxy's issue
mode, the ring hops fused per launch and, for a quarter, bf16 partials
rounded at every hop, run through the C ABI and compared bit for bit with
the oracle (its per-hop-rounding sums where that mode meets bf16)."""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import NAME, TORCH, assert_bitwise, from_dev, to_dev

pytestmark = pytest.mark.gpu

NPDT = {hc.INT32: np.int32, hc.FP32: np.float32, hc.BF16: np.uint16, hc.UINT8: np.uint8}
ES = {hc.INT32: 4, hc.FP32: 4, hc.BF16: 2, hc.UINT8: 1}


def draw(i):
    g = np.random.default_rng([9001, i])
    R = int(g.choice([1, 2, 3, 4, 5, 7, 8, 13, 64], p=[.04, .12, .12, .14, .08, .1, .25, .08, .07]))
    n = int(g.integers(1, 40_000 if R <= 8 else 600))
    c = dict(
        op=str(g.choice(["allreduce", "reduce_scatter", "allgather", "sendrecv", "alltoall", "alltoallv"])),
        dt=[hc.INT32, hc.FP32, hc.BF16][int(g.integers(0, 3))], R=R, n=n,
        lead=int(g.choice([0, 1, 3, 8])),
        cfg=dict(copy_path=str(g.choice(["auto", "hip", "engines", "kernel"])),
                 reduce_algo=str(g.choice(["ring", "direct"])),
                 workgroups_per_step=int(g.choice([0, 0, 1, 7, 300])),
                 threads_per_workgroup=int(g.choice([64, 256, 256, 1024])),
                 ring_group_bytes=int(g.choice([0, 0, 4096])),
                 allreduce_chunk_groups=int(g.choice([0, 1, 3])),
                 allgather_direct=int(g.choice([0, 1])),
                 chunk_bytes=int(g.choice([0, 0, 8192])),
                 a2a_schedule=int(g.choice([0, 0, 1, 2]))),
        seed=int(g.integers(0, 1 << 30)))
    # Drawn last so the earlier fields keep their values: the engine
    # proxy's balanced issue (automatic, 64 KiB pieces) or all at once.
    c["cfg"]["proxy_slice_bytes"] = int(g.choice([0, 0, 64 << 10, (1 << 64) - 1]))
    # A quarter of the copy collectives move single bytes instead.
    if g.random() < 0.25 and c["op"] in ("allgather", "sendrecv", "alltoall", "alltoallv"):
        c["dt"] = hc.UINT8
    # A quarter of the cases keep bf16 partials in bf16 (rounded every hop).
    c["cfg"]["bf16_partials"] = int(g.random() < 0.25)
    # Ring hops folded per launch (the same bits as one per launch).
    c["cfg"]["fused_hops"] = int(g.choice([1, 1, 2, 3, 8]))
    return c


def dev_views(arrays, dt, lead):
    """Device copies of `arrays`, each a view starting `lead` elements into
    its own allocation (so most windows are not 16-byte aligned)."""
    out = []
    for a in arrays:
        full = torch.empty(lead + a.size + 8, dtype=TORCH[dt], device="cuda")
        v = full[lead:lead + a.size]
        v.copy_(to_dev(a, dt))
        out.append(v)
    return out


def empty_views(n, R, dt, lead):
    return [torch.empty(lead + n + 8, dtype=TORCH[dt], device="cuda")[lead:lead + n] for _ in range(R)]


# 160 cases by default; HOCCL_RANDOM_CASES=N runs N (the same first 160).
CASES = int(os.environ.get("HOCCL_RANDOM_CASES", "160"))


@pytest.mark.parametrize("i", range(CASES))
def test_random_case(i):
    c = draw(i)
    op, dt, R, n, lead, seed = c["op"], c["dt"], c["R"], c["n"], c["lead"], c["seed"]
    if c["cfg"]["copy_path"] == "engines" and hc.sdma_engine_count() == 0:
        c["cfg"]["copy_path"] = "hip"
    # stages run one after another are refused on the engine path (AUTO's)
    if c["cfg"]["a2a_schedule"] == 2 and c["cfg"]["copy_path"] in ("engines", "auto"):
        c["cfg"]["a2a_schedule"] = 1
    es = ES[dt]
    hops = dt == hc.BF16 and c["cfg"]["bf16_partials"] == 1
    with hc.config(**c["cfg"]):
        if op == "allreduce":
            x = [W.random_values(NAME[dt], seed, r, n) for r in range(R)]
            ref = oracle.allreduce_bf16_hops_new(x) if hops else oracle.allreduce_new(x, dt)
            out = hc.allreduce(dev_views(x, dt, lead), empty_views(n, R, dt, lead))
        elif op == "reduce_scatter":
            x = [W.random_values(NAME[dt], seed, r, R * n) for r in range(R)]
            ref = oracle.reduce_scatter_bf16_hops_new(x) if hops else oracle.reduce_scatter_new(x, dt)
            out = hc.reduce_scatter(dev_views(x, dt, lead), empty_views(n, R, dt, lead))
        elif op == "allgather":
            x = [W.random_bits(seed, r, n, es).view(NPDT[dt]) for r in range(R)]
            ref = oracle.allgather_new(x, dt)
            out = hc.allgather(dev_views(x, dt, lead), empty_views(R * n, R, dt, lead))
        elif op == "sendrecv":
            g = np.random.default_rng(seed)
            perm = list(g.permutation(R))
            peers = [int(perm[r]) if g.random() < 0.8 else -1 for r in range(R)]
            x = [W.random_bits(seed, r, n, es).view(NPDT[dt]) for r in range(R)]
            ref = [np.zeros(n, NPDT[dt]) for _ in range(R)]
            oracle.sendrecv(x, ref, peers, n, dt)
            out = empty_views(n, R, dt, lead)
            for o in out:
                o.zero_()
            hc.sendrecv(dev_views(x, dt, lead), out, peers)
        elif op == "alltoall":
            x = [W.random_bits(seed, r, R * n, es).view(NPDT[dt]) for r in range(R)]
            ref = [np.zeros(R * n, NPDT[dt]) for _ in range(R)]
            oracle.alltoall(x, ref, n, dt)
            out = hc.alltoall(dev_views(x, dt, lead), empty_views(R * n, R, dt, lead))
        else:
            g = np.random.default_rng(seed)
            C = g.integers(0, max(2, n // R), size=(R, R))
            sd = np.zeros((R, R), np.int64)
            rd = np.zeros((R, R), np.int64)
            for s in range(R):
                sd[s] = np.concatenate([[0], np.cumsum(C[s])[:-1]])
            for d in range(R):
                rd[:, d] = np.concatenate([[0], np.cumsum(C[:, d])[:-1]])
            ssz = [int(C[s].sum()) for s in range(R)]
            rsz = [int(C[:, d].sum()) for d in range(R)]
            x = [W.random_bits(seed, r, max(1, ssz[r]), es).view(NPDT[dt]) for r in range(R)]
            ref = [np.zeros(max(1, rsz[d]), NPDT[dt]) for d in range(R)]
            flat = lambda a: [int(v) for v in a.reshape(-1)]
            oracle.alltoallv(x, flat(C), flat(sd), ref, flat(rd), dt)
            out = [torch.zeros(lead + max(1, rsz[d]) + 8, dtype=TORCH[dt], device="cuda")[lead:lead + max(1, rsz[d])]
                   for d in range(R)]
            hc.alltoallv(dev_views(x, dt, lead), flat(C), flat(sd), out, flat(rd))
        torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(out[r], dt), ref[r], f"case {i} {c} rank {r}")
