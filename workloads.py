"""Seeded synthetic inputs for the HOCCL collectives.

This module holds only input generation: random draws, shapes and the
packing of all-to-all send buffers by destination.  It contains none of the
collectives' arithmetic, so both the CPU oracle and the HIP library can be fed
from it without sharing any of the method.

Every array is a numpy array on the host: int32, float32, or uint16 holding
bf16 bit patterns.  bf16 values are drawn in float64, cast to float32, then
rounded to bf16 (round to nearest even) by torch's CPU conversion.

Workload shapes (sizes of the paper's training traffic; GPT-6.7B has hidden
4096 and ffn 16384, sequence 2048, bf16; DeepSeek-V2-Lite has hidden 2048 and
64 routed experts with top-6 routing):

* ``allreduce_fp32``  -- R=4, 1,048,576 fp32 per rank, uniform[-1, 1), seed 1.
* ``rs_gradients``    -- DP gradient bucket, R=8, 25,165,824 bf16 per rank
  (6 x 4096 x 1024), normal(0, 1e-3), seed 2; recvcount 3,145,728.
* ``ag_parameters``   -- FSDP parameter all-gather of one transformer block:
  4h^2 + 2h*ffn = 201,326,592 bf16 split over R=8 (25,165,824 per rank),
  normal(0, 0.02), seed 3.
* ``p2p_activations`` -- PP activations [1, 2048, 4096] bf16 per message,
  R=8 stages, normal(0, 1), seed 4.
* ``a2a_tokens``      -- EP dispatch, R=8, 4096 tokens x hidden 2048 bf16 per
  rank, 64 experts (8 per rank), top-6 drawn uniformly without replacement,
  seed 5; a token goes once to every rank hosting at least one of its experts.
"""
import numpy as np
import torch

SEEDS = {"allreduce_fp32": 1, "rs_gradients": 2, "ag_parameters": 3,
         "p2p_activations": 4, "a2a_tokens": 5}


def to_bf16_bits(x):
    """float array -> uint16 bf16 bit patterns (round to nearest even)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_f32(h):
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def rng_for(seed, rank=0):
    return np.random.default_rng([seed, rank])


def uniform_f32(seed, rank, n, lo=-1.0, hi=1.0):
    return rng_for(seed, rank).uniform(lo, hi, n).astype(np.float32)


def normal_f32(seed, rank, n, std):
    return rng_for(seed, rank).normal(0.0, std, n).astype(np.float32)


def normal_bf16(seed, rank, n, std):
    return to_bf16_bits(normal_f32(seed, rank, n, std))


def random_int32(seed, rank, n, lo=-(2 ** 31), hi=2 ** 31):
    return rng_for(seed, rank).integers(lo, hi, n, dtype=np.int64).astype(np.int32)


def random_bits(seed, rank, n, itemsize):
    """Arbitrary bit patterns (NaN, Inf and subnormals included) for copies."""
    raw = rng_for(seed, rank).integers(0, 256, n * itemsize, dtype=np.uint8)
    return raw.view({1: np.uint8, 2: np.uint16, 4: np.uint32}[itemsize]).copy()


def random_values(dtype, seed, rank, n):
    """Finite random inputs for reductions: dtype in {'int32','fp32','bf16'}."""
    if dtype == "int32":
        return random_int32(seed, rank, n)
    if dtype == "fp32":
        return uniform_f32(seed, rank, n)
    if dtype == "bf16":
        return normal_bf16(seed, rank, n, 1.0)
    raise ValueError(dtype)


# ---- the benchmark workloads ----------------------------------------------

def allreduce_fp32(R=4, n=1_048_576):
    s = SEEDS["allreduce_fp32"]
    return [uniform_f32(s, r, n) for r in range(R)]


def rs_gradients(R=8, n=25_165_824):
    s = SEEDS["rs_gradients"]
    return [normal_bf16(s, r, n, 1e-3) for r in range(R)]


def ag_parameters(R=8, total=201_326_592):
    s = SEEDS["ag_parameters"]
    assert total % R == 0
    return [normal_bf16(s, r, total // R, 0.02) for r in range(R)]


def p2p_activations(R=8, shape=(1, 2048, 4096)):
    s = SEEDS["p2p_activations"]
    n = int(np.prod(shape))
    return [normal_bf16(s, r, n, 1.0) for r in range(R)]


def a2a_routing(R=8, tokens=4096, experts=64, topk=6, seed=None):
    """Top-k expert choice per token, uniform without replacement.
    Returns a list over source ranks of int arrays [tokens, topk]."""
    seed = SEEDS["a2a_tokens"] if seed is None else seed
    out = []
    for r in range(R):
        u = rng_for(seed, r).random((tokens, experts))
        out.append(np.argsort(u, axis=1)[:, :topk])
    return out


def a2a_plan(routing, R=8, experts=64, hidden=2048):
    """Token packing for all-to-all(v) with one copy per destination rank.

    Expert e lives on rank e // (experts // R).  Rank s sends token t to rank
    d when d hosts at least one of t's experts; tokens of a block are in
    ascending id order and the receive blocks are ordered by source rank.
    Returns (token_lists[s][d], counts[s*R+d], sdispls, rdispls) with counts
    and displacements in elements (tokens * hidden).
    """
    per_rank = experts // R
    token_lists = []
    for s in range(R):
        dest = routing[s] // per_rank
        hit = np.zeros((dest.shape[0], R), dtype=bool)
        hit[np.arange(dest.shape[0])[:, None], dest] = True
        token_lists.append([np.nonzero(hit[:, d])[0] for d in range(R)])
    counts = [len(token_lists[s][d]) * hidden for s in range(R) for d in range(R)]
    sdispls, rdispls = [0] * (R * R), [0] * (R * R)
    for s in range(R):
        off = 0
        for d in range(R):
            sdispls[s * R + d] = off
            off += counts[s * R + d]
    for d in range(R):
        off = 0
        for s in range(R):
            rdispls[s * R + d] = off
            off += counts[s * R + d]
    return token_lists, counts, sdispls, rdispls


def a2a_tokens(R=8, tokens=4096, hidden=2048, experts=64, topk=6):
    """Per-rank token activations [tokens, hidden] bf16 plus the packed send
    buffers and counts for the dispatch all-to-all(v)."""
    seed = SEEDS["a2a_tokens"]
    acts = [normal_bf16(seed + 100, r, tokens * hidden, 1.0).reshape(tokens, hidden)
            for r in range(R)]
    routing = a2a_routing(R, tokens, experts, topk, seed)
    token_lists, counts, sdispls, rdispls = a2a_plan(routing, R, experts, hidden)
    send = [np.ascontiguousarray(np.concatenate([acts[s][token_lists[s][d]]
                                                 for d in range(R)]).reshape(-1))
            for s in range(R)]
    recv_sizes = [sum(counts[s * R + d] for s in range(R)) for d in range(R)]
    return send, counts, sdispls, rdispls, recv_sizes


def device_normal_bf16(seed, rank, n, std=1.0):
    """Seeded normal(0, std) bf16 values generated on the current GPU (for
    inputs too large to draw on the host); returns a torch tensor."""
    g = torch.Generator(device="cuda")
    g.manual_seed(seed * 1_000_003 + rank)
    return (torch.randn(n, generator=g, device="cuda") * std).to(torch.bfloat16)

