"""Randomised plan replay (CPU): random collectives, dtypes, rank counts up to
64, ragged counts and every planner option, each replayed step by step and
compared with the oracle bit for bit.  Complements the fixed grids of
test_plan_replay.py with shapes nobody chose by hand."""
import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import paper_2609_34334_amd as hc
import workloads as W
from test_plan_replay import ES, NAME, as_bytes, replay

OPS = [hc.OP_ALLREDUCE, hc.OP_REDUCE_SCATTER, hc.OP_ALLGATHER, hc.OP_ALLTOALL]

configs = st.fixed_dictionaries({
    "allreduce_chunk_groups": st.sampled_from([1, 2, 3, 5]),
    "chunk_bytes": st.sampled_from([0, 4096, 12288]),
    "ring_group_bytes": st.sampled_from([0, 1000, 4096, 65536]),
    "reduce_algo": st.sampled_from(["ring", "direct"]),
    "allgather_direct": st.sampled_from([0, 1]),
    "fused_hops": st.sampled_from([1, 2, 3, 64]),
    "a2a_schedule": st.sampled_from([0, 1, 2]),
    "bf16_partials": st.sampled_from([0, 1]),
})


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow],
          derandomize=True)
@given(op=st.sampled_from(OPS), dt=st.sampled_from([hc.INT32, hc.FP32, hc.BF16]),
       R=st.one_of(st.integers(1, 9), st.sampled_from([13, 16, 31, 64])),
       n=st.integers(1, 700), seed=st.integers(0, 10_000), cfg=configs)
def test_random_plans_replay_to_oracle(op, dt, R, n, seed, cfg):
    if R >= 16:
        n = min(n, 97)                     # keep R * R * n small
    es = ES[dt]
    hops = dt == hc.BF16 and cfg["bf16_partials"] == 1
    with hc.config(**cfg):
        plan = hc.plan_json(op, n, dt, R)
    if op == hc.OP_ALLREDUCE:
        x = [W.random_values(NAME[dt], seed, r, n) for r in range(R)]
        ref = oracle.allreduce_bf16_hops_new(x) if hops else oracle.allreduce_new(x, dt)
        recv = [np.zeros(n * es, np.uint8) for _ in range(R)]
    elif op == hc.OP_REDUCE_SCATTER:
        x = [W.random_values(NAME[dt], seed, r, R * n) for r in range(R)]
        ref = oracle.reduce_scatter_bf16_hops_new(x) if hops else oracle.reduce_scatter_new(x, dt)
        recv = [np.zeros(n * es, np.uint8) for _ in range(R)]
    elif op == hc.OP_ALLGATHER:
        x = [W.random_bits(seed, r, n, es) for r in range(R)]
        ref = oracle.allgather_new(x, dt)
        recv = [np.zeros(R * n * es, np.uint8) for _ in range(R)]
    else:
        x = [W.random_bits(seed, r, R * n, es) for r in range(R)]
        ref = [np.zeros_like(a) for a in x]
        oracle.alltoall(x, ref, n, dt)
        recv = [np.zeros(R * n * es, np.uint8) for _ in range(R)]
    replay(plan, as_bytes(x), recv)
    for r in range(R):
        assert np.array_equal(recv[r], as_bytes([ref[r]])[0]), (op, NAME[dt], R, n, cfg, r)
