"""Plan replay on the CPU: the planner's schedule, executed step by step with
numpy, must equal the oracle bit for bit.

This checks step order, phases, chunk offsets, workspace placement, copy
chains and chunking without a GPU.  The replayer is scaffolding for the HIP
path's schedules and shares nothing with the oracle: it does plain numpy
float32 / uint32 adds and torch's fp32 -> bf16 rounding.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34334_amd as hc
import workloads as W

NP = {hc.INT32: np.int32, hc.FP32: np.float32, hc.BF16: np.uint16}
ES = {hc.INT32: 4, hc.FP32: 4, hc.BF16: 2, hc.UINT8: 1}
NAME = {hc.INT32: "int32", hc.FP32: "fp32", hc.BF16: "bf16"}


def widen(raw, dt, is_acc):
    if dt == hc.INT32:
        return raw.view(np.uint32)
    if dt == hc.FP32 or is_acc:
        return raw.view(np.float32)
    return (raw.view(np.uint16).astype(np.uint32) << 16).view(np.float32)


def narrow(vals, dt, is_acc):
    if dt == hc.INT32:
        return vals.astype(np.uint32).view(np.uint8)
    if dt == hc.FP32 or is_acc:
        return vals.astype(np.float32).view(np.uint8)
    t = torch.from_numpy(np.ascontiguousarray(vals, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint8)


def replay(plan, send, recv):
    dt = plan["dtype"]
    es = ES[dt]
    ws = np.zeros(plan["ws_bytes"], np.uint8)
    bufs = {"send": send, "recv": recv, "ws": [ws]}

    def region(ref, nbytes):
        kind, rank, off = ref
        arr = bufs[kind][0 if kind == "ws" else rank]
        assert off + nbytes <= arr.size, (ref, nbytes, arr.size)
        return arr[off:off + nbytes]

    # bf16 partials: the partials are bf16 like the operands, and every
    # addition's result is rounded (narrow then widen) before the next.
    bf16p = bool(plan["bf16_partials"])

    def rounded(v):
        if not bf16p:
            return v
        return widen(narrow(v, dt, False).view(np.uint16), dt, False)

    for st in plan["reduce_steps"]:
        ph = st["phase"]
        in0_acc = ph in ("middle", "last") and not bf16p
        out_acc = ph in ("first", "middle") and not bf16p
        for g in st["segs"]:
            n = g["n"]
            r = widen(region(g["in0"], n * (4 if in0_acc else es)).copy(), dt, in0_acc)
            # a fused step adds in1 and then its further contributions in order
            for ref in [g["in1"]] + g["more"]:
                b = widen(region(ref, n * es).copy(), dt, False)
                if dt == hc.INT32:
                    r = (r.astype(np.uint64) + b.astype(np.uint64)) & 0xFFFFFFFF
                else:
                    r = rounded(r + b)
            region(g["out"], n * (4 if out_acc else es))[:] = narrow(r, dt, out_acc)
    f = plan["fold"]
    if f is not None:
        R = plan["R"]
        c, total = f["c"], f["total"]
        for j in range(R):
            e0 = j * c
            if e0 >= total:
                continue
            n = min(c, total - e0)
            acc = None
            for k in range(1, R + 1):
                x = widen(send[(j + k) % R][e0 * es:(e0 + n) * es].copy(), dt, False)
                if acc is None:
                    acc = x.astype(np.uint64) if dt == hc.INT32 else x
                elif dt == hc.INT32:
                    acc = (acc + x.astype(np.uint64)) & 0xFFFFFFFF
                else:
                    acc = rounded(acc + x)
            y = narrow(acc, dt, False)
            oe = 0 if f["out_at_chunk"] else e0
            outs = range(R) if f["write_all"] else [j]
            for r in outs:
                recv[r][oe * es:(oe + n) * es] = y
    for cp in plan["copies"]:
        region(cp["dst"], cp["bytes"])[:] = region(cp["src"], cp["bytes"]).copy()


def as_bytes(arrays):
    return [np.ascontiguousarray(a).view(np.uint8).copy() for a in arrays]


CONFIGS = [
    dict(),
    dict(allreduce_chunk_groups=3),
    dict(chunk_bytes=4096),
    dict(allgather_direct=1, chunk_bytes=4096, allreduce_chunk_groups=2),
    dict(reduce_algo="direct"),
    dict(ring_group_bytes=1000),                      # many cache groups, ragged last group
    dict(ring_group_bytes=4096, allreduce_chunk_groups=2, chunk_bytes=4096),
    dict(fused_hops=2),                               # fused ring hops, a one-hop remainder at R=4, 8
    dict(fused_hops=3, ring_group_bytes=1000, allreduce_chunk_groups=2),
    dict(fused_hops=64),                              # every hop in one launch (capped at 8 per launch)
    dict(reduce_algo="auto"),
    dict(a2a_schedule=1),                             # all-to-all by the scheduler's stages
    dict(a2a_schedule=2, chunk_bytes=4096),
]


@pytest.fixture(params=range(len(CONFIGS)), ids=lambda i: "cfg%d" % i)
def cfg(request):
    with hc.config(**CONFIGS[request.param]):
        yield CONFIGS[request.param]


@pytest.mark.parametrize("dt", [hc.INT32, hc.FP32, hc.BF16], ids=lambda d: NAME[d])
@pytest.mark.parametrize("R", [1, 2, 3, 4, 5, 8])
def test_reduction_plans_replay_to_oracle(cfg, dt, R):
    for n in [1, 7, R * 5 + 3, 64, 3001]:
        seed = 500 + R * 7 + n
        # all-reduce of n elements
        x = [W.random_values(NAME[dt], seed, r, n) for r in range(R)]
        ref = oracle.allreduce_new(x, dt)
        recv = [np.zeros(n * ES[dt], np.uint8) for _ in range(R)]
        replay(hc.plan_json(hc.OP_ALLREDUCE, n, dt, R), as_bytes(x), recv)
        for r in range(R):
            assert np.array_equal(recv[r], as_bytes([ref[r]])[0]), ("allreduce", n, r)
        # reduce-scatter with recvcount n
        x = [W.random_values(NAME[dt], seed + 1, r, R * n) for r in range(R)]
        ref = oracle.reduce_scatter_new(x, dt)
        recv = [np.zeros(n * ES[dt], np.uint8) for _ in range(R)]
        replay(hc.plan_json(hc.OP_REDUCE_SCATTER, n, dt, R), as_bytes(x), recv)
        for r in range(R):
            assert np.array_equal(recv[r], as_bytes([ref[r]])[0]), ("reduce_scatter", n, r)


@pytest.mark.parametrize("R", [1, 2, 3, 8])
def test_copy_plans_replay_to_oracle(cfg, R):
    for dt in [hc.FP32, hc.BF16, hc.UINT8]:
        for n in [1, 5, 3001]:
            x = [W.random_bits(600 + n, r, n, ES[dt]) for r in range(R)]
            # all-gather
            ref = oracle.allgather_new(x, dt)
            recv = [np.zeros(R * n * ES[dt], np.uint8) for _ in range(R)]
            replay(hc.plan_json(hc.OP_ALLGATHER, n, dt, R), as_bytes(x), recv)
            for r in range(R):
                assert np.array_equal(recv[r], as_bytes([ref[r]])[0])
            # all-to-all with blocks of n
            xs = [W.random_bits(700 + n, r, R * n, ES[dt]) for r in range(R)]
            ref = [np.zeros_like(a) for a in xs]
            oracle.alltoall(xs, ref, n, dt)
            recv = [np.zeros(R * n * ES[dt], np.uint8) for _ in range(R)]
            replay(hc.plan_json(hc.OP_ALLTOALL, n, dt, R), as_bytes(xs), recv)
            for r in range(R):
                assert np.array_equal(recv[r], as_bytes([ref[r]])[0])
            # send/recv pipeline r -> r+1
            peers = [r + 1 if r + 1 < R else -1 for r in range(R)]
            ref = [np.zeros_like(a) for a in x]
            oracle.sendrecv(x, ref, peers, n, dt)
            recv = [np.zeros(n * ES[dt], np.uint8) for _ in range(R)]
            replay(hc.plan_json(hc.OP_SENDRECV, n, dt, R), as_bytes(x), recv)
            for r in range(R):
                assert np.array_equal(recv[r], as_bytes([ref[r]])[0])


@pytest.mark.parametrize("op", [hc.OP_ALLGATHER, hc.OP_ALLTOALL, hc.OP_SENDRECV, hc.OP_ALLREDUCE])
def test_copies_cover_each_destination_byte_once(cfg, op):
    """Completeness (every flow of the traffic matrix is realised) and no
    destination byte is written twice."""
    R, n, dt = 8, 3001, hc.BF16
    plan = hc.plan_json(op, n, dt, R)
    written = {}
    for cp in plan["copies"]:
        kind, rank, off = cp["dst"]
        assert kind == "recv"
        cov = written.setdefault(rank, np.zeros(R * n * 2 + 1, np.int32))
        cov[off:off + cp["bytes"]] += 1
    for rank, cov in written.items():
        assert cov.max() <= 1, rank
    total = sum(int(c.sum()) for c in written.values())
    expect = {hc.OP_ALLGATHER: R * R * n * 2, hc.OP_ALLTOALL: R * R * n * 2,
              hc.OP_SENDRECV: (R - 1) * n * 2}
    if op == hc.OP_ALLREDUCE:
        # the ring's gather phase writes every rank's copy of every chunk but
        # the owner's; the direct fold writes all outputs itself
        assert total == (0 if plan["fold"] else (R - 1) * n * 2)
    else:
        assert total == expect[op]


def test_chains_are_ordered_by_level():
    with hc.config(chunk_bytes=4096):
        plan = hc.plan_json(hc.OP_ALLGATHER, 5000, hc.BF16, 8)
    last = {}
    for cp in plan["copies"]:
        ch = cp["chain"]
        assert cp["level"] >= last.get(ch, -1)
        last[ch] = cp["level"]


def test_algorithmic_bytes():
    # reduce-scatter of bf16 with fp32 partials: 8 + 10*(R-3) + 8 bytes per
    # element of each of the R chunks, i.e. 66 n bytes at R = 8
    n = 3_145_728
    plan = hc.plan_json(hc.OP_REDUCE_SCATTER, n, hc.BF16, 8)
    assert plan["hbm_bytes"] == 8 * n * (8 + 5 * 10 + 8)
    assert plan["ws_bytes"] == 8 * n * 4


def test_cache_groups_bound_partials_and_keep_bytes():
    """Ring groups: each group's fp32 partials stay within the budget, the
    algorithmic bytes do not change, and every group runs its R-1 steps in
    order before the next group starts."""
    R, n = 8, 3_145_728
    with hc.config(ring_group_bytes=(1 << 64) - 1):
        one = hc.plan_json(hc.OP_REDUCE_SCATTER, n, hc.BF16, R)
    with hc.config(ring_group_bytes=16 << 20):
        p = hc.plan_json(hc.OP_REDUCE_SCATTER, n, hc.BF16, R)
    assert one["ngroups"] == 1 and p["ngroups"] == 6            # 96 MiB of partials / 16 MiB
    assert p["hbm_bytes"] == one["hbm_bytes"]
    steps = p["reduce_steps"]
    assert [s["group"] for s in steps] == [g for g in range(6) for _ in range(R - 1)]
    for s in steps:
        assert sum(seg["n"] for seg in s["segs"]) * 4 <= 16 << 20
    with hc.config(ring_group_bytes=16 << 20):
        ar = hc.plan_json(hc.OP_ALLREDUCE, R * n, hc.BF16, R)
    assert ar["ngroups"] == 6


def test_automatic_allreduce_groups():
    """allreduce_chunk_groups 0 (the default) plans two groups once each
    rank holds at least 32 MiB and one below, on an engine budget of 8 or
    more; on the automatic budget of 4 it plans one (plan dumps assume the
    engine path); an explicit count wins."""
    assert hc.get_config()["allreduce_chunk_groups"] == 0
    R = 8
    at_default = hc.plan_json(hc.OP_ALLREDUCE, (32 << 20) // 2, hc.BF16, R)
    assert at_default["ngroups"] == 1
    for engines in (8, 16):
        with hc.config(sdma_engines=engines):
            below = hc.plan_json(hc.OP_ALLREDUCE, (16 << 20) // 2, hc.BF16, R)
            at = hc.plan_json(hc.OP_ALLREDUCE, (32 << 20) // 2, hc.BF16, R)
        assert below["ngroups"] == 1 and at["ngroups"] == 2
        assert [s["group"] for s in at["reduce_steps"]] == [g for g in range(2) for _ in range(R - 1)]
        assert {c["group"] for c in at["copies"]} == {0, 1}
    with hc.config(sdma_engines=7):
        assert hc.plan_json(hc.OP_ALLREDUCE, (32 << 20) // 2, hc.BF16, R)["ngroups"] == 1
    with hc.config(allreduce_chunk_groups=1, sdma_engines=16):
        assert hc.plan_json(hc.OP_ALLREDUCE, (32 << 20) // 2, hc.BF16, R)["ngroups"] == 1
    with hc.config(allreduce_chunk_groups=2):
        assert hc.plan_json(hc.OP_ALLREDUCE, (32 << 20) // 2, hc.BF16, R)["ngroups"] == 2


@pytest.mark.parametrize("hops,per_element,launches", [(1, 66, 7), (2, 42, 4), (4, 26, 2), (7, 18, 1)])
def test_fused_hops_bytes_and_launches(hops, per_element, launches):
    """bf16 at R = 8, bytes per element of each chunk, worked out by hand:
    one hop per launch 8 + 5*10 + 8 = 66; two, hops [0,2) [2,4) [4,6) [6,7):
    (3*2 + 4) + 2*(4 + 2*2 + 4) + (4 + 2 + 2) = 42; four, [0,4) [4,7):
    (5*2 + 4) + (4 + 3*2 + 2) = 26; seven: 8*2 + 2 = 18, the direct fold's
    bytes, with no partial in memory at all."""
    n = 3_145_728
    with hc.config(fused_hops=hops):
        plan = hc.plan_json(hc.OP_REDUCE_SCATTER, n, hc.BF16, 8)
    assert plan["hbm_bytes"] == 8 * n * per_element
    assert len(plan["reduce_steps"]) == launches
    assert [s["hops"] for s in plan["reduce_steps"]] == [min(hops, 7 - k * hops) for k in range(launches)]
    assert plan["ws_bytes"] == (0 if hops >= 7 else 8 * n * 4)


@pytest.mark.parametrize("R", [2, 3, 5, 8])
def test_alltoall_stages_are_matchings_and_complete(R):
    """With a2a_schedule the all-to-all's copies carry the stages of the
    collective scheduler's decomposition: inside each stage every rank sends
    at most one piece and receives at most one (the per-stage degree bound,
    Eq. 8, here over the single memory domain), except the last stage of
    copies to self; stages are numbered in order; and every byte of every
    flow is copied exactly once (completeness, Eq. 7)."""
    n, dt = 1001, hc.BF16
    with hc.config(a2a_schedule=1):
        plan = hc.plan_json(hc.OP_ALLTOALL, n, dt, R)
    stages = sorted({c["stage"] for c in plan["copies"]})
    assert stages == list(range(len(stages)))
    for st in stages[:-1]:
        cps = [c for c in plan["copies"] if c["stage"] == st]
        srcs = [c["src"][1] for c in cps]
        dsts = [c["dst"][1] for c in cps]
        assert len(set(srcs)) == len(srcs) and len(set(dsts)) == len(dsts), st
        assert all(a != b for a, b in zip(srcs, dsts))
    last = [c for c in plan["copies"] if c["stage"] == stages[-1]]
    assert all(c["src"][1] == c["dst"][1] for c in last) and len(last) == R
    cov = {}
    for c in plan["copies"]:
        arr = cov.setdefault(c["dst"][1], np.zeros(R * n * 2, np.int32))
        arr[c["dst"][2]:c["dst"][2] + c["bytes"]] += 1
    assert all((a == 1).all() for a in cov.values()) and len(cov) == R


BF16P_CONFIGS = [
    dict(bf16_partials=1, reduce_algo="ring"),
    dict(bf16_partials=1, reduce_algo="direct"),
    dict(bf16_partials=1, reduce_algo="auto"),
    dict(bf16_partials=1, reduce_algo="ring", fused_hops=3, allreduce_chunk_groups=2),
    dict(bf16_partials=1, reduce_algo="ring", fused_hops=64),
    dict(bf16_partials=1, reduce_algo="ring", ring_group_bytes=1000, chunk_bytes=4096),
]


@pytest.mark.parametrize("ci", range(len(BF16P_CONFIGS)), ids=lambda i: "bf16p%d" % i)
@pytest.mark.parametrize("R", [1, 2, 3, 4, 5, 8])
def test_bf16_partial_plans_replay_to_oracle(ci, R):
    """With bf16 partials, bf16 plans replay to the oracle's sums whose every
    hop is rounded to bf16; fp32 and int32 plans are the usual ones."""
    with hc.config(**BF16P_CONFIGS[ci]):
        for n in [1, 7, R * 5 + 3, 3001]:
            seed = 900 + R * 7 + n
            x = [W.random_values("bf16", seed, r, n) for r in range(R)]
            plan = hc.plan_json(hc.OP_ALLREDUCE, n, hc.BF16, R)
            assert plan["bf16_partials"] == 1
            k = max(1, min(BF16P_CONFIGS[ci].get("fused_hops", 1), 8))
            assert all(st["hops"] <= k for st in plan["reduce_steps"])
            ref = oracle.allreduce_bf16_hops_new(x)
            recv = [np.zeros(n * 2, np.uint8) for _ in range(R)]
            replay(plan, as_bytes(x), recv)
            for r in range(R):
                assert np.array_equal(recv[r], as_bytes([ref[r]])[0]), ("allreduce", n, r)
            x = [W.random_values("bf16", seed + 1, r, R * n) for r in range(R)]
            ref = oracle.reduce_scatter_bf16_hops_new(x)
            recv = [np.zeros(n * 2, np.uint8) for _ in range(R)]
            replay(hc.plan_json(hc.OP_REDUCE_SCATTER, n, hc.BF16, R), as_bytes(x), recv)
            for r in range(R):
                assert np.array_equal(recv[r], as_bytes([ref[r]])[0]), ("reduce_scatter", n, r)
            for dt in (hc.FP32, hc.INT32):
                plan = hc.plan_json(hc.OP_REDUCE_SCATTER, n, dt, R)
                assert plan["bf16_partials"] == 0
                x = [W.random_values(NAME[dt], seed + 2, r, R * n) for r in range(R)]
                ref = oracle.reduce_scatter_new(x, dt)
                recv = [np.zeros(n * 4, np.uint8) for _ in range(R)]
                replay(plan, as_bytes(x), recv)
                for r in range(R):
                    assert np.array_equal(recv[r], as_bytes([ref[r]])[0]), (NAME[dt], n, r)


def test_bf16_partial_bytes():
    """bf16 ring reduce-scatter with bf16 partials moves 2+2+2 bytes per
    element on each of its R-1 hops and keeps R*n bf16 partials; with 4
    hops per launch, 2+2+3*2+2 and then 2+2+2*2+2 bytes in 2 launches."""
    R, n = 8, 1 << 20
    with hc.config(bf16_partials=1, reduce_algo="ring", ring_group_bytes=(1 << 64) - 1, fused_hops=1):
        plan = hc.plan_json(hc.OP_REDUCE_SCATTER, n, hc.BF16, R)
        assert plan["hbm_bytes"] == R * n * 6 * (R - 1)
        assert plan["ws_bytes"] == R * n * 2
        assert len(plan["reduce_steps"]) == R - 1
    with hc.config(bf16_partials=1, reduce_algo="ring", ring_group_bytes=(1 << 64) - 1, fused_hops=4):
        plan = hc.plan_json(hc.OP_REDUCE_SCATTER, n, hc.BF16, R)
        assert plan["hbm_bytes"] == R * n * (12 + 10)
        assert plan["ws_bytes"] == R * n * 2
        assert [st["hops"] for st in plan["reduce_steps"]] == [4, 3]
