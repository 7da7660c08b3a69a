"""GPU parity: every collective through the C ABI against the CPU oracle,
bit for bit, across dtypes, rank counts, ragged and misaligned sizes, in-place
forms, copy paths, reduction algorithms and launch shapes."""
import ctypes
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import (ES, NAME, TORCH, assert_bitwise, check_canaries, from_dev, padded,
                      to_dev)

pytestmark = pytest.mark.gpu

DTS = [hc.INT32, hc.FP32, hc.BF16]
# Stages run one after another on the SDMA engines (every copy of a stage
# waiting on all copies of the previous one through dependency signals)
# ended its first GPU run in a host segmentation fault whose cause is not
# established; the library refuses that form and its cases stay off.
SERIAL_STAGES_OFF = "a2a_schedule 2 on the SDMA engines is refused (host fault of unknown cause)"
PATHS = ["hip", "engines", "kernel"]


@pytest.fixture(autouse=True)
def _fresh_config():
    saved = hc.get_config()
    yield
    hc.set_config(**saved)


def run_ar(x, dt, lead=0):
    R, n = len(x), x[0].size
    outs = [padded(n, dt, lead) for _ in range(R)]
    send = [to_dev(a, dt) for a in x]
    hc.allreduce(send, [o[1] for o in outs])
    torch.cuda.synchronize()
    for full, _ in outs:
        check_canaries(full, lead, n, dt)
    return [from_dev(o[1], dt) for o in outs]


def run_rs(x, dt, lead=0):
    R = len(x)
    n = x[0].size // R
    outs = [padded(n, dt, lead) for _ in range(R)]
    send = [to_dev(a, dt) for a in x]
    hc.reduce_scatter(send, [o[1] for o in outs])
    torch.cuda.synchronize()
    for full, _ in outs:
        check_canaries(full, lead, n, dt)
    return [from_dev(o[1], dt) for o in outs]


# ---------------------------------------------------------------- reductions

@pytest.mark.parametrize("dt", [hc.INT32, hc.FP32, hc.BF16], ids=lambda d: NAME[d])
@pytest.mark.parametrize("R", [3, 8])
def test_ring_in_cache_groups(dt, R):
    """The ring run group by group (a tiny partial budget forces many groups
    with a ragged last one) gives the oracle's bits, for reduce-scatter and
    all-reduce, also with the all-reduce's own gather groups."""
    n = 30_011
    for budget, ar_groups in ((1 << 16, 1), (12_345, 3)):
        with hc.config(ring_group_bytes=budget, allreduce_chunk_groups=ar_groups):
            x = [W.random_values(NAME[dt], 700 + R, r, R * n) for r in range(R)]
            ref = oracle.reduce_scatter_new(x, dt)
            got = run_rs(x, dt, lead=3)
            for r in range(R):
                assert_bitwise(got[r], ref[r], f"grouped RS budget={budget} r={r}")
            xa = [W.random_values(NAME[dt], 710 + R, r, n) for r in range(R)]
            refa = oracle.allreduce_new(xa, dt)
            gota = run_ar(xa, dt, lead=5)
            for r in range(R):
                assert_bitwise(gota[r], refa[r], f"grouped AR budget={budget} r={r}")


@pytest.mark.parametrize("R", [2, 5, 8, 16])
def test_auto_reduction_folds_and_matches_the_oracle(R):
    """The default reduction (AUTO) folds directly on one GPU, reports that
    choice, and gives the oracle's bits for reduce-scatter and all-reduce,
    ragged, on the default copy path."""
    hc.set_config(reduce_algo="auto", copy_path="auto")
    for dt in DTS:
        n = R * 37 + 3
        x = [W.random_values(NAME[dt], 720 + R, r, R * n) for r in range(R)]
        got = run_rs(x, dt, lead=1)
        assert hc.last_stats()["reduce_algo_used"] == hc.REDUCE_DIRECT
        ref = oracle.reduce_scatter_new(x, dt)
        for r in range(R):
            assert_bitwise(got[r], ref[r], f"AUTO RS {NAME[dt]} R={R} r={r}")
        xa = [W.random_values(NAME[dt], 730 + R, r, 4099) for r in range(R)]
        gota = run_ar(xa, dt, lead=2)
        assert hc.last_stats()["reduce_algo_used"] == hc.REDUCE_DIRECT
        refa = oracle.allreduce_new(xa, dt)
        for r in range(R):
            assert_bitwise(gota[r], refa[r], f"AUTO AR {NAME[dt]} R={R} r={r}")


@pytest.mark.parametrize("hops", [2, 3, 4, 7, 64])
@pytest.mark.parametrize("dt", DTS, ids=lambda d: NAME[d])
@pytest.mark.parametrize("R", [3, 4, 8, 13])
def test_fused_ring_hops(hops, dt, R):
    """The ring with several hops folded per launch gives the oracle's bits
    (the ring's order), ragged, with misaligned outputs and with inputs
    misaligned against each other, and takes ceil((R-1)/k) launches of at
    most 8 hops each."""
    hc.set_config(reduce_algo="ring", fused_hops=hops, copy_path="hip")
    k = min(hops, 8)
    for n in [1, 7, R * 37 + 3, 65536 + 5]:
        x = [W.random_values(NAME[dt], 740 + R + hops, r, R * n) for r in range(R)]
        ref = oracle.reduce_scatter_new(x, dt)
        got = run_rs(x, dt, lead=3)
        assert hc.last_stats()["reduce_launches"] == -(-(R - 1) // k)
        for r in range(R):
            assert_bitwise(got[r], ref[r], f"fused RS k={hops} n={n} r={r}")
        xa = [W.random_values(NAME[dt], 750 + R + hops, r, n) for r in range(R)]
        refa = oracle.allreduce_new(xa, dt)
        gota = run_ar(xa, dt, lead=1)
        for r in range(R):
            assert_bitwise(gota[r], refa[r], f"fused AR k={hops} n={n} r={r}")
    # inputs at different offsets from 16-byte alignment (every operand of
    # a launch must then take the element-wise path)
    n = 4099
    x = [W.random_values(NAME[dt], 760 + R, r, R * n) for r in range(R)]
    ref = oracle.reduce_scatter_new(x, dt)
    bufs = [to_dev(np.concatenate([np.zeros(r % 3, x[r].dtype), x[r]]), dt) for r in range(R)]
    send = [bufs[r][r % 3:] for r in range(R)]
    out = hc.reduce_scatter(send)
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(out[r], dt), ref[r], f"fused RS misaligned inputs k={hops} r={r}")


@pytest.mark.parametrize("algo", ["ring", "direct"])
@pytest.mark.parametrize("dt", DTS, ids=lambda d: NAME[d])
@pytest.mark.parametrize("R", [1, 2, 3, 4, 8])
def test_allreduce_and_reduce_scatter(algo, dt, R):
    hc.set_config(reduce_algo=algo, copy_path="hip")
    for n in [1, 7, R * 37 + 3, 4099, 65536 + 5]:
        seed = 9000 + 13 * R + n
        x = [W.random_values(NAME[dt], seed, r, n) for r in range(R)]
        ref = oracle.allreduce_new(x, dt)
        got = run_ar(x, dt)
        for r in range(R):
            assert_bitwise(got[r], ref[r], f"allreduce R={R} n={n} r={r}")
        x = [W.random_values(NAME[dt], seed + 1, r, R * n) for r in range(R)]
        ref = oracle.reduce_scatter_new(x, dt)
        got = run_rs(x, dt)
        for r in range(R):
            assert_bitwise(got[r], ref[r], f"reduce_scatter R={R} n={n} r={r}")


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("groups", [1, 4])
def test_allreduce_copy_paths_and_groups(path, groups):
    hc.set_config(copy_path=path, allreduce_chunk_groups=groups)
    for dt in DTS:
        R, n = 4, 262_147
        x = [W.random_values(NAME[dt], 77, r, n) for r in range(R)]
        ref = oracle.allreduce_new(x, dt)
        got = run_ar(x, dt)
        for r in range(R):
            assert_bitwise(got[r], ref[r], f"{path} groups={groups} {NAME[dt]} r={r}")


@pytest.mark.parametrize("wg,threads", [(1, 64), (7, 256), (256, 256), (2048, 512), (4096, 1024)])
def test_launch_shapes(wg, threads):
    hc.set_config(workgroups_per_step=wg, threads_per_workgroup=threads)
    for algo in ["ring", "direct"]:
        hc.set_config(reduce_algo=algo)
        R, n = 8, 20_011
        x = [W.random_values("bf16", 31, r, R * n) for r in range(R)]
        ref = oracle.reduce_scatter_new(x, hc.BF16)
        got = run_rs(x, hc.BF16)
        for r in range(R):
            assert_bitwise(got[r], ref[r], f"wg={wg} threads={threads} {algo} r={r}")


@pytest.mark.parametrize("lead", [1, 3, 5])
def test_misaligned_buffers(lead):
    """Output windows that start off a 16-byte boundary take the scalar head
    and tail paths; inputs are sub-views at an element offset too."""
    for dt in DTS:
        R, n = 4, 10_007
        x = [W.random_values(NAME[dt], 41 + lead, r, n) for r in range(R)]
        ref = oracle.allreduce_new(x, dt)
        send_full = [to_dev(np.concatenate([np.zeros(lead, a.dtype), a]), dt) for a in x]
        send = [t[lead:] for t in send_full]
        outs = [padded(n, dt, lead) for _ in range(R)]
        hc.allreduce(send, [o[1] for o in outs])
        torch.cuda.synchronize()
        for r in range(R):
            check_canaries(outs[r][0], lead, n, dt)
            assert_bitwise(from_dev(outs[r][1], dt), ref[r], f"misaligned {NAME[dt]} r={r}")


def test_mixed_alignment_across_ranks():
    # rank buffers with different misalignments force the all-scalar path
    R, n, dt = 3, 5003, hc.FP32
    x = [W.random_values("fp32", 51, r, n) for r in range(R)]
    ref = oracle.allreduce_new(x, dt)
    send = []
    for r, a in enumerate(x):
        t = to_dev(np.concatenate([np.zeros(r, a.dtype), a]), dt)
        send.append(t[r:])
    recv = [torch.empty(n + 4, dtype=torch.float32, device="cuda")[r:r + n] for r in range(R)]
    hc.allreduce(send, recv)
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(recv[r], dt), ref[r], f"r={r}")


@pytest.mark.parametrize("dt", DTS, ids=lambda d: NAME[d])
def test_in_place_forms(dt):
    R, n = 4, 9001
    # all-reduce in place
    x = [W.random_values(NAME[dt], 61, r, n) for r in range(R)]
    ref = oracle.allreduce_new(x, dt)
    bufs = [to_dev(a, dt) for a in x]
    hc.allreduce(bufs, bufs)
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(bufs[r], dt), ref[r], f"AR in place r={r}")
    # reduce-scatter in place: recv[r] = send[r] + r*n
    x = [W.random_values(NAME[dt], 62, r, R * n) for r in range(R)]
    ref = oracle.reduce_scatter_new(x, dt)
    bufs = [to_dev(a, dt) for a in x]
    hc.reduce_scatter(bufs, [b[r * n:(r + 1) * n] for r, b in enumerate(bufs)])
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(bufs[r][r * n:(r + 1) * n], dt), ref[r], f"RS in place r={r}")
    # all-gather in place: send[r] = recv[r] + r*n
    x = [W.random_bits(63, r, n, ES[dt]).view(np.uint16 if dt == hc.BF16 else np.int32)
         for r in range(R)]
    if dt == hc.FP32:
        x = [a.view(np.float32) for a in x]
    ref = oracle.allgather_new(x, dt)
    recv = [torch.zeros(R * n, dtype=TORCH[dt], device="cuda") for _ in range(R)]
    for r in range(R):
        recv[r][r * n:(r + 1) * n] = to_dev(x[r], dt)
    for path in PATHS:
        hc.set_config(copy_path=path)
        hc.allgather([recv[r][r * n:(r + 1) * n] for r in range(R)], recv)
        torch.cuda.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(recv[r], dt), ref[r], f"AG in place {path} r={r}")


def test_special_values_in_reductions():
    # subnormal sums (no flush to zero), signed zeros, infinities
    R, n = 4, 4096
    rng = np.random.default_rng(5)
    k = [rng.integers(0, 1 << 18, n) for _ in range(R)]
    x = [(kr * 2.0 ** -149).astype(np.float32) for kr in k]
    x[1][:8] = -0.0
    x[0][:8] = -0.0
    x[2][:8] = -0.0
    x[3][:8] = -0.0
    x[0][8] = np.inf
    x[2][9] = -np.inf
    for algo in ["ring", "direct"]:
        hc.set_config(reduce_algo=algo)
        ref = oracle.allreduce_new(x, hc.FP32)
        got = run_ar(x, hc.FP32)
        for r in range(R):
            assert_bitwise(got[r], ref[r], f"special {algo} r={r}")
    xb = [(kr % 32).astype(np.uint16) for kr in k]       # bf16 subnormals
    ref = oracle.allreduce_new(xb, hc.BF16)
    got = run_ar(xb, hc.BF16)
    assert_bitwise(got[0], ref[0], "bf16 subnormal")


# ---------------------------------------------------------------- copies

@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("direct", [0, 1])
@pytest.mark.parametrize("R", [1, 2, 3, 8])
def test_allgather(path, direct, R):
    hc.set_config(copy_path=path, allgather_direct=direct)
    for dt in [hc.FP32, hc.BF16]:
        for n in [1, 13, 100_003]:
            x = [W.random_bits(71 + n, r, n, ES[dt]) for r in range(R)]
            x = [a.view(np.float32) if dt == hc.FP32 else a for a in x]
            ref = oracle.allgather_new(x, dt)
            outs = [padded(R * n, dt, 2) for _ in range(R)]
            hc.allgather([to_dev(a, dt) for a in x], [o[1] for o in outs])
            torch.cuda.synchronize()
            for r in range(R):
                check_canaries(outs[r][0], 2, R * n, dt)
                assert_bitwise(from_dev(outs[r][1], dt), ref[r], f"AG {path} n={n} r={r}")


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("chunk", [0, 65536])
def test_sendrecv_and_alltoall(path, chunk):
    hc.set_config(copy_path=path, chunk_bytes=chunk)
    R = 8
    for n in [5, 300_001]:
        x = [W.random_bits(81, r, n, 2) for r in range(R)]
        for peers in ([r + 1 if r + 1 < R else -1 for r in range(R)],
                      [r - 1 for r in range(R)],
                      [(r + 3) % R for r in range(R)],
                      [r for r in range(R)]):
            ref = [np.full(n, 0x7A5A, np.uint16) for _ in range(R)]
            oracle.sendrecv(x, ref, peers, n, hc.BF16)
            outs = [padded(n, hc.BF16, 0, 0) for _ in range(R)]
            recv = [o[1] for o in outs]
            hc.sendrecv([to_dev(a, hc.BF16) for a in x], recv, peers)
            torch.cuda.synchronize()
            for r in range(R):
                assert_bitwise(from_dev(recv[r], hc.BF16), ref[r], f"P2P {peers} r={r}")
        xs = [W.random_bits(82, r, R * n, 4).view(np.float32) for r in range(R)]
        ref = [np.zeros_like(a) for a in xs]
        oracle.alltoall(xs, ref, n, hc.FP32)
        got = hc.alltoall([to_dev(a, hc.FP32) for a in xs])
        torch.cuda.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(got[r], hc.FP32), ref[r], f"A2A n={n} r={r}")


@pytest.mark.parametrize("path", PATHS)
def test_uint8_copies(path):
    """Bytes on every copy path: odd counts, odd offsets (the kernel's
    single-byte path), all four copy collectives, canaries untouched."""
    hc.set_config(copy_path=path)
    dt = hc.UINT8
    for R, n in [(3, 1), (8, 4097), (5, 1_000_003)]:
        lead = 1 + R % 3
        x = [W.random_bits(95 + n, r, n, 1) for r in range(R)]
        ref = oracle.allgather_new(x, dt)
        outs = [padded(R * n, dt, lead) for _ in range(R)]
        hc.allgather([padded(n, dt, r % 2, 1)[1].copy_(to_dev(x[r], dt)) for r in range(R)],
                     [o[1] for o in outs])
        torch.cuda.synchronize()
        for r in range(R):
            check_canaries(outs[r][0], lead, R * n, dt)
            assert_bitwise(from_dev(outs[r][1], dt), ref[r], f"AG u8 {path} R={R} n={n} r={r}")
        peers = [(r + 1) % R for r in range(R)]
        ref = [np.full(n, 0x5A, np.uint8) for _ in range(R)]
        oracle.sendrecv(x, ref, peers, n, dt)
        outs = [padded(n, dt, lead) for _ in range(R)]
        hc.sendrecv([to_dev(a, dt) for a in x], [o[1] for o in outs], peers)
        torch.cuda.synchronize()
        for r in range(R):
            check_canaries(outs[r][0], lead, n, dt)
            assert_bitwise(from_dev(outs[r][1], dt), ref[r], f"P2P u8 {path} R={R} n={n} r={r}")
        xs = [W.random_bits(96 + n, r, R * n, 1) for r in range(R)]
        ref = [np.zeros_like(a) for a in xs]
        oracle.alltoall(xs, ref, n, dt)
        got = hc.alltoall([to_dev(a, dt) for a in xs])
        torch.cuda.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(got[r], dt), ref[r], f"A2A u8 {path} R={R} n={n} r={r}")
    R = 4
    rng = np.random.default_rng(97)
    C = rng.integers(0, 5000, size=(R, R))
    send = [W.random_bits(98, s, int(C[s].sum()), 1) for s in range(R)]
    counts = [int(C[s][d]) for s in range(R) for d in range(R)]
    sd = [int(C[s][:d].sum()) for s in range(R) for d in range(R)]
    rd = [int(C[:s, d].sum()) for s in range(R) for d in range(R)]
    ref = [np.zeros(int(C[:, d].sum()), np.uint8) for d in range(R)]
    oracle.alltoallv(send, counts, sd, ref, rd, dt)
    recv = [torch.zeros(int(C[:, d].sum()), dtype=torch.uint8, device="cuda") for d in range(R)]
    hc.alltoallv([to_dev(a, dt) for a in send], counts, sd, recv, rd)
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(recv[r], dt), ref[r], f"A2Av u8 {path} r={r}")


def test_uint8_reductions_refused():
    x = [torch.zeros(8, dtype=torch.uint8, device="cuda") for _ in range(2)]
    with pytest.raises(TypeError):
        hc.allreduce(x)
    p = (ctypes.c_void_p * 2)(*[t.data_ptr() for t in x])
    assert hc.lib().hoccl_allreduce(p, p, 8, hc.UINT8, 2, None) == hc.ERR_INVALID_ARG
    assert hc.lib().hoccl_reduce_scatter(p, p, 4, hc.UINT8, 2, None) == hc.ERR_INVALID_ARG


@pytest.mark.parametrize("sched", [0, 1, 2])
@pytest.mark.parametrize("path", PATHS)
def test_alltoallv_routing(path, sched):
    """EP routing (one copy per destination rank), with the byte-balanced
    schedule and with the collective scheduler's stages (in order, and run
    one after another)."""
    if path == "engines" and sched == 2:
        pytest.skip(SERIAL_STAGES_OFF)
    hc.set_config(copy_path=path, a2a_schedule=sched)
    R = 8
    send, counts, sd, rd, rsz = W.a2a_tokens(R=R, tokens=512, hidden=256)
    ref = [np.zeros(s, np.uint16) for s in rsz]
    oracle.alltoallv(send, counts, sd, ref, rd, hc.BF16)
    recv = [torch.zeros(s, dtype=torch.bfloat16, device="cuda") for s in rsz]
    hc.alltoallv([to_dev(a, hc.BF16) for a in send], counts, sd, recv, rd)
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(recv[r], hc.BF16), ref[r], f"A2Av r={r}")


@pytest.mark.parametrize("sched", [1, 2])
@pytest.mark.parametrize("path", PATHS)
def test_alltoall_by_stages(path, sched):
    """Uniform all-to-all through the scheduler's stages, ragged and odd
    rank counts, every element against the oracle."""
    if path == "engines" and sched == 2:
        pytest.skip(SERIAL_STAGES_OFF)
    hc.set_config(copy_path=path, a2a_schedule=sched)
    for R, n in ((3, 7), (5, 4099), (8, 65537)):
        xs = [W.random_bits(83 + R, r, R * n, 2) for r in range(R)]
        ref = [np.zeros_like(a) for a in xs]
        oracle.alltoall(xs, ref, n, hc.BF16)
        got = hc.alltoall([to_dev(a, hc.BF16) for a in xs])
        torch.cuda.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(got[r], hc.BF16), ref[r], f"A2A stages R={R} n={n} r={r}")


def test_serial_stages_refused_on_the_engines():
    """a2a_schedule 2 on the SDMA path is refused before anything is
    enqueued (its outputs keep their contents); stage order (1) runs."""
    R = 4
    xs = [W.random_bits(88, r, R * 100, 2) for r in range(R)]
    send = [to_dev(a, hc.BF16) for a in xs]
    out = [torch.full((R * 100,), 0x5A, dtype=torch.int16, device="cuda").view(torch.bfloat16) for _ in range(R)]
    torch.cuda.synchronize()
    for path in ("engines", "auto"):
        hc.set_config(copy_path=path, a2a_schedule=2)
        with pytest.raises(hc.HocclError) as ei:
            hc.alltoall(send, out)
        assert ei.value.status == hc.ERR_UNSUPPORTED
    torch.cuda.synchronize()
    for r in range(R):
        assert (out[r].view(torch.int16) == 0x5A).all()


def test_copy_paths_report_their_cus():
    """Copy-only collectives launch no kernel of the library on the engine
    proxy or the HIP runtime path.  The stats report the CUs each path may
    occupy: none for the engine proxy with the host-function handshake
    (the default, and what AUTO resolves to), one for its handshake
    kernel, and every CU for the HIP runtime's copies, which the runtime may
    run as a kernel of its own."""
    if hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    R, n = 8, 1 << 16
    x = [torch.randn(n, device="cuda").to(torch.bfloat16) for _ in range(R)]
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    for path, hs, cus, used in [("auto", -1, 0, hc.COPY_SDMA), ("engines", -1, 0, hc.COPY_SDMA),
                                ("engines", 0, 1, hc.COPY_SDMA), ("hip", -1, ncu, hc.COPY_HIP)]:
        hc.set_config(copy_path=path, proxy_handshake=hs)
        hc.allgather(x)
        s = hc.last_stats()
        assert s["cus_used_max"] == cus and s["reduce_launches"] == 0, (path, hs, s)
        assert s["copy_kernel_launches"] == 0 and s["copy_ops"] > 0
        assert s["copy_path_used"] == used, (path, s)
    torch.cuda.synchronize()


def test_kernel_timing_reports_each_launch():
    hc.set_config(kernel_timing=1)
    R, n = 8, 1 << 18
    x = [torch.randn(R * n, device="cuda").to(torch.bfloat16) for _ in range(R)]
    hc.reduce_scatter(x)
    t = hc.kernel_times()
    assert len(t) == R - 1 and all(v > 0 for v in t)


# ---------------------------------------------------------------- stream order

@pytest.mark.parametrize("path", PATHS)
def test_stream_order_with_delayed_producer(path):
    """The inputs are written by a kernel queued behind a long spin on the
    same stream; the collective must not start before them, and a consumer
    queued after it must see its results."""
    hc.set_config(copy_path=path)
    R, n = 4, 1 << 20
    x = [W.random_values("fp32", 91, r, n) for r in range(R)]
    ref = oracle.allreduce_new(x, hc.FP32)
    host = [torch.from_numpy(a).pin_memory() for a in x]
    send = [torch.full((n,), float("nan"), device="cuda") for _ in range(R)]
    recv = [torch.zeros(n, device="cuda") for _ in range(R)]
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        torch.cuda._sleep(50_000_000)                 # ~20 ms spin
        for r in range(R):
            send[r].copy_(host[r], non_blocking=True)
        hc.allreduce(send, recv, stream=s)
        out = [t.clone() for t in recv]
    s.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(out[r], hc.FP32), ref[r], f"{path} r={r}")
    # all-gather too (pure copies)
    shards = [torch.full((n,), float("nan"), device="cuda") for _ in range(R)]
    with torch.cuda.stream(s):
        torch.cuda._sleep(50_000_000)
        for r in range(R):
            shards[r].copy_(host[r], non_blocking=True)
        ag = hc.allgather(shards, stream=s)
        ag = [t.clone() for t in ag]
    s.synchronize()
    cat = np.concatenate(x)
    for r in range(R):
        assert_bitwise(from_dev(ag[r], hc.FP32), cat, f"AG {path} r={r}")


def test_back_to_back_calls_on_two_streams_share_workspace_safely():
    R, n = 8, 1 << 18
    xa = [W.random_values("bf16", 95, r, R * n) for r in range(R)]
    xb = [W.random_values("bf16", 96, r, R * n) for r in range(R)]
    ra = oracle.reduce_scatter_new(xa, hc.BF16)
    rb = oracle.reduce_scatter_new(xb, hc.BF16)
    da = [to_dev(a, hc.BF16) for a in xa]
    db = [to_dev(a, hc.BF16) for a in xb]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for _ in range(3):
        with torch.cuda.stream(s1):
            torch.cuda._sleep(5_000_000)
            oa = hc.reduce_scatter(da, stream=s1)
        with torch.cuda.stream(s2):
            ob = hc.reduce_scatter(db, stream=s2)
        torch.cuda.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(oa[r], hc.BF16), ra[r], f"s1 r={r}")
            assert_bitwise(from_dev(ob[r], hc.BF16), rb[r], f"s2 r={r}")


@pytest.mark.parametrize("handshake", [0, 1, 2])
def test_engine_proxy_handshakes(handshake):
    """Every form of the engine proxy's start/finish flag handshake: the
    kernel on the caller's stream (default), the kernel on the proxy's
    private stream joined by events, and a host function.  Checked behind a delayed producer, with a consumer queued
    after the collective, and for ring chains (dependent hops)."""
    hc.set_config(copy_path="engines", proxy_handshake=handshake)
    R, n = 4, 1 << 20
    x = [W.random_values("fp32", 97, r, n) for r in range(R)]
    ref = oracle.allreduce_new(x, hc.FP32)
    host = [torch.from_numpy(a).pin_memory() for a in x]
    s = torch.cuda.Stream()
    for direct in (1, 0):
        hc.set_config(allgather_direct=direct)
        send = [torch.full((n,), float("nan"), device="cuda") for _ in range(R)]
        recv = [torch.zeros(n, device="cuda") for _ in range(R)]
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            torch.cuda._sleep(20_000_000)
            for r in range(R):
                send[r].copy_(host[r], non_blocking=True)
            for _ in range(3):
                hc.allreduce(send, recv, stream=s)
            out = [t.clone() for t in recv]
        s.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(out[r], hc.FP32), ref[r], f"handshake={handshake} direct={direct} r={r}")


def watchdog_allgather(slice_bytes):
    """An all-gather whose copies make no progress for longer than a 1 ms
    watchdog: 128 MiB shards on one engine, about 2 ms per copy."""
    R, n = 8, 1 << 26
    x = [torch.randn(n, device="cuda").to(torch.bfloat16) for _ in range(R)]
    recv = [torch.empty(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    hc.set_config(copy_path="engines", sdma_engines=1, proxy_timeout_ms=1, proxy_slice_bytes=slice_bytes)
    hc.allgather(x, recv)
    return R, n, x, recv


@pytest.mark.parametrize("slice_bytes", [4 << 20, (1 << 64) - 1])
def test_proxy_watchdog_reports_timeout_then_recovers(slice_bytes):
    """Failure handling forced from the host: a 1 ms watchdog on copies that
    each take about 2 ms, with balanced issue and with every copy issued at
    once.  The copies still complete (results are right), the next call
    reports HOCCL_ERR_TIMEOUT once, and the call after that works."""
    if hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    R, n, x, recv = watchdog_allgather(slice_bytes)
    torch.cuda.synchronize()
    for r in (0, R - 1):
        for s in range(R):
            assert torch.equal(recv[r][s * n:(s + 1) * n], x[s])
    with pytest.raises(hc.HocclError) as ei:
        hc.allgather(x, recv)
    assert ei.value.status == hc.ERR_TIMEOUT
    torch.cuda.synchronize()
    hc.set_config(proxy_timeout_ms=0)
    hc.allgather(x, recv)
    torch.cuda.synchronize()
    assert torch.equal(recv[3][5 * n:6 * n], x[5])


def test_stored_timeout_reported_before_anything_is_enqueued():
    """Failure handling forced from the host: a 1 ms watchdog expires on an
    all-gather's copies.  The next engine call, a ring all-reduce that would
    reduce on the CUs before handing its gather to the proxy, reports the
    timeout and enqueues nothing: its outputs keep their contents.  Then the
    same all-reduce runs and matches the oracle."""
    if hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    R = watchdog_allgather(4 << 20)[0]
    hc.set_config(reduce_algo="ring")
    torch.cuda.synchronize()
    m = 300_007
    xa = [W.random_values("fp32", 97, r, m) for r in range(R)]
    send = [to_dev(a, hc.FP32) for a in xa]
    outs = [torch.full((m,), 7.0, device="cuda") for _ in range(R)]
    torch.cuda.synchronize()
    with pytest.raises(hc.HocclError) as ei:
        hc.allreduce(send, outs)
    assert ei.value.status == hc.ERR_TIMEOUT
    torch.cuda.synchronize()
    for r in range(R):
        assert bool((outs[r] == 7.0).all()), f"rank {r}'s output changed under a reported error"
    hc.set_config(proxy_timeout_ms=0)
    hc.allreduce(send, outs)
    torch.cuda.synchronize()
    ref = oracle.allreduce_new(xa, hc.FP32)
    for r in (0, R - 1):
        assert_bitwise(from_dev(outs[r], hc.FP32), ref[r], f"all-reduce after the error, rank {r}")


def test_finalize_and_reinit():
    R, n = 4, 4096
    x = [W.random_values("fp32", 98, r, n) for r in range(R)]
    ref = oracle.allreduce_new(x, hc.FP32)
    for _ in range(2):
        got = run_ar(x, hc.FP32)
        assert_bitwise(got[0], ref[0], "before finalize")
        hc.finalize()
    hc.init(0)
    got = run_ar(x, hc.FP32)
    assert_bitwise(got[3], ref[3], "after re-init")


@pytest.mark.parametrize("handshake", [0, 2])
def test_handshake_wait_gives_up_then_recovers(handshake):
    """Failure handling forced from the host: a 1 us limit on the handshake
    kernel's own bounded wait.  The kernel stops waiting at once, so its
    dispatch ends and the stream drains; the proxy still runs the copies
    through, reports HOCCL_ERR_TIMEOUT at the next engine call, clears the
    slot, and the calls after that are correct again."""
    if hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    R, n = 8, 1 << 22
    x = [torch.randn(n, device="cuda").to(torch.bfloat16) for _ in range(R)]
    recv = [torch.empty(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    hc.set_config(copy_path="engines", proxy_wait_limit_us=1, proxy_handshake=handshake)
    hc.allgather(x, recv)
    torch.cuda.synchronize()                     # returns: the wait gave up
    err = None
    t0 = time.time()
    while err is None and time.time() - t0 < 10:  # the proxy retires the op
        time.sleep(0.05)
        try:
            hc.allgather(x, recv)
        except hc.HocclError as e:
            err = e
        torch.cuda.synchronize()
    assert err is not None and err.status == hc.ERR_TIMEOUT, err
    assert "stopped waiting" in str(err)
    hc.set_config(proxy_wait_limit_us=0)
    time.sleep(0.2)                               # every limited call retires
    for _ in range(5):                            # late reports, if any, first
        try:
            hc.allgather(x, recv)
            break
        except hc.HocclError as e:
            assert e.status == hc.ERR_TIMEOUT
    else:
        raise AssertionError("the proxy kept reporting timeouts")
    torch.cuda.synchronize()
    for _ in range(3):
        for t in recv:
            t.fill_(0)
        hc.allgather(x, recv)
        torch.cuda.synchronize()
        for r in (0, 5, R - 1):
            for s in range(R):
                assert torch.equal(recv[r][s * n:(s + 1) * n], x[s])


def test_host_function_handshake_refused_under_a_profiler():
    """With a profiler announced (HOCCL_ASSUME_PROFILER stands in for one in
    a child process) the host-function handshake is refused before anything
    is enqueued; the kernel handshake still works there."""
    import subprocess
    import sys
    import os
    code = (
        "import torch, paper_2609_34334_amd as hc\n"
        "x = [torch.ones(4096, device='cuda') for _ in range(4)]\n"
        "hc.set_config(copy_path='engines', proxy_handshake=2)\n"
        "try:\n"
        "    hc.allgather(x)\n"
        "    print('not refused')\n"
        "except hc.HocclError as e:\n"
        "    print('refused', e.status, 'profiler' in str(e))\n"
        "hc.set_config(proxy_handshake=0)\n"
        "y = hc.allgather(x); torch.cuda.synchronize()\n"
        "print('kernel handshake ok', bool(torch.equal(y[2][:4096], x[0])))\n")
    env = dict(os.environ, HOCCL_ASSUME_PROFILER="1")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stderr[-2000:]
    if hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    assert f"refused {hc.ERR_UNSUPPORTED} True" in r.stdout, r.stdout
    assert "kernel handshake ok True" in r.stdout, r.stdout


@pytest.mark.parametrize("streams", [1, 2, 16])
def test_sdma_copy_stream_counts(streams):
    """Every copy collective on the HIP SDMA path with 1, 2 and all 16 copy
    streams (the largest count joins through the last copy stream's event)."""
    R, n = 8, 20_011
    with hc.config(copy_path="hip", copy_streams=streams):
        x = [W.random_bits(800 + streams, r, n, 2) for r in range(R)]
        ref = oracle.allgather_new(x, hc.BF16)
        got = hc.allgather([to_dev(a, hc.BF16) for a in x])
        torch.cuda.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(got[r], hc.BF16), ref[r], f"allgather streams={streams} r={r}")
        xa = [W.random_bits(810 + streams, r, R * n, 4).view(np.int32) for r in range(R)]
        refa = [np.zeros(R * n, np.int32) for _ in range(R)]
        oracle.alltoall(xa, refa, n, hc.INT32)
        gota = hc.alltoall([to_dev(a, hc.INT32) for a in xa])
        torch.cuda.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(gota[r], hc.INT32), refa[r], f"alltoall streams={streams} r={r}")
        xr = [W.random_values("fp32", 820 + streams, r, n) for r in range(R)]
        refr = oracle.allreduce_new(xr, hc.FP32)
        gotr = run_ar(xr, hc.FP32)
        for r in range(R):
            assert_bitwise(gotr[r], refr[r], f"allreduce streams={streams} r={r}")
