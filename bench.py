"""Benchmark of the HOCCL collective hot path on one MI355X.

Headline (`value`): algorithmic bandwidth of the DP gradient reduce-scatter
-- bf16 gradients, 25,165,824 elements per rank (6 x 4096 x 1024), R = 8
virtual ranks, fp32 accumulation, 1/8 shard out per rank -- with inputs
resident in HBM.  One step is one reduce-scatter; W untimed steps, then K
timed steps bracketed by device synchronisation.

Also printed in the same JSON line:
  * roofline of the dominant kernel (the ring reduce-step kernel), from HIP
    events recorded around every launch on the stream it is launched on;
  * cpu_baseline: the CPU oracle on the same workload, single thread;
  * extra: the other collectives of the hot path on their own workloads
    (all-reduce fp32, FSDP all-gather, PP send/recv, EP all-to-all(v) with a
    concurrent bf16 GEMM), each with algbw/busbw, %HBM peak and CUs used;
    the direct fold; the reduce-scatter at fixed workgroup budgets and on
    reserved CUs beside the GEMM; the bucket all-reduce in chunk groups; one
    rank's ring hop; single messages and small-message round trips; the
    engines right after a large device-memory free, static against
    balanced issue.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--quick]
       python bench.py --sweep            (algbw against message size)
Profiling workloads (one phase each): --pmc-workload, --occupancy-workload,
--copy-workload, --ar-groups-workload, --interference-workload,
--ceilings-workload, --after-free-workload, --copy-kernel-workload,
--backend-workload (the torch.distributed backend's per-call time over rank
processes).
"""
import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, GB/s


_T0 = time.perf_counter()


def log(*a):
    print(f"[bench {time.perf_counter() - _T0:6.1f} s]", *a, file=sys.stderr, flush=True)


def bf16_dev(a):
    import numpy as np
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def time_op(fn, steps, warmup, stream=None):
    """Median-free total timing: W warmup calls, then K calls between two
    synchronisations.  Returns seconds per call."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps


def event_time(fn, reps, warmup=2):
    """Per-call device time from HIP events on the current stream (median)."""
    import torch
    for _ in range(warmup):
        fn()
    ts = []
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        b.synchronize()
        ts.append(a.elapsed_time(b) / 1e3)
    return statistics.median(ts), min(ts)


_FLUSH = []


def queued_time(fn, reps, flush, warmup=2):
    """Device time of fn alone: each timed call is enqueued behind a 50 us
    spin, so the host's launch latency stays outside the events.  With
    `flush`, 1 GiB (four times the 256 MB Infinity Cache) is written before
    the spin, so the call starts with a cold last-level cache."""
    import torch
    if flush and not _FLUSH:
        _FLUSH.append(torch.empty(1 << 28, dtype=torch.float32, device="cuda"))
    for _ in range(warmup):
        fn()
    ts = []
    for k in range(reps):
        if flush:
            _FLUSH[0].fill_(float(k))
        torch.cuda._sleep(120_000)
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        b.synchronize()
        ts.append(a.elapsed_time(b) / 1e3)
    return statistics.median(ts), min(ts)


# ---- the headline: reduce-scatter ------------------------------------------

def bench_reduce_scatter(hc, W, steps, warmup):
    import torch
    R, n_in = 8, 25_165_824
    n = n_in // R
    x = W.rs_gradients(R, n_in)
    send = [bf16_dev(a) for a in x]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    hc.set_config(reduce_algo="ring", kernel_timing=0)
    stream = torch.cuda.current_stream()

    def step():
        hc.reduce_scatter(send, recv, stream=stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    # The timed region: K steps between two synchronisations, bracketed by
    # HIP events on the stream every kernel of the step is launched on.
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t0) / steps
    stats = hc.last_stats()
    launches_per_op = stats["reduce_launches"]
    bytes_per_op = stats["hbm_bytes_algorithmic"]
    avg_launch_s = e0.elapsed_time(e1) / 1e3 / (steps * launches_per_op)
    achieved = bytes_per_op / launches_per_op / avg_launch_s / 1e9
    # Per-step detail: events around each launch (they add the dispatch gap).
    hc.set_config(kernel_timing=1)
    hc.kernel_times()
    for _ in range(steps):
        step()
    kt = hc.kernel_times()
    hc.set_config(kernel_timing=0)
    per_step = [round(statistics.mean(kt[i::launches_per_op]) * 1e3, 2) for i in range(launches_per_op)]
    S = R * n * 2
    algbw = S / sec / 1e9
    return dict(x=x, recv=recv, sec=sec, stats=stats, S=S, algbw=algbw,
                busbw=algbw * (R - 1) / R, bytes_per_op=bytes_per_op,
                launches=launches_per_op, avg_launch_us=avg_launch_s * 1e6,
                achieved=achieved, per_step_us=per_step)


def direct_reduce_scatter(hc, send_np, steps, warmup):
    """The same reduce-scatter with the one-pass fold (bit-identical)."""
    import torch
    R = len(send_np)
    n = send_np[0].size // R
    send = [bf16_dev(a) for a in send_np]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    hc.set_config(reduce_algo="direct")
    sec = time_op(lambda: hc.reduce_scatter(send, recv), steps, warmup)
    st = hc.last_stats()
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        hc.reduce_scatter(send, recv, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    hc.set_config(reduce_algo="ring")
    launch = e0.elapsed_time(e1) / 1e3 / steps
    achieved = st["hbm_bytes_algorithmic"] / launch / 1e9
    return recv, dict(algbw_GBs=round(R * n * 2 / sec / 1e9, 2), busbw_GBs=round(R * n * 2 / sec / 1e9 * (R - 1) / R, 2),
                      ms=round(sec * 1e3, 4), cus_used=st["cus_used_max"],
                      roofline={"kernel": "fold_kernel (all 8 ranks folded in ring order, one launch)",
                                "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                                "traffic": measured_traffic(FOLD_TRAFFIC_SUMMARY),
                                "traffic_dram_destined": measured_traffic(
                                    FOLD_TRAFFIC_SUMMARY, key="dram_destined_bytes_per_launch"),
                                "avg_launch_us": round(launch * 1e6, 2),
                                "bytes_per_launch": st["hbm_bytes_algorithmic"]})


def host_cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(x, recvcount, budget_s=12.0):
    """The oracle (single-threaded C) on the same reduce-scatter, repeated
    until about budget_s seconds of CPU work, with this thread pinned to one
    host core for the timing."""
    import numpy as np
    import oracle
    R = len(x)
    out = [np.empty(recvcount, np.uint16) for _ in range(R)]
    saved = os.sched_getaffinity(0)
    core = min(saved)
    os.sched_setaffinity(0, {core})
    try:
        t0 = time.perf_counter()
        reps = 0
        while True:
            oracle.reduce_scatter(x, out, recvcount, oracle.BF16)
            reps += 1
            if time.perf_counter() - t0 > budget_s:
                break
        sec = (time.perf_counter() - t0) / reps
    finally:
        os.sched_setaffinity(0, saved)
    return out, sec, reps, core, len(saved)


# ---- the other collectives ---------------------------------------------------

def dedicated_stream():
    """A stream with a hardware queue of its own.  HIP folds streams onto a
    few shared queues (four per process here), and two streams on one queue
    run one after the other; a stream created with a CU mask (every CU) is
    never shared, so the GEMM and the collective can overlap."""
    import ctypes
    import torch
    hip = ctypes.CDLL("libamdhip64.so.7")    # the HIP runtime torch has loaded
    s = ctypes.c_void_p()
    mask = (ctypes.c_uint32 * 8)(*([0xFFFFFFFF] * 8))
    if hip.hipExtStreamCreateWithCUMask(ctypes.byref(s), 8, mask) != 0:
        return torch.cuda.Stream()
    return torch.cuda.ExternalStream(s.value)


def masked_stream(cus):
    """A stream with a hardware queue of its own whose kernels run only on
    the logical CUs in `cus` (bit i of the runtime's 256-bit CU mask); None
    if the runtime refuses the mask (it needs a CU in every XCD: logical
    CUs 0-7 are one per XCD)."""
    import ctypes
    import torch
    hip = ctypes.CDLL("libamdhip64.so.7")    # the HIP runtime torch has loaded
    words = [0] * 8
    for c in cus:
        words[c // 32] |= 1 << (c % 32)
    s = ctypes.c_void_p()
    if hip.hipExtStreamCreateWithCUMask(ctypes.byref(s), 8, (ctypes.c_uint32 * 8)(*words)) != 0:
        return None
    return torch.cuda.ExternalStream(s.value)


def _gemm_run(gemm, k=20):
    import torch
    A, B, C, _, gs, _ = gemm
    ts = []
    with torch.cuda.stream(gs):
        g0 = torch.cuda.Event(enable_timing=True)
        g0.record(gs)
        for _ in range(k):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(gs)
            torch.matmul(A, B, out=C)
            b.record(gs)
            ts.append((a, b))
        g1 = torch.cuda.Event(enable_timing=True)
        g1.record(gs)
    return g0, g1, ts


_GATE = {}


def host_gate():
    """A gate the host opens: returns (event, open).  `event` completes once
    `open()` has been called, so work on several streams that waits on it
    starts together, however long the host takes to enqueue that work.  An
    own-queue stream waits (hipStreamWaitValue32, equality) on a token in
    coherent host memory; a timer opens the gate after 5 s in any case, so
    the wait always ends.  `open()` returns True when the timer had opened
    it: the host was held up while enqueueing (the HIP runtime makes the
    enqueueing thread wait once too much work is queued), the streams did
    not start together and the measurement is void."""
    import ctypes
    import threading
    import torch
    if not _GATE:
        hip = ctypes.CDLL("libamdhip64.so.7")    # the HIP runtime torch has loaded
        V = ctypes.c_void_p
        hip.hipHostMalloc.argtypes = [ctypes.POINTER(V), ctypes.c_size_t, ctypes.c_uint]
        hip.hipStreamWaitValue32.argtypes = [V, V, ctypes.c_uint32, ctypes.c_uint, ctypes.c_uint32]
        p = V()
        if hip.hipHostMalloc(ctypes.byref(p), 64, 0x2 | 0x40000000) != 0:   # mapped | coherent
            raise RuntimeError("hipHostMalloc of the gate flag failed")
        _GATE.update(hip=hip, flag=p.value, cell=ctypes.c_uint32.from_address(p.value),
                     stream=dedicated_stream(), token=0)
    g = _GATE
    g["token"] = g["token"] % 1_000_000 + 1
    k = g["token"]
    g["cell"].value = 0
    s = g["stream"]
    if g["hip"].hipStreamWaitValue32(ctypes.c_void_p(s.cuda_stream), ctypes.c_void_p(g["flag"]), k,
                                     0x1, 0xFFFFFFFF) != 0:
        raise RuntimeError("hipStreamWaitValue32 failed")
    ev = torch.cuda.Event()
    ev.record(s)
    fired = []

    def on_timer():
        fired.append(True)
        g["cell"].value = k

    timer = threading.Timer(5.0, on_timer)
    timer.start()

    def open_gate():
        timer.cancel()
        g["cell"].value = k
        return bool(fired)

    return ev, open_gate


def _gated(gemm, collective=None, n_coll=0, k=20):
    """k GEMMs and `n_coll` collectives (an event after each), all enqueued
    behind one host gate, which then opens so that both loops start
    together; then the host synchronises.  The host thread does the same
    thing while the GPU runs whether or not collectives are enqueued: GEMM
    time depends on it by several percent (a host that sleeps, spins or
    records events while the GEMMs run sees 0.80-0.87 ms).  Returns the
    collective window start c0, the collective's end events, the GEMM
    event pairs and whether the gate's timer had to open it."""
    import torch
    gs, cs = gemm[4], gemm[5]
    torch.cuda.synchronize()
    gate, open_gate = host_gate()
    c0 = None
    ends = []
    try:
        gs.wait_event(gate)
        if collective is not None:
            cs.wait_event(gate)
            with torch.cuda.stream(cs):
                c0 = torch.cuda.Event(enable_timing=True)
                c0.record(cs)
                for _ in range(n_coll):
                    collective(cs)
                    e = torch.cuda.Event(enable_timing=True)
                    e.record(cs)
                    ends.append(e)
        _, _, ts = _gemm_run(gemm, k)
    finally:
        blocked = open_gate()
    torch.cuda.synchronize()
    return c0, ends, ts, blocked


def _boot_ci(x, reps=4000, seed=1):
    """Bootstrap 95% interval of the mean of x (resampling its items)."""
    import numpy as np
    x = np.asarray(x, dtype=np.float64)
    rng = np.random.default_rng(seed)
    means = x[rng.integers(0, len(x), size=(reps, len(x)))].mean(axis=1)
    lo, hi = np.percentile(means, [2.5, 97.5])
    return float(lo), float(hi)


def interference(hc, collective, med, gemm, pairs=100, k=4, seed=0):
    """Slowdown of a bf16 8192^3 GEMM loop on one queue while `collective`
    loops on another, resolved by pairing.  Each of `pairs` pairs is one run
    of k GEMMs alone and one run of k GEMMs beside back-to-back collectives,
    both under the same host gate (so the host thread does the same in both
    arms), in an order drawn at random per pair.  A pair's ratio is the mean
    time of the GEMMs that ran entirely inside the collective window over
    the mean time of the same GEMMs (by position) alone; adjacent runs
    cancel the drift of the clocks.  Reports the mean ratio - 1 with a
    bootstrap 95% interval over pairs, the collective's own slowdown (its
    time per call while the GEMMs ran, against `med` alone; median over
    pairs) and the pairs voided because the host was held up while
    enqueueing (the collectives then could not start with the GEMMs)."""
    import random
    import torch
    t_alone, cs = gemm[3], gemm[5]
    n_coll = int(1.5 * k * t_alone / max(med, 1e-6)) + 2
    with torch.cuda.stream(cs):
        collective(cs)
    torch.cuda.synchronize()
    rng = random.Random(seed)
    ratios, colls, overlaps = [], [], []
    void = 0
    for _ in range(pairs):
        order = [False, True] if rng.random() < 0.5 else [True, False]
        runs = {}
        for conc in order:
            runs[conc] = _gated(gemm, collective if conc else None, n_coll if conc else 0, k)
        if runs[True][3] or runs[False][3]:
            void += 1
            if void >= 3 and not ratios:
                break
            continue
        c0, ends, ts, _ = runs[True]
        alone = runs[False][2]
        end = c0.elapsed_time(ends[-1])
        inside = [i for i, (a, b) in enumerate(ts)
                  if c0.elapsed_time(a) >= 0 and c0.elapsed_time(b) <= end]
        overlaps.append(len(inside) / k)
        if not inside:
            continue
        tc = statistics.mean(ts[i][0].elapsed_time(ts[i][1]) for i in inside)
        ta = statistics.mean(alone[i][0].elapsed_time(alone[i][1]) for i in inside)
        ratios.append(tc / ta)
        g_hi = c0.elapsed_time(ts[-1][1])
        done = [t for t in (c0.elapsed_time(e) for e in ends) if t <= g_hi]
        if done:
            colls.append(done[-1] / len(done) / 1e3 / med - 1)
    out = dict(gemm_slowdown=None, gemm_slowdown_ci95=None, pairs=len(ratios), pairs_void=void,
               gemms_per_run=k, gemm_overlap=round(statistics.mean(overlaps), 3) if overlaps else None,
               collective_slowdown=round(statistics.median(colls), 4) if colls else None,
               collectives_queued=n_coll)
    if len(ratios) >= 2:
        lo, hi = _boot_ci(ratios)
        out.update(gemm_slowdown=round(statistics.mean(ratios) - 1, 4),
                   gemm_slowdown_ci95=[round(lo - 1, 4), round(hi - 1, 4)])
    if void and not ratios:
        out["gemm_slowdown_void"] = ("the enqueueing thread was held up with the collectives queued "
                                     "behind the gate, so they could not start with the GEMMs")
    return out


def null_interference(gemm, pairs=100, k=4, seed=0):
    """The harness's resolution: the same pairs with nothing beside the
    GEMMs in either arm (an A/A test).  Its interval should hold 0 and its
    half-width is what `interference` can resolve."""
    import random
    rng = random.Random(seed)
    ratios = []
    for _ in range(pairs):
        a = _gated(gemm, None, 0, k)
        b = _gated(gemm, None, 0, k)
        if a[3] or b[3]:
            continue
        if rng.random() < 0.5:
            a, b = b, a
        ta = statistics.mean(x.elapsed_time(y) for x, y in a[2])
        tb = statistics.mean(x.elapsed_time(y) for x, y in b[2])
        ratios.append(tb / ta)
    lo, hi = _boot_ci(ratios)
    return dict(gemm_slowdown=round(statistics.mean(ratios) - 1, 4),
                gemm_slowdown_ci95=[round(lo - 1, 4), round(hi - 1, 4)], pairs=len(ratios), gemms_per_run=k)


def interference_workload(hc, W, engines=(16, 8, 6, 4, 2), pairs=100):
    """GEMM interference of the zero-CU copy collectives against the SDMA
    engines they may use: the FSDP all-gather, the PP schedule and the EP
    all-to-all(v) on the engine proxy beside the bf16 8192^3 GEMM, each at
    several engine budgets, plus the harness's own null (A/A) interval."""
    import torch
    gemm = make_gemm()
    out = {"gemm_alone_ms": round(gemm[3] * 1e3, 4), "null": null_interference(gemm, pairs)}
    R = 8
    x = W.ag_parameters(R)
    ag_send = [bf16_dev(a) for a in x]
    ag_recv = [torch.empty(R * x[0].size, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    p = W.p2p_activations(R)
    pp_send = [bf16_dev(a) for a in p]
    pp_recv = [torch.empty(p[0].size, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    fwd = [r + 1 if r + 1 < R else -1 for r in range(R)]
    bwd = [r - 1 for r in range(R)]

    def pp(s):
        for _ in range(16):
            hc.sendrecv(pp_send, pp_recv, fwd, stream=s)
            hc.sendrecv(pp_send, pp_recv, bwd, stream=s)
    send_np, counts, sd, rd, rsz = W.a2a_tokens(R)
    a2a_send = [bf16_dev(a) for a in send_np]
    a2a_recv = [torch.empty(q, dtype=torch.bfloat16, device="cuda") for q in rsz]
    work = [("allgather_fsdp", lambda s: hc.allgather(ag_send, ag_recv, stream=s),
             R * x[0].size * 2 * (R - 1)),
            ("p2p_pp", pp, 224 * p[0].size * 2),
            ("alltoallv_ep", lambda s: hc.alltoallv(a2a_send, counts, sd, a2a_recv, rd, stream=s),
             sum(counts) * 2)]
    for name, run, copied in work:
        rows = {}
        for E in engines:
            with hc.config(copy_path="engines", sdma_engines=E):
                med, _ = event_time(lambda: run(None), 5)
                row = dict(ms=round(med * 1e3, 4), copy_GBs=round(copied / med / 1e9, 1))
                row.update(interference(hc, run, med, gemm, pairs=pairs))
            rows[f"engines{E}"] = row
            log(f"  {name} engines={E}: {row['ms']} ms, GEMM {row['gemm_slowdown']} {row['gemm_slowdown_ci95']}")
        out[name] = rows
    return out


def make_gemm():
    """The victim: a bf16 8192 x 8192 x 8192 matmul on its own queue."""
    import torch
    A = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    B = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    C = torch.empty(8192, 8192, device="cuda", dtype=torch.bfloat16)
    gs, cs = dedicated_stream(), dedicated_stream()
    for _ in range(5):
        torch.matmul(A, B, out=C)
    torch.cuda.synchronize()
    gemm = (A, B, C, 0.0, gs, cs)
    _, _, ts = _gemm_run(gemm)
    torch.cuda.synchronize()
    t = statistics.median(x.elapsed_time(y) for x, y in ts) / 1e3
    return (A, B, C, t, gs, cs)


# Copy paths compared by the copy workloads.  "engines" is the engine proxy
# with its default host-function handshake and engine budget (4): what AUTO
# resolves to; "engines16" the same on all 16 engines.
PATHS = [("engines", {"copy_path": "engines"}),
         ("engines16", {"copy_path": "engines", "sdma_engines": 16}),
         ("engines_kernel_handshake", {"copy_path": "engines", "proxy_handshake": 0}),
         ("hip", {"copy_path": "hip"}),
         ("kernel", {"copy_path": "kernel"})]


# Paths whose GEMM interference is resolved with 100 pairs (the zero-CU
# paths, whose target is a loss of at most 2%); the CU paths cost tens of
# percent and get 20.
INTERFERENCE_PATHS = ("engines", "engines16", "engines_ring", "auto")


def copy_paths(hc, run, S, f, reps, gemm=None, extra_paths=()):
    """Time `run(stream)` under every copy path: algbw = S / t, busbw = algbw * f."""
    res = {}
    saved = hc.get_config()
    for name, kw in list(PATHS) + list(extra_paths):
        hc.set_config(**kw)
        med, mn = event_time(lambda: run(None), reps)
        st = hc.last_stats()
        r = dict(algbw_GBs=round(S / med / 1e9, 2), busbw_GBs=round(S / med / 1e9 * f, 2),
                 ms=round(med * 1e3, 4), copy_GBs=round(st["copy_bytes"] / med / 1e9, 1),
                 hbm_frac=round(st["hbm_bytes_algorithmic"] / med / 1e9 / HBM_PEAK_GBS, 4),
                 path_used=hc.COPY_PATH_NAMES[st["copy_path_used"]],
                 cus_used=st["cus_used_max"], host_enqueue_us=round(st["host_enqueue_us"], 1))
        if gemm is not None:
            r.update(interference(hc, run, med, gemm, pairs=100 if name in INTERFERENCE_PATHS else 20))
        res[name] = r
        hc.set_config(**saved)
    return res


def bench_allreduce(hc, W, reps, gemm):
    import torch
    R, n = 4, 1_048_576
    x = W.allreduce_fp32(R, n)
    send = [torch.from_numpy(a).cuda() for a in x]
    recv = [torch.empty(n, device="cuda") for _ in range(R)]
    res = copy_paths(hc, lambda s: hc.allreduce(send, recv, stream=s), n * 4, 2 * (R - 1) / R, reps)
    hc.set_config(reduce_algo="direct")
    med, _ = event_time(lambda: hc.allreduce(send, recv), reps)
    st = hc.last_stats()
    res["direct_fold"] = dict(algbw_GBs=round(n * 4 / med / 1e9, 2), us=round(med * 1e6, 2),
                              hbm_frac=round(st["hbm_bytes_algorithmic"] / med / 1e9 / HBM_PEAK_GBS, 4),
                              cus_used=st["cus_used_max"])
    hc.set_config(reduce_algo="ring")
    # The 33.6 MB working set fits the last-level cache.  Device time alone
    # (each call queued behind a spin), with the cache warm and flushed.
    dev = {}
    for name, kw in (("kernel", {"copy_path": "kernel"}), ("hip", {"copy_path": "hip"}),
                     ("engines", {"copy_path": "engines"}), ("direct_fold", {"reduce_algo": "direct"}),
                     ("auto", {"reduce_algo": "auto", "copy_path": "auto"})):
        with hc.config(**kw):
            warm, _ = queued_time(lambda: hc.allreduce(send, recv), reps, flush=False)
            cold, _ = queued_time(lambda: hc.allreduce(send, recv), reps, flush=True)
        dev[name] = dict(warm_us=round(warm * 1e6, 2), flushed_us=round(cold * 1e6, 2),
                         warm_algbw_GBs=round(n * 4 / warm / 1e9, 2),
                         flushed_algbw_GBs=round(n * 4 / cold / 1e9, 2))
    res["device_only"] = dev
    return dict(workload="all-reduce fp32 R=4, 1,048,576 elements per rank (ring reduction + gather copies; "
                         "direct_fold: one kernel writes all outputs)", **res)


def bench_allreduce_bucket(hc, W, reps):
    """All-reduce of one GPT-6.7B gradient bucket (bf16, R=8, 25,165,824
    elements per rank): the ring reduction on CUs, then the gather as copies.
    With G chunk groups the gather of group g overlaps the reduction of
    group g+1 (copies beside CU kernels); the direct fold for scale."""
    import torch
    R, n = 8, 25_165_824
    x = W.rs_gradients(R, n)
    send = [bf16_dev(a) for a in x]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    S = n * 2
    out = {}
    for path in ("engines", "hip", "kernel"):
        for G in (1, 2, 4, 8):
            with hc.config(copy_path=path, allreduce_chunk_groups=G):
                med, _ = event_time(lambda: hc.allreduce(send, recv), reps)
                st = hc.last_stats()
            out[f"{path}_groups{G}"] = dict(ms=round(med * 1e3, 4), algbw_GBs=round(S / med / 1e9, 1),
                                            busbw_GBs=round(S / med / 1e9 * 2 * (R - 1) / R, 1),
                                            copy_ops=st["copy_ops"], reduce_launches=st["reduce_launches"])
    with hc.config(reduce_algo="direct"):
        med, _ = event_time(lambda: hc.allreduce(send, recv), reps)
    out["direct_fold"] = dict(ms=round(med * 1e3, 4), algbw_GBs=round(S / med / 1e9, 1))
    return dict(workload="all-reduce bf16 R=8, 25,165,824 elements per rank (ring reduction + gather; "
                         "G chunk groups overlap the gather of group g with the reduction of group g+1)", **out)


def bench_allgather(hc, W, reps, gemm):
    import torch
    R, total = 8, 201_326_592
    x = W.ag_parameters(R, total)
    send = [bf16_dev(a) for a in x]
    recv = [torch.empty(total, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    res = copy_paths(hc, lambda s: hc.allgather(send, recv, stream=s), total * 2, (R - 1) / R, reps, gemm,
                     extra_paths=[("engines_ring", {"copy_path": "engines", "allgather_direct": 0}),
                                  ("hip_ring", {"copy_path": "hip", "allgather_direct": 0}),
                                  ("kernel_wg8", {"copy_path": "kernel", "workgroups_per_step": 8}),
                                  ("kernel_wg64", {"copy_path": "kernel", "workgroups_per_step": 64})])
    hc.set_config(allgather_direct=1)
    # Roofline of the engine path: HBM bytes (each copied byte read once and
    # written once) against the 8 TB/s peak, and its copy rate against what
    # the 16 engines move when each copies one 256 MiB message of its own
    # (16 independent sends, 4 GiB in all, so the operation's fixed costs
    # weigh under 1%), this path's own ceiling.
    with hc.config(copy_path="engines", sdma_engines=16):
        E, m = 16, 1 << 27
        src = [torch.empty(m, dtype=torch.bfloat16, device="cuda") for _ in range(E)]
        dst = [torch.empty_like(t) for t in src]
        ring = [(r + 1) % E for r in range(E)]
        med, _ = event_time(lambda: hc.sendrecv(src, dst, ring), 5)
        del src, dst
    ceiling = E * m * 2 / med / 1e9
    roof = {}
    for name in ("engines", "engines16"):
        r = res[name]
        copied = total * 2 * R                     # out-of-place: every rank's 8 shards
        achieved = 2 * copied / (r["ms"] / 1e3) / 1e9
        roof[name] = {"bound": "hbm", "kernel": "SDMA engine copies (no kernel)", "achieved": round(achieved, 1),
                      "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                      "copy_GBs": round(copied / (r["ms"] / 1e3) / 1e9, 1),
                      "engine_ceiling_copy_GBs": round(ceiling, 1),
                      "frac_of_engine_ceiling": round(copied / (r["ms"] / 1e3) / 1e9 / ceiling, 4),
                      "bytes_per_op": 2 * copied}
    return dict(workload="FSDP all-gather bf16 R=8, 25,165,824-element shards (one GPT-6.7B block, "
                         "201,326,592 params), out-of-place", roofline=roof,
                cpu_baseline=allgather_cpu_baseline(x), **res)


def allgather_cpu_baseline(x, budget_s=10.0):
    """The oracle all-gather (single-threaded C, bit copies) on the FSDP
    workload, repeated for about budget_s seconds on one pinned host core."""
    import numpy as np
    import oracle
    R, n = len(x), x[0].size
    out = [np.empty(R * n, np.uint16) for _ in range(R)]
    saved = os.sched_getaffinity(0)
    core = min(saved)
    os.sched_setaffinity(0, {core})
    try:
        t0 = time.perf_counter()
        reps = 0
        while True:
            oracle.allgather(x, out, n, oracle.BF16)
            reps += 1
            if time.perf_counter() - t0 > budget_s:
                break
        sec = (time.perf_counter() - t0) / reps
    finally:
        os.sched_setaffinity(0, saved)
    S = R * n * 2
    return {"value": round(S / sec / 1e9, 4), "unit": "GB/s (algbw)", "cores": 1, "kind": "oracle",
            "sample": f"the full FSDP all-gather, {reps} repetitions, {sec:.2f} s each, pinned to host "
                      f"core {core}", "ms": round(sec * 1e3, 1)}


def bench_p2p(hc, W, reps, gemm):
    import torch
    R = 8
    x = W.p2p_activations(R)
    n = x[0].size
    send = [bf16_dev(a) for a in x]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    fwd = [r + 1 if r + 1 < R else -1 for r in range(R)]
    bwd = [r - 1 for r in range(R)]

    def schedule(s):
        for _ in range(16):            # 16 microbatches, forward then backward
            hc.sendrecv(send, recv, fwd, stream=s)
            hc.sendrecv(send, recv, bwd, stream=s)

    # S: one message per round of 7 concurrent hops; 32 rounds per schedule
    res = copy_paths(hc, schedule, 32 * n * 2, 1.0, max(3, reps // 3), gemm)
    for k, r in res.items():
        r["per_message_algbw_GBs"] = r.pop("algbw_GBs")
        r.pop("busbw_GBs")
        r["aggregate_GBs"] = round(r["per_message_algbw_GBs"] * (R - 1), 2)
    return dict(workload="PP send/recv bf16 [1,2048,4096] per message, 8 stages, 16 microbatches fwd+bwd "
                         "(224 messages in 32 rounds of 7 concurrent hops)", **res)


def bench_a2a(hc, W, reps, gemm):
    import torch
    R = 8
    send_np, counts, sd, rd, rsz = W.a2a_tokens(R)
    send = [bf16_dev(a) for a in send_np]
    recv = [torch.empty(s, dtype=torch.bfloat16, device="cuda") for s in rsz]
    sent = sum(counts) * 2
    res = copy_paths(hc, lambda s: hc.alltoallv(send, counts, sd, recv, rd, stream=s), sent // R, (R - 1) / R,
                     reps, gemm, extra_paths=[("kernel_wg8", {"copy_path": "kernel", "workgroups_per_step": 8}),
                                              ("kernel_wg64", {"copy_path": "kernel", "workgroups_per_step": 64})])
    # The collective scheduler's stages (Algorithm 1 on this traffic
    # matrix, one memory domain) against the byte-balanced schedule.
    C = [[counts[s * R + d] * 2 if s != d else 0 for d in range(R)] for s in range(R)]
    nstages = len(hc.schedule(C, [0] * R, [-1] * R, 1.0, 1.0)["stages"])
    ab = {"stages": nstages}
    for E in (0, 16):
        for sched, name in ((0, "byte_balanced"), (1, "stages")):
            with hc.config(copy_path="engines", sdma_engines=E, a2a_schedule=sched):
                med, mn = event_time(lambda: hc.alltoallv(send, counts, sd, recv, rd), reps)
            ab[f"{name}_engines{E or 4}"] = dict(ms=round(med * 1e3, 4), min_ms=round(mn * 1e3, 4),
                                                 copy_GBs=round(sent / med / 1e9, 1))
    for sched, name in ((0, "byte_balanced"), (2, "stages_serial")):
        with hc.config(copy_path="kernel", a2a_schedule=sched):
            med, mn = event_time(lambda: hc.alltoallv(send, counts, sd, recv, rd), reps)
            st = hc.last_stats()
        ab[f"{name}_cu_kernel"] = dict(ms=round(med * 1e3, 4), min_ms=round(mn * 1e3, 4),
                                       copy_GBs=round(sent / med / 1e9, 1),
                                       launches=st["copy_kernel_launches"])
    return dict(workload="EP all-to-all(v) bf16, 4096 tokens x 2048 per rank, 64 experts over R=8, top-6 "
                         "(one copy per destination rank), gemm_slowdown against a concurrent 8192^3 bf16 GEMM",
                bytes_sent_total=sent, schedule_ab=ab, **res)


def bench_p2p_sizes(hc, reps, bufs=None):
    """One message 0 -> 1 over the paper's microbenchmark range: the engine
    proxy and the HIP runtime's copies against the CU copy kernel at 1 ... 256
    workgroups (the analog of NCCL's 1/2/4/8-SM budgets).  `bufs`: two 1 GiB
    bf16 device buffers to copy between (allocated here if not given)."""
    import torch
    if bufs is None:
        bufs = [torch.empty(1 << 29, dtype=torch.bfloat16, device="cuda") for _ in range(2)]
    big, big2 = bufs
    # The first pass over the sizes sometimes caught the engine copies of
    # 32-48 MiB at less than half their rate for some milliseconds (a
    # transient of the engines themselves: the handshake kernel saw it too);
    # a second pass never did.  The loop runs twice and the second is kept.
    for _ in range(2):
        rows = _p2p_size_rows(hc, reps, big, big2)
    return dict(workload="single bf16 message rank 0 -> 1, algbw GB/s", rows=rows)


def _p2p_size_rows(hc, reps, big, big2):
    rows = []
    # 50,331,648 B: one all-gather hop, a 25,165,824-element bf16 shard.
    for sz in [2 << 20, 32 << 20, 50_331_648, 512 << 20]:
        ne = sz // 2
        s0, d1 = big[:ne], big2[:ne]
        row = {"bytes": sz}
        for name, kw in [("hip", dict(copy_path="hip")), ("engines", dict(copy_path="engines")),
                         ("engines16", dict(copy_path="engines", sdma_engines=16)),
                         ("engines_kernel_handshake", dict(copy_path="engines", proxy_handshake=0)),
                         ("engines_striped", dict(copy_path="engines", chunk_bytes=max(1 << 20, sz // 16)))] + \
                        [(f"kernel_wg{w}", dict(copy_path="kernel", workgroups_per_step=w)) for w in (1, 2, 4, 8, 64, 256)]:
            hc.set_config(**kw)
            med, _ = event_time(lambda: hc.sendrecv([s0, s0], [d1, d1], [1, -1]), reps)
            row[name] = round(sz / med / 1e9, 1)
            hc.set_config(copy_path="auto", chunk_bytes=0, workgroups_per_step=0, proxy_handshake=-1,
                          sdma_engines=0)
        rows.append(row)
    return rows


def bench_ring_hop(hc, x, reps):
    """One rank's share of a ring step: the unit each GPU would run per hop
    with the ranks on separate GPUs.  The middle hop over one 3,145,728-
    element block of the headline input (fp32 partial updated in place with
    a bf16 local block: 10 bytes per element, 31.5 MB) at several workgroup
    budgets, and the first and last hops at the automatic budget; device
    time alone (each call queued behind a spin), with the last-level cache
    warm and after writing 1 GiB (flushed)."""
    import torch
    R = len(x)
    n = x[0].size // R
    j = 3
    loc = bf16_dev(x[j][j * n:(j + 1) * n])
    prev = bf16_dev(x[j - 1][j * n:(j + 1) * n])
    part = loc.float()
    dst = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    cases = [("middle_auto" if w == 0 else f"middle_wg{w}", w,
              lambda: hc.ring_hop(part, loc, out=part, hop="middle")) for w in (0, 256, 64, 8)]
    cases += [("first", 0, lambda: hc.ring_hop(prev, loc, out=part, hop="first")),
              ("last", 0, lambda: hc.ring_hop(part, loc, out=dst, hop="last"))]
    out = {}
    for name, w, fn in cases:
        with hc.config(workgroups_per_step=w):
            warm, _ = queued_time(fn, reps, flush=False)
            cold, _ = queued_time(fn, reps, flush=True)
            st = hc.last_stats()
        b = st["hbm_bytes_algorithmic"]
        out[name] = dict(bytes=b, warm_us=round(warm * 1e6, 2), flushed_us=round(cold * 1e6, 2),
                        warm_GBs=round(b / warm / 1e9, 1), flushed_GBs=round(b / cold / 1e9, 1),
                        workgroups=st["workgroups_per_step"], cus_used=st["cus_used_max"])
    return dict(workload="one rank's ring hop of the headline reduce-scatter: 3,145,728 elements, "
                         "bf16 local block, fp32 partial (hoccl_ring_hop)", **out)


def bench_rs_launch_shapes(hc, x, steps=20):
    """The headline ring reduce-scatter at other launch shapes and ring-group
    sizes than the automatic ones: workgroups per launch x threads per
    workgroup, and the fp32 partials' group budget.  Per point the best of
    3 runs of `steps` back-to-back reduce-scatters (HIP events, current
    stream), in microseconds per reduce-scatter."""
    import torch
    R = len(x)
    n = x[0].size // R
    send = [bf16_dev(a) for a in x]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]

    def run():
        for _ in range(5):
            hc.reduce_scatter(send, recv)
        torch.cuda.synchronize()
        best = None
        for _ in range(3):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(steps):
                hc.reduce_scatter(send, recv)
            b.record()
            b.synchronize()
            t = a.elapsed_time(b) / steps * 1e3
            best = t if best is None else min(best, t)
        return round(best, 2)
    shapes, groups = {}, {}
    for w in (0, 1024, 4096, 8192):
        for t in (256, 512, 1024):
            with hc.config(reduce_algo="ring", workgroups_per_step=w, threads_per_workgroup=t):
                shapes[f"{'auto' if w == 0 else w}x{t}"] = run()
    for g, name in ((0, "default"), ((1 << 64) - 1, "one_group"), (32 << 20, "32MiB"), (64 << 20, "64MiB"),
                    (128 << 20, "128MiB")):
        with hc.config(reduce_algo="ring", ring_group_bytes=g):
            groups[name] = run()
    return dict(workload="the headline ring reduce-scatter (bf16, R=8, 25,165,824 elements per rank), "
                         "us per reduce-scatter", workgroups_x_threads=shapes, ring_group_bytes=groups)


def back_to_back_time(fn, reps, warmup=3, runs=3):
    """Device time per call of `reps` calls enqueued back to back between two
    HIP events on the current stream, as the headline is timed (the host's
    launch latency overlaps the previous call); the best of `runs`."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    best = None
    for _ in range(runs):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        b.synchronize()
        t = a.elapsed_time(b) / 1e3 / reps
        best = t if best is None else min(best, t)
    return best


def bench_rs_variants(hc, reps):
    """The ring reduce-scatter beyond the headline: the same 25,165,824
    elements per rank in fp32 and int32 (12 bytes per element per step), and
    bf16 at R = 2 ... 64 virtual ranks with the same bytes per rank.  Timed
    back to back like the headline: at R = 2 one call is a single 27 us
    launch, and timing calls one by one would add the host's launch latency
    to it."""
    import torch
    n_in = 25_165_824
    out = {"dtypes": {}, "ranks": {}}

    def run(send, recv, R, dt_bytes):
        med = back_to_back_time(lambda: hc.reduce_scatter(send, recv), reps)
        st = hc.last_stats()
        return dict(ms=round(med * 1e3, 4), algbw_GBs=round(n_in * dt_bytes / med / 1e9, 1),
                    hbm_TBs=round(st["hbm_bytes_algorithmic"] / med / 1e12, 3),
                    hbm_frac=round(st["hbm_bytes_algorithmic"] / med / 1e9 / HBM_PEAK_GBS, 4),
                    launches=st["reduce_launches"])
    for name, dtype in (("fp32", torch.float32), ("int32", torch.int32)):
        R = 8
        if dtype == torch.int32:
            send = [torch.randint(-1000, 1000, (n_in,), dtype=dtype, device="cuda") for _ in range(R)]
        else:
            send = [torch.randn(n_in, device="cuda") for _ in range(R)]
        recv = [torch.empty(n_in // R, dtype=dtype, device="cuda") for _ in range(R)]
        out["dtypes"][name] = run(send, recv, R, 4)
        del send, recv
    for R in (2, 4, 16, 32, 64):
        n = n_in // R
        send = [torch.randn(R * n, device="cuda").to(torch.bfloat16) for _ in range(R)]
        recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
        out["ranks"][f"R{R}"] = run(send, recv, R, 2)
        del send, recv
        torch.cuda.empty_cache()
    out["workload"] = ("ring reduce-scatter, 25,165,824 elements per rank: fp32 and int32 at R=8; "
                       "bf16 at other R (the headline is bf16 at R=8)")
    return out


def bench_fused_hops(hc, send_np, steps, warmup):
    """The headline ring reduce-scatter with k ring hops folded per launch
    (fused_hops = k; k = 7 folds a whole chunk in one launch): algorithmic
    bytes against time.  Per point: HIP events on the launching stream over
    `steps` back-to-back calls, as for the headline, and per-launch kernel
    times from the library's kernel timing."""
    import torch
    R = len(send_np)
    n = send_np[0].size // R
    send = [bf16_dev(a) for a in send_np]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    stream = torch.cuda.current_stream()
    out = {}
    for k in (1, 2, 4, 7):
        with hc.config(reduce_algo="ring", fused_hops=k, kernel_timing=0):
            def step():
                hc.reduce_scatter(send, recv, stream=stream)
            for _ in range(warmup):
                step()
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(steps):
                step()
            e1.record(stream)
            torch.cuda.synchronize()
            st = hc.last_stats()
            t = e0.elapsed_time(e1) / 1e3 / steps
            hc.set_config(kernel_timing=1)
            hc.kernel_times()
            for _ in range(10):
                step()
            kt = hc.kernel_times()
            hc.set_config(kernel_timing=0)
        b = st["hbm_bytes_algorithmic"]
        L = st["reduce_launches"]
        out[f"k{k}"] = dict(hops_per_launch=k, launches=L, bytes_per_op=b,
                            bytes_per_element=round(b / (R * n), 3), us=round(t * 1e6, 2),
                            algbw_GBs=round(R * n * 2 / t / 1e9, 1), achieved_GBs=round(b / t / 1e9, 1),
                            frac=round(b / t / 1e9 / HBM_PEAK_GBS, 4),
                            launch_us=[round(statistics.mean(kt[i::L]) * 1e3, 2) for i in range(L)])
    return dict(workload="ring reduce-scatter bf16 R=8, 25,165,824 elements per rank, k ring hops "
                         "folded per launch (bit-identical to k = 1)", **out)


def bench_bf16_partials(hc, send_np, steps, warmup, samples=8192):
    """The headline reduce-scatter with bf16 partials (every hop's sum
    rounded to bf16) against fp32 partials (one rounding), on the ring and
    the direct fold: time per call (HIP events on the launching stream over
    `steps` back-to-back calls), algorithmic bytes, and the error of sampled
    outputs against the exact fp64 sum, in units of 2^-8 * sum |x| (the
    bound of one bf16 rounding of the sum's magnitude)."""
    import numpy as np
    import torch
    R = len(send_np)
    n = send_np[0].size // R
    send = [bf16_dev(a) for a in send_np]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    stream = torch.cuda.current_stream()
    g = np.random.default_rng(5)
    ranks = g.integers(0, R, samples)
    idx = g.integers(0, n, samples)
    pos = ranks * n + idx
    vals = np.stack([((a.view(np.uint16)[pos].astype(np.uint32) << 16).view(np.float32))
                     for a in send_np]).astype(np.float64)     # R x samples
    exact = vals.sum(axis=0)
    scale = np.abs(vals).sum(axis=0) * 2.0 ** -8
    out = {}
    for algo, k in (("ring", 1), ("ring", 2), ("ring", 7), ("direct", 1)):
        for bp in (0, 1):
            with hc.config(reduce_algo=algo, bf16_partials=bp, fused_hops=k, kernel_timing=0):
                def step():
                    hc.reduce_scatter(send, recv, stream=stream)
                for _ in range(warmup):
                    step()
                torch.cuda.synchronize()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for _ in range(steps):
                    step()
                e1.record(stream)
                torch.cuda.synchronize()
                st = hc.last_stats()
            t = e0.elapsed_time(e1) / 1e3 / steps
            got = torch.stack(recv).float().cpu().numpy()[ranks, idx].astype(np.float64)
            err = np.abs(got - exact) / np.where(scale > 0, scale, 1.0)
            b = st["hbm_bytes_algorithmic"]
            label = algo if k == 1 else f"{algo}_k{k}"
            out[f"{label}_{'bf16' if bp else 'fp32'}_partials"] = dict(
                us=round(t * 1e6, 2), bytes_per_op=b, achieved_GBs=round(b / t / 1e9, 1),
                frac=round(b / t / 1e9 / HBM_PEAK_GBS, 4), launches=st["reduce_launches"],
                err_max=round(float(err.max()), 4), err_mean=round(float(err.mean()), 5))
    return dict(workload="reduce-scatter bf16 R=8, 25,165,824 elements per rank: bf16 partials "
                         "(rounded at every hop) against fp32 partials (rounded once), ring (one, "
                         "two or seven hops per launch: k2, k7) and direct fold; error of %d sampled "
                         "outputs against the exact sum, in units of 2^-8 * sum |x|" % samples, **out)


def bench_rs_graph(hc, send_np, steps):
    """The headline ring reduce-scatter captured ten steps at a time into a
    HIP graph and replayed, against the same steps issued eagerly on the
    same stream; the replayed results must equal the eager ones bit for
    bit."""
    import torch
    R = len(send_np)
    n = send_np[0].size // R
    send = [bf16_dev(a) for a in send_np]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    s = torch.cuda.Stream()

    def step():
        hc.reduce_scatter(send, recv, stream=s)

    def timed(fn, k):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(k):
            fn()
        e1.record(s)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / 1e3 / k

    with torch.cuda.stream(s):
        for _ in range(3):
            step()
        torch.cuda.synchronize()
        eager = timed(step, steps)
    ref = [t.clone() for t in recv]
    per_graph = 10
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for _ in range(per_graph):
            step()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        g.replay()
        torch.cuda.synchronize()
        replay = timed(g.replay, max(1, steps // per_graph)) / per_graph
    same = all(torch.equal(a.view(torch.int16), b.view(torch.int16)) for a, b in zip(ref, recv))
    S = R * n * 2
    return {"workload": "headline ring reduce-scatter, 10 steps per captured graph",
            "eager_us": round(eager * 1e6, 1), "graph_replay_us": round(replay * 1e6, 1),
            "eager_algbw_GBs": round(S / eager / 1e9, 1), "graph_algbw_GBs": round(S / replay / 1e9, 1),
            "same_bits": same}


def copy_ceiling(hc):
    """The measured streaming ceiling the reduction kernels are also judged
    against: the library's CU copy kernel at its automatic budget moving
    2 GiB (4 GiB of HBM traffic per copy), ten copies back to back between
    two events; 2 GiB per buffer keeps the data well outside the 256 MB
    last-level cache.  Returns HBM GB/s."""
    import torch
    src = torch.empty(1 << 29, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    with hc.config(copy_path="kernel", workgroups_per_step=0):
        for _ in range(2):
            hc.sendrecv([src, src], [dst, dst], [1, -1])
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(10):
            hc.sendrecv([src, src], [dst, dst], [1, -1])
        b.record()
        b.synchronize()
    t = a.elapsed_time(b) / 1e3 / 10
    del src, dst
    torch.cuda.empty_cache()
    return 2 * (1 << 31) / t / 1e9


def bench_after_free(hc, W):
    """The SDMA engines right after a large device-memory free, the
    caching-allocator case: torch's empty_cache (or any hipFree of a large
    allocation) hands memory back, and while the driver releases it one
    engine runs at about half rate.  Per workload on all 16 engines: every
    copy issued at once on its scheduled engine (proxy_slice_bytes =
    SIZE_MAX) against balanced issue with 4 MiB pieces (what the automatic
    setting picks for these sizes on 16 engines), settled (1.5 s after the
    last free) and in the first milliseconds after freeing 2 GiB.  Then each
    of four engines alone, settled and right after a free: which engine the
    release slows."""
    import numpy as np
    import torch
    MiB = 1 << 20
    SMAX = (1 << 64) - 1
    R = 8

    def one(fn):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        b.synchronize()
        return a.elapsed_time(b) / 1e3

    def free_2gib():
        F = [torch.empty(64 * MiB, dtype=torch.uint8, device="cuda") for _ in range(32)]
        torch.cuda.synchronize()
        time.sleep(0.3)
        del F
        torch.cuda.empty_cache()

    def measure(fn, per_rank, **cfg):
        with hc.config(proxy_timeout_ms=3000, **cfg):
            time.sleep(1.5)
            for _ in range(2):
                one(fn)
            steady = statistics.median(one(fn) for _ in range(7))
            free_2gib()
            after = statistics.median(one(fn) for _ in range(3))
        return dict(ms=round(steady * 1e3, 4), after_free_ms=round(after * 1e3, 4),
                    GBs_per_rank=round(per_rank / steady / 1e9, 1),
                    after_free_GBs_per_rank=round(per_rank / after / 1e9, 1))

    out = {}
    n = (1 << 30) // 4 // R
    x = W.ag_parameters(R)
    for name in ("allgather_1GiB", "alltoall_1GiB", "allgather_fsdp"):
        if name == "allgather_1GiB":
            send = [torch.full((n,), r, dtype=torch.int32, device="cuda") for r in range(R)]
            recv = [torch.empty(R * n, dtype=torch.int32, device="cuda") for _ in range(R)]
            fn, per_rank = (lambda: hc.allgather(send, recv)), R * n * 4
        elif name == "alltoall_1GiB":
            send = [torch.full((R * n,), r, dtype=torch.int32, device="cuda") for r in range(R)]
            recv = [torch.empty(R * n, dtype=torch.int32, device="cuda") for _ in range(R)]
            fn, per_rank = (lambda: hc.alltoall(send, recv)), R * n * 4
        else:
            send = [bf16_dev(a) for a in x]
            recv = [torch.empty(R * x[0].size, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
            fn, per_rank = (lambda: hc.allgather(send, recv)), R * x[0].size * 2
        row = {}
        for mode, sl in (("static", SMAX), ("balanced", 4 * MiB)):
            row[mode] = measure(fn, per_rank, copy_path="engines", sdma_engines=16, proxy_slice_bytes=sl)
        log(f"  after free, {name}: static {row['static']['ms']} / {row['static']['after_free_ms']} ms, "
            f"balanced {row['balanced']['ms']} / {row['balanced']['after_free_ms']} ms")
        out[name] = row
        del send, recv
        torch.cuda.empty_cache()
    # Which engine: each alone (the proxy restricted to it), 256 MiB copies.
    saved = hc.get_config()
    src = torch.empty(64 * MiB, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    engines = {}
    try:
        for eng in (0, 1, 5, 14):
            os.environ["HOCCL_SDMA_ENGINE_IDS"] = str(eng)
            hc.finalize()
            hc.init(0)
            r = measure(lambda: hc.sendrecv([src, src], [None, dst], [1, -1]), 256 * MiB,
                        copy_path="engines", sdma_engines=1)
            engines[str(eng)] = dict(GBs=r["GBs_per_rank"], after_free_GBs=r["after_free_GBs_per_rank"])
    finally:
        os.environ.pop("HOCCL_SDMA_ENGINE_IDS", None)
        hc.finalize()
        hc.init(0)
        hc.set_config(**saved)
    out["single_engine_256MiB"] = engines
    # What one engine command costs: 64 MiB on one engine as N commands,
    # every copy issued at once (no balanced issue, no gaps).
    cost = {}
    with hc.config(copy_path="engines", sdma_engines=1, proxy_slice_bytes=SMAX):
        for nc in (1, 4, 16, 64):
            with hc.config(chunk_bytes=(64 * MiB) // nc):
                f = lambda: hc.sendrecv([src[:16 * MiB], src[:16 * MiB]], [None, dst[:16 * MiB]], [1, -1])
                for _ in range(2):
                    one(f)
                cost[str(nc)] = round(statistics.median(one(f) for _ in range(9)) * 1e6, 1)
    out["one_engine_64MiB_us_by_commands"] = cost
    del src, dst
    torch.cuda.empty_cache()
    time.sleep(1.5)
    # The default engine budget (4 engines, which the release never slows,
    # and which issues every copy at once by default): what balanced issue
    # would cost or gain there, settled.
    dflt = {}
    send_np, counts, sd, rd, rsz = W.a2a_tokens(R)
    ep_s = [bf16_dev(a) for a in send_np]
    ep_r = [torch.zeros(q, dtype=torch.bfloat16, device="cuda") for q in rsz]
    pp_s = [torch.full((2048 * 4096,), r, dtype=torch.int32, device="cuda") for r in range(R)]
    pp_r = [torch.zeros(2048 * 4096, dtype=torch.int32, device="cuda") for _ in range(R)]
    fwd = [r + 1 if r + 1 < R else -1 for r in range(R)]
    fs = [bf16_dev(a) for a in x]
    fr = [torch.empty(R * x[0].size, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    for name, fn in (("sendrecv_32MiB", lambda: hc.sendrecv([pp_s[0], pp_s[0]], [None, pp_r[1]], [1, -1])),
                     ("pp_round_7x32MiB", lambda: hc.sendrecv(pp_s, pp_r, fwd)),
                     ("ep_alltoallv", lambda: hc.alltoallv(ep_s, counts, sd, ep_r, rd)),
                     ("allgather_fsdp", lambda: hc.allgather(fs, fr))):
        row = {}
        for mode, sl in (("static", SMAX), ("balanced", 4 * MiB)):
            with hc.config(copy_path="engines", sdma_engines=0, proxy_slice_bytes=sl):
                for _ in range(2):
                    one(fn)
                row[mode + "_ms"] = round(statistics.median(one(fn) for _ in range(11)) * 1e3, 4)
        dflt[name] = row
    out["default_budget_settled"] = dflt
    del ep_s, ep_r, pp_s, pp_r, fs, fr
    torch.cuda.empty_cache()
    time.sleep(1.5)
    out["workload"] = ("R=8 on all 16 SDMA engines: all-gather and all-to-all with 1 GiB per rank (int32), "
                       "the FSDP all-gather (bf16, 25,165,824-element shards); settled, then right after "
                       "freeing 2 GiB (the median of the first 3 calls); GB/s = bytes each rank receives "
                       "over time.  default_budget_settled: the automatic 4 engines, a 32 MiB send/recv, one "
                       "pipeline round of seven 32 MiB messages, the EP all-to-all(v), the FSDP all-gather")
    return out


def bench_callback_thread(hc, reps=5):
    """What the host-function handshake does to other host callbacks.  An
    all-gather on the engine proxy (AUTO: host-function handshake) is
    enqueued on stream 1, then a host function on stream 2, which has no
    other work, and a host function on stream 1 after the all-gather.  The
    host functions record when they run (host clock).  If stream 2's
    callback runs only once the all-gather's handshake has returned, the
    two share the HIP runtime's callback thread.  Control: the same stream-2
    callback with stream 1 idle.  All times in us from stream 2's enqueue."""
    import ctypes
    import torch
    hip = ctypes.CDLL("libamdhip64.so.7")    # the HIP runtime torch has loaded
    CB = ctypes.CFUNCTYPE(None, ctypes.c_void_p)
    hip.hipLaunchHostFunc.argtypes = [ctypes.c_void_p, CB, ctypes.c_void_p]
    stamps = {}

    def mk(key):
        return CB(lambda _arg: stamps.__setitem__(key, time.perf_counter()))
    cb2, cb1 = mk("other_stream"), mk("after_allgather")
    R, n = 8, 1 << 23                         # 16 MiB shards: 56 copies of 16 MiB
    send = [torch.randn(n, device="cuda").to(torch.bfloat16) for _ in range(R)]
    recv = [torch.empty(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    rows = {"busy": [], "idle": []}
    hc.allgather(send, recv, stream=s1)
    torch.cuda.synchronize()
    for _ in range(reps):
        for case in ("busy", "idle"):
            stamps.clear()
            if case == "busy":
                hc.allgather(send, recv, stream=s1)
                assert hip.hipLaunchHostFunc(ctypes.c_void_p(s1.cuda_stream), cb1, None) == 0
            t0 = time.perf_counter()
            assert hip.hipLaunchHostFunc(ctypes.c_void_p(s2.cuda_stream), cb2, None) == 0
            # Poll with sleeps (which release the interpreter lock the
            # callbacks need) rather than block in a synchronisation.
            while not (s1.query() and s2.query()) and time.perf_counter() - t0 < 10:
                time.sleep(20e-6)
            torch.cuda.synchronize()
            rows[case].append({k: round((v - t0) * 1e6, 1) for k, v in stamps.items()})
    # Does the proxy's polling of copy gates (hipEventQuery) need that
    # thread?  A ring all-reduce whose gather copies the proxy starts on gate
    # events, with the handshake kernel (no host function of its own), on
    # stream 2 while a host function on stream 1 holds the callback thread
    # for 5 ms (sleeping: no engine and no CU is used); its device time
    # against the same all-reduce alone.
    hold = CB(lambda _arg: time.sleep(0.005))
    ar_send = [torch.randn(1 << 23, device="cuda").to(torch.bfloat16) for _ in range(R)]
    ar_recv = [torch.empty_like(t) for t in ar_send]
    gate_rows = {"busy": [], "idle": []}

    def ar():
        with hc.config(reduce_algo="ring", allreduce_chunk_groups=2, proxy_handshake=0):
            hc.allreduce(ar_send, ar_recv, stream=s2)
    ar()
    torch.cuda.synchronize()
    for _ in range(reps):
        for case in ("busy", "idle"):
            if case == "busy":
                assert hip.hipLaunchHostFunc(ctypes.c_void_p(s1.cuda_stream), hold, None) == 0
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s2)
            ar()
            e1.record(s2)
            t0 = time.perf_counter()
            while not (s1.query() and s2.query()) and time.perf_counter() - t0 < 10:
                time.sleep(20e-6)
            torch.cuda.synchronize()
            gate_rows[case].append(round(e0.elapsed_time(e1) * 1e3, 1))
    # Do ROCr's asynchronous signal handlers (hsa_amd_signal_async_handler,
    # which is how a tool completes a copy it traces) run on that thread
    # too?  A handler registered on a fresh signal, the signal set while a
    # host function holds the callback thread for 5 ms: when does it fire?
    hsa = ctypes.CDLL("libhsa-runtime64.so.1")

    class Sig(ctypes.Structure):
        _fields_ = [("handle", ctypes.c_uint64)]
    HANDLER = ctypes.CFUNCTYPE(ctypes.c_bool, ctypes.c_int64, ctypes.c_void_p)
    hsa.hsa_signal_create.argtypes = [ctypes.c_int64, ctypes.c_uint32, ctypes.c_void_p, ctypes.POINTER(Sig)]
    hsa.hsa_amd_signal_async_handler.argtypes = [Sig, ctypes.c_int, ctypes.c_int64, HANDLER, ctypes.c_void_p]
    hsa.hsa_signal_store_screlease.argtypes = [Sig, ctypes.c_int64]
    hsa.hsa_signal_destroy.argtypes = [Sig]
    fired = {}
    handler = HANDLER(lambda _v, _a: (fired.__setitem__("t", time.perf_counter()), False)[1])
    began = {}
    hold2 = CB(lambda _arg: (began.__setitem__("t", time.perf_counter()), time.sleep(0.005)))
    hsa_rows = {"busy": [], "idle": []}
    for _ in range(reps):
        for case in ("busy", "idle"):
            sig = Sig()
            assert hsa.hsa_signal_create(1, 0, None, ctypes.byref(sig)) == 0
            fired.clear()
            began.clear()
            assert hsa.hsa_amd_signal_async_handler(sig, 0, 0, handler, None) == 0  # EQ 0
            if case == "busy":
                assert hip.hipLaunchHostFunc(ctypes.c_void_p(s1.cuda_stream), hold2, None) == 0
                t0 = time.perf_counter()
                while "t" not in began and time.perf_counter() - t0 < 10:
                    time.sleep(20e-6)
            t_set = time.perf_counter()
            hsa.hsa_signal_store_screlease(sig, 0)
            while "t" not in fired and time.perf_counter() - t_set < 10:
                time.sleep(20e-6)
            while not s1.query() and time.perf_counter() - t_set < 10:
                time.sleep(20e-6)
            torch.cuda.synchronize()
            hsa_rows[case].append(round((fired.get("t", float("nan")) - t_set) * 1e6, 1))
            hsa.hsa_signal_destroy(sig)
    med = lambda xs: round(statistics.median(xs), 1)
    busy_other = med([r["other_stream"] for r in rows["busy"]])
    busy_end = med([r["after_allgather"] for r in rows["busy"]])
    return dict(workload="host function on an idle stream while an engine-path all-gather (8 x 16 MiB "
                         "shards, host-function handshake) runs on another",
                other_stream_callback_us=busy_other, allgather_done_callback_us=busy_end,
                idle_control_callback_us=med([r["other_stream"] for r in rows["idle"]]),
                other_waited_for_allgather=bool(busy_other >= 0.5 * busy_end), runs=rows,
                gated_allreduce_us=dict(beside_held_callback_thread=med(gate_rows["busy"]),
                                        alone=med(gate_rows["idle"]), runs=gate_rows),
                hsa_async_handler_us=dict(beside_5ms_host_function=med(hsa_rows["busy"]),
                                          alone=med(hsa_rows["idle"]), runs=hsa_rows))


def bench_small_message(hc, reps, gemm=None):
    """Latency of one 4 KiB send/recv (rank 0 -> 1) through each copy path:
    the engine proxy's flag handshake (host function, and the one-lane
    kernel), the HIP runtime's copy, and the CU copy kernel; plus the host
    time of the call.  With `gemm`: the slowdown of the bf16 GEMM beside a
    loop of 40 such messages on the engines, per handshake form (why AUTO
    keeps the host function, whose copies need no CU, although the kernel
    form's round trip is shorter)."""
    import torch
    src = torch.zeros(2048, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    out = {}
    for name, kw in PATHS:
        hc.set_config(**kw)
        med, mn = event_time(lambda: hc.sendrecv([src, src], [dst, dst], [1, -1]), reps, warmup=5)
        host = []
        for _ in range(reps):
            t0 = time.perf_counter()
            hc.sendrecv([src, src], [dst, dst], [1, -1])
            host.append(time.perf_counter() - t0)
            torch.cuda.synchronize()
        out[name] = dict(device_us=round(med * 1e6, 2), device_min_us=round(mn * 1e6, 2),
                         host_call_us=round(statistics.median(host) * 1e6, 2))
    hc.set_config(copy_path="auto", proxy_handshake=-1)
    if gemm is not None:
        loop = {}
        for name, hs in (("host_function", 2), ("kernel", 0)):
            with hc.config(copy_path="engines", proxy_handshake=hs):
                run = lambda st: [hc.sendrecv([src, src], [dst, dst], [1, -1], stream=st) for _ in range(40)]
                med, _ = event_time(lambda: run(None), 3)
                row = interference(hc, run, med, gemm, pairs=60)
            loop[name] = dict(ms_per_40=round(med * 1e3, 3), gemm_slowdown=row["gemm_slowdown"],
                              gemm_slowdown_ci95=row["gemm_slowdown_ci95"])
        out["loop_of_40_beside_gemm"] = loop
    return dict(workload="one 4 KiB message rank 0 -> 1 (stream-manager round trip)", **out)


def bench_rs_workgroups(hc, x, reps, gemm=None):
    """Ring reduce-scatter of the headline at a fixed workgroup budget: the
    CU footprint / bandwidth trade-off of the reduction kernels, and, with
    `gemm`, the slowdown of a bf16 8192^3 GEMM running beside it."""
    import torch
    R = len(x)
    n = x[0].size // R
    send = [bf16_dev(a) for a in x]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    out = {}
    for w in (8, 16, 64, 256, 1024, 0):
        hc.set_config(workgroups_per_step=w)
        med, _ = event_time(lambda: hc.reduce_scatter(send, recv), reps)
        st = hc.last_stats()
        row = dict(ms=round(med * 1e3, 4), algbw_GBs=round(R * n * 2 / med / 1e9, 2),
                   hbm_GBs=round(st["hbm_bytes_algorithmic"] / med / 1e9, 1),
                   cus_used=st["cus_used_max"])
        if gemm is not None:
            row.update(interference(hc, lambda s: hc.reduce_scatter(send, recv, stream=s), med, gemm,
                                    pairs=20))
        out[f"wg{st['workgroups_per_step']}"] = row
    hc.set_config(workgroups_per_step=0)
    return out


def bench_cu_partition(hc, x, gemm):
    """CUs set aside for the reduction, the analog of a collective library
    that owns a fixed set of SMs: the GEMM's stream is masked to the other
    CUs, and the headline ring reduce-scatter runs with K workgroups per
    step on a stream masked to K CUs of its own (two or four per XCD).
    Reports the masked GEMM alone against the full chip, the reduction alone
    on its K CUs, and the gated pair: the GEMM against the masked GEMM
    alone, the reduction against itself alone."""
    import torch
    R = len(x)
    n = x[0].size // R
    send = [bf16_dev(a) for a in x]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    A, B, C, t_full = gemm[:4]
    out = {"gemm_full_chip_ms": round(t_full * 1e3, 4)}
    for K in (16, 32):
        gs, cs = masked_stream(range(K, ncu)), masked_stream(range(K))
        if gs is None or cs is None:
            out[f"cus{K}"] = {"error": "CU mask refused"}
            continue
        _, _, ts = _gemm_run((A, B, C, 0.0, gs, cs))
        torch.cuda.synchronize()
        t_masked = statistics.median(a.elapsed_time(b) for a, b in ts) / 1e3
        g2 = (A, B, C, t_masked, gs, cs)
        with hc.config(workgroups_per_step=K):
            with torch.cuda.stream(cs):
                med, _ = event_time(lambda: hc.reduce_scatter(send, recv, stream=cs), 5)
            row = dict(gemm_masked_ms=round(t_masked * 1e3, 4),
                       gemm_cost_of_the_mask=round(t_masked / t_full - 1, 4),
                       reduce_scatter_alone_ms=round(med * 1e3, 4))
            row.update(interference(hc, lambda s: hc.reduce_scatter(send, recv, stream=s), med, g2,
                                    pairs=20))
        out[f"cus{K}"] = row
    return dict(workload="headline ring reduce-scatter on K reserved CUs (K workgroups per step) beside "
                         "a bf16 8192^3 GEMM masked to the other CUs", **out)


def size_sweep(hc):
    """algbw against message size, 2 MiB .. 1 GiB, as in the paper's
    microbenchmarks: send/recv (one message 0 -> 1), all-gather and
    all-to-all over R = 8 (size = bytes each rank receives), per copy path,
    and the CU copy kernel at 8 and 256 workgroups."""
    import torch
    R = 8
    sizes = [2 << 20, 8 << 20, 32 << 20, 128 << 20, 512 << 20, 1 << 30]
    paths = [("hip", {"copy_path": "hip"}), ("engines", {"copy_path": "engines"}),
             ("engines16", {"copy_path": "engines", "sdma_engines": 16}),
             ("kernel_wg8", {"copy_path": "kernel", "workgroups_per_step": 8}),
             ("kernel_wg256", {"copy_path": "kernel", "workgroups_per_step": 256})]
    out = {"sendrecv": [], "allgather": [], "alltoall": []}
    big = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    big2 = torch.empty_like(big)
    # Two passes, the second kept: the first engine copies of a fresh
    # process ran slow for some milliseconds (the single-message benchmark
    # saw the same transient).
    for _ in range(2):
        out["sendrecv"] = []
        for sz in sizes:
            row = {"bytes": sz}
            for name, kw in paths:
                hc.set_config(**kw)
                s0, d1 = big[:sz].view(torch.int32), big2[:sz].view(torch.int32)
                med, _ = event_time(lambda: hc.sendrecv([s0, s0], [d1, d1], [1, -1]), 5)
                row[name] = round(sz / med / 1e9, 1)
                hc.set_config(copy_path="auto", workgroups_per_step=0, sdma_engines=0)
            out["sendrecv"].append(row)
    del big, big2
    for op in ("allgather", "alltoall"):
        for sz in sizes:
            n = sz // 4 // R
            send = [torch.zeros(n if op == "allgather" else R * n, dtype=torch.int32, device="cuda")
                    for _ in range(R)]
            recv = [torch.empty(R * n, dtype=torch.int32, device="cuda") for _ in range(R)]
            row = {"bytes": R * n * 4}
            for name, kw in paths:
                hc.set_config(**kw)
                fn = (lambda: hc.allgather(send, recv)) if op == "allgather" else \
                     (lambda: hc.alltoall(send, recv))
                med, _ = event_time(fn, 3, warmup=1)
                row[name] = round(R * n * 4 / med / 1e9, 1)
                hc.set_config(copy_path="auto", workgroups_per_step=0, sdma_engines=0)
            out[op].append(row)
            del send, recv
            torch.cuda.empty_cache()
    # Reduce-scatter, bf16, R = 8 (size = each rank's input): the ring at the
    # automatic budget and at 8 workgroups, and the direct fold.
    out["reduce_scatter"] = []
    for sz in sizes:
        n = sz // 2 // R
        send = [torch.zeros(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
        recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
        row = {"bytes": R * n * 2}
        for name, kw in (("ring", {"reduce_algo": "ring"}),
                         ("ring_wg8", {"reduce_algo": "ring", "workgroups_per_step": 8}),
                         ("direct", {"reduce_algo": "direct"})):
            with hc.config(**kw):
                med, _ = event_time(lambda: hc.reduce_scatter(send, recv), 3, warmup=1)
            row[name] = round(R * n * 2 / med / 1e9, 1)
        out["reduce_scatter"].append(row)
        del send, recv
        torch.cuda.empty_cache()
    return out


TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "reduce_step_kernel_rs_bf16_R8_traffic.txt")
FOLD_TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "fold_kernel_rs_bf16_R8_traffic.txt")


def kernel_source_hash():
    """SHA-256 (16 hex digits) of the kernels' source (kernels.hip and the
    header with their argument structs) without // comments and blank
    lines: any change to the code voids the committed counter figures, an
    edit of a comment does not."""
    import hashlib
    import re
    lines = []
    for name in ("kernels.hip", "hoccl_internal.h"):
        with open(os.path.join(ROOT, "paper_2609_34334_amd", "csrc", name), encoding="utf-8") as f:
            lines += [re.sub(r"//.*", "", line).rstrip() for line in f]
    code = "\n".join(line for line in lines if line)
    return hashlib.sha256(code.encode()).hexdigest()[:16]


CEILINGS_SUMMARY = os.path.join(ROOT, "profiles", "stream_ceilings_kernel_durations.txt")
TRAFFIC_NOTE = ("FETCH_SIZE + WRITE_SIZE: bytes crossing the L2-to-fabric boundary, scaled by a 1 GiB copy; "
                "an upper bound on HBM bytes, since no counter separates what the 256 MB Infinity Cache "
                "behind that boundary serves (the DRAM-destined request counters read the same)")


def stream_ceilings():
    """Kernel-time streaming ceilings (GB/s moved) at the 2 GiB operand size
    from the committed profile summary, or None."""
    if not os.path.exists(CEILINGS_SUMMARY):
        return None
    for line in open(CEILINGS_SUMMARY):
        if line.startswith("| 2048 MiB |"):
            cells = [c.strip().split()[0] for c in line.strip().strip("|").split("|")[1:]]
            return dict(zip(("read", "write", "copy", "copy_nt_stores", "two_reads_one_write",
                             "two_reads_one_write_nt_stores", "in_place_rmw"), (float(c) for c in cells)))
    return None


def measured_traffic(summary=TRAFFIC_SUMMARY, key="traffic_bytes_per_launch"):
    """Bytes per launch from a committed rocprofv3 counter summary (`key`:
    FETCH_SIZE + WRITE_SIZE by default), or None when it is missing or the
    kernels changed since."""
    if not os.path.exists(summary):
        return None
    kv = {}
    for line in open(summary):
        if ":" in line and not line.startswith(("#", " ", "|")):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    try:
        return int(float(kv[key]))
    except (KeyError, ValueError):
        return None


def copy_workload(hc, W):
    """What the copy-path kernel trace profiles: the FSDP all-gather, the EP
    all-to-all(v) and one PP send/recv round, once each on the default (AUTO)
    copy path, after the inputs are resident.  Under a profiler AUTO's
    engine proxy uses its one-lane handshake kernel, which the trace shows;
    the copies themselves are SDMA commands.  Whether copies need CUs is
    shown by tests/test_gpu_zero_cu.py, not by a trace."""
    import torch
    R = 8
    ag = [bf16_dev(a) for a in W.ag_parameters(R)]
    send_np, counts, sd, rd, rsz = W.a2a_tokens(R)
    a2a = [bf16_dev(a) for a in send_np]
    a2a_out = [torch.empty(s, dtype=torch.bfloat16, device="cuda") for s in rsz]
    act = [bf16_dev(a) for a in W.p2p_activations(R)]
    act_out = [torch.empty_like(t) for t in act]
    torch.cuda.synchronize()
    marker = torch.cuda.Event()
    hc.set_config(copy_path="auto")
    ag_out = hc.allgather(ag)
    hc.alltoallv(a2a, counts, sd, a2a_out, rd)
    hc.sendrecv(act, act_out, [r + 1 if r + 1 < R else -1 for r in range(R)])
    marker.record()
    torch.cuda.synchronize()
    print(json.dumps({"copy_workload": "done", "copy_ops": hc.last_stats()["copy_ops"],
                      "allgather_bytes": sum(t.numel() * 2 for t in ag_out)}))


def ar_groups_workload(hc, W):
    """What the all-reduce overlap trace profiles: the bf16 R=8 bucket
    all-reduce (25,165,824 elements per rank) in 2 chunk groups on the
    engine proxy, three calls after one warm-up.  The trace shows group 1's
    ring-step launches running while the engines copy group 0."""
    import torch
    R, n = 8, 25_165_824
    send = [bf16_dev(a) for a in W.rs_gradients(R, n)]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    hc.set_config(copy_path="engines", allreduce_chunk_groups=2)
    hc.allreduce(send, recv)
    torch.cuda.synchronize()
    for _ in range(3):
        hc.allreduce(send, recv)
    torch.cuda.synchronize()
    print(json.dumps({"ar_groups_workload": "done", "copy_ops": hc.last_stats()["copy_ops"],
                      "reduce_launches": hc.last_stats()["reduce_launches"]}))


def pmc_workload(hc, W):
    """What the counter runs profile: a 1 GiB CU copy of known size (to
    scale FETCH_SIZE / WRITE_SIZE), then five headline reduce-scatters on
    the ring, five with the direct fold, and five each with 2 and 4 ring
    hops fused per launch."""
    import torch
    src = torch.empty(1 << 28, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    with hc.config(copy_path="kernel"):
        hc.sendrecv([src], [dst], [0])
    torch.cuda.synchronize()
    del src, dst
    R, n_in = 8, 25_165_824
    send = [bf16_dev(a) for a in W.rs_gradients(R, n_in)]
    recv = [torch.empty(n_in // R, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    for _ in range(5):
        hc.reduce_scatter(send, recv)
    with hc.config(reduce_algo="direct"):
        for _ in range(5):
            hc.reduce_scatter(send, recv)
    for k in (2, 4):
        with hc.config(reduce_algo="ring", fused_hops=k):
            for _ in range(5):
                hc.reduce_scatter(send, recv)
    torch.cuda.synchronize()
    print(json.dumps({"pmc_workload": "done", "kernel_source_sha256_16": kernel_source_hash()}))


def ceilings_workload(hc, sizes=(64 << 20, 128 << 20, 256 << 20, 2 << 30), reps=50):
    """The memory system's streaming ceilings (hoccl_debug_stream_ceiling):
    read only, write only, copy, two reads and a write (fp32 add), the two
    with non-temporal stores too, and an in-place fp32 read-modify-write,
    per operand size: 64, 128 and 256 MiB,
    which the 256 MB Infinity Cache holds once warm, and 2 GiB, which it
    cannot.  Each: 3 warm-up launches, then `reps` back-to-back launches
    between two events (per-launch time includes the launch gap; the
    rocprofv3 trace of this workload gives kernel time alone).  GB/s of
    bytes moved (read + written)."""
    import torch
    big = max(sizes)
    A = torch.zeros(big, dtype=torch.uint8, device="cuda")
    B = torch.zeros(big, dtype=torch.uint8, device="cuda")
    C = torch.zeros(big, dtype=torch.uint8, device="cuda")
    out = {}
    for size in sizes:
        row = {}
        for mode in ("read", "write", "copy", "copy_nt", "add", "add_nt", "rmw"):
            a = A[:size] if mode in ("read", "copy", "copy_nt", "add", "add_nt") else None
            b = B[:size] if mode in ("add", "add_nt") else None
            c = C[:size]

            def fn():
                hc.stream_ceiling(mode, a, b, c, nbytes=size)
            for _ in range(3):
                fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            t = e0.elapsed_time(e1) / 1e3 / reps
            moved = hc.last_stats()["hbm_bytes_algorithmic"]
            row[mode] = dict(us=round(t * 1e6, 2), GBs=round(moved / t / 1e9, 1))
        out[f"{size >> 20}MiB"] = row
        log(f"  ceilings {size >> 20} MiB: " + ", ".join(f"{m} {v['GBs']}" for m, v in row.items()))
    return out


def occupancy_workload(hc, W):
    """What the occupancy counter pass profiles, in this order: the headline
    reduce-scatter three times at each workgroup budget 8, 16, 64, 256 and
    automatic (7 ring-step launches each), then a 512 MiB CU-kernel copy at
    8 workgroups and at the automatic budget."""
    import torch
    R, n_in = 8, 25_165_824
    send = [bf16_dev(a) for a in W.rs_gradients(R, n_in)]
    recv = [torch.empty(n_in // R, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    budgets = [8, 16, 64, 256, 0]
    for wg in budgets:
        with hc.config(workgroups_per_step=wg):
            for _ in range(3):
                hc.reduce_scatter(send, recv)
    torch.cuda.synchronize()
    del send, recv
    src = torch.empty(1 << 27, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    for wg in (8, 0):
        with hc.config(copy_path="kernel", workgroups_per_step=wg):
            hc.sendrecv([src], [dst], [0])
    torch.cuda.synchronize()
    print(json.dumps({"occupancy_workload": "done", "rs_budgets": budgets, "copy_budgets": [8, 0],
                      "kernel_source_sha256_16": kernel_source_hash()}))


def copy_kernel_workload(hc, W):
    """The CU copy kernel on the copy workloads, back to back (median of
    HIP events per call): a 2 GiB and a 64 MiB copy, the FSDP all-gather,
    the PP schedule (32 rounds of seven 16 MiB hops) and the EP
    all-to-all(v), all on copy path `kernel`.  Run once per build of the
    kernel's knobs (HOCCL_COPY_UNROLL, HOCCL_COPY_NT_IN, HOCCL_COPY_NT_OUT)
    to compare them."""
    import torch
    res = {}
    hc.set_config(copy_path="kernel")

    def t(label, fn, reps=20):
        med, _ = event_time(fn, reps)
        res[label] = round(med * 1e6, 1)
    a = torch.empty(1 << 30, dtype=torch.bfloat16, device="cuda")
    b = torch.empty_like(a)
    t("copy_2GiB_us", lambda: hc.sendrecv([a, a], [b, b], [1, -1]))
    a2, b2 = a[:1 << 25], b[:1 << 25]
    t("copy_64MiB_us", lambda: hc.sendrecv([a2, a2], [b2, b2], [1, -1]), 50)
    del a, b, a2, b2
    R, total = 8, 201_326_592
    send = [bf16_dev(v) for v in W.ag_parameters(R, total)]
    recv = [torch.empty(total, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    t("fsdp_allgather_us", lambda: hc.allgather(send, recv))
    del send, recv
    ps = [bf16_dev(v) for v in W.p2p_activations(R)]
    pr = [torch.empty_like(v) for v in ps]
    fwd, bwd = [r + 1 if r + 1 < R else -1 for r in range(R)], [r - 1 for r in range(R)]

    def pp():
        for _ in range(16):
            hc.sendrecv(ps, pr, fwd)
            hc.sendrecv(ps, pr, bwd)
    t("pp_schedule_us", pp, 5)
    s_np, counts, sd, rd, rsz = W.a2a_tokens(R)
    asend = [bf16_dev(v) for v in s_np]
    arecv = [torch.empty(z, dtype=torch.bfloat16, device="cuda") for z in rsz]
    t("ep_alltoallv_us", lambda: hc.alltoallv(asend, counts, sd, arecv, rd))
    return res


def backend_rank():
    """One rank of --backend-workload (started by torchrun with
    HOCCL_BACKEND=1): per-call host time of the torch.distributed backend,
    rank 0 printing one JSON line."""
    from datetime import timedelta

    import torch
    import torch.distributed as dist

    from paper_2609_34334_amd import distributed as hdist
    rank, R = int(os.environ["RANK"]), int(os.environ["WORLD_SIZE"])
    torch.cuda.set_device(0)
    hdist.init_process_group(backend="nccl", timeout=timedelta(seconds=60))
    reps, out = 50, {"ranks": R}

    def per_call(fn):
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        return round((time.perf_counter() - t0) / reps * 1e6, 1)
    for n in (1024, 1 << 20, 16 << 20):
        t = torch.ones(n, device="cuda")
        out[f"all_reduce_fp32_{n * 4 >> 10}KiB_us"] = per_call(lambda: dist.all_reduce(t))
    g = torch.empty(R << 20, dtype=torch.bfloat16, device="cuda")
    x = torch.ones(1 << 20, dtype=torch.bfloat16, device="cuda")
    out["all_gather_bf16_2MiB_shard_us"] = per_call(lambda: dist.all_gather_into_tensor(g, x))
    b = torch.ones(1 << 20, device="cuda")
    out["broadcast_fp32_4MiB_us"] = per_call(lambda: dist.broadcast(b, 0))
    out["barrier_us"] = per_call(lambda: dist.barrier())
    for name, m in (("4KiB", torch.ones(1024, device="cuda")),
                    ("16MiB", torch.ones(1 << 23, dtype=torch.bfloat16, device="cuda"))):
        def ping():
            if rank == 0:
                dist.send(m, 1)
                dist.recv(m, 1)
            elif rank == 1:
                dist.recv(m, 0)
                dist.send(m, 0)
        out[f"send_recv_{name}_round_trip_us"] = per_call(ping)
    dist.barrier()
    hdist.destroy_process_group()
    if rank == 0:
        print(json.dumps(out), flush=True)


def bench_backend(ranks=(2, 4)):
    """Per-call time of the torch.distributed backend with R processes
    sharing the GPU: torchrun starts this file with --backend-rank."""
    import socket
    import subprocess
    res = {}
    for R in ranks:
        with socket.socket() as so:
            so.bind(("127.0.0.1", 0))
            port = so.getsockname()[1]
        env = dict(os.environ, HOCCL_BACKEND="1", OMP_NUM_THREADS="1")
        cmd = [sys.executable, "-m", "torch.distributed.run", "--nnodes=1", f"--nproc-per-node={R}",
               "--master-addr=127.0.0.1", f"--master-port={port}", os.path.abspath(__file__),
               "--backend-rank"]
        r = subprocess.run(cmd, env=env, capture_output=True, text=True, timeout=300)
        lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
        res[f"R{R}"] = json.loads(lines[-1]) if r.returncode == 0 and lines else {
            "error": (r.stderr or r.stdout)[-800:]}
        log(f"backend R={R}: {res[f'R{R}']}")
    return res


def main():
    if "--backend-rank" in sys.argv:
        backend_rank()
        return
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--quick", action="store_true", help="headline only, no extras")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--pmc-workload", action="store_true",
                    help="run only the workload the counter profiles are taken on")
    ap.add_argument("--occupancy-workload", action="store_true",
                    help="run only the workload the occupancy counter pass is taken on")
    ap.add_argument("--sweep", action="store_true",
                    help="print algbw against message size per copy path instead")
    ap.add_argument("--ar-groups-workload", action="store_true",
                    help="run only the grouped all-reduce the overlap trace profiles")
    ap.add_argument("--interference-workload", action="store_true",
                    help="GEMM interference of the engine-path collectives against the engine budget")
    ap.add_argument("--ceilings-workload", action="store_true",
                    help="the memory system's streaming ceilings (read, write, copy, 2R+1W, RMW)")
    ap.add_argument("--copy-workload", action="store_true",
                    help="run only the copy collectives the zero-CU trace is taken on")
    ap.add_argument("--after-free-workload", action="store_true",
                    help="the SDMA engines right after a large device-memory free, static against balanced")
    ap.add_argument("--copy-kernel-workload", action="store_true",
                    help="the CU copy kernel on the copy workloads (to compare its build knobs)")
    ap.add_argument("--backend-workload", action="store_true",
                    help="per-call time of the torch.distributed backend, 2 and 4 rank processes")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the R virtual ranks of every collective live in "
              "that GPU's HBM; run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if args.backend_workload:
        print(json.dumps({"backend": bench_backend()}), flush=True)
        return

    import numpy as np
    import torch

    import paper_2609_34334_amd as hc
    import workloads as W

    torch.cuda.set_device(0)
    hc.init(0)
    # The benchmark studies the ring schedule (the step each GPU runs when the
    # ranks are GPUs); rows that measure the direct fold or AUTO ask for it.
    hc.set_config(reduce_algo="ring")
    if args.pmc_workload:
        pmc_workload(hc, W)
        return
    if args.occupancy_workload:
        occupancy_workload(hc, W)
        return
    if args.ar_groups_workload:
        ar_groups_workload(hc, W)
        return
    if args.copy_workload:
        copy_workload(hc, W)
        return
    if args.ceilings_workload:
        print(json.dumps({"ceilings": ceilings_workload(hc)}), flush=True)
        return
    if args.interference_workload:
        print(json.dumps({"interference": interference_workload(hc, W)}), flush=True)
        return
    if args.sweep:
        print(json.dumps({"sweep": size_sweep(hc)}), flush=True)
        return
    if args.after_free_workload:
        print(json.dumps({"sdma_after_free": bench_after_free(hc, W)}), flush=True)
        return
    if args.copy_kernel_workload:
        print(json.dumps({"copy_kernel": copy_kernel_workload(hc, W)}), flush=True)
        return
    log("reduce-scatter headline")
    rs = bench_reduce_scatter(hc, W, args.steps, args.warmup)
    log(f"RS algbw {rs['algbw']:.1f} GB/s, {rs['sec'] * 1e3:.3f} ms/step, "
        f"kernel {rs['achieved']:.0f} GB/s")
    got = [rs["recv"][r].cpu().view(torch.int16).numpy().view(np.uint16) for r in range(8)]

    extra = {}
    drecv, extra["reduce_scatter_direct"] = direct_reduce_scatter(hc, rs["x"], args.steps, args.warmup)
    dgot = [t.cpu().view(torch.int16).numpy().view(np.uint16) for t in drecv]

    cpu = None
    parity = None
    if not args.no_cpu:
        log("oracle CPU baseline")
        ref, csec, reps, core, ncores = cpu_baseline(rs["x"], 25_165_824 // 8)
        parity = all(np.array_equal(got[r], ref[r]) and np.array_equal(dgot[r], ref[r])
                     for r in range(8))
        cpu = {"value": round(rs["S"] / csec / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
               "sample": f"the full reduce-scatter workload, {reps} repetitions, "
                         f"{csec:.2f} s each, pinned to host core {core}",
               "host_cpu": host_cpu_model(), "host_cores_available": ncores}
    if not args.quick:
        gemm = make_gemm()
        extra["gemm_alone"] = dict(ms=round(gemm[3] * 1e3, 4), tflops=round(2 * 8192 ** 3 / gemm[3] / 1e12, 1))
        extra["reduce_scatter_workgroups"] = bench_rs_workgroups(hc, rs["x"], 3, gemm)
        log("reduce-scatter on reserved CUs")
        try:
            extra["reduce_scatter_reserved_cus"] = bench_cu_partition(hc, rs["x"], gemm)
        except Exception as e:
            extra["reduce_scatter_reserved_cus"] = {"error": repr(e)}
        for name, fn in [("allreduce_fp32_R4", bench_allreduce), ("allgather_fsdp", bench_allgather),
                         ("p2p_pp", bench_p2p), ("alltoallv_ep", bench_a2a)]:
            log(name)
            try:
                extra[name] = fn(hc, W, 10, gemm)
            except Exception as e:  # report, do not hide the headline
                extra[name] = {"error": repr(e)}
        log("allreduce bucket")
        try:
            extra["allreduce_bf16_R8_bucket"] = bench_allreduce_bucket(hc, W, 10)
        except Exception as e:
            extra["allreduce_bf16_R8_bucket"] = {"error": repr(e)}
        log("reduce-scatter variants")
        try:
            extra["reduce_scatter_variants"] = bench_rs_variants(hc, 10)
        except Exception as e:
            extra["reduce_scatter_variants"] = {"error": repr(e)}
        log("reduce-scatter launch shapes")
        try:
            extra["reduce_scatter_launch_shapes"] = bench_rs_launch_shapes(hc, rs["x"])
        except Exception as e:
            extra["reduce_scatter_launch_shapes"] = {"error": repr(e)}
        log("reduce-scatter with fused ring hops")
        try:
            extra["reduce_scatter_fused_hops"] = bench_fused_hops(hc, rs["x"], args.steps, args.warmup)
        except Exception as e:
            extra["reduce_scatter_fused_hops"] = {"error": repr(e)}
        log("reduce-scatter with bf16 partials")
        try:
            extra["reduce_scatter_bf16_partials"] = bench_bf16_partials(hc, rs["x"], args.steps,
                                                                        args.warmup)
        except Exception as e:
            extra["reduce_scatter_bf16_partials"] = {"error": repr(e)}
        log("reduce-scatter in a graph")
        try:
            extra["reduce_scatter_graph"] = bench_rs_graph(hc, rs["x"], args.steps)
        except Exception as e:
            extra["reduce_scatter_graph"] = {"error": repr(e)}
        log("ring hop, one rank")
        try:
            extra["ring_hop_one_rank"] = bench_ring_hop(hc, rs["x"], 20)
        except Exception as e:
            extra["ring_hop_one_rank"] = {"error": repr(e)}
        log("p2p sizes")
        extra["p2p_single_message"] = bench_p2p_sizes(hc, 11)
        extra["small_message_latency"] = bench_small_message(hc, 30, gemm)
        log("host callbacks beside the host-function handshake")
        try:
            extra["callback_thread"] = bench_callback_thread(hc)
        except Exception as e:
            extra["callback_thread"] = {"error": repr(e)}
        # Last: its 2 GiB frees slow one engine for a while after each.
        log("SDMA engines after a large free")
        try:
            extra["sdma_after_free"] = bench_after_free(hc, W)
        except Exception as e:
            extra["sdma_after_free"] = {"error": repr(e)}

    ceiling = round(copy_ceiling(hc), 1)
    st = rs["stats"]
    out = {
        "metric": "collective algbw/busbw GB/s (1 GPU, R virtual ranks), % HBM peak, CUs used",
        "value": round(rs["algbw"], 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(rs["sec"] * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "DP gradient reduce-scatter, ring, bf16 with fp32 accumulation, R=8 virtual "
                               "ranks, 25,165,824 elements per rank (6x4096x1024), recvcount 3,145,728",
                   "R": 8, "elements_per_rank": 25_165_824, "algorithm": "ring",
                   "workgroups_per_step": st["workgroups_per_step"]},
        "busbw": round(rs["busbw"], 3),
        "hbm_GBs": round(rs["bytes_per_op"] / rs["sec"] / 1e9, 1),
        "hbm_frac": round(rs["bytes_per_op"] / rs["sec"] / 1e9 / HBM_PEAK_GBS, 4),
        "cus_used": st["cus_used_max"],
        "cus_available": st["cus_available"],
        "host_enqueue_us": round(st["host_enqueue_us"], 1),
        "parity_vs_oracle": parity,
        "roofline": {"bound": "hbm", "kernel": "reduce_step_kernel (ring step, all 8 ranks per launch)",
                     "achieved": round(rs["achieved"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(rs["achieved"] / HBM_PEAK_GBS, 4), "traffic": measured_traffic(),
                     "traffic_dram_destined": measured_traffic(key="dram_destined_bytes_per_launch"),
                     "traffic_counts": TRAFFIC_NOTE,
                     "stream_ceilings_2GiB_GBs": stream_ceilings(),
                     "avg_launch_us": round(rs["avg_launch_us"], 2),
                     "bytes_per_launch": rs["bytes_per_op"] // rs["launches"],
                     "launches_per_step": rs["launches"],
                     "per_launch_event_us": rs["per_step_us"],
                     "measured_copy_ceiling": ceiling,
                     "frac_of_measured_copy_ceiling": round(rs["achieved"] / ceiling, 4)},
        "cpu_baseline": cpu,
        "extra": extra,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
