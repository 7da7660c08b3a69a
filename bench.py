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
    concurrent bf16 GEMM), each with algbw/busbw, %HBM peak and CUs used.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--quick]
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


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


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


# ---- the headline: reduce-scatter ------------------------------------------

def bench_reduce_scatter(hc, W, steps, warmup):
    import torch
    R, n_in = 8, 25_165_824
    n = n_in // R
    x = W.rs_gradients(R, n_in)
    send = [bf16_dev(a) for a in x]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    hc.set_config(reduce_algo="ring", kernel_timing=0)

    def step():
        hc.reduce_scatter(send, recv)

    sec = time_op(step, steps, warmup)
    stats = hc.last_stats()
    # Per-launch durations of the reduce-step kernel over a second timed run.
    hc.set_config(kernel_timing=1)
    hc.kernel_times()
    for _ in range(steps):
        step()
    kt = hc.kernel_times()
    hc.set_config(kernel_timing=0)
    launches_per_op = stats["reduce_launches"]
    bytes_per_op = stats["hbm_bytes_algorithmic"]
    avg_launch_s = statistics.mean(kt) / 1e3
    achieved = bytes_per_op / launches_per_op / avg_launch_s / 1e9
    S = R * n * 2
    algbw = S / sec / 1e9
    return dict(x=x, recv=recv, sec=sec, stats=stats, S=S, algbw=algbw,
                busbw=algbw * (R - 1) / R, bytes_per_op=bytes_per_op,
                launches=launches_per_op, avg_launch_us=avg_launch_s * 1e6,
                achieved=achieved, kernel_ms=kt)


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
    hc.set_config(reduce_algo="ring")
    return recv, dict(algbw_GBs=round(R * n * 2 / sec / 1e9, 2), ms=round(sec * 1e3, 4),
                      hbm_GBs=round(st["hbm_bytes_algorithmic"] / sec / 1e9, 1),
                      hbm_frac=round(st["hbm_bytes_algorithmic"] / sec / 1e9 / HBM_PEAK_GBS, 4))


def cpu_baseline(x, recvcount, budget_s=12.0):
    """The oracle (single-threaded C) on the same reduce-scatter, repeated
    until about budget_s seconds of CPU work."""
    import numpy as np
    import oracle
    R = len(x)
    out = [np.empty(recvcount, np.uint16) for _ in range(R)]
    t0 = time.perf_counter()
    reps = 0
    while True:
        oracle.reduce_scatter(x, out, recvcount, oracle.BF16)
        reps += 1
        if time.perf_counter() - t0 > budget_s:
            break
    sec = (time.perf_counter() - t0) / reps
    return out, sec, reps


# ---- the other collectives ---------------------------------------------------

def bench_allreduce(hc, W, reps):
    import torch
    R, n = 4, 1_048_576
    x = W.allreduce_fp32(R, n)
    send = [torch.from_numpy(a).cuda() for a in x]
    recv = [torch.empty(n, device="cuda") for _ in range(R)]
    res = {}
    for path in ["sdma", "engines", "kernel"]:
        hc.set_config(copy_path=path)
        med, mn = event_time(lambda: hc.allreduce(send, recv), reps)
        st = hc.last_stats()
        S = n * 4
        res[path] = dict(algbw_GBs=round(S / med / 1e9, 2),
                         busbw_GBs=round(S / med / 1e9 * 2 * (R - 1) / R, 2),
                         us=round(med * 1e6, 2), hbm_frac=round(st["hbm_bytes_algorithmic"] / med / 1e9 / HBM_PEAK_GBS, 4),
                         cus_used=st["cus_used_max"])
    hc.set_config(copy_path="auto")
    return dict(workload="all-reduce ring fp32 R=4, 1,048,576 elements per rank", **res)


def bench_allgather(hc, W, reps):
    import torch
    R, total = 8, 201_326_592
    x = W.ag_parameters(R, total)
    n = total // R
    send = [bf16_dev(a) for a in x]
    recv = [torch.empty(total, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    res = {}
    for path, extra in [("sdma", {}), ("engines", {}), ("engines", {"allgather_direct": 1, "chunk_bytes": 8 << 20}),
                        ("kernel", {})]:
        key = path + ("_direct_8MiB" if extra else "")
        hc.set_config(copy_path=path, **extra)
        med, mn = event_time(lambda: hc.allgather(send, recv), reps, warmup=1)
        st = hc.last_stats()
        S = total * 2
        res[key] = dict(algbw_GBs=round(S / med / 1e9, 2), busbw_GBs=round(S / med / 1e9 * (R - 1) / R, 2),
                        ms=round(med * 1e3, 3), hbm_frac=round(st["hbm_bytes_algorithmic"] / med / 1e9 / HBM_PEAK_GBS, 4),
                        cus_used=st["cus_used_max"])
        hc.set_config(allgather_direct=0, chunk_bytes=0)
    hc.set_config(copy_path="auto")
    return dict(workload="FSDP all-gather bf16 R=8, 25,165,824-element shards (201,326,592 params)", **res)


def bench_p2p(hc, W, reps):
    import torch
    R = 8
    x = W.p2p_activations(R)
    n = x[0].size
    send = [bf16_dev(a) for a in x]
    recv = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    fwd = [r + 1 if r + 1 < R else -1 for r in range(R)]
    bwd = [r - 1 for r in range(R)]
    res = {}
    for path in ["sdma", "engines", "kernel"]:
        hc.set_config(copy_path=path)

        def schedule():
            for _ in range(16):            # 16 microbatches, forward then backward
                hc.sendrecv(send, recv, fwd)
                hc.sendrecv(send, recv, bwd)

        med, mn = event_time(schedule, max(3, reps // 4), warmup=1)
        st = hc.last_stats()
        msgs = 16 * 2 * (R - 1)
        # 32 rounds (16 microbatches x fwd/bwd) of 7 concurrent messages
        res[path] = dict(per_message_algbw_GBs=round(n * 2 / (med / 32) / 1e9, 2),
                         aggregate_GBs=round(msgs * n * 2 / med / 1e9, 2),
                         schedule_ms=round(med * 1e3, 3), cus_used=st["cus_used_max"])
    hc.set_config(copy_path="auto")
    return dict(workload="PP send/recv bf16 [1,2048,4096], 8 stages, 16 microbatches fwd+bwd "
                         "(224 messages in rounds of 7 concurrent hops)", **res)


def bench_a2a_gemm(hc, W, reps):
    import torch
    R = 8
    send_np, counts, sd, rd, rsz = W.a2a_tokens(R)
    send = [bf16_dev(a) for a in send_np]
    recv = [torch.empty(s, dtype=torch.bfloat16, device="cuda") for s in rsz]
    sent = sum(counts) * 2
    A = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    B = torch.randn(8192, 8192, device="cuda").to(torch.bfloat16)
    C = torch.empty(8192, 8192, device="cuda", dtype=torch.bfloat16)
    gemm_s = torch.cuda.Stream()
    coll_s = torch.cuda.Stream()

    def gemm_alone(ngemm=20):
        ts = []
        with torch.cuda.stream(gemm_s):
            for _ in range(ngemm):
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                a.record()
                torch.matmul(A, B, out=C)
                b.record()
                ts.append((a, b))
        torch.cuda.synchronize()
        return statistics.median(a.elapsed_time(b) for a, b in ts) / 1e3

    gemm_alone(3)
    t_alone = gemm_alone()
    res = dict(gemm_ms_alone=round(t_alone * 1e3, 4),
               gemm_tflops_alone=round(2 * 8192 ** 3 / t_alone / 1e12, 1))
    for path in ["sdma", "engines", "kernel"]:
        hc.set_config(copy_path=path)
        med, mn = event_time(lambda: hc.alltoallv(send, counts, sd, recv, rd), reps)
        st = hc.last_stats()
        # concurrent: keep the all-to-all looping on its own stream for the
        # whole GEMM window
        torch.cuda.synchronize()
        n_coll = int(20 * t_alone / med) + 4
        with torch.cuda.stream(coll_s):
            for _ in range(n_coll):
                hc.alltoallv(send, counts, sd, recv, rd, stream=coll_s)
        t_conc = gemm_alone()
        torch.cuda.synchronize()
        res[path] = dict(algbw_GBs=round(sent / R / med / 1e9, 2), aggregate_GBs=round(sent / med / 1e9, 2),
                         ms=round(med * 1e3, 3), cus_used=st["cus_used_max"],
                         gemm_ms_concurrent=round(t_conc * 1e3, 4),
                         gemm_slowdown=round(t_conc / t_alone - 1, 4))
    hc.set_config(copy_path="auto")
    return dict(workload="EP all-to-all(v) bf16, 4096 tokens x 2048 per rank, 64 experts over R=8, "
                         "top-6 (one copy per destination rank), with a concurrent 8192^3 bf16 GEMM",
                bytes_sent_total=sent, **res)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--quick", action="store_true", help="headline only, no extras")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the R virtual ranks of every collective live in "
              "that GPU's HBM; run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_34334_amd as hc
    import workloads as W

    torch.cuda.set_device(0)
    hc.init(0)
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
        ref, csec, reps = cpu_baseline(rs["x"], 25_165_824 // 8)
        parity = all(np.array_equal(got[r], ref[r]) and np.array_equal(dgot[r], ref[r])
                     for r in range(8))
        cpu = {"value": round(rs["S"] / csec / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
               "sample": f"the full reduce-scatter workload, {reps} repetitions, "
                         f"{csec:.2f} s each on one host core"}
    if not args.quick:
        for name, fn in [("allreduce_fp32_R4", bench_allreduce), ("allgather_fsdp", bench_allgather),
                         ("p2p_pp", bench_p2p), ("alltoallv_ep_with_gemm", bench_a2a_gemm)]:
            log(name)
            try:
                extra[name] = fn(hc, W, 10)
            except Exception as e:  # report, do not hide the headline
                extra[name] = {"error": repr(e)}

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
        "parity_vs_oracle": parity,
        "roofline": {"bound": "hbm", "kernel": "reduce_step_kernel (ring step, all 8 ranks per launch)",
                     "achieved": round(rs["achieved"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(rs["achieved"] / HBM_PEAK_GBS, 4), "traffic": None,
                     "avg_launch_us": round(rs["avg_launch_us"], 2),
                     "bytes_per_launch": rs["bytes_per_op"] // rs["launches"],
                     "launches_per_step": rs["launches"]},
        "cpu_baseline": cpu,
        "extra": extra,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
