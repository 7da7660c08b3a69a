"""One rank of the randomised test of the "hoccl" backend
(tests/test_gpu_backend.py launches WORLD_SIZE of these with torchrun, all
on GPU 0, with HOCCL_BACKEND=1).  Every rank draws the same seeded sequence
of calls: all_reduce, reduce_scatter_tensor, all_gather_into_tensor,
all_to_all_single with random splits, broadcast from a random root, and
asynchronous send/recv between random pairs, over random dtypes and sizes
(odd byte counts included).  Every rank computes every rank's inputs, so it
checks its own outputs against the oracle (reductions) or the bytes it must
hold (copies).  Prints "rank r: random ok"."""
import os
import sys
from datetime import timedelta

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))
sys.path.insert(0, HERE)

import numpy as np  # noqa: E402
import torch  # noqa: E402
import torch.distributed as dist  # noqa: E402

import oracle  # noqa: E402
import paper_2609_34334_amd as hc  # noqa: E402
import workloads as W  # noqa: E402
from backend_worker import assert_same_bytes, byte_tensor  # noqa: E402
from gpu_util import NAME, TORCH, assert_bitwise, from_dev, to_dev  # noqa: E402
from paper_2609_34334_amd import distributed as hdist  # noqa: E402

COPY_DTYPES = [torch.float32, torch.bfloat16, torch.int64, torch.uint8, torch.float16, torch.int32]


def main():
    rank, R = int(os.environ["RANK"]), int(os.environ["WORLD_SIZE"])
    cases = int(sys.argv[1]) if len(sys.argv) > 1 else 100
    torch.cuda.set_device(0)
    hdist.init_process_group(backend="nccl", timeout=timedelta(seconds=60))
    g = np.random.default_rng(4242)                     # the same draws on every rank
    for k in range(cases):
        op = str(g.choice(["all_reduce", "reduce_scatter", "all_gather", "all_to_all", "broadcast", "p2p"]))
        n = int(g.integers(0, 20_000))
        seed = 5000 + k
        if op in ("all_reduce", "reduce_scatter"):
            dt = [hc.INT32, hc.FP32, hc.BF16][int(g.integers(0, 3))]
            if op == "all_reduce":
                xs = [W.random_values(NAME[dt], seed, r, n) for r in range(R)]
                t = to_dev(xs[rank], dt)
                dist.all_reduce(t)
                assert_bitwise(from_dev(t, dt), oracle.allreduce_new(xs, dt)[rank], f"case {k} {op}")
            else:
                xs = [W.random_values(NAME[dt], seed, r, R * n) for r in range(R)]
                out = torch.empty(n, dtype=TORCH[dt], device="cuda")
                dist.reduce_scatter_tensor(out, to_dev(xs[rank], dt))
                assert_bitwise(from_dev(out, dt), oracle.reduce_scatter_new(xs, dt)[rank], f"case {k} {op}")
            continue
        dtype = COPY_DTYPES[int(g.integers(0, len(COPY_DTYPES)))]
        if op == "all_gather":
            xs = [byte_tensor(seed, r, n, dtype) for r in range(R)]
            out = torch.empty(R * n, dtype=dtype, device="cuda")
            dist.all_gather_into_tensor(out, xs[rank])
            assert_same_bytes(out, torch.cat(xs), f"case {k} {op} {dtype}")
        elif op == "all_to_all":
            C = g.integers(0, 300, size=(R, R))
            xs = [byte_tensor(seed, s, int(C[s].sum()), dtype) for s in range(R)]
            out = torch.empty(int(C[:, rank].sum()), dtype=dtype, device="cuda")
            dist.all_to_all_single(out, xs[rank], output_split_sizes=[int(c) for c in C[:, rank]],
                                   input_split_sizes=[int(c) for c in C[rank]])
            want = torch.cat([xs[s][int(C[s][:rank].sum()):int(C[s][:rank + 1].sum())] for s in range(R)])
            assert_same_bytes(out, want, f"case {k} {op} {dtype}")
        elif op == "broadcast":
            root = int(g.integers(0, R))
            want = byte_tensor(seed, root, n, dtype)
            t = want.clone() if rank == root else torch.zeros_like(want)
            dist.broadcast(t, root)
            assert_same_bytes(t, want, f"case {k} {op} {dtype} root {root}")
        else:
            src, dst = (int(v) for v in g.permutation(R)[:2]) if R > 1 else (0, 0)
            if R == 1:
                continue
            msgs = int(g.integers(1, 4))
            sizes = [int(g.integers(0, 9000)) for _ in range(msgs)]
            if rank == src:
                reqs = [dist.isend(byte_tensor(seed + j, src, m, dtype), dst) for j, m in enumerate(sizes)]
            elif rank == dst:
                bufs = [torch.empty(m, dtype=dtype, device="cuda") for m in sizes]
                reqs = [dist.irecv(b, src) for b in bufs]
            else:
                reqs = []
            for q in reversed(reqs):
                q.wait()
            if rank == dst:
                for j, m in enumerate(sizes):
                    assert_same_bytes(bufs[j], byte_tensor(seed + j, src, m, dtype), f"case {k} p2p {j}")
    dist.barrier()
    hdist.destroy_process_group()
    print(f"rank {rank}: random ok", flush=True)


if __name__ == "__main__":
    main()
