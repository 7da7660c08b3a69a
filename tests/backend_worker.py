"""One rank of the multi-process test of the "hoccl" torch.distributed
backend (tests/test_gpu_backend.py launches WORLD_SIZE of these with
torchrun, all on GPU 0, with HOCCL_BACKEND=1).  Every rank generates every
rank's seeded inputs, so it can compute the oracle's result itself and
compare its own output with it bit for bit: all_reduce, reduce_scatter_tensor,
reduce_scatter (list), all_gather_into_tensor, all_gather (list),
all_to_all_single with uneven splits, send/recv around the ring (blocking,
and asynchronous in orders that deadlock with synchronous sends, and
batch_isend_irecv as a pipeline stage uses it), broadcast
from every root, gather, scatter, reduce, all_to_all (lists), the object
collectives, barrier, and torch's functional collectives (all_reduce,
reduce_scatter_tensor, all_gather_tensor, all_to_all_single, broadcast);
an all-reduce and an all-gather in a subgroup of the odd ranks.  The copy collectives also run on dtypes the
library has no arithmetic for (int64, uint8, float16), whose bytes they
move in 4-, 2- or 1-byte units.
Prints "rank r: backend ok" when everything matched."""
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
from gpu_util import NAME, assert_bitwise, from_dev, to_dev  # noqa: E402
from paper_2609_34334_amd import distributed as hdist  # noqa: E402


def byte_tensor(seed, rank, n, dtype):
    """n seeded elements of `dtype` on the GPU, arbitrary bit patterns."""
    nbytes = n * torch.empty(0, dtype=dtype).element_size()
    raw = W.random_bits(seed, rank, (nbytes + 1) // 2, 2).view(np.uint8)[:nbytes]
    return torch.from_numpy(raw.copy()).view(dtype).to("cuda") if nbytes else torch.empty(0, dtype=dtype, device="cuda")


def assert_same_bytes(got, want, what):
    a = got.cpu().reshape(-1).view(torch.uint8).numpy()
    b = want.cpu().reshape(-1).view(torch.uint8).numpy()
    assert a.shape == b.shape and np.array_equal(a, b), (what, np.flatnonzero(a != b)[:8])


def main():
    rank, R = int(os.environ["RANK"]), int(os.environ["WORLD_SIZE"])
    torch.cuda.set_device(0)
    # HOCCL_BACKEND=1 selects hoccl; every store wait ends within 60 s
    hdist.init_process_group(backend="nccl", timeout=timedelta(seconds=60))
    assert dist.get_backend() == hdist.BACKEND, dist.get_backend()
    print(f"rank {rank}: {dist.get_backend()} over {R} ranks", flush=True)
    for dt in (hc.INT32, hc.FP32, hc.BF16):
        for n in (1, 4099, 3 * 65536 + 7):
            xs = [W.random_values(NAME[dt], 900 + n, r, n) for r in range(R)]
            t = to_dev(xs[rank], dt)
            dist.all_reduce(t)
            assert_bitwise(from_dev(t, dt), oracle.allreduce_new(xs, dt)[rank], f"all_reduce {NAME[dt]} n={n}")
            xr = [W.random_values(NAME[dt], 910 + n, r, R * n) for r in range(R)]
            ref = oracle.reduce_scatter_new(xr, dt)[rank]
            out = torch.empty(n, dtype=t.dtype, device="cuda")
            dist.reduce_scatter_tensor(out, to_dev(xr[rank], dt))
            assert_bitwise(from_dev(out, dt), ref, f"reduce_scatter_tensor {NAME[dt]} n={n}")
            out2 = torch.empty(n, dtype=t.dtype, device="cuda")
            dist.reduce_scatter(out2, list(to_dev(xr[rank], dt).chunk(R)))
            assert_bitwise(from_dev(out2, dt), ref, f"reduce_scatter {NAME[dt]} n={n}")
            xg = [W.random_values(NAME[dt], 920 + n, r, n) for r in range(R)]
            refg = oracle.allgather_new(xg, dt)[rank]
            g = torch.empty(R * n, dtype=t.dtype, device="cuda")
            dist.all_gather_into_tensor(g, to_dev(xg[rank], dt))
            assert_bitwise(from_dev(g, dt), refg, f"all_gather_into_tensor {NAME[dt]} n={n}")
            parts = [torch.empty(n, dtype=t.dtype, device="cuda") for _ in range(R)]
            dist.all_gather(parts, to_dev(xg[rank], dt))
            assert_bitwise(from_dev(torch.cat(parts), dt), refg, f"all_gather {NAME[dt]} n={n}")
    # all_to_all_single, uneven rows: rank s sends C[s][d] rows of 96 bf16 to d
    rng = np.random.default_rng(77)
    C = rng.integers(0, 9, size=(R, R))
    row = 96
    xs = [W.random_bits(930, s, int(C[s].sum()) * row, 2) for s in range(R)]
    counts = [int(C[s][d]) * row for s in range(R) for d in range(R)]
    sd = [int(C[s][:d].sum()) * row for s in range(R) for d in range(R)]
    rd = [int(C[:s, d].sum()) * row for s in range(R) for d in range(R)]
    ref = [np.zeros(int(C[:, d].sum()) * row, np.uint16) for d in range(R)]
    oracle.alltoallv(xs, counts, sd, ref, rd, hc.BF16)
    inp = to_dev(xs[rank], hc.BF16).view(-1, row)
    out = torch.empty(int(C[:, rank].sum()), row, dtype=torch.bfloat16, device="cuda")
    dist.all_to_all_single(out, inp, output_split_sizes=[int(c) for c in C[:, rank]],
                           input_split_sizes=[int(c) for c in C[rank]])
    assert_bitwise(from_dev(out.reshape(-1), hc.BF16), ref[rank], "all_to_all_single")
    # send/recv around the ring, three rounds (even ranks send first)
    for k in range(3):
        mine = W.random_bits(940 + k, rank, 70_001, 2)
        prev = W.random_bits(940 + k, (rank - 1) % R, 70_001, 2)
        src, got = to_dev(mine, hc.BF16), torch.empty(70_001, dtype=torch.bfloat16, device="cuda")
        if rank % 2 == 0:
            dist.send(src, (rank + 1) % R)
            dist.recv(got, (rank - 1) % R)
        else:
            dist.recv(got, (rank - 1) % R)
            dist.send(src, (rank + 1) % R)
        assert_bitwise(from_dev(got, hc.BF16), prev, f"recv round {k}")
    # asynchronous point to point: orders that deadlock with synchronous sends
    for k in range(2):
        mine = byte_tensor(1100 + k, rank, 50_001, torch.bfloat16)
        got = torch.empty_like(mine)
        rq = dist.irecv(got, (rank - 1) % R)          # every rank receives first ...
        sq = dist.isend(mine, (rank + 1) % R)         # ... then sends, and waits for the send first
        sq.wait()
        rq.wait()
        assert_same_bytes(got, byte_tensor(1100 + k, (rank - 1) % R, 50_001, torch.bfloat16),
                          f"ring, receives first, round {k}")
    # a pipeline stage: gradient to the previous stage, activation from it,
    # activation to the next, gradient from it (the first and last stages
    # have one neighbour)
    nxt, prv = rank + 1, rank - 1
    a = byte_tensor(1110, rank, 4099, torch.float32)
    b = byte_tensor(1111, rank, 777, torch.float32)
    fa, fb = torch.empty_like(a), torch.empty_like(b)
    ops = []
    if prv >= 0:
        ops += [dist.P2POp(dist.isend, b, prv), dist.P2POp(dist.irecv, fa, prv)]
    if nxt < R:
        ops += [dist.P2POp(dist.isend, a, nxt), dist.P2POp(dist.irecv, fb, nxt)]
    for req in dist.batch_isend_irecv(ops):
        req.wait()
    if prv >= 0:
        assert_same_bytes(fa, byte_tensor(1110, prv, 4099, torch.float32), "batch_isend_irecv forward")
    if nxt < R:
        assert_same_bytes(fb, byte_tensor(1111, nxt, 777, torch.float32), "batch_isend_irecv backward")
    if R >= 2 and rank < 2:                           # two stages exchanging, both sending first
        peer = 1 - rank
        mine = byte_tensor(1120, rank, 12_345, torch.int32)
        got = torch.empty_like(mine)
        sq = dist.isend(mine, peer)
        rq = dist.irecv(got, peer)
        sq.wait()
        rq.wait()
        assert_same_bytes(got, byte_tensor(1120, peer, 12_345, torch.int32), "exchange, both send first")
    # more receives outstanding from one sender than a pair has slots, of
    # different sizes, waited for newest first
    if rank < 2:
        sizes = [3, 70_000, 1, 4099, 65_536, 17]
        if rank == 1:
            reqs = [dist.irecv(torch.empty(m, dtype=torch.bfloat16, device="cuda"), 0) for m in sizes]
            for k in reversed(range(len(sizes))):
                reqs[k].wait()
                got = reqs[k].get_future().value()[0]
                assert_same_bytes(got, byte_tensor(1130 + k, 0, sizes[k], torch.bfloat16), f"queued receive {k}")
        else:
            sends = [dist.isend(byte_tensor(1130 + k, 0, m, torch.bfloat16), 1) for k, m in enumerate(sizes)]
            for q in sends:
                q.wait()
    # broadcast from every root; dtypes beyond the library's move as bytes
    for root in range(R):
        for k, (dtype, n) in enumerate(((torch.float32, 4099), (torch.bfloat16, 3 * 65536 + 7),
                                        (torch.int32, 1), (torch.int64, 33), (torch.uint8, 1000),
                                        (torch.float16, 77), (torch.float32, 0))):
            want = byte_tensor(950 + k, root, n, dtype)
            t = want.clone() if rank == root else torch.full_like(want, 7)
            dist.broadcast(t, root)
            assert_same_bytes(t, want, f"broadcast {dtype} n={n} root={root}")
    # all_gather_into_tensor, all_to_all_single and send/recv of int64 and uint8
    for k, (dtype, n) in enumerate(((torch.int64, 1001), (torch.uint8, 6))):
        xs = [byte_tensor(960 + k, r, n, dtype) for r in range(R)]
        g = torch.empty(R * n, dtype=dtype, device="cuda")
        dist.all_gather_into_tensor(g, xs[rank])
        assert_same_bytes(g, torch.cat(xs), f"all_gather_into_tensor {dtype}")
        ys = [byte_tensor(970 + k, r, R * n, dtype) for r in range(R)]
        out = torch.empty(R * n, dtype=dtype, device="cuda")
        dist.all_to_all_single(out, ys[rank])
        assert_same_bytes(out, torch.cat([ys[s][rank * n:(rank + 1) * n] for s in range(R)]),
                          f"all_to_all_single {dtype}")
        got = torch.empty(n, dtype=dtype, device="cuda")
        if rank % 2 == 0:
            dist.send(xs[rank], (rank + 1) % R)
            dist.recv(got, (rank - 1) % R)
        else:
            dist.recv(got, (rank - 1) % R)
            dist.send(xs[rank], (rank + 1) % R)
        assert_same_bytes(got, xs[(rank - 1) % R], f"recv {dtype}")
    # torch's functional collectives (what DTensor uses) reach the backend too
    import torch.distributed._functional_collectives as funcol
    grp = dist.group.WORLD
    done = lambda x: x.wait() if hasattr(x, "wait") else x
    for dt in (hc.INT32, hc.FP32, hc.BF16):
        n = 4099
        xs = [W.random_values(NAME[dt], 980, r, n) for r in range(R)]
        got = done(funcol.all_reduce(to_dev(xs[rank], dt), "sum", grp))
        assert_bitwise(from_dev(got, dt), oracle.allreduce_new(xs, dt)[rank], f"funcol all_reduce {NAME[dt]}")
        xr = [W.random_values(NAME[dt], 981, r, R * n) for r in range(R)]
        got = done(funcol.reduce_scatter_tensor(to_dev(xr[rank], dt), "sum", 0, grp))
        assert_bitwise(from_dev(got, dt), oracle.reduce_scatter_new(xr, dt)[rank],
                       f"funcol reduce_scatter_tensor {NAME[dt]}")
        got = done(funcol.all_gather_tensor(to_dev(xs[rank], dt), 0, grp))
        assert_bitwise(from_dev(got, dt), oracle.allgather_new(xs, dt)[rank], f"funcol all_gather {NAME[dt]}")
        got = done(funcol.all_to_all_single(to_dev(xr[rank], dt), None, None, grp))
        want = np.concatenate([xr[s][rank * n:(rank + 1) * n] for s in range(R)])
        assert_bitwise(from_dev(got, dt), want, f"funcol all_to_all_single {NAME[dt]}")
        got = done(funcol.broadcast(to_dev(xs[rank], dt), R - 1, grp))
        assert_bitwise(from_dev(got, dt), xs[R - 1], f"funcol broadcast {NAME[dt]}")
    # a subgroup of the odd ranks (every rank creates it; only members call)
    odd = list(range(1, R, 2))
    sub = dist.new_group(odd)
    if rank in odd:
        n = 1000
        xs = [W.random_values("fp32", 990, r, n) for r in odd]
        t = to_dev(xs[odd.index(rank)], hc.FP32)
        dist.all_reduce(t, group=sub)
        assert_bitwise(from_dev(t, hc.FP32), oracle.allreduce_new(xs, hc.FP32)[odd.index(rank)],
                       "subgroup all_reduce")
        g = torch.empty(len(odd) * n, dtype=torch.float32, device="cuda")
        dist.all_gather_into_tensor(g, t, group=sub)
        assert_bitwise(from_dev(g, hc.FP32), np.concatenate([from_dev(t, hc.FP32)] * len(odd)),
                       "subgroup all_gather")
    dist.barrier()
    # odd byte counts move as single bytes
    want = byte_tensor(1000, 0, 3, torch.uint8)
    t = want.clone() if rank == 0 else torch.zeros(3, dtype=torch.uint8, device="cuda")
    dist.broadcast(t, 0)
    assert_same_bytes(t, want, "broadcast of 3 bytes")
    xs = [byte_tensor(1001, r, 5, torch.uint8) for r in range(R)]
    g = torch.empty(R * 5, dtype=torch.uint8, device="cuda")
    dist.all_gather_into_tensor(g, xs[rank])
    assert_same_bytes(g, torch.cat(xs), "all_gather of 5 bytes")
    # object collectives (pickles of odd length, through the byte path)
    objs = [None] * R
    dist.all_gather_object(objs, {"rank": rank, "pad": "x" * (rank * 7 + 1)})
    assert objs == [{"rank": r, "pad": "x" * (r * 7 + 1)} for r in range(R)], objs
    lst = [("config", 3.5, list(range(rank + 3)))] if rank == R - 1 else [None]
    dist.broadcast_object_list(lst, src=R - 1)
    assert lst == [("config", 3.5, list(range(R + 2)))], lst
    # gather, scatter, reduce and the list all-to-all, rooted at the last rank
    root, n = R - 1, 1001
    xs = [byte_tensor(1010, r, n, torch.float32) for r in range(R)]
    parts = [torch.empty(n, device="cuda") for _ in range(R)] if rank == root else None
    dist.gather(xs[rank], parts, dst=root)
    if rank == root:
        assert_same_bytes(torch.cat(parts), torch.cat(xs), "gather")
    blocks = [byte_tensor(1020 + d, root, n, torch.int64) for d in range(R)]
    got = torch.empty(n, dtype=torch.int64, device="cuda")
    dist.scatter(got, blocks if rank == root else None, src=root)
    assert_same_bytes(got, blocks[rank], "scatter")
    vals = [W.random_values("fp32", 1030, r, n) for r in range(R)]
    t = to_dev(vals[rank], hc.FP32)
    dist.reduce(t, dst=root)
    want = oracle.allreduce_new(vals, hc.FP32)[root] if rank == root else vals[rank]
    assert_bitwise(from_dev(t, hc.FP32), want, "reduce")
    ins = [byte_tensor(1040 + d, rank, d + 2, torch.bfloat16) for d in range(R)]
    outs = [torch.empty(rank + 2, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    dist.all_to_all(outs, ins)
    for s in range(R):
        assert_same_bytes(outs[s], byte_tensor(1040 + rank, s, rank + 2, torch.bfloat16),
                          f"all_to_all from {s}")
    # a check failing on one rank only: every rank fails at once, none waits
    import time
    t0 = time.perf_counter()
    bad = torch.zeros(8, dtype=torch.int64 if rank == R - 1 else torch.float32, device="cuda")
    try:
        dist.all_reduce(bad)
        raise AssertionError("an int64 all_reduce was accepted")
    except RuntimeError as e:
        assert f"rank {R - 1}" in str(e) and "int32, float32 or bfloat16" in str(e), e
    assert time.perf_counter() - t0 < 10, "a rank waited for the failing one"
    x = torch.ones(4, device="cuda")
    dist.all_reduce(x)                      # the group goes on afterwards
    assert bool((x == R).all()), x
    dist.barrier()
    hdist.destroy_process_group()
    print(f"rank {rank}: backend ok", flush=True)


if __name__ == "__main__":
    main()
