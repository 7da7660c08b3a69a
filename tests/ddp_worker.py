"""One rank of the DistributedDataParallel test of the "hoccl" backend
(tests/test_gpu_backend.py launches WORLD_SIZE of these with torchrun, all
on GPU 0, with HOCCL_BACKEND=1).

Every rank starts from different parameters and buffers; DDP's constructor
broadcasts rank 0's (parameters fp32, buffers fp32 and int64), which every
rank rebuilds from rank 0's seed and compares bit for bit.  Then three SGD
steps on per-rank seeded batches, with small gradient buckets so that each
backward all-reduces several of them (and the second step rebuilds the
buckets, broadcasting their layout).  After each backward every gradient is
checked against the sum over ranks of the local gradients divided by the
world size, which every rank computes itself on a plain copy of the model:
bit for bit at 2 ranks (one fp32 add, so order-free), within the recursive
summation bound otherwise (the ring's element order depends on where DDP's
bucket boundaries fall).  After each step the parameters must agree bit for
bit across ranks.  Prints "rank r: ddp ok"."""
import os
import sys
from datetime import timedelta

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))

import torch  # noqa: E402
import torch.distributed as dist  # noqa: E402
import torch.nn.functional as F  # noqa: E402

from paper_2609_34334_amd import distributed as hdist  # noqa: E402

IN, HID, OUT, BATCH = 256, 512, 10, 32


class Net(torch.nn.Module):
    def __init__(self):
        super().__init__()
        self.fc1 = torch.nn.Linear(IN, HID)
        self.fc2 = torch.nn.Linear(HID, HID)
        self.head = torch.nn.Linear(HID, OUT)
        self.register_buffer("scale", torch.ones(HID))
        self.register_buffer("calls", torch.zeros((), dtype=torch.int64))

    def forward(self, x):
        self.calls += 1
        h = torch.relu(self.fc1(x)) * self.scale
        return self.head(torch.relu(self.fc2(h)))


def initial_model(rank):
    """Rank `rank`'s model before DDP: its own seed, its own buffers."""
    torch.manual_seed(1000 + rank)
    m = Net()
    m.scale.fill_(1.0 + rank)
    m.calls.fill_(100 * rank)
    return m.cuda()


def batch(rank, step):
    g = torch.Generator().manual_seed(2000 + 100 * step + rank)
    x = torch.randn(BATCH, IN, generator=g)
    y = torch.randint(0, OUT, (BATCH,), generator=g)
    return x.cuda(), y.cuda()


def same_bits(a, b):
    return a.shape == b.shape and torch.equal(a.reshape(-1).view(torch.uint8), b.reshape(-1).view(torch.uint8))


def main():
    rank, R = int(os.environ["RANK"]), int(os.environ["WORLD_SIZE"])
    torch.cuda.set_device(0)
    hdist.init_process_group(backend="nccl", timeout=timedelta(seconds=60))
    assert dist.get_backend() == hdist.BACKEND, dist.get_backend()
    ddp = torch.nn.parallel.DistributedDataParallel(initial_model(rank), device_ids=[0],
                                                    bucket_cap_mb=0.25)
    want = initial_model(0).state_dict()
    for k, v in ddp.module.state_dict().items():
        assert same_bits(v, want[k]), f"rank {rank}: {k} differs from rank 0's after DDP's broadcast"
    print(f"rank {rank}: parameters and buffers broadcast", flush=True)
    opt = torch.optim.SGD(ddp.parameters(), lr=0.05)
    gamma = (R - 1) * 2.0 ** -24 / (1 - (R - 1) * 2.0 ** -24)
    for step in range(3):
        plain = Net().cuda()                       # the same parameters, no hooks
        plain.load_state_dict(ddp.module.state_dict())
        local = []
        for r in range(R):
            plain.zero_grad(set_to_none=True)
            x, y = batch(r, step)
            F.cross_entropy(plain(x), y).backward()
            local.append({n: p.grad.clone() for n, p in plain.named_parameters()})
        opt.zero_grad(set_to_none=True)
        x, y = batch(rank, step)
        F.cross_entropy(ddp(x), y).backward()
        for n, p in ddp.module.named_parameters():
            parts = [g[n] / R for g in local]
            if R == 2:
                assert same_bits(p.grad, parts[0] + parts[1]), f"step {step}: {n} gradient"
            else:
                exact = sum(t.double() for t in parts)
                bound = gamma * sum(t.double().abs() for t in parts) + 1e-45
                err = (p.grad.double() - exact).abs()
                assert bool((err <= bound).all()), f"step {step}: {n} gradient off by {float(err.max())}"
        opt.step()
        flat = torch.cat([p.detach().reshape(-1) for p in ddp.module.parameters()])
        every = torch.empty(R * flat.numel(), device="cuda")
        dist.all_gather_into_tensor(every, flat)
        for r in range(R):
            assert same_bits(every[r * flat.numel():(r + 1) * flat.numel()], flat), \
                f"step {step}: rank {r}'s parameters differ from rank {rank}'s"
        assert int(ddp.module.calls) == step + 1, int(ddp.module.calls)
        print(f"rank {rank}: step {step} ok", flush=True)
    hdist.destroy_process_group()
    print(f"rank {rank}: ddp ok", flush=True)


if __name__ == "__main__":
    main()
