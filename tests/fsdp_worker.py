"""One rank of the FSDP2 (torch.distributed.fsdp.fully_shard) test of the
"hoccl" backend (tests/test_gpu_backend.py launches WORLD_SIZE of these with
torchrun, all on GPU 0, with HOCCL_BACKEND=1).

Every rank builds the same model from one seed and shards it layer by layer
with fully_shard on the default device mesh, so that every forward
all-gathers the parameters (all_gather_into_tensor) and every backward
reduce-scatters the gradients with an average (reduce_scatter_tensor, AVG).
With argument "bf16" the parameters are gathered and the gradients reduced
in bfloat16 (MixedPrecisionPolicy), otherwise in float32.

Three SGD steps on per-rank seeded batches.  After each backward the
gradients, gathered with DTensor.full_tensor() (torch's functional
all-gather, which reaches the backend too), are compared with the average over ranks of the local
gradients, which every rank computes itself on a plain copy of the model
(in the parameter dtype, as FSDP computes them): within the recursive
summation bound of a fold over the ranks in float32, plus the final
rounding to the reduce dtype.  The plain copy then takes the same SGD step
with the gathered gradients, and the parameters must agree with FSDP's.
Prints "rank r: fsdp ok"."""
import os
import sys
from datetime import timedelta

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))

import torch  # noqa: E402
import torch.distributed as dist  # noqa: E402
import torch.nn.functional as F  # noqa: E402
from torch.distributed.fsdp import MixedPrecisionPolicy, fully_shard  # noqa: E402

from paper_2609_34334_amd import distributed as hdist  # noqa: E402

WIDTH, OUT, BATCH, LAYERS = 256, 10, 32, 3


class Net(torch.nn.Module):
    def __init__(self):
        super().__init__()
        self.layers = torch.nn.ModuleList(torch.nn.Linear(WIDTH, WIDTH) for _ in range(LAYERS))
        self.head = torch.nn.Linear(WIDTH, OUT)

    def forward(self, x):
        for layer in self.layers:
            x = torch.relu(layer(x))
        return self.head(x)


def build():
    torch.manual_seed(1234)
    return Net().cuda()


def batch(rank, step):
    g = torch.Generator().manual_seed(3000 + 100 * step + rank)
    return torch.randn(BATCH, WIDTH, generator=g).cuda(), torch.randint(0, OUT, (BATCH,), generator=g).cuda()


def main():
    rank, R = int(os.environ["RANK"]), int(os.environ["WORLD_SIZE"])
    low = len(sys.argv) > 1 and sys.argv[1] == "bf16"
    pdt = torch.bfloat16 if low else torch.float32
    torch.cuda.set_device(0)
    hdist.init_process_group(backend="nccl", timeout=timedelta(seconds=60))
    assert dist.get_backend() == hdist.BACKEND, dist.get_backend()
    model = build()
    mp = MixedPrecisionPolicy(param_dtype=pdt, reduce_dtype=pdt)
    for layer in model.layers:
        fully_shard(layer, mp_policy=mp)
    fully_shard(model, mp_policy=mp)
    plain = build()                                   # the same initial parameters, unsharded
    opt = torch.optim.SGD(model.parameters(), lr=0.05)
    gamma = (R - 1) * 2.0 ** -24 / (1 - (R - 1) * 2.0 ** -24)
    ulp = 2.0 ** -8 if low else 2.0 ** -24            # half an ulp of the reduce dtype, relative
    for step in range(3):
        local = []
        lowered = build().to(pdt)
        lowered.load_state_dict({k: v.to(pdt) for k, v in plain.state_dict().items()})
        for r in range(R):
            lowered.zero_grad(set_to_none=True)
            x, y = batch(r, step)
            F.cross_entropy(lowered(x.to(pdt)).float(), y).backward()
            local.append({n: p.grad.float() for n, p in lowered.named_parameters()})
        opt.zero_grad(set_to_none=True)
        x, y = batch(rank, step)
        F.cross_entropy(model(x).float(), y).backward()
        grads = {}
        for n, p in model.named_parameters():
            full = p.grad.full_tensor()           # torch's functional all-gather, over the backend
            g = full.double()
            exact = sum(t[n].double() for t in local) / R
            bound = (gamma + ulp) * sum(t[n].double().abs() for t in local) / R + 1e-30
            err = (g - exact).abs()
            assert bool((err <= bound).all()), f"step {step}: {n} gradient off by {float(err.max())}"
            grads[n] = full
        opt.step()
        with torch.no_grad():
            for n, p in plain.named_parameters():
                p.add_(grads[n], alpha=-0.05)
        for n, p in model.named_parameters():
            full = p.full_tensor()
            ref = dict(plain.named_parameters())[n]
            assert torch.allclose(full, ref, rtol=2 ** -22, atol=1e-9), \
                f"step {step}: {n} parameters off by {float((full - ref).abs().max())}"
        print(f"rank {rank}: step {step} ok", flush=True)
    hdist.destroy_process_group()
    print(f"rank {rank}: fsdp ok", flush=True)


if __name__ == "__main__":
    main()
