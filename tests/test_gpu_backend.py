"""The "hoccl" torch.distributed backend across processes sharing the one
GPU: ranks launched by torchrun (HOCCL_BACKEND=1 turns the requested
backend into hoccl).  Every collective's output compared with the oracle by
each rank (tests/backend_worker.py), a seeded random sequence of calls
(tests/backend_random_worker.py); DistributedDataParallel training
(tests/ddp_worker.py) and FSDP2 training (tests/fsdp_worker.py) over the
backend."""
import os
import signal
import socket
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def free_port():
    with socket.socket() as s:
        s.bind(("127.0.0.1", 0))
        return s.getsockname()[1]


def run_ranks(worker, ranks, done, *args):
    env = dict(os.environ, HOCCL_BACKEND="1", MASTER_ADDR="127.0.0.1", OMP_NUM_THREADS="1")
    cmd = [sys.executable, "-m", "torch.distributed.run", "--nnodes=1", f"--nproc-per-node={ranks}",
           "--master-addr=127.0.0.1", f"--master-port={free_port()}",
           os.path.join(ROOT, "tests", worker), *args]
    print("launching", " ".join(cmd[3:]), flush=True)
    p = subprocess.Popen(cmd, env=env, cwd=ROOT, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True,
                         start_new_session=True)
    try:
        out, err = p.communicate(timeout=240)
    except subprocess.TimeoutExpired:
        os.killpg(p.pid, signal.SIGKILL)      # torchrun and every worker it started
        out, err = p.communicate()
        raise AssertionError(("timed out", out[-3000:], err[-3000:]))
    assert p.returncode == 0, (out[-3000:], err[-4000:])
    assert out.count(done) == ranks, out[-3000:]


@pytest.mark.parametrize("ranks", [2, 4])
def test_backend_across_processes_on_one_gpu(ranks):
    run_ranks("backend_worker.py", ranks, "backend ok")


@pytest.mark.parametrize("ranks", [2, 4])
def test_ddp_over_the_backend(ranks):
    run_ranks("ddp_worker.py", ranks, "ddp ok")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("ranks", [2, 4])
def test_fsdp_over_the_backend(ranks, dtype):
    run_ranks("fsdp_worker.py", ranks, "fsdp ok", dtype)


@pytest.mark.parametrize("ranks", [2, 4])
def test_random_calls_over_the_backend(ranks):
    run_ranks("backend_random_worker.py", ranks, "random ok", "120")
