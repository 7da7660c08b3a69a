"""The reduce-scatter entry point that allocates nothing
(hoccl_reduce_scatter_noalloc), called through the C ABI and compared bit
for bit with the ordinary hoccl_reduce_scatter on the same inputs, over two
calls in a row, the second with a smaller input; plus its size limit.  The
ordinary entry point is itself held to the oracle by the parity tests."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import NAME, TORCH, assert_bitwise, from_dev, to_dev

pytestmark = pytest.mark.gpu

L = hc.lib()
V = ctypes.c_void_p


@pytest.fixture(autouse=True)
def _defaults():
    saved = hc.get_config()
    yield
    hc.set_config(**saved)


def call(fn, send, recv, n, dt):
    R = len(send)
    sp = (V * R)(*[t.data_ptr() for t in send])
    rp = (V * R)(*[t.data_ptr() for t in recv])
    return getattr(L, fn)(sp, rp, n, dt, R, V(torch.cuda.current_stream().cuda_stream))


def canary_like(n, dt, R):
    return [torch.full((n,), 0x5A, dtype=torch.int16 if dt == hc.BF16 else torch.int32,
                       device="cuda").view(TORCH[dt]) for _ in range(R)]


# (R, recvcount, dtype, in place): the first is the DP gradient bucket
# (bf16, R = 8, 3,145,728 per rank out: 100.7 MB of fp32 partials in the
# scratch); the second is smaller and ragged; the third is an in-place
# int32 reduce-scatter, whose partials also go to the scratch.
CASES = [(8, 3_145_728, hc.BF16, False), (5, 4099, hc.FP32, False), (3, 1031, hc.INT32, True)]


@pytest.mark.parametrize("algo", ["ring", "auto"])
def test_noalloc_matches_reduce_scatter_on_calls_in_a_row(algo):
    hc.init(0)
    hc.set_config(reduce_algo=algo)
    for R, n, dt, in_place in CASES:
        print(f"noalloc case algo={algo} R={R} n={n} dt={NAME[dt]} in_place={in_place}", flush=True)
        x = [W.random_values(NAME[dt], 31 + R, r, R * n) for r in range(R)]
        if in_place:
            send_a = [to_dev(a, dt) for a in x]
            send_b = [to_dev(a, dt) for a in x]
            want = [send_a[r][r * n:(r + 1) * n] for r in range(R)]
            got = [send_b[r][r * n:(r + 1) * n] for r in range(R)]
        else:
            send_a = send_b = [to_dev(a, dt) for a in x]
            want, got = canary_like(n, dt, R), canary_like(n, dt, R)
        assert call("hoccl_reduce_scatter", send_a, want, n, dt) == hc.OK
        torch.cuda.synchronize()
        assert call("hoccl_reduce_scatter_noalloc", send_b, got, n, dt) == hc.OK, \
            hc.lib().hoccl_last_error_string()
        st = hc.last_stats()
        torch.cuda.synchronize()
        assert st["reduce_algo_used"] == (hc.REDUCE_RING if algo == "ring" else hc.REDUCE_DIRECT)
        for r in range(R):
            assert_bitwise(from_dev(got[r], dt), from_dev(want[r], dt), f"rank {r}")


def test_noalloc_bf16_partials_fit_twice_the_elements():
    """bf16 partials take 2 bytes per element: a bf16 ring reduce-scatter
    whose fp32 partials would overflow the scratch fits with them, and
    matches hoccl_reduce_scatter in that mode, on two calls in a row, the
    second smaller."""
    hc.init(0)
    hc.set_config(reduce_algo="ring", bf16_partials=1)
    for R, n in ((8, 4_200_000), (5, 3001)):
        print(f"noalloc bf16 partials R={R} n={n}", flush=True)
        x = [W.random_values("bf16", 77 + R, r, R * n) for r in range(R)]
        send = [to_dev(a, hc.BF16) for a in x]
        want, got = canary_like(n, hc.BF16, R), canary_like(n, hc.BF16, R)
        assert call("hoccl_reduce_scatter", send, want, n, hc.BF16) == hc.OK
        torch.cuda.synchronize()
        assert call("hoccl_reduce_scatter_noalloc", send, got, n, hc.BF16) == hc.OK, \
            hc.lib().hoccl_last_error_string()
        torch.cuda.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(got[r], hc.BF16), from_dev(want[r], hc.BF16), f"rank {r}")


def test_noalloc_rejects_what_the_scratch_cannot_hold():
    """A bf16 ring reduce-scatter whose fp32 partials (R * recvcount * 4
    bytes) exceed the 128 MiB scratch is refused before anything is
    enqueued; the outputs keep their contents."""
    hc.init(0)
    hc.set_config(reduce_algo="ring")
    R, n = 8, 4_200_000                      # 134.4 MB of partials
    send = [torch.zeros(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    out = canary_like(n, hc.BF16, R)
    torch.cuda.synchronize()
    assert call("hoccl_reduce_scatter_noalloc", send, out, n, hc.BF16) == hc.ERR_INVALID_ARG
    assert b"scratch" in hc.lib().hoccl_last_error_string()
    torch.cuda.synchronize()
    for r in range(R):
        assert (out[r].view(torch.int16) == 0x5A).all()
