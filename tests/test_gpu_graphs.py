"""Collectives captured into a HIP graph: each replay must equal the eager
result (and the oracle), with eager work and synchronisations between the
replays.  The library clears nothing with hipMemsetAsync, so capture records
only kernels, copies and events."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import assert_bitwise, from_dev, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _defaults():
    saved = hc.get_config()
    yield
    hc.set_config(**saved)


def replay_check(run, outs, ref, dt, label):
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        run(s)                       # eager: allocates the workspace, warms up
    torch.cuda.synchronize()
    for o in outs:
        o.zero_()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        run(s)
    torch.cuda.synchronize()
    for k in range(3):
        for o in outs:
            o.fill_(7)                   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for r, o in enumerate(outs):
            assert_bitwise(from_dev(o, dt), ref[r], f"{label} replay {k} rank {r}")


@pytest.mark.parametrize("algo", ["ring", "direct"])
def test_reduce_scatter_in_a_graph(algo):
    hc.set_config(reduce_algo=algo)
    R, n = 8, 100_003
    x = [W.random_values("bf16", 301, r, R * n) for r in range(R)]
    ref = oracle.reduce_scatter_new(x, hc.BF16)
    send = [to_dev(a, hc.BF16) for a in x]
    outs = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    replay_check(lambda s: hc.reduce_scatter(send, outs, stream=s), outs, ref, hc.BF16, algo)


@pytest.mark.parametrize("algo", ["ring", "direct"])
def test_bf16_partials_in_a_graph(algo):
    """bf16 partials rounded at every hop: reduce-scatter and all-reduce
    (whose gather copies go to the default copy path) replay to the
    oracle's per-hop-rounding sums."""
    hc.set_config(reduce_algo=algo, bf16_partials=1)
    R, n = 8, 100_003
    x = [W.random_values("bf16", 304, r, R * n) for r in range(R)]
    ref = oracle.reduce_scatter_bf16_hops_new(x)
    send = [to_dev(a, hc.BF16) for a in x]
    outs = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    replay_check(lambda s: hc.reduce_scatter(send, outs, stream=s), outs, ref, hc.BF16,
                 "RS bf16 partials " + algo)
    xa = [W.random_values("bf16", 305, r, 70_001) for r in range(R)]
    refa = oracle.allreduce_bf16_hops_new(xa)
    senda = [to_dev(a, hc.BF16) for a in xa]
    outa = [torch.empty(70_001, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    replay_check(lambda s: hc.allreduce(senda, outa, stream=s), outa, refa, hc.BF16,
                 "AR bf16 partials " + algo)


@pytest.mark.parametrize("path", ["auto", "engines", "hip", "kernel"])
def test_allgather_and_allreduce_in_a_graph(path):
    """On AUTO and the engine proxy the copies are recorded as a host node
    that issues them on the SDMA engines at every replay."""
    if path == "engines" and hc.sdma_engine_count() == 0:
        pytest.skip("engine proxy unavailable")
    hc.set_config(copy_path=path)
    R, n = 8, 50_021
    x = [W.random_bits(302, r, n, 2) for r in range(R)]
    ref = oracle.allgather_new(x, hc.BF16)
    send = [to_dev(a, hc.BF16) for a in x]
    outs = [torch.empty(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    replay_check(lambda s: hc.allgather(send, outs, stream=s), outs, ref, hc.BF16, "AG " + path)
    xa = [W.random_values("fp32", 303, r, 40_000) for r in range(4)]
    refa = oracle.allreduce_new(xa, hc.FP32)
    senda = [to_dev(a, hc.FP32) for a in xa]
    outa = [torch.empty(40_000, device="cuda") for _ in range(4)]
    replay_check(lambda s: hc.allreduce(senda, outa, stream=s), outa, refa, hc.FP32, "AR " + path)


def test_eager_calls_after_a_captured_call():
    """The copy streams a capture forked into are usable eagerly afterwards,
    and the captured graph keeps replaying correctly after an eager call made
    the workspace grow (the captured workspace is retired, not freed)."""
    R, n = 8, 30_011
    x = [W.random_values("bf16", 304, r, R * n) for r in range(R)]
    ref = oracle.reduce_scatter_new(x, hc.BF16)
    send = [to_dev(a, hc.BF16) for a in x]
    outs = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    hc.finalize()                                 # start from an empty workspace
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        hc.reduce_scatter(send, outs, stream=s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        hc.reduce_scatter(send, outs, stream=s)
    torch.cuda.synchronize()
    # An eager call 8x larger grows the workspace.
    m = 8 * n
    xb = [W.random_values("bf16", 305, r, R * m) for r in range(R)]
    refb = oracle.reduce_scatter_new(xb, hc.BF16)
    sendb = [to_dev(a, hc.BF16) for a in xb]
    outb = hc.reduce_scatter(sendb)
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(outb[r], hc.BF16), refb[r], f"eager larger rank {r}")
    for k in range(2):
        for o in outs:
            o.fill_(3)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(outs[r], hc.BF16), ref[r], f"replay after growth {k} rank {r}")
    # Eager SDMA all-gather with several copy chains after the capture.
    xa = [W.random_bits(306, r, 4099, 2) for r in range(R)]
    refa = oracle.allgather_new(xa, hc.BF16)
    outa = hc.allgather([to_dev(a, hc.BF16) for a in xa])
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(outa[r], hc.BF16), refa[r], f"eager allgather rank {r}")
    del g


def _capture(stream, fn):
    """Runs fn between hipStreamBeginCapture (relaxed mode) and
    hipStreamEndCapture on `stream`, returns fn's exception (or None)."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so.7")          # the HIP runtime torch has loaded
    h = ctypes.c_void_p(stream.cuda_stream)
    assert hip.hipStreamBeginCapture(h, 2) == 0
    err = None
    try:
        fn()
    except hc.HocclError as e:
        err = e
    graph = ctypes.c_void_p()
    assert hip.hipStreamEndCapture(h, ctypes.byref(graph)) == 0
    if graph.value:
        assert hip.hipGraphDestroy(graph) == 0
    return err


def test_capture_refuses_to_allocate_or_to_record_the_handshake_kernel():
    R, n = 8, 20_000
    send = [torch.ones(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    outs = [torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
    hc.finalize()                                  # no library state at all
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    err = _capture(s, lambda: hc.reduce_scatter(send, outs, stream=s))
    assert err is not None and err.status == hc.ERR_UNSUPPORTED, err
    assert "not initialised" in str(err)
    hc.init()                                      # state, but no workspace yet
    err = _capture(s, lambda: hc.reduce_scatter(send, outs, stream=s))
    assert err is not None and err.status == hc.ERR_UNSUPPORTED, err
    assert "workspace" in str(err)
    # The refusal enqueued nothing; the same call now runs eagerly.
    hc.reduce_scatter(send, outs, stream=s)
    torch.cuda.synchronize()
    assert torch.equal(outs[3], torch.full((n,), 8.0, dtype=torch.bfloat16, device="cuda"))
    if hc.sdma_engine_count() > 0:
        # The engine proxy's handshake kernel waits for copies its thread
        # issues at call time: it cannot be recorded.  (The default
        # host-function form can.)
        hc.set_config(copy_path="engines", proxy_handshake=0)
        a = [torch.ones(n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
        b = [torch.empty(R * n, dtype=torch.bfloat16, device="cuda") for _ in range(R)]
        err = _capture(s, lambda: hc.allgather(a, b, stream=s))
        assert err is not None and err.status == hc.ERR_UNSUPPORTED, err
        assert "captured" in str(err)
