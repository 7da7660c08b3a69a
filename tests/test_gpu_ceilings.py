"""The streaming-ceiling kernels the roofline context is measured with
compute what they claim: a write fills, a copy copies, an add adds, a
read-modify-write adds one, a read leaves its sink alone."""
import pytest
import torch

import paper_2609_34334_amd as hc

pytestmark = pytest.mark.gpu


def test_stream_ceiling_kernels():
    n = (1 << 20) + 64                    # floats: not a multiple of the launch's stride
    a = torch.randn(n, device="cuda")
    b = torch.randn(n, device="cuda")
    c = torch.zeros(n + 16, device="cuda")
    hc.stream_ceiling("write", c=c, nbytes=n * 4)
    torch.cuda.synchronize()
    assert bool((c[:n] == 1.0).all()) and bool((c[n:] == 0).all())
    hc.stream_ceiling("copy", a=a, c=c, nbytes=n * 4)
    torch.cuda.synchronize()
    assert torch.equal(c[:n], a) and bool((c[n:] == 0).all())
    c.zero_()
    hc.stream_ceiling("copy_nt", a=a, c=c, nbytes=n * 4)
    torch.cuda.synchronize()
    assert torch.equal(c[:n], a) and bool((c[n:] == 0).all())
    hc.stream_ceiling("add_nt", a=a, b=b, c=c, nbytes=n * 4)
    torch.cuda.synchronize()
    assert torch.equal(c[:n], a + b) and bool((c[n:] == 0).all())
    assert hc.last_stats()["hbm_bytes_algorithmic"] == 3 * n * 4
    c.zero_()
    hc.stream_ceiling("add", a=a, b=b, c=c, nbytes=n * 4)
    torch.cuda.synchronize()
    assert torch.equal(c[:n], a + b)
    before = c.clone()
    hc.stream_ceiling("rmw", c=c, nbytes=n * 4)
    torch.cuda.synchronize()
    assert torch.equal(c[:n], before[:n] + 1.0) and bool((c[n:] == 0).all())
    sink = torch.full((4,), 7, dtype=torch.int32, device="cuda")
    hc.stream_ceiling("read", a=a, c=sink, nbytes=n * 4)
    torch.cuda.synchronize()
    assert bool((sink == 7).all())
    assert hc.last_stats()["hbm_bytes_algorithmic"] == n * 4
