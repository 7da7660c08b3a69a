"""Helpers shared by the GPU tests: numpy (oracle representation) <-> torch
device tensors."""
import numpy as np
import torch

import paper_2609_34334_amd as hc

NAME = {hc.INT32: "int32", hc.FP32: "fp32", hc.BF16: "bf16", hc.UINT8: "uint8"}
TORCH = {hc.INT32: torch.int32, hc.FP32: torch.float32, hc.BF16: torch.bfloat16, hc.UINT8: torch.uint8}
NPDT = {hc.INT32: np.int32, hc.FP32: np.float32, hc.BF16: np.uint16, hc.UINT8: np.uint8}
ES = {hc.INT32: 4, hc.FP32: 4, hc.BF16: 2, hc.UINT8: 1}
CANARY = {hc.INT32: 0x7A5A7A5A, hc.FP32: 0x7A5A7A5A, hc.BF16: 0x7A5A, hc.UINT8: 0x5A}


def to_dev(a, dt):
    a = np.ascontiguousarray(a)
    if dt == hc.BF16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).cuda()
    return torch.from_numpy(a.copy()).cuda()


def from_dev(t, dt):
    t = t.detach().cpu()
    if dt == hc.BF16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()


def bits(a):
    a = np.ascontiguousarray(a)
    return a.view({1: np.uint8, 2: np.uint16, 4: np.uint32}[a.dtype.itemsize])


def assert_bitwise(got, ref, what=""):
    g, r = bits(got), bits(ref)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    if not np.array_equal(g, r):
        bad = np.nonzero(g != r)[0]
        raise AssertionError(f"{what}: {bad.size} mismatches, first at {bad[:5]}: "
                             f"got {g[bad[:5]]} expected {r[bad[:5]]}")


def padded(n, dt, lead=0, trail=16, canary=None):
    """A device buffer with `lead` and `trail` canary elements around an
    n-element window; returns (full buffer, window view)."""
    full = torch.empty(lead + n + trail, dtype=TORCH[dt], device="cuda")
    if canary is None:
        canary = CANARY[dt]
    if dt == hc.UINT8:
        full.fill_(canary)
    else:
        full.view(torch.int16 if dt == hc.BF16 else torch.int32).fill_(
            canary - (1 << 16) if dt == hc.BF16 and canary >= (1 << 15) else canary)
    return full, full[lead:lead + n]


def check_canaries(full, lead, n, dt):
    raw = from_dev(full, dt)
    raw = bits(raw)
    want = CANARY[dt]
    assert (raw[:lead] == want).all() and (raw[lead + n:] == want).all(), "canary overwritten"
