"""torch.distributed backend "hoccl": the library's collectives as a PyTorch
process group, selected by an environment variable (the paper's
Implementation section: a backend matching torch.distributed's abstraction,
switched in by one variable).

Setting.  Every process is one rank and all ranks share one GPU (launch them
with torchrun; each calls ``torch.cuda.set_device(0)``).  The library runs a
collective over R device pointers in one process, so each call goes like the
paper's intra-node path (Zero-SM Point-to-Point Executor):

* runtime IPC-handle exchange: every rank exports the allocations that hold
  its buffers (``hoccl_ipc_export``) and publishes the handles in the c10d
  store under the call's sequence number;
* rank 0 opens the other ranks' handles (``hoccl_ipc_open``, cached per
  allocation), runs the collective through the C ABI on its current stream
  over all ranks' buffers, waits for it and publishes completion;
* CPU-based cross-process synchronisation: every rank waits for that
  completion key in the store before the call returns, so its later work
  sees the results.

Point-to-point: the receiver publishes its buffer's handle; the sender opens
it, copies straight into it through the library (the engine proxy by
default) and publishes completion, which the receiver waits for.

Every call synchronises the calling rank's current stream before it
publishes (its inputs are complete and its outputs free) and returns once
the operation has completed: the returned work is already done.  Reductions
are sums.  Buffers must be contiguous CUDA tensors of int32, float32 or
bfloat16 on the shared GPU, in allocations below 2 GiB (larger ones are not
shared), and must not be freed (``torch.cuda.empty_cache``) while the group
lives.  ``destroy_process_group`` closes the opened handles before any rank
may free its memory.

Use::

    from paper_2609_34334_amd import distributed as hdist
    hdist.init_process_group(backend="nccl")   # "hoccl" when HOCCL_BACKEND=1
    torch.distributed.all_reduce(t)
    hdist.destroy_process_group()
"""
import ctypes
import json
import os
from datetime import timedelta

import torch
import torch.distributed as dist

from . import (BF16, FP32, INT32, _check, _DTYPES, ipc_close_all, ipc_export, ipc_open, lib)

BACKEND = "hoccl"
ENV = "HOCCL_BACKEND"
_VP = ctypes.c_void_p
_GROUPS = []


def selected_backend(requested):
    """The backend init_process_group uses: "hoccl" when the environment
    variable HOCCL_BACKEND is set to anything but 0 or empty, else
    `requested`."""
    return BACKEND if os.environ.get(ENV, "0") not in ("", "0") else requested


def register():
    """Register "hoccl" with torch.distributed (idempotent)."""
    if getattr(dist.Backend, BACKEND.upper(), None) == BACKEND:
        return
    dist.Backend.register_backend(BACKEND, _create, devices=["cuda"])


def init_process_group(backend="nccl", **kwargs):
    """torch.distributed.init_process_group with the backend the
    environment selects (see selected_backend)."""
    b = selected_backend(backend)
    if b == BACKEND:
        register()
    dist.init_process_group(backend=b, **kwargs)


def destroy_process_group():
    """Close every IPC mapping the hoccl groups opened, wait until every rank
    has, then destroy the default group."""
    for g in list(_GROUPS):
        g.close()
    dist.destroy_process_group()


def _create(store, rank, world_size, timeout):
    g = HocclProcessGroup(store, rank, world_size, timeout)
    _GROUPS.append(g)
    return g


class _Done(dist._Work):
    """A work item that has already completed."""

    def __init__(self, result=None):
        super().__init__()
        self._fut = torch.futures.Future()
        self._fut.set_result(result)

    def wait(self, timeout=None):
        return True

    def is_completed(self):
        return True

    def get_future(self):
        return self._fut


def _dtype(t):
    if t.dtype not in _DTYPES:
        raise TypeError(f"hoccl: unsupported dtype {t.dtype}")
    if t.device.type != "cuda" or not t.is_contiguous():
        raise ValueError("hoccl: buffers must be contiguous CUDA tensors")
    return _DTYPES[t.dtype]


def _export(t):
    h, off, size = ipc_export(t)
    return {"h": h.hex(), "o": off, "n": size, "dev": t.device.index}


def _open(d):
    return ipc_open(bytes.fromhex(d["h"]), d["o"], d["n"])


def _ptrs(vals):
    return (_VP * len(vals))(*vals)


def _stream():
    return _VP(torch.cuda.current_stream().cuda_stream)


def _sum_only(opts):
    op = getattr(opts, "reduceOp", dist.ReduceOp.SUM)
    if op != dist.ReduceOp.SUM:
        raise ValueError("hoccl: only sum reductions")


class HocclProcessGroup(dist.ProcessGroup):
    """The process group of the "hoccl" backend (see the module docstring)."""

    def __init__(self, store, rank, size, timeout):
        super().__init__(rank, size)
        self._store = dist.PrefixStore("hoccl", store)
        if timeout is not None:
            self._store.set_timeout(timeout if isinstance(timeout, timedelta) else timedelta(seconds=timeout))
        self._r, self._n = rank, size
        self._seq = 0
        self._p2p = {}
        self._closed = False

    def getBackendName(self):
        return BACKEND

    # ---- the collective protocol ----------------------------------------------

    def _call(self, desc, run):
        """Publish this rank's `desc`; rank 0 gathers every rank's and runs
        `run(descs)`; every rank waits for completion."""
        k = self._seq
        self._seq += 1
        torch.cuda.current_stream().synchronize()
        self._store.set(f"c{k}/{self._r}", json.dumps(desc))
        if self._r == 0:
            try:
                descs = [json.loads(self._store.get(f"c{k}/{r}")) for r in range(self._n)]
                if len({d["dev"] for d in descs if "dev" in d}) > 1:
                    raise ValueError("hoccl: all ranks must use the same GPU")
                run(descs)
                torch.cuda.current_stream().synchronize()
                status = "ok"
            except Exception as e:  # every rank must learn of it, not only rank 0
                status = f"error: {e}"
            self._store.set(f"c{k}/done", status)
        status = self._store.get(f"c{k}/done").decode()
        if self._store.add(f"c{k}/ack", 1) == self._n:     # the last reader cleans up
            for key in [f"c{k}/{r}" for r in range(self._n)] + [f"c{k}/done", f"c{k}/ack"]:
                self._store.delete_key(key)
        if status != "ok":
            raise RuntimeError(status)
        return _Done()

    def _resolve(self, descs, field, mine):
        """Device pointers of every rank's `field`: rank 0's own, the others
        through their IPC handles."""
        return [mine if r == 0 else _open(d[field]) for r, d in enumerate(descs)]

    # ---- collectives ---------------------------------------------------------------

    def allreduce(self, tensors, opts=None):
        _sum_only(opts)
        (t,) = tensors
        dt = _dtype(t)
        desc = {"t": _export(t), "numel": t.numel(), "dt": dt, "dev": t.device.index}

        def run(descs):
            if any(d["numel"] != t.numel() or d["dt"] != dt for d in descs):
                raise ValueError("hoccl: all_reduce tensors differ between ranks")
            p = _ptrs(self._resolve(descs, "t", t.data_ptr()))
            _check(lib().hoccl_allreduce(p, p, t.numel(), dt, self._n, _stream()), "hoccl_allreduce")
        return self._call(desc, run)

    def _reduce_scatter_base(self, output, input, opts=None):
        _sum_only(opts)
        dt = _dtype(input)
        if _dtype(output) != dt or input.numel() != self._n * output.numel():
            raise ValueError("hoccl: reduce_scatter needs an input of world_size times the output")
        desc = {"in": _export(input), "out": _export(output), "numel": output.numel(), "dt": dt,
                "dev": input.device.index}

        def run(descs):
            if any(d["numel"] != output.numel() or d["dt"] != dt for d in descs):
                raise ValueError("hoccl: reduce_scatter tensors differ between ranks")
            s = _ptrs(self._resolve(descs, "in", input.data_ptr()))
            r = _ptrs(self._resolve(descs, "out", output.data_ptr()))
            _check(lib().hoccl_reduce_scatter(s, r, output.numel(), dt, self._n, _stream()),
                   "hoccl_reduce_scatter")
        return self._call(desc, run)

    def reduce_scatter(self, output_tensors, input_tensors, opts=None):
        (out,) = output_tensors
        (ins,) = input_tensors
        flat = torch.cat([x.reshape(-1) for x in ins])
        return self._reduce_scatter_base(out, flat, opts)

    def _allgather_base(self, output, input, opts=None):
        dt = _dtype(input)
        if _dtype(output) != dt or output.numel() != self._n * input.numel():
            raise ValueError("hoccl: all_gather needs an output of world_size times the input")
        desc = {"in": _export(input), "out": _export(output), "numel": input.numel(), "dt": dt,
                "dev": input.device.index}

        def run(descs):
            if any(d["numel"] != input.numel() or d["dt"] != dt for d in descs):
                raise ValueError("hoccl: all_gather tensors differ between ranks")
            s = _ptrs(self._resolve(descs, "in", input.data_ptr()))
            r = _ptrs(self._resolve(descs, "out", output.data_ptr()))
            _check(lib().hoccl_allgather(s, r, input.numel(), dt, self._n, _stream()), "hoccl_allgather")
        return self._call(desc, run)

    def allgather(self, output_tensors, input_tensors, opts=None):
        (outs,) = output_tensors
        (inp,) = input_tensors
        flat = torch.empty(self._n * inp.numel(), dtype=inp.dtype, device=inp.device)
        w = self._allgather_base(flat, inp.reshape(-1) if inp.is_contiguous() else inp.contiguous(), opts)
        for r, o in enumerate(outs):
            o.copy_(flat[r * inp.numel():(r + 1) * inp.numel()].view_as(o))
        return w

    def alltoall_base(self, output, input, output_split_sizes, input_split_sizes, opts=None):
        dt = _dtype(input)
        if _dtype(output) != dt:
            raise ValueError("hoccl: all_to_all tensors differ in dtype")
        row_in = input.numel() // max(1, input.size(0)) if input.dim() else 1
        row_out = output.numel() // max(1, output.size(0)) if output.dim() else 1
        if row_in != row_out:
            raise ValueError("hoccl: all_to_all rows differ in size")
        split_in = list(input_split_sizes) or [input.size(0) // self._n] * self._n
        split_out = list(output_split_sizes) or [output.size(0) // self._n] * self._n
        desc = {"in": _export(input), "out": _export(output), "dt": dt, "dev": input.device.index,
                "sin": [s * row_in for s in split_in], "sout": [s * row_out for s in split_out]}

        def run(descs):
            R = self._n
            if any(d["dt"] != dt for d in descs):
                raise ValueError("hoccl: all_to_all dtypes differ between ranks")
            counts, sd, rd = [], [], []
            for s in range(R):
                off = 0
                for d in range(R):
                    c = descs[s]["sin"][d]
                    if descs[d]["sout"][s] != c:
                        raise ValueError(f"hoccl: rank {s} sends {c} elements to rank {d}, which expects "
                                         f"{descs[d]['sout'][s]}")
                    counts.append(c)
                    sd.append(off)
                    off += c
            for s in range(R):
                for d in range(R):
                    rd.append(sum(descs[d]["sout"][:s]))
            S = ctypes.c_size_t * (R * R)
            sp = _ptrs(self._resolve(descs, "in", input.data_ptr()))
            rp = _ptrs(self._resolve(descs, "out", output.data_ptr()))
            _check(lib().hoccl_alltoallv(sp, S(*counts), S(*sd), rp, S(*rd), dt, R, _stream()),
                   "hoccl_alltoallv")
        return self._call(desc, run)

    def barrier(self, opts=None):
        return self._call({}, lambda descs: None)

    # ---- point to point ----------------------------------------------------------------

    def _p2p_key(self, src, dst):
        n = self._p2p.get((src, dst), 0)
        self._p2p[(src, dst)] = n + 1
        return f"p{src}-{dst}/{n}"

    def send(self, tensors, dst, tag=0):
        (t,) = tensors
        dt = _dtype(t)
        key = self._p2p_key(self._r, dst)
        torch.cuda.current_stream().synchronize()
        d = json.loads(self._store.get(key + "/recv"))          # the receiver's buffer
        status = "ok"
        try:
            if d["numel"] != t.numel() or d["dt"] != dt:
                raise ValueError(f"hoccl: send of {t.numel()} elements to a receive of {d['numel']}")
            dst_ptr = _open(d["t"])
            _check(lib().hoccl_sendrecv(_ptrs([t.data_ptr(), None]), _ptrs([None, dst_ptr]),
                                        (ctypes.c_int * 2)(1, -1), t.numel(), dt, 2, _stream()),
                   "hoccl_sendrecv")
            torch.cuda.current_stream().synchronize()
        except Exception as e:
            status = f"error: {e}"
        self._store.set(key + "/done", status)
        if status != "ok":
            raise RuntimeError(status)
        return _Done()

    def recv(self, tensors, src, tag=0):
        (t,) = tensors
        dt = _dtype(t)
        key = self._p2p_key(src, self._r)
        torch.cuda.current_stream().synchronize()
        self._store.set(key + "/recv", json.dumps({"t": _export(t), "numel": t.numel(), "dt": dt}))
        status = self._store.get(key + "/done").decode()
        self._store.delete_key(key + "/recv")
        self._store.delete_key(key + "/done")
        if status != "ok":
            raise RuntimeError(status)
        return _Done()

    # ---- teardown ----------------------------------------------------------------------

    def close(self):
        """Every rank closes the mappings it opened (rank 0 those of the
        collectives, senders those of their receivers) and waits until all
        have, before any may free its memory."""
        if self._closed:
            return
        self.barrier()
        ipc_close_all()
        self.barrier()
        self._closed = True
        if self in _GROUPS:
            _GROUPS.remove(self)


__all__ = ["BACKEND", "ENV", "HocclProcessGroup", "destroy_process_group", "init_process_group",
           "register", "selected_backend", "BF16", "FP32", "INT32"]
