"""torch.distributed backend "hoccl": the library's collectives as a PyTorch
process group, selected by an environment variable (the paper's
Implementation section: a backend matching torch.distributed's abstraction,
switched in by one variable).

Setting.  Every process is one rank and all ranks share one GPU (launch them
with torchrun; each calls ``torch.cuda.set_device(0)``).  The library runs a
collective over R device pointers in one process, so each call goes like the
paper's intra-node path (Zero-SM Point-to-Point Executor):

* runtime IPC-handle exchange: every rank exports the allocations that hold
  its buffers (``hoccl_ipc_export``) and posts the handles, with the call's
  sequence number, into its slot of the group's shared-memory mailbox
  (``hoccl_mailbox_*``);
* rank 0 waits for every rank's slot, opens the other ranks' handles
  (``hoccl_ipc_open``, cached per allocation), runs the collective through
  the C ABI on its current stream over all ranks' buffers, waits for it and
  posts the status into the mailbox's status slot;
* CPU-based cross-process synchronisation: every rank waits for that status
  before the call returns, so its later work sees the results.  The
  mailbox is the paper's shared-memory semaphores: a waiter polls briefly,
  then sleeps on a futex.

Point-to-point: the receiver posts its buffer's handle into the mailbox
slot of the (sender, receiver) pair and returns; the sender hands its
buffer to the group's send thread and returns.  That thread opens the
receiver's handle as soon as it is posted, copies straight into it through
the library (the engine proxy by default) and posts completion, which both
sides' waits wait for.  Both calls return at once, so batch_isend_irecv,
and any order of sends, receives and waits across ranks, cannot deadlock.
The library serialises calls from several host threads on one device, so
the calling thread's collectives and the send thread's copies take turns.

The c10d store is used once, when the group is created: rank 0 creates the
mailboxes and publishes their names, every rank opens them, and once all
have, rank 0 removes the names (the mappings stay, and nothing is left in
/dev/shm when the processes exit).

Broadcast is a one-row all-to-all(v): the root's buffer is copied into every
other rank's.  Scatter and gather are the same with the root's buffer cut
into blocks (one column for gather); reduce is an all-reduce of copies;
the list forms of all-gather and all-to-all stage through flat buffers.

Every call synchronises the calling rank's current stream before it
publishes (its inputs are complete and its outputs free) and returns once
the operation has completed: the returned work is already done, and its
future holds the output tensors (as DistributedDataParallel's reducer
expects).  Reductions are sums of int32, float32 or bfloat16, or averages
of float32 or bfloat16 (FSDP's gradient reduce-scatter): the sum, rounded
once to the dtype, then divided by the world size in that dtype on the
caller's stream (exact when the world size is a power of two).  The copy
collectives (broadcast, all-gather, all-to-all, send/recv) move bytes, so
they take any dtype; the library copies them in 4-, 2- or 1-byte units,
the widest that divides every count and offset (so all_gather_object and
broadcast_object_list work too).  Buffers must be contiguous CUDA
tensors on the shared GPU, in allocations below 2 GiB (larger ones are not
shared), and must not be freed (``torch.cuda.empty_cache``) while the group
lives.  ``destroy_process_group`` closes the opened handles before any rank
may free its memory.  With these, torch.nn.parallel.DistributedDataParallel
(parameter and buffer broadcast, gradient buckets) and FSDP2's fully_shard
(parameter all-gathers, averaging gradient reduce-scatters) run over the
backend, and so do torch's functional collectives (all_gather_tensor,
reduce_scatter_tensor, all_reduce(_coalesced), all_to_all_single,
broadcast), which DTensor redistribution such as ``full_tensor()`` uses.

Use::

    from paper_2609_34334_amd import distributed as hdist
    hdist.init_process_group(backend="nccl")   # "hoccl" when HOCCL_BACKEND=1
    torch.distributed.all_reduce(t)
    hdist.destroy_process_group()
"""
import ctypes
import functools
import json
import os
import secrets
import threading
import time
from datetime import timedelta

import torch
import torch.distributed as dist

from . import (BF16, FP32, INT32, UINT8, Mailbox, _check, _DTYPES, ipc_close_all, ipc_export, ipc_open,
               lib)

BACKEND = "hoccl"
ENV = "HOCCL_BACKEND"
_VP = ctypes.c_void_p
_GROUPS = []
COLL_SLOT_BYTES = 64 << 10    # one rank's call description (handles, split sizes)
P2P_SLOT_BYTES = 512          # a receive buffer's handle, or a completion status
P2P_DEPTH = 4                 # receives a rank may have outstanding per sender
SEND_SPIN_S = 50e-6           # how long a send waits for its receiver before handing off


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


class _SendWork(dist._Work):
    """A send: done once the group's send thread has copied the buffer
    into the receiver's and posted completion."""

    def __init__(self, t, timeout_s):
        super().__init__()
        self._t, self._timeout_s = t, timeout_s
        self._event, self._status = threading.Event(), None
        self._fut = torch.futures.Future()

    def _finish(self, status):
        self._status = status
        self._event.set()
        if status == "ok":
            self._fut.set_result([self._t])
        else:
            self._fut.set_exception(RuntimeError(status))

    def wait(self, timeout=None):
        if not self._event.wait(self._timeout_s):
            raise RuntimeError("hoccl: send not completed: no matching receive was posted in time")
        if self._status != "ok":
            raise RuntimeError(self._status)
        return True

    def is_completed(self):
        return self._event.is_set()

    def get_future(self):
        return self._fut


class _RecvWork(dist._Work):
    """A receive: done once the sender has posted completion."""

    def __init__(self, box, slot, n, t, timeout_ms):
        super().__init__()
        self._box, self._slot, self._n, self._t, self._timeout_ms = box, slot, n, t, timeout_ms
        self._status = None
        self._fut = torch.futures.Future()

    def wait(self, timeout=None):
        if self._status is None:
            self._box.wait(self._slot, self._n, self._timeout_ms)
            self._status = self._box.read(self._slot).decode(errors="replace")
            if self._status == "ok":
                self._fut.set_result([self._t])
            else:
                self._fut.set_exception(RuntimeError(self._status))
        if self._status != "ok":
            raise RuntimeError(self._status)
        return True

    def is_completed(self):
        return self._status is not None or self._box.ready(self._slot, self._n)

    def get_future(self):
        return self._fut


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


def _check_buffer(t):
    if t.device.type != "cuda" or not t.is_contiguous():
        raise ValueError("hoccl: buffers must be contiguous CUDA tensors")


def _dtype(t):
    """The library dtype of a reduction's buffer."""
    if t.dtype not in _DTYPES:
        raise TypeError(f"hoccl: reductions take int32, float32 or bfloat16, not {t.dtype}")
    _check_buffer(t)
    return _DTYPES[t.dtype]


def _nbytes(t):
    _check_buffer(t)
    return t.numel() * t.element_size()


def _unit(byte_counts):
    """(library dtype, unit bytes) of a copy: copies move bits, so the dtype
    only sets the unit, the largest of 4, 2 and 1 bytes that divides every
    count and offset."""
    for size, dt in ((4, INT32), (2, BF16)):
        if all(b % size == 0 for b in byte_counts):
            return dt, size
    return UINT8, 1


def _export(t):
    if t.numel() == 0:
        return None                           # no allocation to share; nothing is copied
    h, off, size = ipc_export(t)
    return {"h": h.hex(), "o": off, "n": size, "dev": t.device.index}


def _open(d):
    return None if d is None else ipc_open(bytes.fromhex(d["h"]), d["o"], d["n"])


def _ptrs(vals):
    return (_VP * len(vals))(*vals)


def _stream():
    return _VP(torch.cuda.current_stream().cuda_stream)


def _average(opts, t):
    """Whether the reduction is an average: SUM, or AVG (FSDP's gradient
    reduce-scatter) of float32 or bfloat16, which is the library's sum
    divided by the world size afterwards."""
    op = getattr(opts, "reduceOp", dist.ReduceOp.SUM)
    if op == dist.ReduceOp.SUM:
        return False
    if op == dist.ReduceOp.AVG and t.dtype in (torch.float32, torch.bfloat16):
        return True
    raise ValueError(f"hoccl: only sums, and averages of float32 or bfloat16 ({op} on {t.dtype})")


def _together(method):
    """A collective whose checks fail on this rank before it joins the call
    still joins it, with the error as its description, so that every rank
    fails at once instead of waiting for this one."""
    @functools.wraps(method)
    def wrapper(self, *args, **kwargs):
        joined = self._seq
        try:
            return method(self, *args, **kwargs)
        except Exception as e:
            if self._seq == joined:
                msg = f"rank {self._r}: {e}"
                self._call(lambda: {"error": msg}, lambda descs: None)
            raise
    return wrapper


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
        self._name, self._desc = "", ""
        t = timeout.total_seconds() if isinstance(timeout, timedelta) else timeout
        self._timeout_ms = int(1000 * t) if t else 30 * 60 * 1000
        self._sends, self._cv, self._sender = [], threading.Condition(), None
        self._recvs = {}                  # (src, dst) -> {message number: its receive}
        self._open_mailboxes()

    def _open_mailboxes(self):
        """Rank 0 creates the collective mailbox (a slot per rank plus the
        status slot) and the point-to-point one (P2P_DEPTH pairs of slots
        per ordered pair of ranks); every rank opens them; rank 0 removes
        the names once all have."""
        if self._r == 0:
            base = f"/hoccl-{os.getpid()}-{secrets.token_hex(6)}"
            try:
                self._coll = Mailbox(base + "-c", self._n + 1, COLL_SLOT_BYTES)
                self._pp = Mailbox(base + "-p", 2 * P2P_DEPTH * self._n * self._n, P2P_SLOT_BYTES)
            except Exception as e:             # the other ranks wait for the name
                self._store.set("mailbox", f"error: {e}")
                raise
            self._store.set("mailbox", base)
        else:
            base = self._store.get("mailbox").decode()
            if base.startswith("error: "):
                raise RuntimeError(f"hoccl: rank 0 could not create the group's mailboxes ({base[7:]})")
            self._coll = Mailbox(base + "-c")
            self._pp = Mailbox(base + "-p")
        if self._store.add("mailbox-opened", 1) == self._n:
            self._store.set("mailbox-all", "1")
        self._store.get("mailbox-all")
        if self._r == 0:
            Mailbox.unlink(base + "-c")
            Mailbox.unlink(base + "-p")

    def getBackendName(self):
        return BACKEND

    # torch keeps a group's name in its C++ backends, which a process group
    # written in Python has none of; these keep it here (DeviceMesh, and so
    # FSDP2, looks groups up by name).
    def getGroupName(self):
        return self._name

    def setGroupName(self, name):
        self._name = name

    def getGroupDesc(self):
        return self._desc

    def setGroupDesc(self, desc):
        self._desc = desc

    @property
    def _device_types(self):
        """The devices the group serves, as torch reads them to place the
        tensors of its object collectives (all_gather_object and the like);
        torch would list its C++ backends, of which this group has none."""
        return [torch.device("cuda")]

    # ---- the collective protocol ----------------------------------------------

    def _call(self, desc, run, result=None):
        """Post this rank's description (`desc()`: its buffers' handles and
        sizes); rank 0 gathers every rank's and runs `run(descs)`; every
        rank waits for completion.  The work's future holds `result` (the
        output tensors).  A rank that cannot describe its buffers posts the
        error instead, so every rank fails at once rather than wait.  A rank
        posts call k + 1 only after it has seen call k's status, so rank 0
        has read every slot before it is written again."""
        self._seq += 1
        k, R, box = self._seq, self._n, self._coll
        torch.cuda.current_stream().synchronize()
        try:
            mine = desc()
        except Exception as e:
            mine = {"error": f"rank {self._r}: {e}"}
        if self._r != 0:
            box.post(self._r, k, json.dumps(mine).encode()[:COLL_SLOT_BYTES])
        else:
            try:
                descs = [mine]
                for r in range(1, R):
                    box.wait(r, k, self._timeout_ms)
                    descs.append(json.loads(box.read(r)))
                for d in descs:
                    if "error" in d:
                        raise ValueError(d["error"])
                if len({d["dev"] for d in descs if "dev" in d}) > 1:
                    raise ValueError("hoccl: all ranks must use the same GPU")
                run(descs)
                torch.cuda.current_stream().synchronize()
                status = "ok"
            except Exception as e:  # every rank must learn of it, not only rank 0
                status = f"error: {e}"
            box.post(R, k, status.encode()[:COLL_SLOT_BYTES])
        box.wait(R, k, self._timeout_ms)
        status = box.read(R).decode(errors="replace")
        if status != "ok":
            raise RuntimeError(status)
        return _Done(result)

    def _resolve(self, descs, field, mine):
        """Device pointers of every rank's `field`: rank 0's own, the others
        through their IPC handles."""
        return [mine if r == 0 else _open(d[field]) for r, d in enumerate(descs)]

    # ---- collectives ---------------------------------------------------------------

    @_together
    def allreduce(self, tensors, opts=None):
        (t,) = tensors
        avg = _average(opts, t)
        dt = _dtype(t)
        desc = lambda: {"t": _export(t), "numel": t.numel(), "dt": dt, "dev": t.device.index}

        def run(descs):
            if any(d["numel"] != t.numel() or d["dt"] != dt for d in descs):
                raise ValueError("hoccl: all_reduce tensors differ between ranks")
            p = _ptrs(self._resolve(descs, "t", t.data_ptr()))
            _check(lib().hoccl_allreduce(p, p, t.numel(), dt, self._n, _stream()), "hoccl_allreduce")
        w = self._call(desc, run, [t])
        if avg:
            t.div_(self._n)
        return w

    def allreduce_coalesced(self, tensors, opts=None):
        for t in tensors:
            self.allreduce([t], opts)
        return _Done(list(tensors))

    @_together
    def broadcast(self, tensors, opts=None):
        """The root's tensor into every rank's: an all-to-all(v) whose only
        nonzero row is the root's, every copy reading the root's whole
        buffer."""
        (t,) = tensors
        root = getattr(opts, "rootRank", 0)
        if not 0 <= root < self._n:
            raise ValueError(f"hoccl: broadcast root {root} outside 0..{self._n - 1}")
        nb = _nbytes(t)
        desc = lambda: {"t": _export(t), "bytes": nb, "type": str(t.dtype), "dev": t.device.index}

        def run(descs):
            R = self._n
            if any(d["bytes"] != nb or d["type"] != str(t.dtype) for d in descs):
                raise ValueError("hoccl: broadcast tensors differ between ranks")
            dt, u = _unit([nb])
            p = _ptrs(self._resolve(descs, "t", t.data_ptr()))
            S = ctypes.c_size_t * (R * R)
            counts = S(*[nb // u if s == root and d != root else 0 for s in range(R) for d in range(R)])
            zero = S()
            _check(lib().hoccl_alltoallv(p, counts, zero, p, zero, dt, R, _stream()), "hoccl_alltoallv")
        return self._call(desc, run, [t])

    @_together
    def _reduce_scatter_base(self, output, input, opts=None):
        avg = _average(opts, input)
        dt = _dtype(input)
        if _dtype(output) != dt or input.numel() != self._n * output.numel():
            raise ValueError("hoccl: reduce_scatter needs an input of world_size times the output")
        desc = lambda: {"in": _export(input), "out": _export(output), "numel": output.numel(), "dt": dt,
                "dev": input.device.index}

        def run(descs):
            if any(d["numel"] != output.numel() or d["dt"] != dt for d in descs):
                raise ValueError("hoccl: reduce_scatter tensors differ between ranks")
            s = _ptrs(self._resolve(descs, "in", input.data_ptr()))
            r = _ptrs(self._resolve(descs, "out", output.data_ptr()))
            _check(lib().hoccl_reduce_scatter(s, r, output.numel(), dt, self._n, _stream()),
                   "hoccl_reduce_scatter")
        w = self._call(desc, run, [output])
        if avg:
            output.div_(self._n)
        return w

    def reduce_scatter_tensor_coalesced(self, outputs, inputs, opts=None):
        """One reduce-scatter per pair (torch's functional reduce_scatter_tensor
        arrives here)."""
        for o, i in zip(outputs, inputs):
            self._reduce_scatter_base(o, i, opts)
        return _Done(list(outputs))

    def reduce_scatter(self, output_tensors, input_tensors, opts=None):
        (out,) = output_tensors
        (ins,) = input_tensors
        flat = torch.cat([x.reshape(-1) for x in ins])
        return self._reduce_scatter_base(out, flat, opts)

    @_together
    def _allgather_base(self, output, input, opts=None):
        nb = _nbytes(input)
        if output.dtype != input.dtype or _nbytes(output) != self._n * nb:
            raise ValueError("hoccl: all_gather needs an output of world_size times the input")
        desc = lambda: {"in": _export(input), "out": _export(output), "bytes": nb, "type": str(input.dtype),
                "dev": input.device.index}

        def run(descs):
            if any(d["bytes"] != nb or d["type"] != str(input.dtype) for d in descs):
                raise ValueError("hoccl: all_gather tensors differ between ranks")
            dt, u = _unit([nb])
            s = _ptrs(self._resolve(descs, "in", input.data_ptr()))
            r = _ptrs(self._resolve(descs, "out", output.data_ptr()))
            _check(lib().hoccl_allgather(s, r, nb // u, dt, self._n, _stream()), "hoccl_allgather")
        return self._call(desc, run, [output])

    def allgather_into_tensor_coalesced(self, outputs, inputs, opts=None):
        """One all-gather per pair (torch's functional all_gather_tensor, and
        so DTensor's full_tensor(), arrives here)."""
        for o, i in zip(outputs, inputs):
            self._allgather_base(o, i, opts)
        return _Done(list(outputs))

    def allgather(self, output_tensors, input_tensors, opts=None):
        (outs,) = output_tensors
        (inp,) = input_tensors
        flat = torch.empty(self._n * inp.numel(), dtype=inp.dtype, device=inp.device)
        w = self._allgather_base(flat, inp.reshape(-1) if inp.is_contiguous() else inp.contiguous(), opts)
        for r, o in enumerate(outs):
            o.copy_(flat[r * inp.numel():(r + 1) * inp.numel()].view_as(o))
        return _Done([outs])

    @_together
    def alltoall_base(self, output, input, output_split_sizes, input_split_sizes, opts=None):
        if output.dtype != input.dtype:
            raise ValueError("hoccl: all_to_all tensors differ in dtype")
        _check_buffer(input)
        _check_buffer(output)
        es = input.element_size()
        row_in = input.numel() // max(1, input.size(0)) if input.dim() else 1
        row_out = output.numel() // max(1, output.size(0)) if output.dim() else 1
        if row_in != row_out:
            raise ValueError("hoccl: all_to_all rows differ in size")
        split_in = list(input_split_sizes) or [input.size(0) // self._n] * self._n
        split_out = list(output_split_sizes) or [output.size(0) // self._n] * self._n
        desc = lambda: {"in": _export(input), "out": _export(output), "type": str(input.dtype),
                "dev": input.device.index,
                "sin": [s * row_in * es for s in split_in], "sout": [s * row_out * es for s in split_out]}

        def run(descs):
            R = self._n
            if any(d["type"] != str(input.dtype) for d in descs):
                raise ValueError("hoccl: all_to_all dtypes differ between ranks")
            counts, sd, rd = [], [], []           # in bytes until the unit is known
            for s in range(R):
                off = 0
                for d in range(R):
                    c = descs[s]["sin"][d]
                    if descs[d]["sout"][s] != c:
                        raise ValueError(f"hoccl: rank {s} sends {c // es} elements to rank {d}, which "
                                         f"expects {descs[d]['sout'][s] // es}")
                    counts.append(c)
                    sd.append(off)
                    off += c
            for s in range(R):
                for d in range(R):
                    rd.append(sum(descs[d]["sout"][:s]))
            dt, u = _unit(counts + sd + rd)
            S = ctypes.c_size_t * (R * R)
            units = lambda v: S(*[b // u for b in v])
            sp = _ptrs(self._resolve(descs, "in", input.data_ptr()))
            rp = _ptrs(self._resolve(descs, "out", output.data_ptr()))
            _check(lib().hoccl_alltoallv(sp, units(counts), units(sd), rp, units(rd), dt, R, _stream()),
                   "hoccl_alltoallv")
        return self._call(desc, run, [output])

    # ---- rooted and list forms, built on the above ------------------------------------
    # They stage through flat buffers (torch copies on the caller's stream)
    # where the library's forms need one buffer per rank.

    @_together
    def _rooted(self, mine, root, to_root):
        """One all-to-all(v) whose only nonzero row (to_root False: the
        root's buffer cut into R blocks, block d to rank d) or column
        (to_root True: every rank's buffer to block r of the root's) is the
        root's.  `mine` is this rank's flat buffer: R blocks on the root and
        one block elsewhere."""
        R = self._n
        if not 0 <= root < R:
            raise ValueError(f"hoccl: root {root} outside 0..{R - 1}")
        nb = _nbytes(mine) // (R if self._r == root else 1)
        desc = lambda: {"t": _export(mine), "bytes": nb, "type": str(mine.dtype), "dev": mine.device.index}

        def run(descs):
            if any(d["bytes"] != nb or d["type"] != str(mine.dtype) for d in descs):
                raise ValueError("hoccl: gather/scatter tensors differ between ranks")
            dt, u = _unit([nb])
            p = _ptrs(self._resolve(descs, "t", mine.data_ptr()))
            S = ctypes.c_size_t * (R * R)
            n = nb // u
            if to_root:      # rank s's block to block s of the root's buffer
                counts = [n if d == root and s != root else 0 for s in range(R) for d in range(R)]
                sd = [0] * (R * R)
                rd = [s * n if d == root else 0 for s in range(R) for d in range(R)]
            else:            # block d of the root's buffer to rank d
                counts = [n if s == root and d != root else 0 for s in range(R) for d in range(R)]
                sd = [d * n if s == root else 0 for s in range(R) for d in range(R)]
                rd = [0] * (R * R)
            _check(lib().hoccl_alltoallv(p, S(*counts), S(*sd), p, S(*rd), dt, R, _stream()),
                   "hoccl_alltoallv")
        return self._call(desc, run)

    def gather(self, output_tensors, input_tensors, opts=None):
        (inp,) = input_tensors
        root = getattr(opts, "rootRank", 0)
        n = inp.numel()
        if self._r == root:
            flat = torch.empty(self._n * n, dtype=inp.dtype, device=inp.device)
            flat[root * n:(root + 1) * n].copy_(inp.reshape(-1))
            self._rooted(flat, root, True)
            (outs,) = output_tensors
            for r, o in enumerate(outs):
                o.copy_(flat[r * n:(r + 1) * n].view_as(o))
            return _Done(output_tensors)
        self._rooted(inp.contiguous().reshape(-1), root, True)
        return _Done([])

    def scatter(self, output_tensors, input_tensors, opts=None):
        (out,) = output_tensors
        root = getattr(opts, "rootRank", 0)
        if self._r == root:
            (ins,) = input_tensors
            flat = torch.cat([x.reshape(-1) for x in ins])
            self._rooted(flat, root, False)
            out.copy_(ins[root].view_as(out))
        else:
            dst = out if out.is_contiguous() else torch.empty_like(out, memory_format=torch.contiguous_format)
            self._rooted(dst.reshape(-1), root, False)
            if dst is not out:
                out.copy_(dst)
        return _Done([out])

    def reduce(self, tensors, opts=None):
        """The sum (or average) into the root's tensor only: an all-reduce of
        copies, the root's result copied back."""
        (t,) = tensors
        tmp = t.clone()
        self.allreduce([tmp], opts)
        if self._r == getattr(opts, "rootRank", 0):
            t.copy_(tmp)
        return _Done([t])

    def alltoall(self, output_tensors, input_tensors, opts=None):
        flat_in = torch.cat([x.reshape(-1) for x in input_tensors])
        flat_out = torch.empty(sum(o.numel() for o in output_tensors), dtype=flat_in.dtype,
                               device=flat_in.device)
        self.alltoall_base(flat_out, flat_in, [o.numel() for o in output_tensors],
                           [x.numel() for x in input_tensors], opts)
        off = 0
        for o in output_tensors:
            o.copy_(flat_out[off:off + o.numel()].view_as(o))
            off += o.numel()
        return _Done(output_tensors)

    def barrier(self, opts=None):
        return self._call(dict, lambda descs: None)

    # ---- point to point ----------------------------------------------------------------

    def _p2p_slot(self, src, dst):
        """(slot of the receiver's buffer, slot of the completion, message
        number) of the next message from src to dst.  Each ordered pair has
        P2P_DEPTH pairs of slots, used in turn, so that a receiver can post
        that many receives from one sender before the first completes."""
        n = self._p2p.get((src, dst), 0) + 1
        self._p2p[(src, dst)] = n
        base = 2 * ((src * self._n + dst) * P2P_DEPTH + n % P2P_DEPTH)
        return base, base + 1, n

    # Point to point is asynchronous on both sides, so that no order of
    # sends, receives and waits across ranks can deadlock: a receive posts
    # its buffer and returns; a send hands its buffer to the group's send
    # thread and returns; that thread copies each pending send as soon as
    # its receiver has posted, and posts completion, which the receive's
    # wait (and the send's) waits for.

    def send(self, tensors, dst, tag=0):
        (t,) = tensors
        _nbytes(t)
        want, done, n = self._p2p_slot(self._r, dst)
        torch.cuda.current_stream().synchronize()          # the buffer is complete
        work = _SendWork(t, self._timeout_ms / 1000)
        with self._cv:
            idle = not self._sends
        inline = False
        if idle:
            # No earlier send waits: if the receiver is there, or arrives
            # within SEND_SPIN_S, copy now on the caller's stream (a hand-off
            # to the send thread costs more than that).
            t0 = time.perf_counter()
            while True:
                if self._pp.ready(want, n):
                    inline = True
                    break
                if time.perf_counter() - t0 > SEND_SPIN_S:
                    break
        if inline:
            status = self._copy_out(t, want, torch.cuda.current_stream())
            self._pp.post(done, n, status.encode()[:P2P_SLOT_BYTES])
            work._finish(status)
            return work
        with self._cv:
            if self._sender is None:
                self._sender = threading.Thread(target=self._send_loop, args=(t.device,),
                                                name="hoccl-send", daemon=True)
                self._sender.start()
            self._sends.append((want, done, n, t, work))
            self._cv.notify()
        return work

    def recv(self, tensors, src, tag=0):
        (t,) = tensors
        nb = _nbytes(t)
        want, done, n = self._p2p_slot(src, self._r)
        mine = self._recvs.setdefault((src, self._r), {})
        older = mine.pop(n - P2P_DEPTH, None)
        if older is not None:
            older.wait()                 # it used the slots this receive reuses
        torch.cuda.current_stream().synchronize()          # the buffer is free
        self._pp.post(want, n, json.dumps({"t": _export(t), "bytes": nb, "type": str(t.dtype)}).encode())
        work = _RecvWork(self._pp, done, n, t, self._timeout_ms)
        mine[n] = work
        return work

    def _send_loop(self, device):
        """Copies every pending send whose receiver has posted, in any order
        across receivers, each on this thread's own stream."""
        torch.cuda.set_device(device)
        stream = torch.cuda.Stream(device)
        while True:
            with self._cv:
                while not self._sends:
                    if self._closed:
                        return
                    self._cv.wait()
                pending = list(self._sends)
            moved = False
            for item in pending:
                want, done, n, t, work = item
                if not self._pp.ready(want, n):
                    continue
                status = self._copy_out(t, want, stream)
                self._pp.post(done, n, status.encode()[:P2P_SLOT_BYTES])
                with self._cv:
                    self._sends.remove(item)
                work._finish(status)
                moved = True
            if not moved:                       # sleep until the oldest receiver posts (or 1 ms)
                try:
                    self._pp.wait(pending[0][0], pending[0][2], 1)
                except Exception:
                    pass

    def _copy_out(self, t, want, stream):
        nb = _nbytes(t)
        try:
            d = json.loads(self._pp.read(want))            # the receiver's buffer
            if d["bytes"] != nb or d["type"] != str(t.dtype):
                raise ValueError(f"hoccl: send of {nb} bytes of {t.dtype} to a receive of "
                                 f"{d['bytes']} bytes of {d['type']}")
            if nb:
                dt, u = _unit([nb])
                with torch.cuda.stream(stream):
                    dst_ptr = _open(d["t"])
                    _check(lib().hoccl_sendrecv(_ptrs([t.data_ptr(), None]), _ptrs([None, dst_ptr]),
                                                (ctypes.c_int * 2)(1, -1), nb // u, dt, 2, _stream()),
                           "hoccl_sendrecv")
                    stream.synchronize()
            return "ok"
        except Exception as e:
            return f"error: {e}"

    # ---- teardown ----------------------------------------------------------------------

    def close(self):
        """Every rank closes the mappings it opened (rank 0 those of the
        collectives, senders those of their receivers) and waits until all
        have, before any may free its memory."""
        if self._closed:
            return
        for *_, work in list(self._sends):              # sends still waiting for their receivers
            work.wait()
        self.barrier()
        ipc_close_all()
        self.barrier()
        with self._cv:
            self._closed = True
            self._cv.notify()
        if self._sender is not None:
            self._sender.join()
        self._coll.close()
        self._pp.close()
        if self in _GROUPS:
            _GROUPS.remove(self)


__all__ = ["BACKEND", "ENV", "HocclProcessGroup", "destroy_process_group", "init_process_group",
           "register", "selected_backend", "BF16", "FP32", "INT32", "UINT8"]
