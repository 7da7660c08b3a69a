"""Python binding of libhoccl (ctypes).

Argument marshalling only: every step of a collective runs in the HIP
library (``libhoccl.so``, built from ``csrc/`` by ``build.py``).  PyTorch is
used for device memory and streams; each call passes raw device pointers and
``torch.cuda.current_stream().cuda_stream`` (or the stream given) to the
C ABI declared in ``include/hoccl.h``.

Importing fails loudly when the library has not been built: there is no
fallback implementation.
"""
import ctypes
import os
import threading

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhoccl.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is not built; run `python -m paper_2609_34334_amd.build` "
        "(or __graft_entry__.build()) first")

_lib = ctypes.CDLL(LIB_PATH)

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_HIP, ERR_NO_MEMORY, ERR_TIMEOUT, ERR_INTERNAL = range(7)
INT32, FP32, BF16, UINT8 = 0, 1, 2, 3
COPY_AUTO, COPY_SDMA, COPY_KERNEL, COPY_HIP = range(4)
REDUCE_RING, REDUCE_DIRECT, REDUCE_AUTO = range(3)
OP_ALLREDUCE, OP_REDUCE_SCATTER, OP_ALLGATHER, OP_SENDRECV, OP_ALLTOALL = range(5)

_DTYPES = {torch.int32: INT32, torch.float32: FP32, torch.bfloat16: BF16}
_COPY_DTYPES = {**_DTYPES, torch.uint8: UINT8}     # the copy-only collectives also move bytes
HOP_FIRST, HOP_MIDDLE, HOP_LAST, HOP_ONLY = range(4)
HOPS = {"first": HOP_FIRST, "middle": HOP_MIDDLE, "last": HOP_LAST, "only": HOP_ONLY}
COPY_PATHS = {"auto": COPY_AUTO, "sdma": COPY_SDMA, "engines": COPY_SDMA,
              "kernel": COPY_KERNEL, "hip": COPY_HIP}
COPY_PATH_NAMES = {COPY_AUTO: "auto", COPY_SDMA: "engines", COPY_KERNEL: "kernel", COPY_HIP: "hip"}
REDUCE_ALGOS = {"ring": REDUCE_RING, "direct": REDUCE_DIRECT, "auto": REDUCE_AUTO}


class Config(ctypes.Structure):
    _fields_ = [("workgroups_per_step", ctypes.c_int),
                ("threads_per_workgroup", ctypes.c_int),
                ("chunk_bytes", ctypes.c_size_t),
                ("copy_streams", ctypes.c_int),
                ("copy_path", ctypes.c_int),
                ("allgather_direct", ctypes.c_int),
                ("allreduce_chunk_groups", ctypes.c_int),
                ("sdma_engines", ctypes.c_int),
                ("reduce_algo", ctypes.c_int),
                ("kernel_timing", ctypes.c_int),
                ("proxy_timeout_ms", ctypes.c_uint),
                ("proxy_handshake", ctypes.c_int),
                ("ring_group_bytes", ctypes.c_size_t),
                ("proxy_wait_limit_us", ctypes.c_uint),
                ("fused_hops", ctypes.c_int),
                ("a2a_schedule", ctypes.c_int),
                ("proxy_slice_bytes", ctypes.c_size_t),
                ("bf16_partials", ctypes.c_int)]


class Stats(ctypes.Structure):
    _fields_ = [("reduce_launches", ctypes.c_int),
                ("copy_ops", ctypes.c_int),
                ("workgroups_per_step", ctypes.c_int),
                ("cus_available", ctypes.c_int),
                ("cus_used_max", ctypes.c_int),
                ("copy_path_used", ctypes.c_int),
                ("hbm_bytes_algorithmic", ctypes.c_ulonglong),
                ("host_enqueue_us", ctypes.c_double),
                ("copy_kernel_launches", ctypes.c_int),
                ("reduce_algo_used", ctypes.c_int),
                ("copy_bytes", ctypes.c_ulonglong)]


_vpp = ctypes.POINTER(ctypes.c_void_p)
_sz = ctypes.c_size_t
_szp = ctypes.POINTER(ctypes.c_size_t)
_i = ctypes.c_int
_SIGS = {
    "hoccl_init": [_i],
    "hoccl_finalize": [],
    "hoccl_set_config": [ctypes.POINTER(Config)],
    "hoccl_get_config": [ctypes.POINTER(Config)],
    "hoccl_get_last_stats": [ctypes.POINTER(Stats)],
    "hoccl_get_kernel_times": [ctypes.POINTER(ctypes.c_float), _i, ctypes.POINTER(_i)],
    "hoccl_allreduce": [_vpp, _vpp, _sz, _i, _i, ctypes.c_void_p],
    "hoccl_reduce_scatter": [_vpp, _vpp, _sz, _i, _i, ctypes.c_void_p],
    "hoccl_reduce_scatter_noalloc": [_vpp, _vpp, _sz, _i, _i, ctypes.c_void_p],
    "hoccl_allgather": [_vpp, _vpp, _sz, _i, _i, ctypes.c_void_p],
    "hoccl_sendrecv": [_vpp, _vpp, ctypes.POINTER(_i), _sz, _i, _i, ctypes.c_void_p],
    "hoccl_alltoall": [_vpp, _vpp, _sz, _i, _i, ctypes.c_void_p],
    "hoccl_alltoallv": [_vpp, _szp, _szp, _vpp, _szp, _i, _i, ctypes.c_void_p],
    "hoccl_ring_hop": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, _sz, _i, _i, ctypes.c_void_p],
    "hoccl_debug_plan_json": [_i, _sz, _i, _i, ctypes.c_char_p, _sz, _szp],
    "hoccl_debug_schedule_json": [_i, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_i),
                                  ctypes.POINTER(_i), ctypes.c_double, ctypes.c_double,
                                  ctypes.c_char_p, _sz, _szp],
    "hoccl_debug_interleave": [_i, ctypes.POINTER(ctypes.c_double), ctypes.c_double,
                               ctypes.POINTER(_i), _sz, _szp],
    "hoccl_debug_stream_ceiling": [_i, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, _sz,
                                   ctypes.c_void_p],
    "hoccl_ipc_export": [ctypes.c_void_p, ctypes.c_void_p, _szp, _szp],
    "hoccl_ipc_open": [ctypes.c_void_p, _sz, _sz, ctypes.POINTER(ctypes.c_void_p)],
    "hoccl_ipc_close_all": [],
    "hoccl_mailbox_create": [ctypes.c_char_p, ctypes.c_uint, _sz, _vpp],
    "hoccl_mailbox_open": [ctypes.c_char_p, _vpp],
    "hoccl_mailbox_unlink": [ctypes.c_char_p],
    "hoccl_mailbox_close": [ctypes.c_void_p],
    "hoccl_mailbox_post": [ctypes.c_void_p, ctypes.c_uint, ctypes.c_uint, ctypes.c_char_p, _sz],
    "hoccl_mailbox_wait": [ctypes.c_void_p, ctypes.c_uint, ctypes.c_uint, ctypes.c_uint],
    "hoccl_mailbox_read": [ctypes.c_void_p, ctypes.c_uint, ctypes.c_char_p, _sz, _szp],
}
for _name, _args in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = ctypes.c_int
_lib.hoccl_status_string.argtypes = [ctypes.c_int]
_lib.hoccl_status_string.restype = ctypes.c_char_p
_lib.hoccl_last_error_string.argtypes = []
_lib.hoccl_last_error_string.restype = ctypes.c_char_p
_lib.hoccl_sdma_engine_count.argtypes = []
_lib.hoccl_sdma_engine_count.restype = ctypes.c_int


class HocclError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        msg = _lib.hoccl_status_string(status).decode()
        detail = _lib.hoccl_last_error_string().decode()
        super().__init__(f"{where}: {msg}" + (f" ({detail})" if detail else ""))


def _check(status, where):
    if status != OK:
        raise HocclError(status, where)


def lib():
    """The loaded ctypes library (for tests that call the C ABI directly)."""
    return _lib


# ---- configuration -------------------------------------------------------------

def get_config():
    c = Config()
    _check(_lib.hoccl_get_config(ctypes.byref(c)), "hoccl_get_config")
    return {k: getattr(c, k) for k, _ in Config._fields_}


def set_config(**kw):
    """Update configuration fields; copy_path also accepts a name
    ('auto', 'sdma' or 'engines', 'kernel', 'hip') and reduce_algo
    'ring', 'direct' or 'auto'."""
    c = Config()
    _check(_lib.hoccl_get_config(ctypes.byref(c)), "hoccl_get_config")
    for k, v in kw.items():
        if k == "copy_path" and isinstance(v, str):
            v = COPY_PATHS[v]
        if k == "reduce_algo" and isinstance(v, str):
            v = REDUCE_ALGOS[v]
        if not hasattr(c, k):
            raise KeyError(k)
        setattr(c, k, v)
    _check(_lib.hoccl_set_config(ctypes.byref(c)), "hoccl_set_config")


class config:
    """Context manager: temporarily change configuration fields."""

    def __init__(self, **kw):
        self.kw = kw

    def __enter__(self):
        self.saved = get_config()
        set_config(**self.kw)
        return self

    def __exit__(self, *exc):
        set_config(**self.saved)


def last_stats():
    s = Stats()
    _check(_lib.hoccl_get_last_stats(ctypes.byref(s)), "hoccl_get_last_stats")
    return {k: getattr(s, k) for k, _ in Stats._fields_}


def kernel_times():
    """Durations (ms) of the kernel launches of the last call (needs
    kernel_timing=1); waits for them."""
    n = ctypes.c_int(0)
    _check(_lib.hoccl_get_kernel_times(None, 0, ctypes.byref(n)), "hoccl_get_kernel_times")
    buf = (ctypes.c_float * max(1, n.value))()
    _check(_lib.hoccl_get_kernel_times(buf, n.value, ctypes.byref(n)), "hoccl_get_kernel_times")
    return list(buf[:n.value])


def sdma_engine_count():
    return _lib.hoccl_sdma_engine_count()


def init(device=-1):
    _check(_lib.hoccl_init(device), "hoccl_init")


def finalize():
    _check(_lib.hoccl_finalize(), "hoccl_finalize")


def plan_json(op, count, dtype, R):
    import json
    need = ctypes.c_size_t(0)
    _check(_lib.hoccl_debug_plan_json(op, count, dtype, R, None, 0, ctypes.byref(need)),
           "hoccl_debug_plan_json")
    buf = ctypes.create_string_buffer(need.value)
    _check(_lib.hoccl_debug_plan_json(op, count, dtype, R, buf, need.value, ctypes.byref(need)),
           "hoccl_debug_plan_json")
    return json.loads(buf.value.decode())


def schedule(C, node, peer, bw_intra, bw_inter):
    """The paper's collective scheduler on a described topology: returns
    {'T', 'stages', 'tau', 'total'} (see hoccl_debug_schedule_json)."""
    import json
    G = len(node)
    flat = [float(C[u][v]) for u in range(G) for v in range(G)]
    Cm = (ctypes.c_double * (G * G))(*flat)
    nd = (ctypes.c_int * G)(*node)
    pr = (ctypes.c_int * G)(*peer)
    need = ctypes.c_size_t(0)
    _check(_lib.hoccl_debug_schedule_json(G, Cm, nd, pr, bw_intra, bw_inter, None, 0,
                                          ctypes.byref(need)), "hoccl_debug_schedule_json")
    buf = ctypes.create_string_buffer(need.value)
    _check(_lib.hoccl_debug_schedule_json(G, Cm, nd, pr, bw_intra, bw_inter, buf, need.value,
                                          ctypes.byref(need)), "hoccl_debug_schedule_json")
    return json.loads(buf.value.decode())


def interleave(bytes_per_flow, chunk_bytes):
    """Flow-size-aware chunk order on one engine: list of flow indices."""
    F = len(bytes_per_flow)
    b = (ctypes.c_double * max(1, F))(*bytes_per_flow)
    n = ctypes.c_size_t(0)
    _check(_lib.hoccl_debug_interleave(F, b, chunk_bytes, None, 0, ctypes.byref(n)),
           "hoccl_debug_interleave")
    out = (ctypes.c_int * max(1, n.value))()
    _check(_lib.hoccl_debug_interleave(F, b, chunk_bytes, out, n.value, ctypes.byref(n)),
           "hoccl_debug_interleave")
    return list(out[:n.value])


# ---- collectives ---------------------------------------------------------------

def _dtype_of(tensors, copy=False):
    dt = tensors[0].dtype
    table = _COPY_DTYPES if copy else _DTYPES
    if dt not in table:
        raise TypeError(f"unsupported dtype {dt}")
    dev = tensors[0].device
    for t in tensors:
        if t.dtype != dt:
            raise TypeError("all buffers must share one dtype")
        if t.device != dev or t.device.type != "cuda":
            raise ValueError("all buffers must live on the same GPU")
        if not t.is_contiguous():
            raise ValueError("buffers must be contiguous")
    return table[dt]


def _ptrs(tensors):
    return (ctypes.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _on_send_device(fn):
    """Runs a collective with its buffers' GPU current (and that GPU's
    current stream as the default): the library keeps its streams and
    workspace per device and acts on the current one."""
    import functools

    @functools.wraps(fn)
    def wrapper(send, *args, **kwargs):
        with torch.cuda.device(send[0].device):
            return fn(send, *args, **kwargs)
    return wrapper


@_on_send_device
def allreduce(send, recv=None, stream=None):
    """Sum of the R tensors `send`, written to every tensor of `recv`
    (defaults to in place)."""
    recv = send if recv is None else recv
    dt = _dtype_of(list(send) + list(recv))
    n = send[0].numel()
    if any(t.numel() != n for t in list(send) + list(recv)):
        raise ValueError("all buffers must have the same number of elements")
    _check(_lib.hoccl_allreduce(_ptrs(send), _ptrs(recv), n, dt, len(send), _stream(stream)),
           "hoccl_allreduce")
    return recv


@_on_send_device
def reduce_scatter(send, recv=None, stream=None):
    """send: R tensors of R*n elements; recv[r] receives block r of the sum."""
    R = len(send)
    if send[0].numel() % R:
        raise ValueError("send buffers must hold R * recvcount elements")
    n = send[0].numel() // R
    if recv is None:
        recv = [torch.empty(n, dtype=send[0].dtype, device=send[0].device) for _ in range(R)]
    dt = _dtype_of(list(send) + list(recv))
    if any(t.numel() != R * n for t in send) or any(t.numel() != n for t in recv):
        raise ValueError("buffer sizes do not match")
    _check(_lib.hoccl_reduce_scatter(_ptrs(send), _ptrs(recv), n, dt, R, _stream(stream)),
           "hoccl_reduce_scatter")
    return recv


@_on_send_device
def reduce_scatter_noalloc(send, recv, stream=None):
    """reduce_scatter through the entry point that allocates nothing: the
    ring's partials live in the library's static device scratch.  `recv`
    must be given; the library must be initialised on the device."""
    R = len(send)
    if send[0].numel() % R:
        raise ValueError("send buffers must hold R * recvcount elements")
    n = send[0].numel() // R
    dt = _dtype_of(list(send) + list(recv))
    if any(t.numel() != R * n for t in send) or any(t.numel() != n for t in recv):
        raise ValueError("buffer sizes do not match")
    _check(_lib.hoccl_reduce_scatter_noalloc(_ptrs(send), _ptrs(recv), n, dt, R, _stream(stream)),
           "hoccl_reduce_scatter_noalloc")
    return recv


@_on_send_device
def allgather(send, recv=None, stream=None):
    """send: R tensors of n elements; every recv[r] gets their concatenation."""
    R = len(send)
    n = send[0].numel()
    if recv is None:
        recv = [torch.empty(R * n, dtype=send[0].dtype, device=send[0].device) for _ in range(R)]
    dt = _dtype_of(list(send) + list(recv), copy=True)
    if any(t.numel() != n for t in send) or any(t.numel() != R * n for t in recv):
        raise ValueError("buffer sizes do not match")
    _check(_lib.hoccl_allgather(_ptrs(send), _ptrs(recv), n, dt, R, _stream(stream)),
           "hoccl_allgather")
    return recv


@_on_send_device
def sendrecv(send, recv, peers, stream=None):
    """Rank r sends send[r] to rank peers[r] (-1: nothing).  recv[d] may be
    None for ranks that receive nothing."""
    R = len(send)
    n = send[0].numel()
    live = [t for t in list(send) + list(recv) if t is not None]
    dt = _dtype_of(live, copy=True)
    rp = (ctypes.c_void_p * R)(*[0 if t is None else t.data_ptr() for t in recv])
    pp = (ctypes.c_int * R)(*peers)
    _check(_lib.hoccl_sendrecv(_ptrs(send), rp, pp, n, dt, R, _stream(stream)), "hoccl_sendrecv")
    return recv


@_on_send_device
def alltoall(send, recv=None, stream=None):
    R = len(send)
    if send[0].numel() % R:
        raise ValueError("send buffers must hold R blocks")
    n = send[0].numel() // R
    if recv is None:
        recv = [torch.empty_like(t) for t in send]
    dt = _dtype_of(list(send) + list(recv), copy=True)
    _check(_lib.hoccl_alltoall(_ptrs(send), _ptrs(recv), n, dt, R, _stream(stream)),
           "hoccl_alltoall")
    return recv


@_on_send_device
def alltoallv(send, counts, sdispls, recv, rdispls, stream=None):
    """counts/sdispls/rdispls: R*R element counts and offsets, [s*R + d]."""
    R = len(send)
    dt = _dtype_of(list(send) + list(recv), copy=True)
    S = ctypes.c_size_t * (R * R)
    _check(_lib.hoccl_alltoallv(_ptrs(send), S(*counts), S(*sdispls), _ptrs(recv), S(*rdispls),
                                dt, R, _stream(stream)), "hoccl_alltoallv")
    return recv


IPC_HANDLE_BYTES = 64


def ipc_export(t):
    """(handle bytes, byte offset, allocation bytes) of the allocation that
    holds tensor `t`'s data (hoccl_ipc_export)."""
    h = ctypes.create_string_buffer(IPC_HANDLE_BYTES)
    off, size = ctypes.c_size_t(0), ctypes.c_size_t(0)
    with torch.cuda.device(t.device):
        _check(_lib.hoccl_ipc_export(t.data_ptr(), h, ctypes.byref(off), ctypes.byref(size)),
               "hoccl_ipc_export")
    return h.raw, off.value, size.value


def ipc_open(handle, offset, alloc_bytes):
    """Device address, in this process, of byte `offset` of an allocation
    another process exported (hoccl_ipc_open; cached per handle)."""
    p = ctypes.c_void_p()
    _check(_lib.hoccl_ipc_open(handle, offset, alloc_bytes, ctypes.byref(p)), "hoccl_ipc_open")
    return p.value


def ipc_close_all():
    _check(_lib.hoccl_ipc_close_all(), "hoccl_ipc_close_all")


class Mailbox:
    """A cross-process mailbox (hoccl_mailbox_*): numbered slots of a
    sequence number and a payload in POSIX shared memory.  Given `slots`, it
    creates the object `name`; otherwise it opens an existing one."""

    def __init__(self, name, slots=None, slot_bytes=None):
        self._h = ctypes.c_void_p()
        self.name = name
        if slots is None:
            _check(_lib.hoccl_mailbox_open(name.encode(), ctypes.byref(self._h)), "hoccl_mailbox_open")
        else:
            _check(_lib.hoccl_mailbox_create(name.encode(), slots, slot_bytes, ctypes.byref(self._h)),
                   "hoccl_mailbox_create")
        self._cap = slot_bytes or (1 << 20)
        self._local = threading.local()     # a read buffer per thread

    @staticmethod
    def unlink(name):
        _check(_lib.hoccl_mailbox_unlink(name.encode()), "hoccl_mailbox_unlink")

    def post(self, slot, seq, data=b""):
        _check(_lib.hoccl_mailbox_post(self._h, slot, seq & 0xFFFFFFFF, data, len(data)),
               "hoccl_mailbox_post")

    def wait(self, slot, seq, timeout_ms):
        _check(_lib.hoccl_mailbox_wait(self._h, slot, seq & 0xFFFFFFFF, int(timeout_ms)),
               "hoccl_mailbox_wait")

    def ready(self, slot, seq):
        """Whether the slot has reached `seq` (one look, no waiting)."""
        return _lib.hoccl_mailbox_wait(self._h, slot, seq & 0xFFFFFFFF, 0) == OK

    def read(self, slot):
        loc = self._local
        if not hasattr(loc, "buf"):
            loc.buf, loc.len = ctypes.create_string_buffer(self._cap), ctypes.c_size_t(0)
        _check(_lib.hoccl_mailbox_read(self._h, slot, loc.buf, self._cap, ctypes.byref(loc.len)),
               "hoccl_mailbox_read")
        return loc.buf.raw[:loc.len.value]

    def close(self):
        if self._h:
            _lib.hoccl_mailbox_close(self._h)
            self._h = ctypes.c_void_p()


CEILING_MODES = {"read": 0, "write": 1, "copy": 2, "add": 3, "rmw": 4, "copy_nt": 5, "add_nt": 6}


def stream_ceiling(mode, a=None, b=None, c=None, nbytes=None, stream=None):
    """One launch of a streaming-ceiling kernel (hoccl_debug_stream_ceiling):
    'read' a, 'write' c, 'copy' a -> c, 'add' c = a + b (fp32), 'rmw' c += 1
    (fp32), 'copy_nt' and 'add_nt' with non-temporal stores.  nbytes
    defaults to the size of the first tensor given."""
    m = CEILING_MODES[mode] if isinstance(mode, str) else int(mode)
    ts = [t for t in (a, b, c) if t is not None]
    if nbytes is None:
        nbytes = ts[0].numel() * ts[0].element_size()
    ptr = lambda t: None if t is None else t.data_ptr()
    with torch.cuda.device(ts[0].device):
        _check(_lib.hoccl_debug_stream_ceiling(m, ptr(a), ptr(b), ptr(c), nbytes, _stream(stream)),
               "hoccl_debug_stream_ceiling")


def ring_hop(partial, local, out=None, hop="middle", stream=None):
    """One ring hop of one rank: out = partial + local in the ring fold's
    arithmetic (hoccl_ring_hop).  With bf16 `local`, `partial` and `out`
    are fp32 or bf16 by hop: "first" bf16 -> fp32, "middle" fp32 -> fp32,
    "last" fp32 -> bf16, "only" bf16 -> bf16; int32 and fp32 use their own
    dtype throughout.  `out` defaults to a new tensor and may be `partial`
    (same dtype) for an in-place update."""
    h = HOPS[hop] if isinstance(hop, str) else int(hop)
    dt = _dtype_of([local])
    bf = local.dtype == torch.bfloat16
    want_in = torch.float32 if bf and h in (HOP_MIDDLE, HOP_LAST) else local.dtype
    want_out = torch.float32 if bf and h in (HOP_FIRST, HOP_MIDDLE) else local.dtype
    if out is None:
        out = torch.empty(local.numel(), dtype=want_out, device=local.device)
    for t, want, name in ((partial, want_in, "partial"), (out, want_out, "out")):
        if t.dtype != want:
            raise TypeError(f"{name} must be {want} for this hop, not {t.dtype}")
        if t.device != local.device:
            raise ValueError("all buffers must live on the same GPU")
        if not t.is_contiguous():
            raise ValueError("buffers must be contiguous")
        if t.numel() != local.numel():
            raise ValueError("partial, local and out must have the same number of elements")
    with torch.cuda.device(local.device):
        _check(_lib.hoccl_ring_hop(partial.data_ptr(), local.data_ptr(), out.data_ptr(), local.numel(),
                                   dt, h, _stream(stream)), "hoccl_ring_hop")
    return out
