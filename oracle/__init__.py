"""CPU oracle for the HOCCL collectives -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never loads it and
shares no code with it.

The arithmetic lives in ``hoccl_oracle.c`` (plain single-threaded C; see its
header for the definition of every collective and the reading of the paper it
follows).  This module only marshals numpy arrays into that library and holds
the build command for it.

Parity status: every function here is pinned by ``tests/test_oracle_pins.py``
(closed forms, invariants, exhaustive conversion check, brute force, the
Higham error bound and hand-derived ring-order fixtures under
``tests/golden/``; the bf16-partials fold by the pure-Python ring that
rounds every hop, a hand-worked example, special cases and its own error
bound).
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hoccl_oracle.c")
_LIB = os.path.join(_HERE, "libhoccl_oracle.so")

INT32, FP32, BF16, UINT8 = 0, 1, 2, 3
_NP = {INT32: np.int32, FP32: np.float32, BF16: np.uint16, UINT8: np.uint8}

_lib = None


def build():
    """Compile the oracle with plain gcc (no fast-math, no FMA contraction)."""
    cmd = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC",
           "-shared", "-std=c11", "-Wall", "-Wextra", "-o", _LIB, _SRC]
    subprocess.run(cmd, check=True)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        vpp = ctypes.POINTER(ctypes.c_void_p)
        sz = ctypes.c_size_t
        for name, args in {
            "oracle_allreduce": [vpp, vpp, sz, ctypes.c_int, ctypes.c_int],
            "oracle_reduce_scatter": [vpp, vpp, sz, ctypes.c_int, ctypes.c_int],
            "oracle_allgather": [vpp, vpp, sz, ctypes.c_int, ctypes.c_int],
            "oracle_sendrecv": [vpp, vpp, ctypes.POINTER(ctypes.c_int), sz,
                                ctypes.c_int, ctypes.c_int],
            "oracle_alltoall": [vpp, vpp, sz, ctypes.c_int, ctypes.c_int],
            "oracle_alltoallv": [vpp, ctypes.POINTER(sz), ctypes.POINTER(sz), vpp,
                                 ctypes.POINTER(sz), ctypes.c_int, ctypes.c_int],
            "oracle_allreduce_bf16_hops": [vpp, vpp, sz, ctypes.c_int],
            "oracle_reduce_scatter_bf16_hops": [vpp, vpp, sz, ctypes.c_int],
        }.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = ctypes.c_int
        L.oracle_f32_to_bf16_array.argtypes = [ctypes.c_void_p, ctypes.c_void_p, sz]
        L.oracle_f32_to_bf16_array.restype = None
        _lib = L
    return _lib


def _ptrs(arrays):
    for a in arrays:
        assert a.flags["C_CONTIGUOUS"]
    return (ctypes.c_void_p * len(arrays))(*[a.ctypes.data for a in arrays])


def _check(rc, name):
    if rc != 0:
        raise ValueError(f"{name}: oracle rejected the arguments (code {rc})")


def dtype_code(np_dtype):
    """int32 -> INT32, float32 -> FP32, uint16 (bf16 bit patterns) -> BF16,
    uint8 -> UINT8 (copies only)."""
    np_dtype = np.dtype(np_dtype)
    for k, v in _NP.items():
        if np.dtype(v) == np_dtype:
            return k
    raise TypeError(f"unsupported dtype {np_dtype}")


def allreduce(send, recv, count, dtype):
    _check(lib().oracle_allreduce(_ptrs(send), _ptrs(recv), count, dtype, len(send)),
           "allreduce")


def reduce_scatter(send, recv, recvcount, dtype):
    _check(lib().oracle_reduce_scatter(_ptrs(send), _ptrs(recv), recvcount, dtype,
                                       len(send)), "reduce_scatter")


def allgather(send, recv, sendcount, dtype):
    _check(lib().oracle_allgather(_ptrs(send), _ptrs(recv), sendcount, dtype,
                                  len(send)), "allgather")


def sendrecv(send, recv, peers, count, dtype):
    p = (ctypes.c_int * len(peers))(*peers)
    _check(lib().oracle_sendrecv(_ptrs(send), _ptrs(recv), p, count, dtype,
                                 len(send)), "sendrecv")


def alltoall(send, recv, count, dtype):
    _check(lib().oracle_alltoall(_ptrs(send), _ptrs(recv), count, dtype, len(send)),
           "alltoall")


def alltoallv(send, sendcounts, sdispls, recv, rdispls, dtype):
    R = len(send)
    S = ctypes.c_size_t * (R * R)
    _check(lib().oracle_alltoallv(_ptrs(send), S(*sendcounts), S(*sdispls),
                                  _ptrs(recv), S(*rdispls), dtype, R), "alltoallv")


def f32_to_bf16(x):
    """Round-to-nearest-even fp32 -> bf16 bit patterns (uint16 array)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    lib().oracle_f32_to_bf16_array(x.ctypes.data, out.ctypes.data, x.size)
    return out


# ---- whole-array conveniences: allocate outputs, return them ----------------

def allreduce_bf16_hops(send, recv, count):
    """bf16 all-reduce with bf16 partials rounded at every hop."""
    _check(lib().oracle_allreduce_bf16_hops(_ptrs(send), _ptrs(recv), count, len(send)),
           "allreduce_bf16_hops")


def reduce_scatter_bf16_hops(send, recv, recvcount):
    """bf16 reduce-scatter with bf16 partials rounded at every hop."""
    _check(lib().oracle_reduce_scatter_bf16_hops(_ptrs(send), _ptrs(recv), recvcount, len(send)),
           "reduce_scatter_bf16_hops")


def allreduce_new(send, dtype):
    count = send[0].size
    recv = [np.zeros_like(s) for s in send]
    allreduce(send, recv, count, dtype)
    return recv


def reduce_scatter_new(send, dtype):
    R = len(send)
    n = send[0].size // R
    recv = [np.zeros(n, dtype=send[0].dtype) for _ in send]
    reduce_scatter(send, recv, n, dtype)
    return recv


def allgather_new(send, dtype):
    R = len(send)
    n = send[0].size
    recv = [np.zeros(R * n, dtype=send[0].dtype) for _ in send]
    allgather(send, recv, n, dtype)
    return recv


def allreduce_bf16_hops_new(send):
    recv = [np.zeros_like(s) for s in send]
    allreduce_bf16_hops(send, recv, send[0].size)
    return recv


def reduce_scatter_bf16_hops_new(send):
    R = len(send)
    n = send[0].size // R
    recv = [np.zeros(n, dtype=np.uint16) for _ in send]
    reduce_scatter_bf16_hops(send, recv, n)
    return recv
