"""The C-ABI library loads on a machine without a GPU, exports every entry
point include/hoccl.h declares, and rejects bad arguments before touching the
device."""
import ctypes
import os
import re

import pytest

import paper_2609_34334_amd as hc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hoccl.h")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hoccl_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_collectives():
    syms = declared_symbols()
    for s in ["hoccl_allreduce", "hoccl_reduce_scatter", "hoccl_allgather", "hoccl_sendrecv",
              "hoccl_alltoall", "hoccl_alltoallv", "hoccl_init", "hoccl_finalize"]:
        assert s in syms


@pytest.mark.parametrize("sym", declared_symbols())
def test_library_exports_symbol(sym):
    assert hasattr(hc.lib(), sym), sym


L = hc.lib()
VP = ctypes.c_void_p


def ptrs(*vals):
    return (VP * len(vals))(*vals)


def test_bad_rank_count_and_dtype():
    p = ptrs(0x1000)
    assert L.hoccl_allreduce(p, p, 4, hc.FP32, 0, None) == hc.ERR_INVALID_ARG
    big = (VP * 65)(*([0x1000] * 65))
    assert L.hoccl_allreduce(big, big, 4, hc.FP32, 65, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_allreduce(p, p, 4, 9, 1, None) == hc.ERR_INVALID_ARG
    # bytes are for the copies: every reduction refuses them before looking further
    assert L.hoccl_allreduce(p, p, 4, hc.UINT8, 1, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_reduce_scatter(p, p, 4, hc.UINT8, 1, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_reduce_scatter_noalloc(p, p, 4, hc.UINT8, 1, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_ring_hop(VP(0x1000), VP(0x2000), VP(0x3000), 4, hc.UINT8, hc.HOP_MIDDLE,
                            None) == hc.ERR_INVALID_ARG
    assert L.hoccl_allgather(p, p, 4, 4, 1, None) == hc.ERR_INVALID_ARG          # no dtype 4
    assert L.hoccl_allreduce(None, p, 4, hc.FP32, 1, None) == hc.ERR_INVALID_ARG


def test_null_buffer_with_count():
    s = ptrs(0x1000, 0)
    r = ptrs(0x10000, 0x20000)
    assert L.hoccl_allgather(s, r, 4, hc.FP32, 2, None) == hc.ERR_INVALID_ARG


def test_zero_count_is_noop_ok():
    s = ptrs(0, 0)
    assert L.hoccl_allreduce(s, s, 0, hc.FP32, 2, None) == hc.OK
    assert L.hoccl_reduce_scatter(s, s, 0, hc.BF16, 2, None) == hc.OK


def test_sendrecv_duplicate_receiver_and_bad_peer():
    s = ptrs(0x1000, 0x2000, 0x3000)
    r = ptrs(0x10000, 0x20000, 0x30000)
    dup = (ctypes.c_int * 3)(1, 1, -1)
    assert L.hoccl_sendrecv(s, r, dup, 4, hc.FP32, 3, None) == hc.ERR_INVALID_ARG
    bad = (ctypes.c_int * 3)(3, -1, -1)
    assert L.hoccl_sendrecv(s, r, bad, 4, hc.FP32, 3, None) == hc.ERR_INVALID_ARG
    neg = (ctypes.c_int * 3)(-2, -1, -1)
    assert L.hoccl_sendrecv(s, r, neg, 4, hc.FP32, 3, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_sendrecv(s, r, None, 4, hc.FP32, 3, None) == hc.ERR_INVALID_ARG


def test_overlapping_outputs_rejected():
    s = ptrs(0x100000, 0x200000)
    r = ptrs(0x300000, 0x300008)                 # 16-byte outputs 8 bytes apart
    assert L.hoccl_allreduce(s, r, 4, hc.FP32, 2, None) == hc.ERR_INVALID_ARG


def test_input_output_overlap_outside_in_place_form():
    # all-reduce: recv[0] overlaps send[1]
    s = ptrs(0x100000, 0x200000)
    r = ptrs(0x200000, 0x300000)
    assert L.hoccl_allreduce(s, r, 4, hc.FP32, 2, None) == hc.ERR_INVALID_ARG
    # all-gather: send[1] must sit at recv[1] + 1*n, not at recv[1]
    s = ptrs(0x100000, 0x300000)
    r = ptrs(0x200000, 0x300000)
    assert L.hoccl_allgather(s, r, 4, hc.FP32, 2, None) == hc.ERR_INVALID_ARG
    # reduce-scatter: recv[1] must be send[1] + 1*n, not send[1] + 0
    s = ptrs(0x100000, 0x200000)
    r = ptrs(0x300000, 0x200000)
    assert L.hoccl_reduce_scatter(s, r, 4, hc.FP32, 2, None) == hc.ERR_INVALID_ARG
    # all-to-all is out-of-place only
    s = ptrs(0x100000, 0x200000)
    assert L.hoccl_alltoall(s, s, 4, hc.FP32, 2, None) == hc.ERR_INVALID_ARG


def test_alltoallv_overlapping_destinations_rejected():
    R = 2
    s = ptrs(0x100000, 0x200000)
    r = ptrs(0x300000, 0x400000)
    S = ctypes.c_size_t * 4
    counts = S(4, 4, 4, 4)
    sd = S(0, 4, 0, 4)
    rd = S(0, 0, 2, 4)       # (0->0) at 0..4 and (1->0) at 2..6 overlap
    assert L.hoccl_alltoallv(s, counts, sd, r, rd, hc.FP32, R, None) == hc.ERR_INVALID_ARG


def test_config_roundtrip_and_validation():
    saved = hc.get_config()
    try:
        hc.set_config(workgroups_per_step=64, copy_path="kernel", allreduce_chunk_groups=4)
        c = hc.get_config()
        assert c["workgroups_per_step"] == 64 and c["copy_path"] == hc.COPY_KERNEL
        with pytest.raises(hc.HocclError):
            hc.set_config(threads_per_workgroup=100)
        with pytest.raises(hc.HocclError):
            hc.set_config(chunk_bytes=100)
        for bad in (-1, 2):
            with pytest.raises(hc.HocclError):
                hc.set_config(bf16_partials=bad)
        assert hc.get_config()["bf16_partials"] == 0
        hc.set_config(bf16_partials=1)
        assert hc.get_config()["bf16_partials"] == 1
        assert hc.get_config()["workgroups_per_step"] == 64
    finally:
        hc.set_config(**saved)


def test_status_strings():
    for st in range(7):
        assert L.hoccl_status_string(st)


def test_debug_env_logs_plans_without_a_gpu_call():
    """HOCCL_DEBUG is read with the rest of the environment; with no GPU the
    library still loads and reports its configuration."""
    import subprocess
    import sys
    code = ("import paper_2609_34334_amd as hc; c = hc.get_config(); "
            "print(c['copy_path'], c['reduce_algo'], c['proxy_wait_limit_us'])")
    env = dict(os.environ, HOCCL_DEBUG="1", HOCCL_COPY_PATH="kernel", HOCCL_REDUCE_ALGO="direct",
               HOCCL_PROXY_WAIT_LIMIT_US="250")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env,
                       cwd=ROOT)
    assert r.returncode == 0, r.stderr
    assert r.stdout.split() == [str(hc.COPY_KERNEL), str(hc.REDUCE_DIRECT), "250"], r.stdout
    env.update(HOCCL_COPY_PATH="sdma", HOCCL_REDUCE_ALGO="auto")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env,
                       cwd=ROOT)
    assert r.returncode == 0, r.stderr
    assert r.stdout.split() == [str(hc.COPY_SDMA), str(hc.REDUCE_AUTO), "250"], r.stdout



def test_size_overflow_rejected_with_a_reason():
    """Counts whose byte size does not fit in size_t are argument errors,
    reported before anything touches a device, with their own message."""
    L = hc.lib()
    send = (ctypes.c_void_p * 2)(1 << 40, 2 << 40)
    recv = (ctypes.c_void_p * 2)(3 << 40, 4 << 40)
    huge = ctypes.c_size_t((1 << 64) - 1)
    for fn in (L.hoccl_allreduce, L.hoccl_reduce_scatter, L.hoccl_allgather, L.hoccl_alltoall):
        assert fn(send, recv, huge, hc.FP32, 2, None) == hc.ERR_INVALID_ARG
        assert b"does not fit" in L.hoccl_last_error_string()


def test_ring_hop_rejects_bad_arguments_before_the_device():
    a, b, o = 0x100000, 0x200000, 0x300000
    assert L.hoccl_ring_hop(a, b, o, 4, 9, hc.HOP_MIDDLE, None) == hc.ERR_INVALID_ARG      # dtype
    assert L.hoccl_ring_hop(a, b, o, 4, hc.BF16, 4, None) == hc.ERR_INVALID_ARG            # hop
    assert L.hoccl_ring_hop(a, b, o, 4, hc.BF16, -1, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_ring_hop(None, b, o, 4, hc.FP32, hc.HOP_MIDDLE, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_ring_hop(a, b, None, 4, hc.FP32, hc.HOP_MIDDLE, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_ring_hop(0, 0, 0, 0, hc.FP32, hc.HOP_MIDDLE, None) == hc.OK             # no work
    # bf16 middle hop: out (fp32, 16 bytes) may be the partial itself, but not
    # the bf16 local (other element size) nor half-overlap the partial.
    assert L.hoccl_ring_hop(a, b, b, 4, hc.BF16, hc.HOP_MIDDLE, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_ring_hop(a, b, a + 8, 4, hc.BF16, hc.HOP_MIDDLE, None) == hc.ERR_INVALID_ARG
    # last hop: bf16 out aliasing the fp32 partial is a different element size
    assert L.hoccl_ring_hop(a, b, a, 4, hc.BF16, hc.HOP_LAST, None) == hc.ERR_INVALID_ARG


def _compile_and_run(tmp_path, name, body):
    import subprocess
    src = tmp_path / f"{name}.c"
    src.write_text('#include <stddef.h>\n#include <stdio.h>\n#include "hoccl.h"\nint main(void){\n'
                   + body + "return 0;}\n")
    exe = tmp_path / name
    subprocess.run(["gcc", "-std=c11", "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROOT, "include"),
                    "-I/opt/rocm/include", str(src), "-o", str(exe)], check=True)
    return subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()


@pytest.mark.parametrize("cls,ctype", [(hc.Config, "hoccl_config_t"), (hc.Stats, "hoccl_stats_t")])
def test_binding_structs_match_header_layout(tmp_path, cls, ctype):
    """The ctypes mirrors of the configuration and statistics structs have
    the header's field offsets and size (a C compiler says what they are)."""
    body = "".join(f'printf("%zu\\n", offsetof({ctype}, {f}));' for f, _ in cls._fields_)
    body += f'printf("%zu\\n", sizeof({ctype}));'
    got = [int(v) for v in _compile_and_run(tmp_path, ctype, body)]
    want = [getattr(cls, f).offset for f, _ in cls._fields_] + [ctypes.sizeof(cls)]
    assert got == want


def test_enum_values_match_binding(tmp_path):
    """Copy paths keep AUTO 0, SDMA 1, KERNEL 2 with HIP appended as 3; the
    binding's constants equal the header's."""
    names = ["HOCCL_COPY_AUTO", "HOCCL_COPY_SDMA", "HOCCL_COPY_KERNEL", "HOCCL_COPY_HIP",
             "HOCCL_REDUCE_RING", "HOCCL_REDUCE_DIRECT", "HOCCL_REDUCE_AUTO",
             "HOCCL_INT32", "HOCCL_FP32", "HOCCL_BF16", "HOCCL_UINT8"]
    got = [int(v) for v in _compile_and_run(tmp_path, "enums",
                                            "".join(f'printf("%d\\n", (int){n});' for n in names))]
    assert got == [0, 1, 2, 3, 0, 1, 2, 0, 1, 2, 3]
    assert [hc.INT32, hc.FP32, hc.BF16, hc.UINT8] == [0, 1, 2, 3]
    assert [hc.COPY_AUTO, hc.COPY_SDMA, hc.COPY_KERNEL, hc.COPY_HIP] == [0, 1, 2, 3]
    assert [hc.REDUCE_RING, hc.REDUCE_DIRECT, hc.REDUCE_AUTO] == [0, 1, 2]


def test_c_abi_check_compiles_with_its_layout_pins():
    """tests/native/c_abi_check.c pins enum values and struct layouts with
    static assertions; it must compile against the header (it runs on the
    GPU)."""
    import subprocess
    subprocess.run(["gcc", "-std=c11", "-fsyntax-only", "-D__HIP_PLATFORM_AMD__",
                    "-I" + os.path.join(ROOT, "include"), "-I/opt/rocm/include",
                    os.path.join(ROOT, "tests", "native", "c_abi_check.c")], check=True)


def test_stream_ceiling_rejects_bad_arguments_without_a_device():
    L = hc.lib()
    V = ctypes.c_void_p
    assert L.hoccl_debug_stream_ceiling(9, V(0x1000), None, V(0x2000), 64, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_debug_stream_ceiling(2, V(0x1000), None, V(0x2008), 64, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_debug_stream_ceiling(2, V(0x1000), None, V(0x2000), 60, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_debug_stream_ceiling(3, V(0x1000), None, V(0x2000), 64, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_debug_stream_ceiling(6, V(0x1000), None, V(0x2000), 64, None) == hc.ERR_INVALID_ARG  # add_nt needs b
    assert L.hoccl_debug_stream_ceiling(5, None, None, V(0x2000), 64, None) == hc.ERR_INVALID_ARG       # copy_nt needs a
    assert L.hoccl_debug_stream_ceiling(7, V(0x1000), V(0x1000), V(0x2000), 64, None) == hc.ERR_INVALID_ARG
    assert L.hoccl_debug_stream_ceiling(1, None, None, V(0x2000), 0, None) == hc.OK


def test_backend_switch_and_registration():
    """HOCCL_BACKEND selects the backend init_process_group uses; the
    backend registers once under its name."""
    import torch.distributed as dist
    from paper_2609_34334_amd import distributed as hdist
    old = os.environ.pop("HOCCL_BACKEND", None)
    try:
        assert hdist.selected_backend("nccl") == "nccl"
        os.environ["HOCCL_BACKEND"] = "0"
        assert hdist.selected_backend("gloo") == "gloo"
        os.environ["HOCCL_BACKEND"] = "1"
        assert hdist.selected_backend("nccl") == "hoccl"
    finally:
        os.environ.pop("HOCCL_BACKEND", None)
        if old is not None:
            os.environ["HOCCL_BACKEND"] = old
    hdist.register()
    hdist.register()
    assert dist.Backend.HOCCL == "hoccl"


def test_backend_copy_units():
    """The backend's copy collectives move any dtype as bytes: 4-byte units
    where every count and offset allows, else 2-byte, else single bytes.
    Reductions keep to the library's three arithmetic dtypes."""
    import torch
    from paper_2609_34334_amd import distributed as hdist
    assert hdist._unit([8, 4, 0]) == (hc.INT32, 4)
    assert hdist._unit([8, 6]) == (hc.BF16, 2)
    assert hdist._unit([]) == (hc.INT32, 4)
    assert hdist._unit([4, 3]) == (hc.UINT8, 1)
    with pytest.raises(TypeError, match="int32, float32 or bfloat16"):
        hdist._dtype(torch.zeros(2, dtype=torch.int64))


def test_backend_reduction_ops():
    """Sums of every library dtype; averages (FSDP2's reduce-scatter) of
    float32 and bfloat16 only; nothing else."""
    import torch
    import torch.distributed as dist
    from paper_2609_34334_amd import distributed as hdist

    def opts(op):
        o = dist.AllreduceOptions()
        o.reduceOp = op
        return o
    assert hdist._average(None, torch.zeros(1)) is False
    assert hdist._average(opts(dist.ReduceOp.SUM), torch.zeros(1, dtype=torch.int32)) is False
    assert hdist._average(opts(dist.ReduceOp.AVG), torch.zeros(1)) is True
    assert hdist._average(opts(dist.ReduceOp.AVG), torch.zeros(1, dtype=torch.bfloat16)) is True
    for op, dt in ((dist.ReduceOp.AVG, torch.int32), (dist.ReduceOp.MAX, torch.float32),
                   (dist.ReduceOp.PRODUCT, torch.bfloat16)):
        with pytest.raises(ValueError, match="only sums"):
            hdist._average(opts(op), torch.zeros(1, dtype=dt))


def test_backend_group_name():
    """DeviceMesh finds a group by the name torch sets on it."""
    import torch.distributed as dist
    from paper_2609_34334_amd import distributed as hdist
    g = hdist.HocclProcessGroup(dist.HashStore(), 0, 1, None)
    g._set_group_name("7")
    g._set_group_desc("mesh_default")
    assert (g.group_name, g.group_desc) == ("7", "mesh_default")
    g._coll.close()
    g._pp.close()


def test_ipc_export_rejects_host_memory():
    import ctypes as C
    buf = C.create_string_buffer(64)
    off, size = C.c_size_t(0), C.c_size_t(0)
    host = (C.c_char * 256)()
    assert hc.lib().hoccl_ipc_export(C.addressof(host), buf, C.byref(off), C.byref(size)) != hc.OK


def _config_under_env(env):
    """The configuration a fresh process reads from HOCCL_* variables."""
    import json
    import subprocess
    import sys
    code = ("import json, paper_2609_34334_amd as hc; "
            "c = hc.get_config(); print(json.dumps({k: c[k] for k in "
            "('bf16_partials', 'fused_hops', 'a2a_schedule')}))")
    e = dict(os.environ)
    for k in list(e):
        if k.startswith("HOCCL_"):
            del e[k]
    e.update(env)
    out = subprocess.run([sys.executable, "-c", code], env=e, cwd=ROOT, capture_output=True,
                         text=True, timeout=300, check=True)
    return json.loads(out.stdout.strip().splitlines()[-1])


def test_environment_sets_bf16_partials_and_invalid_sets_fall_back():
    assert _config_under_env({}) == {"bf16_partials": 0, "fused_hops": 1, "a2a_schedule": 0}
    assert _config_under_env({"HOCCL_BF16_PARTIALS": "1", "HOCCL_FUSED_HOPS": "3"}) == \
        {"bf16_partials": 1, "fused_hops": 3, "a2a_schedule": 0}
    # one invalid value discards the whole set, as the header states
    assert _config_under_env({"HOCCL_BF16_PARTIALS": "2", "HOCCL_FUSED_HOPS": "3"}) == \
        {"bf16_partials": 0, "fused_hops": 1, "a2a_schedule": 0}
