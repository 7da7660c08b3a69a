"""Pins for the CPU oracle (no GPU).

The oracle is checked against things other than itself:
  * hand-derived ring-order fixtures (tests/golden/ring_order.txt);
  * a simulation of the ring protocol in pure Python (oracle/brute.py);
  * closed forms for int32 sums, subnormal sums and signed zeros;
  * Higham's bound for recursive summation against the exact rational sum;
  * the exhaustive fp32 -> bf16 round-to-nearest-even table of torch;
  * numpy library routines (concatenate, float32 add of two operands);
  * collective invariants (RS = slice of AR, AG = concatenation, A2A is an
    involution, send/recv leaves other receivers untouched).
"""
import math
import os
import struct
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from oracle import brute
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "ring_order.txt")
CODE = {"int32": oracle.INT32, "fp32": oracle.FP32, "bf16": oracle.BF16}
NPT = {"int32": np.int32, "fp32": np.float32, "bf16": np.uint16}


def _bits(a):
    a = np.asarray(a)
    return a.view({2: np.uint16, 4: np.uint32}[a.dtype.itemsize])


def _to_py(a, dtype):
    if dtype == "fp32":
        return [float(v) for v in a]
    return [int(v) for v in a]


def _from_py(vals, dtype):
    return np.array(vals, dtype=NPT[dtype])


# ---------------------------------------------------------------- golden order

def _golden():
    rows = []
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if not line:
            continue
        f = line.split()
        dtype, R = f[0], int(f[1])
        vals = [int(v, 16) for v in f[2:2 + R]]
        rows.append((dtype, R, vals, int(f[2 + R], 16)))
    return rows


@pytest.mark.parametrize("row", _golden(), ids=lambda r: f"{r[0]}-R{r[1]}")
def test_ring_order_reduce_scatter(row):
    dtype, R, vals, expect = row
    bt = np.uint32 if dtype == "fp32" else np.uint16
    n = 5
    x = [np.zeros(R * n, dtype=bt) for _ in range(R)]
    for j in range(R):                      # block j's fold starts at rank j+1
        for m in range(1, R + 1):
            x[(j + m) % R][j * n:(j + 1) * n] = vals[m - 1]
    x = [a.view(NPT[dtype]) for a in x]
    out = oracle.reduce_scatter_new(x, CODE[dtype])
    for r in range(R):
        assert (_bits(out[r]) == expect).all(), (r, _bits(out[r]))


@pytest.mark.parametrize("row", _golden(), ids=lambda r: f"{r[0]}-R{r[1]}")
@pytest.mark.parametrize("count", [1, 2, 7, 10, 13, 31])
def test_ring_order_allreduce_ragged(row, count):
    dtype, R, vals, expect = row
    bt = np.uint32 if dtype == "fp32" else np.uint16
    c = -(-count // R)                      # chunk length ceil(count / R)
    x = [np.zeros(count, dtype=bt) for _ in range(R)]
    for i in range(count):
        j = i // c
        for m in range(1, R + 1):
            x[(j + m) % R][i] = vals[m - 1]
    x = [a.view(NPT[dtype]) for a in x]
    out = oracle.allreduce_new(x, CODE[dtype])
    for r in range(R):
        assert (_bits(out[r]) == expect).all(), (r, _bits(out[r]))


# ------------------------------------------------------- brute-force ring model

@pytest.mark.parametrize("dtype", ["int32", "fp32", "bf16"])
@pytest.mark.parametrize("R", [1, 2, 3, 4, 5, 8])
def test_ring_simulation_matches_oracle(dtype, R):
    for n in list(range(0, 18)) + [29]:
        seed = 1000 + 37 * R + n
        # reduce-scatter with recvcount n
        x = [W.random_values(dtype, seed, r, R * n) for r in range(R)]
        got = oracle.reduce_scatter_new(x, CODE[dtype])
        ref = brute.ring_reduce_scatter([_to_py(a, dtype) for a in x], n, dtype=CODE[dtype])
        for r in range(R):
            assert np.array_equal(_bits(got[r]), _bits(_from_py(ref[r], dtype))), (n, r)
        # all-reduce with count n
        x = [W.random_values(dtype, seed + 1, r, n) for r in range(R)]
        got = oracle.allreduce_new(x, CODE[dtype])
        ref = brute.ring_allreduce([_to_py(a, dtype) for a in x], CODE[dtype])
        for r in range(R):
            assert np.array_equal(_bits(got[r]), _bits(_from_py(ref[r], dtype))), (n, r)


@pytest.mark.parametrize("R", [1, 2, 3, 4, 6])
def test_copy_collectives_match_flow_lists(R):
    for n in [0, 1, 5, 17]:
        for es, code in [(4, oracle.FP32), (2, oracle.BF16), (1, oracle.UINT8)]:
            x = [W.random_bits(77 + n, r, R * n, es) for r in range(R)]
            # all-to-all
            got = [np.zeros(R * n, dtype=x[0].dtype) for _ in range(R)]
            oracle.alltoall(x, got, n, code)
            ref = brute.alltoall([list(a) for a in x], n)
            for r in range(R):
                assert [int(v) for v in got[r]] == [int(v) for v in ref[r]]
            # all-gather of the first n elements
            s = [np.ascontiguousarray(a[:n]) for a in x]
            got = oracle.allgather_new(s, code)
            ref = brute.allgather([list(a) for a in s])
            for r in range(R):
                assert [int(v) for v in got[r]] == [int(v) for v in ref[r]]


# --------------------------------------------------------------- closed forms

@pytest.mark.parametrize("R", [1, 2, 3, 4, 7, 8, 16, 64])
def test_int32_closed_form(R):
    n = 1000
    x = [(r * n + np.arange(n)).astype(np.int32) for r in range(R)]
    out = oracle.allreduce_new(x, oracle.INT32)
    i = np.arange(n, dtype=np.int64)
    expect = n * R * (R - 1) // 2 + R * i
    for r in range(R):
        assert np.array_equal(out[r].astype(np.int64), expect)
    # reduce-scatter of R blocks of m elements: element k of the flat input
    m = 37
    x = [(r * R * m + np.arange(R * m)).astype(np.int32) for r in range(R)]
    out = oracle.reduce_scatter_new(x, oracle.INT32)
    for r in range(R):
        k = r * m + np.arange(m, dtype=np.int64)
        assert np.array_equal(out[r].astype(np.int64), R * m * R * (R - 1) // 2 + R * k)


@pytest.mark.parametrize("R", [2, 3, 8])
def test_int32_wraps_mod_2_32(R):
    n = 4096
    x = [W.random_int32(5, r, n, 2 ** 31 - 2 ** 20, 2 ** 31) for r in range(R)]
    x[0][:n // 2] = W.random_int32(6, 0, n // 2, -(2 ** 31), -(2 ** 31) + 2 ** 20)
    out = oracle.allreduce_new(x, oracle.INT32)
    tot = sum(a.astype(object) for a in x)
    expect = [((int(t) + 2 ** 31) % 2 ** 32) - 2 ** 31 for t in tot]
    assert [int(v) for v in out[0]] == expect


def test_fp32_subnormal_sums_are_exact():
    # k * 2^-149 values: sums of subnormals are exact (no flush to zero)
    R, n = 5, 64
    rng = np.random.default_rng(9)
    k = [rng.integers(0, 1 << 18, n) for _ in range(R)]
    tiny = 2.0 ** -149
    x = [(kr * tiny).astype(np.float32) for kr in k]
    out = oracle.allreduce_new(x, oracle.FP32)
    expect = (sum(k) * tiny).astype(np.float32)
    assert np.array_equal(_bits(out[0]), _bits(expect))
    assert (out[0] != 0).any()


def test_bf16_subnormal_sums_are_exact():
    R, n = 4, 64
    rng = np.random.default_rng(10)
    k = [rng.integers(0, 32, n) for _ in range(R)]          # k * 2^-133
    x = [(kr.astype(np.uint16)) for kr in k]                # bf16 bits of k*2^-133
    out = oracle.allreduce_new(x, oracle.BF16)
    total = sum(k)                                          # < 128: representable
    assert np.array_equal(out[0].astype(np.int64), total)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_signed_zero(dtype):
    R = 4
    neg = 0x80000000 if dtype == "fp32" else 0x8000
    bt = np.uint32 if dtype == "fp32" else np.uint16
    x = [np.full(8, neg, dtype=bt).view(NPT[dtype]) for _ in range(R)]
    out = oracle.allreduce_new(x, CODE[dtype])
    assert (_bits(out[0]) == neg).all()                     # -0 + -0 = -0
    x[2] = np.zeros(8, dtype=bt).view(NPT[dtype])
    out = oracle.allreduce_new(x, CODE[dtype])
    assert (_bits(out[0]) == 0).all()                       # any +0 gives +0


def test_inf_and_nan():
    x = [np.array([np.inf, np.inf, 1.0], np.float32),
         np.array([1.0, -np.inf, np.nan], np.float32)]
    out = oracle.allreduce_new(x, oracle.FP32)
    assert out[0][0] == np.inf and np.isnan(out[0][1]) and np.isnan(out[0][2])


# --------------------------------------------------------- error bound (Higham)

def _gamma(k, u):
    return k * u / (1 - k * u)


@pytest.mark.parametrize("R", [2, 3, 5, 8])
def test_fp32_within_recursive_summation_bound(R):
    n = 400
    x = [W.uniform_f32(21, r, n) for r in range(R)]
    out = oracle.allreduce_new(x, oracle.FP32)
    g = _gamma(R - 1, 2.0 ** -24)
    for i in range(n):
        vals = [Fraction(float(a[i])) for a in x]
        exact = sum(vals)
        bound = Fraction(g) * sum(abs(v) for v in vals)
        assert abs(Fraction(float(out[0][i])) - exact) <= bound


@pytest.mark.parametrize("R", [2, 4, 8])
def test_bf16_within_bound(R):
    n = 300
    x = [W.normal_bf16(22, r, n, 1.0) for r in range(R)]
    out = oracle.allreduce_new(x, oracle.BF16)
    g = _gamma(R - 1, 2.0 ** -24)
    for i in range(n):
        vals = [Fraction(float(W.bf16_bits_to_f32(a[i]))) for a in x]
        exact = sum(vals)
        o = float(W.bf16_bits_to_f32(out[0][i]))
        ulp = 2.0 ** (math.frexp(max(abs(o), 2.0 ** -126))[1] - 8)
        bound = Fraction(ulp) / 2 + Fraction(g) * sum(abs(v) for v in vals) * 2
        assert abs(Fraction(o) - exact) <= bound


def test_small_integer_sums_exact():
    R, n = 8, 500
    rng = np.random.default_rng(3)
    ints = [rng.integers(-1000, 1000, n) for _ in range(R)]
    out = oracle.allreduce_new([a.astype(np.float32) for a in ints], oracle.FP32)
    assert np.array_equal(out[0], sum(ints).astype(np.float32))
    ints = [rng.integers(-32, 32, n) for _ in range(R)]     # |sum| <= 256
    out = oracle.allreduce_new([W.to_bf16_bits(a) for a in ints], oracle.BF16)
    assert np.array_equal(W.bf16_bits_to_f32(out[0]), sum(ints).astype(np.float32))


def test_two_ranks_equal_numpy_float32_add():
    x = [W.uniform_f32(23, r, 10000) for r in range(2)]
    out = oracle.allreduce_new(x, oracle.FP32)
    assert np.array_equal(_bits(out[1]), _bits(x[0] + x[1]))


# ------------------------------------------------------------------ invariants

@pytest.mark.parametrize("dtype", ["int32", "fp32", "bf16"])
@pytest.mark.parametrize("R", [1, 2, 3, 8])
def test_rs_is_slice_of_ar_and_ar_outputs_identical(dtype, R):
    n = 53
    x = [W.random_values(dtype, 31, r, R * n) for r in range(R)]
    rs = oracle.reduce_scatter_new(x, CODE[dtype])
    ar = oracle.allreduce_new(x, CODE[dtype])
    for r in range(R):
        assert np.array_equal(_bits(ar[r]), _bits(ar[0]))
        assert np.array_equal(_bits(rs[r]), _bits(ar[0][r * n:(r + 1) * n]))


@pytest.mark.parametrize("R", [1, 3, 8])
def test_allgather_is_concatenation(R):
    x = [W.random_bits(41, r, 1001, 2) for r in range(R)]
    out = oracle.allgather_new(x, oracle.BF16)
    cat = np.concatenate(x)
    for r in range(R):
        assert np.array_equal(out[r], cat)


@pytest.mark.parametrize("R", [2, 5, 8])
def test_alltoall_involution(R):
    n = 33
    x = [W.random_bits(42, r, R * n, 4) for r in range(R)]
    y = [np.zeros_like(a) for a in x]
    z = [np.zeros_like(a) for a in x]
    oracle.alltoall(x, y, n, oracle.FP32)
    oracle.alltoall(y, z, n, oracle.FP32)
    for r in range(R):
        assert np.array_equal(z[r], x[r])
    # not the identity map for R > 1
    assert any(not np.array_equal(y[r], x[r]) for r in range(R))


def test_alltoallv_transposed_restores():
    R = 8
    send, counts, sd, rd, rsz = W.a2a_tokens(R=R, tokens=64, hidden=16, experts=64, topk=6)
    recv = [np.zeros(s, dtype=np.uint16) for s in rsz]
    oracle.alltoallv(send, counts, sd, recv, rd, oracle.BF16)
    countsT = [counts[d * R + s] for s in range(R) for d in range(R)]
    sdT = [rd[d * R + s] for s in range(R) for d in range(R)]
    rdT = [sd[d * R + s] for s in range(R) for d in range(R)]
    back = [np.zeros_like(s) for s in send]
    oracle.alltoallv(recv, countsT, sdT, back, rdT, oracle.BF16)
    for r in range(R):
        assert np.array_equal(back[r], send[r])
    ref = brute.alltoallv([list(a) for a in send], counts, sd,
                          [[None] * s for s in rsz], rd)
    for r in range(R):
        assert [int(v) for v in recv[r]] == ref[r]


def test_uint8_copies_and_no_uint8_sums():
    """Bytes move like any element (odd counts and offsets included); the
    reductions refuse them, as the sum is defined for int32, fp32 and bf16."""
    R = 3
    rng = np.random.default_rng(5)
    C = rng.integers(0, 6, size=(R, R))
    send = [W.random_bits(88, s, int(C[s].sum()), 1) for s in range(R)]
    counts = [int(C[s][d]) for s in range(R) for d in range(R)]
    sd = [int(C[s][:d].sum()) for s in range(R) for d in range(R)]
    rd = [int(C[:s, d].sum()) for s in range(R) for d in range(R)]
    rsz = [int(C[:, d].sum()) for d in range(R)]
    recv = [np.zeros(s, dtype=np.uint8) for s in rsz]
    oracle.alltoallv(send, counts, sd, recv, rd, oracle.UINT8)
    ref = brute.alltoallv([list(a) for a in send], counts, sd, [[None] * s for s in rsz], rd)
    for r in range(R):
        assert [int(v) for v in recv[r]] == ref[r]
    x = [W.random_bits(89, r, 7, 1) for r in range(R)]
    got = [np.full(7, 0xA5, np.uint8) for _ in range(R)]
    oracle.sendrecv(x, got, [2, -1, 0], 7, oracle.UINT8)
    ref = brute.sendrecv([list(a) for a in x], [[0xA5] * 7 for _ in range(R)], [2, -1, 0])
    for r in range(R):
        assert [int(v) for v in got[r]] == [int(v) for v in ref[r]]
    assert oracle.dtype_code(np.uint8) == oracle.UINT8
    with pytest.raises(ValueError):
        oracle.allreduce_new(x, oracle.UINT8)
    with pytest.raises(ValueError):
        oracle.reduce_scatter_new([W.random_bits(90, r, 6, 1) for r in range(R)], oracle.UINT8)


def test_sendrecv_pipeline_and_canaries():
    R, n = 8, 100
    x = [W.random_bits(43, r, n, 2) for r in range(R)]
    peers = [r + 1 if r + 1 < R else -1 for r in range(R)]  # forward pipeline
    canary = np.uint16(0xDEAD)
    recv = [np.full(n, canary, dtype=np.uint16) for _ in range(R)]
    oracle.sendrecv(x, recv, peers, n, oracle.BF16)
    assert (recv[0] == canary).all()
    for r in range(1, R):
        assert np.array_equal(recv[r], x[r - 1])
    with pytest.raises(ValueError):
        oracle.sendrecv(x, recv, [1, 1] + [-1] * (R - 2), n, oracle.BF16)


def test_argument_errors():
    x = [np.zeros(4, np.float32)]
    with pytest.raises(ValueError):
        oracle.allreduce(x * 65, x * 65, 4, oracle.FP32)
    with pytest.raises(ValueError):
        oracle.allreduce(x, x, 4, 7)


# ---------------------------------------------------------- fp32 -> bf16 table

def test_bf16_rounding_matches_python_model():
    rng = np.random.default_rng(44)
    pats = rng.integers(0, 2 ** 32, 20000, dtype=np.uint64).astype(np.uint32)
    edge = np.array([0, 0x80000000, 0x7F7FFFFF, 0x7F7F8000, 0x7F800000, 0xFF800000,
                     0x00000001, 0x00008000, 0x00018000, 0x3F808000, 0x3F818000,
                     0x7FC00001, 0xFFA00000, 0x007FFFFF], dtype=np.uint32)
    pats = np.concatenate([pats, edge])
    got = oracle.f32_to_bf16(pats.view(np.float32))
    for p, g in zip(pats, got):
        f = struct.unpack("<f", struct.pack("<I", int(p)))[0]
        if math.isnan(f):
            assert (int(g) & 0x7F80) == 0x7F80 and (int(g) & 0x7F)
        else:
            assert int(g) == brute.float_to_bf16_bits(f), hex(int(p))


def test_bf16_rounding_exhaustive_against_torch():
    step = 1 << 23                                  # one sign+exponent per chunk
    base = np.arange(step, dtype=np.uint32)
    u = np.empty(step, dtype=np.uint32)
    ours = np.empty(step, dtype=np.uint16)
    L = oracle.lib()
    for start in range(0, 1 << 32, step):
        np.add(base, np.uint32(start), out=u)
        f = u.view(np.float32)
        L.oracle_f32_to_bf16_array(f.ctypes.data, ours.ctypes.data, step)
        ref = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        if (start >> 23) & 0xFF == 0xFF:            # exponent all ones: Inf/NaN
            nan = np.isnan(f)
            assert np.array_equal(ours[~nan], ref[~nan]), hex(start)
            o = ours[nan]
            assert ((o & 0x7F80) == 0x7F80).all() and ((o & 0x7F) != 0).all()
        else:
            assert np.array_equal(ours, ref), hex(start)


# ------------------------------------------- bf16 partials rounded at every hop

@pytest.mark.parametrize("R", [1, 2, 3, 4, 6])
def test_bf16_hops_ring_simulation_matches_oracle(R):
    """The fold with bf16 partials against the pure-Python ring that rounds
    every partial it passes on (reduce-scatter and ragged all-reduce)."""
    for n in list(range(0, 12)) + [29]:
        x = [W.random_values("bf16", 3000 + 7 * R + n, r, R * n) for r in range(R)]
        got = oracle.reduce_scatter_bf16_hops_new(x)
        ref = brute.ring_reduce_scatter([_to_py(a, "bf16") for a in x], n, dtype=oracle.BF16, bf16_hops=True)
        for r in range(R):
            assert np.array_equal(got[r], _from_py(ref[r], "bf16")), (n, r)
        x = [W.random_values("bf16", 3100 + 7 * R + n, r, n) for r in range(R)]
        got = oracle.allreduce_bf16_hops_new(x)
        ref = brute.ring_allreduce([_to_py(a, "bf16") for a in x], oracle.BF16, bf16_hops=True)
        for r in range(R):
            assert np.array_equal(got[r], _from_py(ref[r], "bf16")), (n, r)


def test_bf16_hops_worked_example():
    """Three ranks, rank 0's block: the fold takes x1 = 1, x2 = 2^-8, x0 = 2^-8.
    With one rounding at the end the sum 1 + 2^-7 is a bf16 value; rounded at
    every hop, 1 + 2^-8 is a tie between 1 and 1 + 2^-7 and goes to the even
    1, twice, so the result is 1."""
    one, eps = 0x3F80, 0x3B80                          # 1.0 and 2^-8 in bf16
    x = [np.array([eps], np.uint16), np.array([one], np.uint16), np.array([eps], np.uint16)]
    x = [np.concatenate([a, np.zeros(2, np.uint16)]) for a in x]      # R * recvcount = 3
    assert oracle.reduce_scatter_new(x, oracle.BF16)[0][0] == 0x3F81  # 1 + 2^-7
    assert oracle.reduce_scatter_bf16_hops_new(x)[0][0] == one


def test_bf16_hops_worked_example_four_ranks():
    """Four ranks, block 0: the ring folds x1 = 1, then x2 = x3 = x0 = 2^-8.
    Rounded at every hop, each 1 + 2^-8 is a tie that goes to the even 1, so
    the result is 1 (0x3F80).  Rounded once, 1 + 3*2^-8 is a tie between
    1 + 2^-7 and 1 + 2^-6 that goes to the even 1 + 2^-6 (0x3F82).  A fold
    that starts one rank later, or runs backwards, adds the three small
    terms first (exactly, 3*2^-8) and also gives 0x3F82, so only the ring's
    order with per-hop rounding gives 0x3F80.  All-reduce's block 0 is the
    same sum."""
    one, eps = 0x3F80, 0x3B80
    vals = [eps, one, eps, eps]                              # x0, x1, x2, x3 at block 0
    x = [np.concatenate([[v], np.zeros(3)]).astype(np.uint16) for v in vals]
    assert oracle.reduce_scatter_new(x, oracle.BF16)[0][0] == 0x3F82
    assert oracle.reduce_scatter_bf16_hops_new(x)[0][0] == 0x3F80
    assert all(r[0] == 0x3F80 for r in oracle.allreduce_bf16_hops_new(x))
    assert all(r[0] == 0x3F82 for r in oracle.allreduce_new(x, oracle.BF16))


def test_bf16_hops_special_cases():
    """Two ranks round once in either mode; sums of small integers are exact
    in either mode; rank-count 1 is the identity."""
    x = [W.normal_bf16(24, r, 5000, 1.0) for r in range(2)]
    assert np.array_equal(oracle.allreduce_bf16_hops_new(x)[0], oracle.allreduce_new(x, oracle.BF16)[0])
    rng = np.random.default_rng(4)
    ints = [rng.integers(-16, 16, 700) for _ in range(8)]   # every partial |.| <= 128
    xs = [W.to_bf16_bits(a) for a in ints]
    assert np.array_equal(W.bf16_bits_to_f32(oracle.allreduce_bf16_hops_new(xs)[3]),
                          sum(ints).astype(np.float32))
    one = [W.normal_bf16(25, 0, 33, 1.0)]
    assert np.array_equal(oracle.allreduce_bf16_hops_new(one)[0], one[0])


@pytest.mark.parametrize("R", [3, 8])
def test_bf16_hops_within_bound(R):
    """Each of the R-1 hops rounds the partial once to bf16 (8 significant
    bits: at most 2^-8 of its magnitude) after an fp32 add (2^-24): the
    result lies within (R-1)(2^-8 + 2^-24) times the sum of magnitudes of
    the exact sum."""
    n = 300
    x = [W.normal_bf16(26, r, n, 1.0) for r in range(R)]
    out = oracle.allreduce_bf16_hops_new(x)
    for i in range(n):
        vals = [Fraction(float(W.bf16_bits_to_f32(a[i]))) for a in x]
        bound = (R - 1) * Fraction(2.0 ** -8 + 2.0 ** -24) * sum(abs(v) for v in vals)
        assert abs(Fraction(float(W.bf16_bits_to_f32(out[0][i]))) - sum(vals)) <= bound
