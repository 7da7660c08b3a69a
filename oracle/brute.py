"""Pure-Python brute force for tiny collectives -- TEST INFRASTRUCTURE ONLY.

Standard library only.  It is a second, independent formulation of the same
collectives that pins the C oracle:

* reductions are computed by *simulating the ring protocol* rank by rank:
  R ranks each hold a buffer, and in each of the R-1 reduce steps every rank
  r receives a partial from rank r-1 and adds its own element (ring direction
  r -> r+1), after which rank j holds the reduced chunk j; all-reduce then
  runs the R-1 forwarding steps of a ring all-gather.  The C oracle instead
  writes the fold for each output element directly, so a wrong start rank, a
  dropped or doubled term, or a wrong chunk partition in either one shows up
  as a mismatch;
* fp32 additions are done in binary64 and rounded to binary32 by
  ``struct.pack('<f', .)``; binary64 has more than 2*24+2 significand bits,
  so by Figueroa's double-rounding result this is the correctly rounded
  binary32 sum;
* fp32 -> bf16 rounding uses ``math.frexp`` and Python's round-half-even
  ``round()`` on the significand scaled to 8 bits (bf16 keeps 8 significant
  bits and the binary32 exponent range), rather than bit manipulation;
* copy collectives are written as explicit lists of flows (source rank,
  source offset, destination rank, destination offset, length): the traffic
  matrix of the collective.

Values are Python ints for int32 (any int; results wrap to [-2^31, 2^31)),
Python floats for fp32 (each must be binary32-representable) and ints in
[0, 65536) holding bf16 bit patterns for bf16.
"""
import math
import struct

INT32, FP32, BF16 = 0, 1, 2


def _wrap32(v):
    v &= 0xFFFFFFFF
    return v - (1 << 32) if v & 0x80000000 else v


def _round_f32(v):
    return struct.unpack("<f", struct.pack("<f", v))[0]


def bf16_bits_to_float(h):
    return struct.unpack("<f", struct.pack("<I", (h & 0xFFFF) << 16))[0]


def float_to_bf16_bits(v):
    """Round a binary32-representable float to the nearest bf16, ties to even."""
    if math.isnan(v):
        bits = struct.unpack("<I", struct.pack("<f", v))[0]
        return ((bits >> 16) | 0x40) & 0xFFFF
    sign = 0x8000 if math.copysign(1.0, v) < 0 else 0
    a = abs(v)
    if math.isinf(a):
        return sign | 0x7F80
    if a == 0.0:
        return sign
    m, e = math.frexp(a)            # a = m * 2**e, 0.5 <= m < 1
    if e - 1 >= -126:               # normal range: 8 significant bits
        q = round(m * 256)          # round half to even
        r = math.ldexp(q, e - 8)
    else:                           # subnormal range: quantum 2**-133
        q = round(math.ldexp(a, 133))
        r = math.ldexp(q, -133)
    if r >= 2.0 ** 128:
        return sign | 0x7F80
    bits = struct.unpack("<I", struct.pack("<f", r))[0]
    assert bits & 0xFFFF == 0
    return sign | (bits >> 16)


def _add(dtype, acc, v):
    if dtype == INT32:
        return _wrap32(acc + v)
    return _round_f32(acc + v)


def _widen(dtype, v):
    return bf16_bits_to_float(v) if dtype == BF16 else v


def _narrow(dtype, v):
    return float_to_bf16_bits(v) if dtype == BF16 else v


def ring_reduce_scatter(x, n, dtype, bf16_hops=False):
    """x: R lists of R*n values.  Returns R lists of n values (rank r owns
    block r).  Simulates the R-1 reduce steps of a ring r -> r+1.  With
    bf16_hops (bf16 only), every partial a rank passes on is rounded to
    bf16 first."""
    R = len(x)
    if R == 1:
        return [list(x[0][:n])]
    # step 0: rank r sends its own contribution to block (r-1) to rank r+1,
    # i.e. rank r receives block (r-2)'s element from rank r-1.
    inbox = [None] * R
    for r in range(R):
        blk = (r - 2) % R
        sender = (r - 1) % R
        inbox[r] = (blk, [_widen(dtype, v) for v in x[sender][blk * n:(blk + 1) * n]])
    for step in range(R - 1):
        outbox = [None] * R
        for r in range(R):
            blk, part = inbox[r]
            mine = x[r][blk * n:(blk + 1) * n]
            part = [_add(dtype, p, _widen(dtype, v)) for p, v in zip(part, mine)]
            if bf16_hops:
                part = [bf16_bits_to_float(float_to_bf16_bits(p)) for p in part]
            outbox[r] = (blk, part)
        if step == R - 2:
            out = [None] * R
            for r in range(R):
                blk, part = outbox[r]
                assert blk == r
                out[r] = [_narrow(dtype, p) for p in part]
            return out
        inbox = [outbox[(r - 1) % R] for r in range(R)]
    raise AssertionError("unreachable")


def ring_allreduce(x, dtype, bf16_hops=False):
    """x: R lists of n values.  Chunk size c = ceil(n / R); ragged chunks are
    simulated as blocks padded to c elements whose pad is discarded."""
    R = len(x)
    n = len(x[0])
    if n == 0:
        return [[] for _ in range(R)]
    c = -(-n // R)
    pad = 0 if dtype != BF16 else 0
    xp = [list(xr) + [pad] * (R * c - n) for xr in x]
    owned = ring_reduce_scatter(xp, c, dtype, bf16_hops)   # rank j owns chunk j
    # ring all-gather: at step s, rank r forwards chunk (r - s) to rank r+1.
    have = [{r: owned[r]} for r in range(R)]
    for s in range(R - 1):
        sends = [((r - s) % R, have[r][(r - s) % R]) for r in range(R)]
        for r in range(R):
            blk, data = sends[r]
            have[(r + 1) % R][blk] = list(data)
    out = []
    for r in range(R):
        flat = []
        for j in range(R):
            flat += have[r][j]
        out.append(flat[:n])
    return out


def _apply_flows(send, recv, flows):
    for (s, so, d, do, ln) in flows:
        recv[d][do:do + ln] = send[s][so:so + ln]


def allgather(send):
    R, n = len(send), len(send[0])
    recv = [[None] * (R * n) for _ in range(R)]
    _apply_flows(send, recv, [(s, 0, d, s * n, n) for s in range(R) for d in range(R)])
    return recv


def alltoall(send, n):
    R = len(send)
    recv = [[None] * (R * n) for _ in range(R)]
    _apply_flows(send, recv, [(s, d * n, d, s * n, n) for s in range(R) for d in range(R)])
    return recv


def alltoallv(send, counts, sdispls, recv, rdispls):
    R = len(send)
    flows = [(s, sdispls[s * R + d], d, rdispls[s * R + d], counts[s * R + d])
             for s in range(R) for d in range(R)]
    _apply_flows(send, recv, flows)
    return recv


def sendrecv(send, recv, peers):
    _apply_flows(send, recv, [(r, 0, d, 0, len(send[r]))
                              for r, d in enumerate(peers) if d >= 0])
    return recv
