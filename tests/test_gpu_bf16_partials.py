"""GPU parity of the bf16-partials mode: bf16 reduce-scatter and all-reduce
whose every ring addition is rounded to bf16 (round to nearest, ties to
even) before the next, bit for bit against the oracle's sums with that
rounding at every hop, on the ring, the direct fold and the automatic
choice; ragged, misaligned, in place, in cache groups, on every copy path
and with few workgroups (several passes per thread)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_34334_amd as hc
import workloads as W
from gpu_util import (assert_bitwise, check_canaries, from_dev, padded, to_dev)

pytestmark = pytest.mark.gpu

BF16 = hc.BF16


@pytest.fixture(autouse=True)
def _fresh_config():
    saved = hc.get_config()
    yield
    hc.set_config(**saved)


def run_rs(x, lead=0):
    R = len(x)
    n = x[0].size // R
    outs = [padded(n, BF16, lead) for _ in range(R)]
    hc.reduce_scatter([to_dev(a, BF16) for a in x], [o[1] for o in outs])
    torch.cuda.synchronize()
    for full, _ in outs:
        check_canaries(full, lead, n, BF16)
    return [from_dev(o[1], BF16) for o in outs]


def run_ar(x, lead=0):
    R, n = len(x), x[0].size
    outs = [padded(n, BF16, lead) for _ in range(R)]
    hc.allreduce([to_dev(a, BF16) for a in x], [o[1] for o in outs])
    torch.cuda.synchronize()
    for full, _ in outs:
        check_canaries(full, lead, n, BF16)
    return [from_dev(o[1], BF16) for o in outs]


@pytest.mark.parametrize("algo", ["ring", "direct", "auto"])
@pytest.mark.parametrize("R", [1, 2, 3, 4, 5, 8, 13, 16])
def test_bf16_partials_match_the_oracle(algo, R):
    """Every size from one element to several tiles with a ragged tail; the
    ring takes R-1 one-hop launches."""
    hc.set_config(bf16_partials=1, reduce_algo=algo, copy_path="hip", fused_hops=1)
    differs = False
    for n in [1, 7, R * 37 + 3, 4099, 65536 + 5]:
        seed = 9400 + 13 * R + n
        x = [W.random_values("bf16", seed, r, R * n) for r in range(R)]
        ref = oracle.reduce_scatter_bf16_hops_new(x)
        got = run_rs(x, lead=3)
        if algo == "ring" and R > 1:
            assert hc.last_stats()["reduce_launches"] == R - 1
        for r in range(R):
            assert_bitwise(got[r], ref[r], f"RS {algo} R={R} n={n} r={r}")
        one = oracle.reduce_scatter_new(x, BF16)
        differs |= any(not np.array_equal(a, b) for a, b in zip(one, ref))
        xa = [W.random_values("bf16", seed + 1, r, n) for r in range(R)]
        refa = oracle.allreduce_bf16_hops_new(xa)
        gota = run_ar(xa, lead=1)
        for r in range(R):
            assert_bitwise(gota[r], refa[r], f"AR {algo} R={R} n={n} r={r}")
    # the mode is observable: from three ranks on, the per-hop roundings
    # change some sums against a single rounding
    assert differs or R <= 2


@pytest.mark.parametrize("hops", [2, 3, 7, 64])
@pytest.mark.parametrize("R", [3, 4, 8, 13])
def test_bf16_partials_with_fused_hops(hops, R):
    """k hops per launch round every addition as k separate hops would:
    the oracle's per-hop-rounding bits, in ceil((R-1)/k) launches of at
    most 8 hops, ragged and misaligned."""
    hc.set_config(bf16_partials=1, reduce_algo="ring", copy_path="hip", fused_hops=hops)
    k = min(hops, 8)
    for n in [1, 7, R * 37 + 3, 65536 + 5]:
        x = [W.random_values("bf16", 9540 + R + hops, r, R * n) for r in range(R)]
        ref = oracle.reduce_scatter_bf16_hops_new(x)
        got = run_rs(x, lead=3)
        assert hc.last_stats()["reduce_launches"] == -(-(R - 1) // k)
        for r in range(R):
            assert_bitwise(got[r], ref[r], f"fused RS k={hops} R={R} n={n} r={r}")
        xa = [W.random_values("bf16", 9550 + R + hops, r, n) for r in range(R)]
        refa = oracle.allreduce_bf16_hops_new(xa)
        gota = run_ar(xa, lead=1)
        for r in range(R):
            assert_bitwise(gota[r], refa[r], f"fused AR k={hops} R={R} n={n} r={r}")


@pytest.mark.parametrize("path", ["hip", "engines", "kernel"])
def test_bf16_partials_in_groups_on_every_copy_path(path):
    """Cache groups with a ragged last group, and all-reduce gather groups,
    change neither the fold order nor the roundings."""
    R, n = 8, 30_011
    hc.set_config(bf16_partials=1, reduce_algo="ring", copy_path=path)
    for budget, groups in ((1 << 16, 1), (12_345, 3)):
        with hc.config(ring_group_bytes=budget, allreduce_chunk_groups=groups):
            x = [W.random_values("bf16", 9500, r, R * n) for r in range(R)]
            ref = oracle.reduce_scatter_bf16_hops_new(x)
            got = run_rs(x, lead=5)
            for r in range(R):
                assert_bitwise(got[r], ref[r], f"grouped RS {path} budget={budget} r={r}")
            xa = [W.random_values("bf16", 9501, r, n) for r in range(R)]
            refa = oracle.allreduce_bf16_hops_new(xa)
            gota = run_ar(xa, lead=2)
            for r in range(R):
                assert_bitwise(gota[r], refa[r], f"grouped AR {path} budget={budget} r={r}")


@pytest.mark.parametrize("algo", ["ring", "direct"])
def test_bf16_partials_in_place_and_misaligned_inputs(algo):
    hc.set_config(bf16_partials=1, reduce_algo=algo)
    R, n = 4, 9001
    x = [W.random_values("bf16", 9510, r, n) for r in range(R)]
    ref = oracle.allreduce_bf16_hops_new(x)
    bufs = [to_dev(a, BF16) for a in x]
    hc.allreduce(bufs, bufs)
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(bufs[r], BF16), ref[r], f"AR in place r={r}")
    x = [W.random_values("bf16", 9511, r, R * n) for r in range(R)]
    ref = oracle.reduce_scatter_bf16_hops_new(x)
    bufs = [to_dev(a, BF16) for a in x]
    hc.reduce_scatter(bufs, [b[r * n:(r + 1) * n] for r, b in enumerate(bufs)])
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(bufs[r][r * n:(r + 1) * n], BF16), ref[r], f"RS in place r={r}")
    # inputs at different offsets from 16-byte alignment: every operand of
    # a launch takes the element-wise path
    R, n = 8, 4099
    x = [W.random_values("bf16", 9512, r, R * n) for r in range(R)]
    ref = oracle.reduce_scatter_bf16_hops_new(x)
    full = [to_dev(np.concatenate([np.zeros(r % 3, np.uint16), x[r]]), BF16) for r in range(R)]
    out = hc.reduce_scatter([full[r][r % 3:] for r in range(R)])
    torch.cuda.synchronize()
    for r in range(R):
        assert_bitwise(from_dev(out[r], BF16), ref[r], f"RS misaligned inputs r={r}")


@pytest.mark.parametrize("wg", [8, 0])
def test_bf16_partials_several_passes_per_thread(wg):
    """Eight workgroups leave every thread many passes (the deeper unroll);
    0 is the automatic launch."""
    hc.set_config(bf16_partials=1, reduce_algo="ring", copy_path="hip", workgroups_per_step=wg)
    R, n = 8, (1 << 20) + 17
    x = [W.random_values("bf16", 9520, r, R * n) for r in range(R)]
    ref = oracle.reduce_scatter_bf16_hops_new(x)
    got = run_rs(x, lead=1)
    for r in range(R):
        assert_bitwise(got[r], ref[r], f"RS wg={wg} r={r}")


def test_bf16_partials_leave_other_dtypes_alone():
    hc.set_config(bf16_partials=1, reduce_algo="ring", copy_path="hip")
    R, n = 5, 3001
    for dt, name in ((hc.FP32, "fp32"), (hc.INT32, "int32")):
        x = [W.random_values(name, 9530, r, R * n) for r in range(R)]
        ref = oracle.reduce_scatter_new(x, dt)
        send = [to_dev(a, dt) for a in x]
        out = hc.reduce_scatter(send)
        torch.cuda.synchronize()
        for r in range(R):
            assert_bitwise(from_dev(out[r], dt), ref[r], f"{name} RS r={r}")
