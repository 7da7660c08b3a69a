"""Planted mistakes in the oracle must fail its pins (CPU only, no GPU).

Each mutant is a copy of ``oracle/hoccl_oracle.c`` with one plausible
mistake written into it: a fold that starts at the wrong rank or runs the
wrong way, a dropped term, a wrong sign, the wrong block or chunk length, an
operand taken from the wrong rank, a truncating or ties-away conversion,
and the same for the fold with bf16 partials.  The
copy is built into a temporary library that stands in for the oracle's own
while the fast pins of ``test_oracle_pins.py`` run against it.  A mutant that
passed every pin would be a mistake the pins cannot see, so each must fail
at least one.  The unmutated copy, built the same way, must pass them all:
otherwise a failing battery would "detect" every mutant for free.

Every planted mistake keeps each access inside its buffer, so a mutant can
give wrong values but never corrupt the test process.
"""
import os
import subprocess

import pytest

import oracle
import test_oracle_pins as P

SRC = os.path.join(os.path.dirname(oracle.__file__), "hoccl_oracle.c")

# (name, text in the oracle, replacement, how many times the text occurs)
MUTANTS = [
    ("fold starts at rank j, not j+1",
     "x[(j + k) % R]", "x[(j + k - 1) % R]", 4),
    ("fold runs backwards (j, j-1, ..., j+1)",
     "x[(j + k) % R]", "x[(j + R + 1 - k) % R]", 4),
    ("fold drops rank j's own term",
     "for (int k = 1; k <= R; ++k)", "for (int k = 1; k < R; ++k)", 3),
    ("int32 partials subtracted",
     "acc = (k == 1) ? v : acc + v;\n        }\n        *(int32_t *)out",
     "acc = (k == 1) ? v : acc - v;\n        }\n        *(int32_t *)out", 1),
    ("fp32 first term counted twice",
     "acc = (k == 1) ? xr[i] : acc + xr[i];", "acc = (k == 1) ? xr[i] + xr[i] : acc + xr[i];", 1),
    ("bf16 widened with the wrong shift",
     "uint32_t u = (uint32_t)h << 16;", "uint32_t u = (uint32_t)h << 15;", 1),
    ("bf16 conversion truncates",
     "if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u)))", "if (0)", 1),
    ("bf16 conversion rounds ties away from zero",
     "if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u)))", "if (dropped >= 0x8000u)", 1),
    ("bf16 conversion turns NaN into infinity",
     "return (uint16_t)((u >> 16) | 0x0040u);", "return (uint16_t)((u >> 16) & 0xff80u);", 1),
    ("all-reduce chunk length one too long",
     "size_t c = (count + (size_t)R - 1) / (size_t)R;", "size_t c = count / (size_t)R + 1;", 2),
    ("all-reduce writes rank 0's output only",
     "for (int r = 0; r < R; ++r)\n            memcpy((unsigned char *)recv[r] + i * es, v, es);",
     "for (int r = 0; r < 1; ++r)\n            memcpy((unsigned char *)recv[r] + i * es, v, es);", 1),
    ("reduce-scatter folds in rank r+1's order",
     "ring_sum_one(send, dtype, R, r, (size_t)r * recvcount + i,",
     "ring_sum_one(send, dtype, R, (r + 1) % R, (size_t)r * recvcount + i,", 1),
    ("reduce-scatter gives rank r block r+1",
     "ring_sum_one(send, dtype, R, r, (size_t)r * recvcount + i,",
     "ring_sum_one(send, dtype, R, r, (size_t)((r + 1) % R) * recvcount + i,", 1),
    ("all-gather copies the receiver's own shard",
     "(const unsigned char *)send[s] + i * es, es);", "(const unsigned char *)send[r] + i * es, es);", 1),
    ("all-to-all block indices transposed",
     "(const unsigned char *)send[s] + ((size_t)d * count + i) * es,",
     "(const unsigned char *)send[d] + ((size_t)s * count + i) * es,", 1),
    ("all-to-all(v) drops each block's last element",
     "for (size_t i = 0; i < sendcounts[k]; ++i)", "for (size_t i = 0; i + 1 < sendcounts[k]; ++i)", 1),
    ("bf16 partials: the fold starts at rank j's own term",
     "uint16_t part = ((const uint16_t *)x[(j + 1) % R])[i];", "uint16_t part = ((const uint16_t *)x[j % R])[i];", 1),
    ("bf16 partials: the fold drops rank j's own term",
     "for (int k = 2; k <= R; ++k)", "for (int k = 2; k < R; ++k)", 1),
    ("bf16 partials: each hop subtracts its contribution",
     "part = oracle_f32_to_bf16(bf16_to_f32(part) + bf16_to_f32(xr[i]));",
     "part = oracle_f32_to_bf16(bf16_to_f32(part) - bf16_to_f32(xr[i]));", 1),
    ("bf16 partials: the hops run backwards (j+1, j, j-1, ..., j+2)",
     "(const uint16_t *)x[(j + k) % R];\n        part =",
     "(const uint16_t *)x[(j + R + 2 - k) % R];\n        part =", 1),
    ("send/recv runs the wrong direction",
     "memcpy((unsigned char *)recv[d] + i * es,\n                   (const unsigned char *)send[r] + i * es, es);",
     "memcpy((unsigned char *)recv[r] + i * es,\n                   (const unsigned char *)send[d] + i * es, es);", 1),
]


def battery():
    """The fast pins, as (name, callable); each raises when the oracle is wrong."""
    rows = P._golden()
    return [
        ("ring-order fixtures, reduce-scatter", lambda: [P.test_ring_order_reduce_scatter(r) for r in rows]),
        ("ring-order fixtures, ragged all-reduce",
         lambda: [P.test_ring_order_allreduce_ragged(r, c) for r in rows for c in (7, 10)]),
        ("int32 closed form", lambda: [P.test_int32_closed_form(R) for R in (3, 8)]),
        ("int32 wraps", lambda: P.test_int32_wraps_mod_2_32(3)),
        ("fp32 subnormal sums", P.test_fp32_subnormal_sums_are_exact),
        ("bf16 subnormal sums", P.test_bf16_subnormal_sums_are_exact),
        ("signed zeros", lambda: [P.test_signed_zero(d) for d in ("fp32", "bf16")]),
        ("Higham bound, fp32", lambda: P.test_fp32_within_recursive_summation_bound(5)),
        ("error bound, bf16", lambda: P.test_bf16_within_bound(4)),
        ("small integer sums", P.test_small_integer_sums_exact),
        ("two ranks = numpy float32 add", P.test_two_ranks_equal_numpy_float32_add),
        ("RS = slice of AR",
         lambda: [P.test_rs_is_slice_of_ar_and_ar_outputs_identical(d, R)
                  for d in ("int32", "fp32", "bf16") for R in (3, 8)]),
        ("AG = concatenation", lambda: P.test_allgather_is_concatenation(3)),
        ("A2A involution", lambda: P.test_alltoall_involution(5)),
        ("copy collectives = flow lists", lambda: P.test_copy_collectives_match_flow_lists(3)),
        ("A2A(v) transposed restores", P.test_alltoallv_transposed_restores),
        ("send/recv pipeline", P.test_sendrecv_pipeline_and_canaries),
        ("bf16 rounding model", P.test_bf16_rounding_matches_python_model),
        ("ring simulation",
         lambda: [P.test_ring_simulation_matches_oracle(d, R) for d in ("int32", "fp32", "bf16") for R in (3, 4)]),
        ("bf16 partials: ring simulation", lambda: [P.test_bf16_hops_ring_simulation_matches_oracle(R) for R in (3, 4)]),
        ("bf16 partials: worked example", P.test_bf16_hops_worked_example),
        ("bf16 partials: four-rank example", P.test_bf16_hops_worked_example_four_ranks),
        ("bf16 partials: special cases", P.test_bf16_hops_special_cases),
        ("bf16 partials: error bound", lambda: P.test_bf16_hops_within_bound(3)),
    ]


def failing_pins(src_text, tmp_path, tag):
    """Builds `src_text` as the oracle, runs the whole battery against it and
    returns the names of the pins that failed."""
    src = tmp_path / f"{tag}.c"
    so = tmp_path / f"lib{tag}.so"
    src.write_text(src_text)
    subprocess.run(["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC", "-shared",
                    "-std=c11", "-o", str(so), str(src)], check=True)
    saved = (oracle._lib, oracle._LIB, oracle._SRC)
    oracle._lib, oracle._LIB, oracle._SRC = None, str(so), str(src)
    failed = []
    try:
        for name, pin in battery():
            try:
                pin()
            except Exception:           # an assertion, or a rejected argument
                failed.append(name)
    finally:
        oracle._lib, oracle._LIB, oracle._SRC = saved
    return failed


def test_unmutated_copy_passes_the_battery(tmp_path):
    assert failing_pins(open(SRC).read(), tmp_path, "pristine") == []


@pytest.mark.parametrize("name,old,new,count", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_fails_a_pin(name, old, new, count, tmp_path):
    text = open(SRC).read()
    assert text.count(old) == count, f"the mutation site of '{name}' no longer matches the oracle"
    failed = failing_pins(text.replace(old, new), tmp_path, "mutant")
    assert failed, f"no pin catches the planted mistake: {name}"
