"""The oracle's pins must reject plausible mistakes in the oracle.

Each case copies the oracle's C source, plants one mistake by a textual edit, compiles the
copy with the same flags into a temporary directory (CPU only), and runs a subset of the pins
against it in a child process that points the oracle module at the copy. A mutant that every pin accepts would mean the pins do
not constrain that part of the oracle, so the test fails.
"""
import json
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

import oracle
import test_oracle_dynamic_pins as dyn_pins
import test_oracle_order_pins as order_pins
import test_oracle_pins as pins

_SRC = os.path.join(os.path.dirname(oracle.__file__), "hccl_oracle.c")

MUTANTS = {
    "fold_descending": (
        "float acc = load_as_f32(src[0], dtype, i);\n"
        "        for (int r = 1; r < P; ++r) acc = combine_f32(op, acc, load_as_f32(src[r], dtype, i));",
        "float acc = load_as_f32(src[P - 1], dtype, i);\n"
        "        for (int r = P - 2; r >= 0; --r) acc = combine_f32(op, acc, load_as_f32(src[r], dtype, i));",
    ),
    "seed_with_positive_zero": (
        "float acc = load_as_f32(src[0], dtype, i);\n        for (int r = 1; r < P; ++r)",
        "float acc = 0.0f;\n        for (int r = 0; r < P; ++r)",
    ),
    "drop_last_contributor": (
        "for (int r = 1; r < P; ++r) acc = combine_f32(op, acc, load_as_f32(src[r], dtype, i));",
        "for (int r = 1; r < P - 1; ++r) acc = combine_f32(op, acc, load_as_f32(src[r], dtype, i));",
    ),
    "bf16_ties_round_down": (
        "if (r > 0x8000u || (r == 0x8000u && (t & 1u))) t += 1u;",
        "if (r > 0x8000u) t += 1u;",
    ),
    "fp16_subnormal_shift_off_by_one": (
        "int shift = 14 - he;",
        "int shift = 13 - he;",
    ),
    "reduce_scatter_wrong_block": (
        "\n            block[r] = (const char*)send[r] + (size_t)c * recvcount * es;",
        "\n            block[r] = (const char*)send[r] + (size_t)r * recvcount * es;",
    ),
    "ordered_reduce_scatter_wrong_block": (
        "++r) block[r] = (const char*)send[r] + (size_t)c * recvcount * es;",
        "++r) block[r] = (const char*)send[r] + (size_t)r * recvcount * es;",
    ),
    "allgather_wrong_block": (
        "memcpy((char*)recv[r] + (size_t)q * bytes, send[q], bytes);",
        "memcpy((char*)recv[r] + (size_t)r * bytes, send[q], bytes);",
    ),
    "alltoallv_transposed_rdispls": (
        "char* to = (char*)recv[d] + rdispls[(size_t)d * P + s] * elem_size;",
        "char* to = (char*)recv[d] + rdispls[(size_t)s * P + d] * elem_size;",
    ),
    "two_level_partials_requantised": (
        "total = (g == 0) ? part : combine_f32(op, total, part);",
        "part = orc_bf16_to_f32(orc_f32_to_bf16(part));\n"
        "        total = (g == 0) ? part : combine_f32(op, total, part);",
    ),
    "int32_sum_saturates": (
        "if (op == ORC_SUM) return (int32_t)((uint32_t)acc + (uint32_t)x);",
        "if (op == ORC_SUM) { long long s = (long long)acc + x; "
        "return s > 2147483647LL ? 2147483647 : (s < -2147483648LL ? (int32_t)-2147483648LL : (int32_t)s); }",
    ),
    "halving_distances_doubling": (
        "for (int d = P / 2; d >= 1; d /= 2)\n            for (int r = 0; r < d; ++r) v[r] = comb_q(op, dtype, q, v[r], v[r + d]);",
        "for (int d = 1; d < P; d *= 2)\n            for (int r = 0; r + d < P; r += 2 * d) v[r] = comb_q(op, dtype, q, v[r], v[r + d]);",
    ),
    "ring_starts_at_the_owner": (
        "int first = (c + 1) % P;\n        float acc",
        "int first = c % P;\n        float acc",
    ),
    "two_level_cross_group_fold_not_requantised": (
        "total = (g == 0) ? part : comb_q(op, dtype, q, total, part);",
        "total = (g == 0) ? part : combine_f32(op, total, part);",
    ),
    "two_level_in_group_fold_not_requantised": (
        "part = comb_q(op, dtype, q, part, load_as_f32(src[r], dtype, i));",
        "part = combine_f32(op, part, load_as_f32(src[r], dtype, i));",
    ),
    "requant_ignored": (
        "return requant ? requantize(dtype, v) : v;",
        "return v;",
    ),
    "dynamic_packed_receive_offset_inclusive": (
        "rd[(size_t)d * P + s] = rdispls ? rdispls[(size_t)d * P + s] : at;",
        "rd[(size_t)d * P + s] = rdispls ? rdispls[(size_t)d * P + s] : at + n;",
    ),
    "dynamic_rows_read_as_elements": (
        "so[(size_t)s * P + d] = (size_t)sd[(size_t)s * P + d] * row_elems;",
        "so[(size_t)s * P + d] = (size_t)sd[(size_t)s * P + d];",
    ),
    "dynamic_exact_fit_rejected": (
        "return (uint64_t)n <= cap - (uint64_t)off;",
        "return (uint64_t)n < cap - (uint64_t)off;",
    ),
    "dynamic_overlap_unchecked": (
        "if (a0 < b0 + nb && b0 < a0 + na) return -2;",
        "if (a0 < b0 + nb && b0 < a0 + na && 0) return -2;",
    ),
    "dynamic_recvcounts_not_transposed": (
        "recvcounts_out[(size_t)d * P + s] = counts[(size_t)s * P + d];",
        "recvcounts_out[(size_t)s * P + d] = counts[(size_t)s * P + d];",
    ),
    "dynamic_zero_count_ranges_checked": (
        "if (n > 0 && !range_fits(sd[(size_t)s * P + d], n, send_cap)) return -2;",
        "if (!range_fits(sd[(size_t)s * P + d], n, send_cap)) return -2;",
    ),
}

# The pins run against every mutant (cheap ones, CPU only).
PIN_CALLS = [
    ("bf16 ties", lambda: pins.test_bf16_narrowing_matches_torch_on_every_tie_class()),
    ("bf16 hand", lambda: pins.test_bf16_hand_values()),
    ("fp16 ties", lambda: pins.test_fp16_narrowing_matches_numpy_on_every_tie_class()),
    ("fp16 subnormal", lambda: pins.test_fp16_narrowing_subnormal_ties()),
    ("fp32 fold", lambda: pins.test_allreduce_fp32_is_the_ascending_numpy_fold(5)),
    ("order", lambda: pins.test_fold_order_is_ascending_rank_not_any_other()),
    ("seed", lambda: pins.test_accumulator_is_seeded_with_the_first_contributor()),
    ("two level", lambda: pins.test_two_level_is_group_folds_then_partial_fold(4, 2)),
    ("triangular", lambda: pins.test_allreduce_of_rank_plus_one_is_triangular_number("fp32", 7)),
    ("int32 wrap", lambda: pins.test_int32_sum_wraps_like_uint32_arithmetic()),
    ("rs brute", lambda: pins.test_reduce_scatter_brute_force(4, 7)),
    ("ag brute", lambda: pins.test_allgather_brute_force(3, 1)),
    ("a2av brute", lambda: pins.test_alltoallv_brute_force_with_gaps_and_zero_blocks()),
    ("ring order", lambda: order_pins.test_ring_order_reduce_scatter_is_the_rotated_numpy_fold(5)),
    ("halving order", lambda: order_pins.test_halving_order_is_the_distance_halving_tree(8)),
    ("order cancellation", lambda: order_pins.test_orders_are_told_apart_by_cancellation()),
    ("requant", lambda: order_pins.test_requant_rounds_every_partial_to_bf16("ascending")),
    ("requant two-level", lambda: order_pins.test_two_level_requant_rounds_inside_and_across_groups(2)),
    ("dynamic example", lambda: dyn_pins.test_worked_example_packed_layout()),
    ("dynamic explicit", lambda: dyn_pins.test_worked_example_explicit_offsets()),
    ("dynamic brute", lambda: dyn_pins.test_packed_layout_is_the_brute_force_row_placement(3, 4, 2)),
    ("dynamic capacity", lambda: dyn_pins.test_capacity_boundaries_packed()),
    ("dynamic overlap", lambda: dyn_pins.test_receive_overlap_boundaries()),
    ("dynamic zero ranges", lambda: dyn_pins.test_zero_count_ranges_are_never_checked()),
]


def _build_mutant(tmpdir, name):
    before, after = MUTANTS[name]
    src = open(_SRC).read()
    assert src.count(before) == 1, f"mutation site for {name} not found exactly once"
    mutated = src.replace(before, after)
    c_path = os.path.join(tmpdir, f"{name}.c")
    so_path = os.path.join(tmpdir, f"{name}.so")
    with open(c_path, "w") as f:
        f.write(mutated)
    inc = os.path.dirname(_SRC)
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                    "-fno-fast-math", "-I", inc, "-o", so_path, c_path], check=True)
    return so_path


def run_pins_against(so_path):
    """Entry point of the child process: every pin against one mutant library; prints the
    labels of the pins that failed as one JSON list."""
    caught = []
    with oracle.use_library(so_path):
        for label, call in PIN_CALLS:
            try:
                call()
            except (AssertionError, ValueError):
                caught.append(label)
    print(json.dumps(caught))


_CHILD = (
    "import sys; sys.path[:0] = [{tests!r}, {root!r}]\n"
    "import test_oracle_mutants as m\n"
    "m.run_pins_against(sys.argv[1])\n"
)


@pytest.fixture(scope="module")
def mutant_results(tmp_path_factory):
    """Builds every mutant and runs the pins against each in a process of its own (a mutant
    may write outside a buffer; that must not corrupt the test process), a few at a time."""
    tmp = str(tmp_path_factory.mktemp("mutants"))
    tests = os.path.dirname(os.path.abspath(__file__))
    child = _CHILD.format(tests=tests, root=os.path.dirname(tests))
    names = sorted(MUTANTS)
    with ThreadPoolExecutor(max_workers=6) as pool:
        libs = dict(zip(names, pool.map(lambda n: _build_mutant(tmp, n), names)))

    def run(name):
        try:
            r = subprocess.run([sys.executable, "-c", child, libs[name]], capture_output=True, text=True,
                               timeout=300)
        except subprocess.TimeoutExpired:
            return ["timed out"]
        if r.returncode != 0:
            return ["crashed"]  # the pins drove the mutant into memory it does not own
        return json.loads(r.stdout.strip().splitlines()[-1])

    with ThreadPoolExecutor(max_workers=6) as pool:
        return dict(zip(names, pool.map(run, names)))


def test_unmutated_source_passes_every_pin():
    for _, call in PIN_CALLS:
        call()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_every_planted_mistake_fails_a_pin(name, mutant_results):
    assert mutant_results[name], f"mutant {name} passed every pin"
