"""Every plausible slip in the oracle must trip at least one pin.

Each mutant is the oracle source with one deliberate mistake (a dropped term,
a wrong sign or index, a transposed operand...), compiled on the CPU; the pin
suite must reject every one of them.
"""
import os

import pytest

import oracle
from tests import oracle_pins

MUTANTS = {
    "skip_first_term": ("for (int64_t k = lo; k < hi; ++k) {", "for (int64_t k = lo + 1; k < hi; ++k) {"),
    "extra_term": ("for (int64_t k = lo; k < hi; ++k) {", "for (int64_t k = lo; k <= hi && k < J->offsets[(int64_t)J->T * J->B]; ++k) {"),
    "ignore_weights": ("const double w = J->weights ? (double)J->weights[k] : 1.0;", "const double w = 1.0;"),
    "dest_transposed": ("const int64_t r = b / S;", "const int64_t r = b % J->R;"),
    "row_transposed": ("const int64_t s = b % S;", "const int64_t s = b / J->R;"),
    "col_off_zero": ("const int64_t out = (r * S + s) * J->sum_dim + J->col_off[t];", "const int64_t out = (r * S + s) * J->sum_dim;"),
    "row_stride_wrong": ("(int64_t)J->indices[k] * D + j", "(int64_t)J->indices[k] + j"),
    "sample_major_offsets": ("const int64_t lo = J->offsets[(int64_t)t * J->B + b];", "const int64_t lo = J->offsets[b * J->T + t];"),
    "abs_not_abs": ("mag += fabs(term);", "mag += term;"),
    "half_bias": ("v = ldexp((double)(f + 1024), e - 25);", "v = ldexp((double)(f + 1024), e - 24);"),
    "half_subnormal": ("v = ldexp((double)f, -24);", "v = ldexp((double)(f + 1024), -24);"),
    "half_sign": ("return sign ? -v : v;", "return v;"),
    "bf16_shift": ("uint32_t bits = (uint32_t)h << 16;", "uint32_t bits = (uint32_t)h << 15;"),
    "no_range_check": ("if (indices[k] < 0 || (int64_t)indices[k] >= rows[t]) return OR_BAD_INDEX;", ""),
    "flags_off_by_one": ("flags[(r * nC + c) * per_slice + t] = epoch;",
                         "flags[(r * nC + c) * per_slice + t] = epoch + (c == 0);"),
    "flags_per_table_index": ("flags[(r * nC + c) * per_slice + t] = epoch;",
                              "flags[(r * nC + c) * per_slice + t * 0] = epoch;"),
    "mean_not_divided": ("          sum /= (double)(hi - lo);\n", ""),
    "mean_divides_by_l_plus_one": ("          sum /= (double)(hi - lo);", "          sum /= (double)(hi - lo + 1);"),
    "gemv_drop_rank": ("for (int32_t r = 0; r < J->R; ++r) {", "for (int32_t r = 0; r + 1 < J->R; ++r) {"),
    "gemv_transposed": ("load_elem(J->A[r], J->dtype, i * K + k)", "load_elem(J->A[r], J->dtype, k * J->M + i)"),
    "gemv_x_reversed": ("load_elem(J->x[r], J->dtype, k)", "load_elem(J->x[r], J->dtype, K - 1 - k)"),
    "gemv_abs_not_abs": ("mag = mag + fabs(term);", "mag = mag + term;"),
    "gemv_no_rounding_to_f32": ("if (J->y) J->y[i] = (float)sum;", "if (J->y) J->y[i] = (float)(sum + 1e-3);"),
    "backward_no_weight": ("            v = (double)weights[k] * v;", "            v = v;"),
    "backward_mean_off_by_one": ("            v = v / (double)(hi - lo);", "            v = v / (double)(hi - lo + 1);"),
    "backward_block_start": ("    block += (offsets[(int64_t)(t + 1) * B] - first) * D;", "    block += (offsets[(int64_t)(t + 1) * B] - first) * D - D;"),
    "backward_column": ("      const float* g = grad + b * sum_dim + col;", "      const float* g = grad + b * sum_dim;"),
    "round_down": ("if (J->send) J->send[out + j] = (float)sum;", "if (J->send) J->send[out + j] = (float)floor(sum);"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    mpath = os.path.join(tmp_path, "oracle_mut.c")
    with open(mpath, "w") as f:
        f.write(src.replace(old, new))
    lib = oracle.load(oracle.build(src=mpath, out=os.path.join(tmp_path, "libmut.so")))
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(lib)
        except (AssertionError, oracle.OracleError, ValueError):
            caught.append(pin.__name__)
    assert caught, f"mutant {name} passed every pin"
