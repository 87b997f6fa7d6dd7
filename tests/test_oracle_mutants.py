"""Mutation check of the oracle's pins, on the CPU.

Each case copies laq_oracle.c, plants one plausible mistake (a wrong sign, a
dropped term, an off-by-one, a wrong rounding, a transposed index, a wrong
bit position), builds the copy and runs every pin against it.  A pin set that
lets a mutant through is too weak.  Nothing here touches the real oracle.
"""
import os
import subprocess

import pytest

import oracle
import oracle_pins as P
from oracle import build as obuild

MUTANTS = [
    ("zero_sign", "float zf = rintf(-lo / s);", "float zf = rintf(lo / s);"),
    ("range_sign", "float range = hi - lo;", "float range = hi + lo;"),
    ("levels_off_by_one", "float s32 = range / (float)qmax;", "float s32 = range / (float)(qmax + 1);"),
    ("code_minus_zero", "int q = (int)t + z;", "int q = (int)t - z;"),
    ("floor_not_rint", "float t = rintf(v / s);", "float t = floorf(v / s);"),
    ("no_zero_widening", "float lo = 0.0f, hi = 0.0f;",
     "float lo = laqo_f16_to_f32(wg[0]), hi = laqo_f16_to_f32(wg[0]);"),
    ("scale_not_rounded", "float s = laqo_f16_to_f32(s16);", "float s = s32 > 0 ? s32 : 5.9604645e-08f;"),
    ("fp16_truncates", "float r = rintf(n);", "float r = truncf(n);"),
    ("w3_field_offsets", "{0, 3, 6, 10, 13}", "{0, 3, 6, 9, 12}"),
    ("w3_spare_bits_swapped", "*bit = (i == 30) ? 9 : 25;", "*bit = (i == 30) ? 25 : 9;"),
    ("w4_nibble_order", "*bit = 16 * (i % 2) + 4 * ((i % 8) / 2) + j;", "*bit = 4 * (i % 8) + j;"),
    ("linear_drops_zero",
     "acc += xv * (s * (double)((int)codes[n * K + k] - z));",
     "acc += xv * (s * (double)((int)codes[n * K + k]));"),
    ("linear_x_transposed", "double xv = (double)laqo_f16_to_f32(x[m * K + k]);",
     "double xv = (double)laqo_f16_to_f32(x[(k % M) * K + (k / M) + m * 0]);"),
    ("linear_wrong_group_scale", "double s = (double)laqo_f16_to_f32(scales[n * G + g]);\n                int z",
     "double s = (double)laqo_f16_to_f32(scales[n * G + (G - 1 - g)]);\n                int z"),
    ("params_floor_not_rint", "float u = rintf(v / s) + z;", "float u = floorf(v / s) + z;"),
    ("params_zero_sign", "float u = rintf(v / s) + z;", "float u = rintf(v / s) - z;"),
    ("params_first_group_scale", "float s = laqo_f16_to_f32(scales[n * G + g]);",
     "float s = laqo_f16_to_f32(scales[n * G]);"),
    ("dequant_wrong_zero", "w_hat[n * K + k] = s * (double)((int)codes[n * K + k] - (int)zeros[n * G + g]);",
     "w_hat[n * K + k] = s * (double)((int)codes[n * K + k] - (int)zeros[n * G + 0]);"),
]


def _all_pins():
    return P.ALL_FP16_PINS + P.ALL_QUANT_PINS + P.ALL_PARAMS_PINS + P.ALL_PACK_PINS + P.ALL_LINEAR_PINS


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    src = open(obuild.SRC).read()
    assert src.count(old) == 1, "mutation anchor not found exactly once: " + name
    mpath = tmp_path / "mutant.c"
    mpath.write_text(src.replace(old, new))
    lib = str(tmp_path / "libmutant.so")
    subprocess.run(["gcc", "-O2", "-std=c11", "-fno-fast-math", "-ffp-contract=off",
                    "-fopenmp", "-fPIC", "-shared", "-o", lib, str(mpath), "-lm"], check=True)
    m = oracle.Oracle(lib)
    caught = []
    for pname, fn in _all_pins():
        try:
            fn(m)
        except (AssertionError, ValueError):
            caught.append(pname)
    assert caught, "no pin caught mutant " + name


def test_unmutated_copy_passes(tmp_path):
    """Control: the same build procedure on the unmodified source passes."""
    lib = str(tmp_path / "libcopy.so")
    subprocess.run(["gcc", "-O2", "-std=c11", "-fno-fast-math", "-ffp-contract=off",
                    "-fopenmp", "-fPIC", "-shared", "-o", lib, obuild.SRC, "-lm"], check=True)
    m = oracle.Oracle(lib)
    for pname, fn in _all_pins():
        fn(m)
