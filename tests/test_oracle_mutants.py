"""The oracle's pins are sensitive: each planted mistake is caught.

Each case copies the oracle's C source, makes one plausible mistake in it (a
flipped or transposed kernel index, a swapped stride, a dropped term, a wrong
lowering offset, a wrong slab offset or row, a short slab, a narrower accumulator, a wrong bf16
widening, and in the training passes a flipped kernel row, a swapped stride,
a fold or slab offset without its stride), builds the copy with gcc and runs
the pin battery of test_oracle_pins.py and test_oracle_training.py against it. At least one pin must fail. Every mutant keeps
all memory accesses in bounds, so a mutant can only give wrong values.
"""
import os
import shutil
import subprocess

import pytest

import oracle
import test_oracle_pins as pins
import test_oracle_training as tpins

SRC = os.path.join(os.path.dirname(oracle.__file__), "mec_oracle.c")

DIRECT_KK = "int64_t kk = ((a * k_w + b) * i_c + c) * k_c + m;"

MUTANTS = {
    "kernel_flipped": (DIRECT_KK,
                       "int64_t kk = (((k_h - 1 - a) * k_w + (k_w - 1 - b)) * i_c + c) * k_c + m;"),
    "kernel_transposed": (DIRECT_KK, "int64_t kk = ((a * k_w + b) * k_c + (m % k_c)) * i_c + c % i_c;"),
    "stride_swapped": ("int64_t ii = ((n * i_h + (y * s_h + a)) * i_w + (x * s_w + b)) * i_c + c;",
                       "int64_t ii = ((n * i_h + (y * s_h + a)) * i_w + (x * s_h + b) % i_w) * i_c + c;"),
    "channel_term_dropped": ("for (int64_t c = 0; c < i_c; ++c) {\n                                int64_t ii",
                             "for (int64_t c = 0; c < i_c - (i_c > 1); ++c) {\n                                int64_t ii"),
    "lower_no_column_stride": ("int64_t src = ((n * i_h + h) * i_w + s_w * w) * i_c;    /* I[n, h, s_w*w, 0] */",
                               "int64_t src = ((n * i_h + h) * i_w + w) * i_c;"),
    "lower_rows_transposed": ("int64_t dst = (((n * o_w + w) * i_h + h) * k_w) * i_c;  /* L[n, w, h, 0, 0] */",
                              "int64_t dst = (((n * i_h + h) * o_w + w) * k_w) * i_c;"),
    "slab_offset_without_channels": ("int64_t start = s_h * R * h;", "int64_t start = s_h * k_w * h;"),
    "slab_rows_transposed": ("int64_t row = (n * o_w + w) * LD;", "int64_t row = (w * i_n + n) % (i_n * o_w) * LD;"),
    "slab_one_row_short": ("for (int64_t j = 0; j < k_h * R; ++j)\n                        acc += elem(L, row + start + j",
                           "for (int64_t j = 0; j < (k_h - 1) * R + (k_h == 1) * R; ++j)\n                        acc += elem(L, row + start + j"),
    "float_accumulator": ("double acc = 0.0;\n                    for (int64_t a = 0; a < k_h; ++a)",
                          "float acc = 0.0f;\n                    for (int64_t a = 0; a < k_h; ++a)"),
    "bf16_widen_wrong": ("uint32_t bits = (uint32_t)((const uint16_t*)base)[idx] << 16;",
                         "uint32_t bits = (uint32_t)((const uint16_t*)base)[idx] << 15;"),
    "vanilla_ld_wrong": ("int64_t ld = i_h * k_w;", "int64_t ld = i_h * k_w - 1;"),
    # training passes
    "dgrad_kernel_flipped": ("g * elem(K, ((a * k_w + b) * i_c + c) * k_c + m, dtype);",
                             "g * elem(K, (((k_h - 1 - a) * k_w + b) * i_c + c) * k_c + m, dtype);"),
    "wgrad_rows_flipped": ("acc += elem(I, ((n * i_h + (y * s_h + a)) * i_w + (x * s_w + b)) * i_c + c, dtype) *",
                           "acc += elem(I, ((n * i_h + (y * s_h + (k_h - 1 - a))) * i_w + (x * s_w + b)) * i_c + c, dtype) *"),
    "wgrad_stride_swapped": ("acc += elem(I, ((n * i_h + (y * s_h + a)) * i_w + (x * s_w + b)) * i_c + c, dtype) *",
                             "acc += elem(I, ((n * i_h + (y * s_h + a)) * i_w + (x * s_h + b) % i_w) * i_c + c, dtype) *"),
    "fold_no_column_stride": ("d[(h * i_w + s_w * w + b) * i_c + c] +=",
                              "d[(h * i_w + (w + b) % i_w) * i_c + c] +="),
    "dL_slab_offset_without_stride": ("row[s_h * R * h + j] += acc;", "row[R * h + j] += acc;"),
    "wgrad_lowered_offset_without_stride": ("acc += elem(L, p * LD + s_h * R * h + j, dtype) *",
                                            "acc += elem(L, p * LD + R * h + j, dtype) *"),
}


def battery():
    """The pin checks, as callables taking the oracle module."""
    o = oracle
    checks = [
        lambda: pins.test_example_lowered_matrix_closed_form(o),
        lambda: pins.test_example_outputs_closed_form_and_no_flip(o),
        lambda: pins.test_example_vertical_partitions(o),
        lambda: pins.test_identity_1x1(o),
        lambda: pins.test_bf16_inputs_widen_exactly(o),
        lambda: pins.test_vanilla_is_algorithm2_special_case(o),
        lambda: pins.test_1x1_reduces_to_matmul(o),
    ]
    for shape in pins.TINY_SHAPES:
        checks.append(lambda shape=shape: pins.test_brute_force_integers_exact(o, shape))
    for shape in pins.TORCH_SHAPES[:3]:
        checks.append(lambda shape=shape: pins.test_against_torch_conv2d_f64(o, shape))
        checks.append(lambda shape=shape: pins.test_mec_equals_im2col(o, shape))
    checks.append(lambda: pins.test_delta_kernel_reproduces_shifted_input(o, (2, 3), (3, 3)))
    # training passes
    checks.append(lambda: tpins.test_worked_example_closed_forms(o))
    for d in tpins.SHAPES[:4]:
        checks.append(lambda d=d: tpins.test_adjoint_identities_exact(o, d))
        checks.append(lambda d=d: tpins.test_mec_forms_equal_direct(o, d))
        checks.append(lambda d=d: tpins.test_fold_is_adjoint_of_lowering(o, d))
    checks.append(lambda: tpins.test_delta_gradients(o, (2, 12, 11, 3, 3, 4, 5, 2, 3)))
    return checks


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path, monkeypatch):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, "mutation anchor not found: %s" % name
    mutated = src.replace(old, new, 1)
    cfile = tmp_path / "mutant.c"
    cfile.write_text(mutated)
    so = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O1", "-fopenmp", "-shared", "-fPIC", str(cfile), "-o", str(so)],
                   check=True)
    monkeypatch.setattr(oracle, "_lib", oracle._load(str(so)))
    caught = 0
    for check in battery():
        try:
            check()
        except AssertionError:
            caught += 1
    assert caught > 0, "mutant %s passed every pin" % name


def test_unmutated_source_passes_battery(tmp_path, monkeypatch):
    so = tmp_path / "libclean.so"
    shutil.copy(SRC, tmp_path / "clean.c")
    subprocess.run(["gcc", "-O1", "-fopenmp", "-shared", "-fPIC", str(tmp_path / "clean.c"),
                    "-o", str(so)], check=True)
    monkeypatch.setattr(oracle, "_lib", oracle._load(str(so)))
    for check in battery():
        check()
