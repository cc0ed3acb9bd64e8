"""Planted mistakes in the oracle must be caught by its pins (CPU only).

Each case rewrites one plausible mistake into a copy of oracle/oracle.c (a
flipped kernel, a dropped bias, a wrong group offset, floor instead of ceil
pooling, last-instead-of-first argmax, ...), compiles the copy, points the
oracle wrappers at it, runs the pin checks of the other oracle test modules
and requires at least one of them to fail.
"""
import os
import subprocess

import pytest

import oracle
import test_oracle_conv_fc as tc
import test_oracle_pool_lrn_net as tp
import test_oracle_softmax as ts

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

# (name, text in oracle.c, replacement)
MUTANTS = [
    ("kernel flipped",
     "w[(((size_t)k * Cg + c) * R + r) * S + s]",
     "w[(((size_t)k * Cg + c) * R + (R - 1 - r)) * S + (S - 1 - s)]"),
    ("conv bias dropped",
     "double acc = bias ? (double)bias[k] : 0.0;", "double acc = 0.0;"),
    ("group offset dropped", "const int ci = g * Cg + c;", "const int ci = c;"),
    ("pad sign", "const int h = p * sh - ph + r;", "const int h = p * sh + ph + r;"),
    ("width stride from height", "const int ww = q * sw - pw + s;", "const int ww = q * sh - pw + s;"),
    ("conv relu keeps negatives", "if (relu) out = relu_f(out);\n                    y[(((size_t)n * K",
     "if (relu) out = out;\n                    y[(((size_t)n * K"),
    ("fc weight transposed", "(double)w[(size_t)o * I + i]", "(double)w[(size_t)i * O + o]"),
    ("fc bias dropped", "double acc = bias ? (double)bias[o] : 0.0;", "double acc = 0.0;"),
    ("pool floor instead of ceil", "int out = ceil_mode ? (span + s - 1) / s + 1 : span / s + 1;",
     "int out = span / s + 1;"),
    ("pool last maximum", "if (plane[(size_t)h * W + ww] > best) {", "if (plane[(size_t)h * W + ww] >= best) {"),
    ("avg divisor clipped to image", "const int h1p = hs + kh < H + ph ? hs + kh : H + ph;",
     "const int h1p = hs + kh < H ? hs + kh : H;"),
    ("avg divides by full window", "out = (float)(sum / count);", "out = (float)(sum / (kh * kw));"),
    ("pool index column-major", "best_i = h * W + ww;", "best_i = ww * H + h;"),
    ("lrn alpha not divided by size", "(double)alpha / size * sq", "(double)alpha * sq"),
    ("lrn window one short", "const int c1 = c + half > C - 1 ? C - 1 : c + half;",
     "const int c1 = c + half - 1 > C - 1 ? C - 1 : c + half - 1;"),
    ("lrn beta sign", "pow(scale, -(double)beta)", "pow(scale, (double)beta)"),
    ("relu keeps negative zero", "return v > 0.0f ? v : 0.0f;", "return v >= 0.0f ? v : 0.0f;"),
    ("conv floor rounds up", "*P = (H + 2 * ph - R) / sh + 1;", "*P = (H + 2 * ph - R + sh - 1) / sh + 1;"),
    ("softmax without the max shift", "double m = xc[0];", "double m = 0.0;"),
    ("softmax not normalized", "- m) / sum);", "- m));"),
    ("softmax sum skips a channel", "for (int c = 0; c < C; ++c) sum +=", "for (int c = 1; c < C; ++c) sum +="),
    ("softmax over the wrong axis", "const int64_t cs = HW;", "const int64_t cs = 1;"),
]


def _pins():
    """The pin checks, as (name, callable) pairs."""
    return [
        ("conv golden 1", tc.test_conv_golden_stride1_bias),
        ("conv golden 2", tc.test_conv_golden_stride2_pad1),
        ("conv delta", lambda: tc.test_conv_delta_kernel_is_shifted_sample(2, 1, 1, 2)),
        ("conv torch", lambda: tc.test_conv_matches_torch_float64(1, 4, 9, 9, 6, 3, 3, 1, 1, 2)),
        ("conv torch stem", lambda: tc.test_conv_matches_torch_float64(1, 3, 23, 23, 8, 11, 11, 4, 0, 1)),
        ("conv anisotropic", tc.test_conv_anisotropic_stride_pad_matches_torch),
        ("conv grouped", tc.test_conv_grouped_is_concatenation),
        ("conv relu", tc.test_conv_relu_flag_is_relu_after),
        ("conv shapes", lambda: tc.test_conv_out_shape_floor(224, 7, 2, 3, 112)),
        ("fc", tc.test_fc_identity_and_matmul_witness),
        ("fc=conv", tc.test_fc_equals_conv_over_whole_image),
        ("pool chain", tp.test_pool_ceil_chain_forced_by_cifar_fc),
        ("pool golden", tp.test_pool_golden_ramp),
        ("pool ties", tp.test_pool_ties_take_first_index),
        ("pool torch", lambda: tp.test_pool_matches_torch(10, 7, 3, 2, 1)),
        ("lrn golden", tp.test_lrn_golden_single_channel),
        ("lrn torch", lambda: tp.test_lrn_matches_torch(7, 5, 1e-4, 0.75, 1.0)),
        ("lrn torch 2", lambda: tp.test_lrn_matches_torch(16, 5, 0.5, 0.75, 2.0)),
        ("relu", tp.test_relu_definition),
        ("softmax logistic", lambda: ts.test_softmax_two_classes_is_logistic(1.0, -2.0)),
        ("softmax overflow", ts.test_softmax_large_inputs_do_not_overflow),
        ("softmax sums", ts.test_softmax_rows_sum_to_one_and_keep_order),
        ("softmax axis", lambda: ts.test_softmax_channel_axis_matches_torch((2, 3, 2, 2))),
    ]


@pytest.fixture(scope="module")
def source():
    with open(SRC) as f:
        return f.read()


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(name, old, new, source, tmp_path):
    assert source.count(old) == 1, f"mutation site for '{name}' not found exactly once"
    mutated = tmp_path / "oracle.c"
    mutated.write_text(source.replace(old, new))
    (tmp_path / "oracle.h").write_text(open(os.path.join(os.path.dirname(SRC), "oracle.h")).read())
    lib = tmp_path / "liboracle_mutant.so"
    subprocess.run(["gcc", "-O1", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-w", "-o", str(lib),
                    str(mutated), "-lm"], check=True)
    saved = oracle.LIB_PATH
    caught = []
    try:
        oracle.use_library(str(lib))
        for pin_name, pin in _pins():
            try:
                pin()
            except (AssertionError, ValueError):
                caught.append(pin_name)
    finally:
        oracle.use_library(saved)
    assert caught, f"no pin caught the planted mistake '{name}'"
