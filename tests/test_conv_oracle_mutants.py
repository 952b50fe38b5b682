"""Planted-mistake check of the convolution oracle's pins (CPU only).

Each mutant is a plausible slip in conv_oracle.c (a padding sign, a stride
on the wrong axis, a dropped divisibility test, a flipped filter, a
truncated sum).  It is planted textually into a copy of the source, built,
and the pins of test_conv_oracle_pins.py run against it: at least one pin
must fail for every mutant, and none for the unmodified source.  Every
mutant keeps its memory accesses inside the arrays.
"""
import pytest

import oracle.conv as conv_mod
import test_conv_oracle_pins as pins

MUTANTS = {
    "fwd_pad_sign": ("const int hi = p * sh - ph + r;", "const int hi = p * sh + ph + r;"),
    "fwd_stride_axes": ("const int wi = q * sw - pw + s;", "const int wi = q * sh - pw + s;"),
    "fwd_channel_sum_short": ("for (int c = 0; c < C; ++c) acc += x[c] * f[c];",
                              "for (int c = 0; c < C - 1; ++c) acc += x[c] * f[c];"),
    "data_pad_sign": ("const int hp = h + ph - r;", "const int hp = h - ph - r;"),
    "data_divisibility_dropped": ("if (hp < 0 || hp % sh != 0) continue;",
                                  "if (hp < 0) continue;"),
    "data_last_column_dropped": ("if (q >= Q) continue;", "if (q >= Q - 1) continue;"),
    "data_filter_flipped": ("acc += g[k] * Wt[(((size_t)k * R + r) * S + s) * C + c];",
                            "acc += g[k] * Wt[(((size_t)k * R + (R - 1 - r)) * S + (S - 1 - s))"
                            " * C + c];"),
    "filter_pad_sign": ("const int w = q * sw - pw + s;", "const int w = q * sw + pw + s;"),
    "filter_batch_dropped": ("    for (int n = 0; n < N; ++n)\n        for (int p = 0; p < P; ++p) {",
                             "    for (int n = 0; n < 1; ++n)\n        for (int p = 0; p < P; ++p) {"),
    "filter_channel_reversed": ("X[(((size_t)n * H + h) * W + w) * C + c];",
                                "X[(((size_t)n * H + h) * W + w) * C + (C - 1 - c)];"),
}

PINS = [
    lambda: pins.test_fwd_matches_scipy_correlation(pins.SHAPES[1]),
    lambda: pins.test_fwd_matches_scipy_correlation(pins.SHAPES[2]),
    lambda: pins.test_all_three_match_torch_autograd_f64(pins.SHAPES[1]),
    lambda: pins.test_all_three_match_torch_autograd_f64(pins.SHAPES[5]),
    lambda: pins.test_adjoint_identity(pins.SHAPES[1]),
    lambda: pins.test_central_differences_of_bilinear_loss(pins.SHAPES[0]),
    pins.test_pointwise_convolution_is_a_matrix_product,
    pins.test_strided_pointwise_data_gradient_skips_pixels,
    pins.test_delta_filter_is_a_shift,
    pins.test_single_output_position_gives_an_outer_product,
]


def _run_pins(lib_path):
    saved = conv_mod._lib
    conv_mod._lib = conv_mod.load_conv_oracle(lib_path)
    failures = 0
    try:
        for pin in PINS:
            try:
                pin()
            except AssertionError:
                failures += 1
    finally:
        conv_mod._lib = saved
    return failures


@pytest.fixture(scope="module")
def source():
    with open(conv_mod.CONV_ORACLE_SRC) as f:
        return f.read()


def _build(tmp_path, name, text):
    src = tmp_path / (name + ".c")
    src.write_text(text)
    return conv_mod.build_conv_oracle(str(src), str(tmp_path / ("lib" + name + ".so")))


def test_unmodified_source_passes_all_pins(tmp_path, source):
    assert _run_pins(_build(tmp_path, "control", source)) == 0


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, source, name):
    old, new = MUTANTS[name]
    assert source.count(old) == 1, "mutation site missing or not unique: " + name
    assert _run_pins(_build(tmp_path, name, source.replace(old, new))) >= 1
