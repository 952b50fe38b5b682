"""Planted-mistake check of the oracle pins (CPU only).

Each mutant below is a plausible slip in the oracle (a dropped term, a wrong
sign, index or operand, an off-by-one mask).  It is planted textually into a
copy of the oracle source, compiled into a temporary library, and the pins of
test_oracle_pins.py are run against that library: at least one pin must fail
for every mutant, and all of them must pass for the unmodified source.
"""
import os

import pytest

import oracle.oracle as oracle_mod
import test_oracle_pins as pins

MUTANTS = {
    "causal_off_by_one": ("return (!causal || j <= i + off) && j < klen;",
                          "return (!causal || j < i + off) && j < klen;"),
    "padding_off_by_one": ("return (!causal || j <= i + off) && j < klen;",
                           "return (!causal || j <= i + off) && j <= klen;"),
    "causal_top_left_for_cross": ("return (!causal || j <= i + off) && j < klen;",
                                  "return (!causal || j <= i) && j < klen;"),
    "cross_offset_sign": ("const int off = Lk - Lq;\n    for (int i = 0; i < Lq; ++i) {",
                          "const int off = Lq - Lk;\n    for (int i = 0; i < Lq; ++i) {"),
    "fwd_scores_unscaled": ("S[j] = scale * dot(q, K + (size_t)j * d, d);",
                            "S[j] = dot(q, K + (size_t)j * d, d);"),
    "lse_base_two": ("LSE[i] = m + log(sum);", "LSE[i] = m + log2(sum);"),
    "max_shift_sign": ("sum += exp(S[j] - m);", "sum += exp(S[j] + m);"),
    "unnormalised_probs": ("double p = exp(S[j] - LSE[i]);", "double p = exp(S[j] - m);"),
    "dS_sign_of_D": ("double dSij = Pij * (dPij - Di);", "double dSij = Pij * (dPij + Di);"),
    "dS_drops_D": ("double dSij = Pij * (dPij - Di);", "double dSij = Pij * dPij;"),
    "dQ_unscaled": ("gq[k] += scale * dSij * kj[k];", "gq[k] += dSij * kj[k];"),
    "dK_wrong_operand": ("gk[k] += scale * dSij * q[k];", "gk[k] += scale * dSij * kj[k];"),
    "dV_uses_dS": ("gv[k] += Pij * go[k];", "gv[k] += dSij * go[k];"),
    "dV_wrong_operand": ("gv[k] += Pij * go[k];", "gv[k] += Pij * q[k];"),
    "D_from_V": ("double Di = dot(go, O + (size_t)i * d, d);",
                 "double Di = dot(go, V + (size_t)i * d, d);"),
    "dP_wrong_operand": ("double dPij = dot(go, vj, d);", "double dPij = dot(go, kj, d);"),
    "bwd_probs_unscaled": ("double Pij = exp(scale * dot(q, kj, d) - LSE[i]);",
                           "double Pij = exp(dot(q, kj, d) - LSE[i]);"),
    "key_len_batch_index": ("key_limit(key_len, bh / H, Lk)", "key_limit(key_len, bh % H, Lk)"),
    "key_len_clamped_to_Lq": ("key_limit(key_len, bh / H, Lk)", "key_limit(key_len, bh / H, Lq)"),
    "bwd_from_first_head_lse": ("O + qo, LSE + (size_t)bh * Lq, dO + qo,", "O + qo, LSE, dO + qo,"),
    "bwd_from_O_dO_swapped": ("O + qo, LSE + (size_t)bh * Lq, dO + qo,",
                              "dO + qo, LSE + (size_t)bh * Lq, O + qo,"),
}

PINS = [
    pins.test_fwd_single_key_returns_value,
    pins.test_fwd_zero_scale_gives_prefix_means,
    pins.test_fwd_two_keys_is_logistic,
    pins.test_fwd_large_scale_is_hard_argmax,
    pins.test_fwd_causal_first_row_is_first_value,
    lambda: pins.test_fwd_matches_scipy_softmax(True, True),
    lambda: pins.test_fwd_matches_scipy_softmax(False, True),
    pins.test_fwd_row_shift_invariance,
    pins.test_fwd_fully_masked_rows,
    lambda: pins.test_bwd_central_finite_differences(5, 2, True, False),
    lambda: pins.test_bwd_central_finite_differences(5, 2, False, True),
    lambda: pins.test_fwd_bwd_match_torch_autograd_f64(True, False, 16, 4),
    lambda: pins.test_fwd_bwd_match_torch_autograd_f64(False, True, 12, 4),
    pins.test_bwd_invariants,
    pins.test_bwd_single_key_special_case,
    pins.test_cross_causal_is_the_bottom_rows_of_square_causal,
    pins.test_cross_single_key,
    lambda: pins.test_cross_matches_torch_autograd_f64(12, 30, False, True),
    lambda: pins.test_cross_central_finite_differences(3, 5, True, False),
    lambda: pins.test_bwd_from_exact_forward_is_the_backward(False, True, 5, 7),
    pins.test_bwd_from_single_key_closed_forms,
    pins.test_bwd_from_linear_in_upstream_gradient,
]


def _build_variant(tmp_path, name, src_text):
    src = tmp_path / (name + ".c")
    src.write_text(src_text)
    return oracle_mod.build_oracle(str(src), str(tmp_path / ("lib" + name + ".so")))


def _run_pins(lib_path):
    """Run every pin against the library at lib_path; returns failure count."""
    saved = oracle_mod._lib
    oracle_mod._lib = oracle_mod.load_oracle(lib_path)
    failures = 0
    try:
        for pin in PINS:
            try:
                pin()
            except AssertionError:
                failures += 1
    finally:
        oracle_mod._lib = saved
    return failures


@pytest.fixture(scope="module")
def source():
    with open(oracle_mod.ORACLE_SRC) as f:
        return f.read()


def test_unmodified_source_passes_all_pins(tmp_path, source):
    assert _run_pins(_build_variant(tmp_path, "control", source)) == 0


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, source, name):
    old, new = MUTANTS[name]
    assert old in source, "mutation site vanished from the oracle: " + name
    mutated = source.replace(old, new)
    assert _run_pins(_build_variant(tmp_path, name, mutated)) >= 1
