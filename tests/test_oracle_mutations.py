"""Plant plausible mistakes in a copy of the oracle's C source (on the CPU)
and check that the pins catch every one of them."""

import ctypes
import os
import subprocess

import pytest

import oracle
import test_oracle_pins as pins

SRC = oracle._SRC

# (name, original text, mutated text)
MUTANTS = [
    ("rotation sign", "y[2 * i] = x0 * c - x1 * s;", "y[2 * i] = x0 * c + x1 * s;"),
    ("transposed M", "ld(m, ((int64_t)h * d_v + i) * d_c + k, dt_m)",
     "ld(m, ((int64_t)h * d_c + k) * d_v + i, dt_m)"),
    ("dropped positional term", "s[t] = scale * (content + positional);", "s[t] = scale * content;"),
    ("scale without d_r", "scale = 1.0 / sqrt((double)(d_c + d_r));", "scale = 1.0 / sqrt((double)d_c);"),
    ("group map", "const int b = bh / H, h = bh % H, g = h / hpg;\n    int L = lens[b];\n    if (L < 0) L = 0;\n    if (L > T_max) L = T_max;\n    int t0",
     "const int b = bh / H, h = bh % H, g = h % G;\n    int L = lens[b];\n    if (L < 0) L = 0;\n    if (L > T_max) L = T_max;\n    int t0"),
    ("query position", "const int64_t p = L > 0 ? L - 1 : 0;", "const int64_t p = L;"),
    ("combine weight", "double w = exp(x - big);", "double w = exp(x - mx);"),
    ("double rounding", "double n = nearbyint(scaled);", "double n = nearbyint((double)(float)scaled);"),
    ("rope-decode key position", "gva_oracle_rope(k, d_c, (int64_t)t + shift, rope_base, krot);",
     "gva_oracle_rope(k, d_c, (int64_t)(L - 1 - t) + shift, rope_base, krot);"),
    ("rope-decode scale", "if (scale <= 0.0) scale = 1.0 / sqrt((double)d_c);",
     "if (scale <= 0.0) scale = 1.0 / sqrt((double)d_v);"),
    ("rope-decode transposed M", "ld(m, ((int64_t)h * d_v + i) * d_c + c, dt_m)",
     "ld(m, ((int64_t)h * d_c + c) * d_v + i, dt_m)"),
    ("prefill query position", "b * N + i, h, p, rope_base, qa, qr);",
     "b * N + i, h, p + 1, rope_base, qa, qr);"),
    ("prefill query row", "b * N + i, h, p, rope_base, qa, qr);",
     "b * N + (N - 1 - i), h, p, rope_base, qa, qr);"),
    ("last row dropped", "for (int t = 0; t < n; ++t) {\n      double w", "for (int t = 0; t < n - 1; ++t) {\n      double w"),
]

PIN_TESTS = [
    lambda o: pins.test_absorbed_matches_explicit_reconstruction(o, 8, 4, 2),
    lambda o: pins.test_absorbed_matches_explicit_reconstruction(o, 4, 6, 3),
    lambda o: pins.test_absorbed_query_is_q_times_m_transpose(o),
    lambda o: pins.test_weights_sum_to_one_and_match_softmax(o),
    lambda o: pins.test_two_rows_closed_form(o),
    lambda o: pins.test_rope_matches_complex_form_and_invariants(o),
    lambda o: pins.test_position_shift_leaves_output_unchanged(o),
    lambda o: pins.test_split_and_combine_equals_unsplit(o, 3, 0),
    lambda o: pins.test_split_and_combine_equals_unsplit(o, 5, 32),
    lambda o: pins.test_round_bf16_single_rounding(o),
    lambda o: pins.test_zero_query_gives_mean_value(o),
    lambda o: pins.test_rope_decode_matches_explicit_construction(o, 4, 2),
    lambda o: pins.test_rope_decode_scores_are_a_relative_rotation(o),
    lambda o: pins.test_rope_decode_shift_and_edge_cases(o),
    lambda o: pins.test_prefill_matches_masked_explicit_attention(o, 4, 2, 8),
    lambda o: pins.test_prefill_rows_are_decode_steps(o),
]


@pytest.mark.parametrize("name,orig,mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_every_planted_mistake_fails_a_pin(tmp_path, monkeypatch, name, orig, mut):
    text = open(SRC).read()
    assert orig in text, f"mutation site for {name!r} not found"
    src = tmp_path / "mutant.c"
    src.write_text(text.replace(orig, mut, 1))
    so = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", str(so),
                    str(src), "-lm"], check=True)
    saved = oracle._lib
    monkeypatch.setattr(oracle, "LIB_PATH", str(so))
    oracle._lib = None
    try:
        oracle._load()
        caught = []
        for pin in PIN_TESTS:
            try:
                pin(oracle)
            except AssertionError:
                caught.append(pin)
        assert caught, f"no pin catches the mutant {name!r}"
    finally:
        oracle._lib = saved
