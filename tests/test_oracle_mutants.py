"""Plant plausible mistakes in a copy of oracle.c (on the CPU) and require the pins to catch each.

This checks the pins rather than the oracle: a pin suite that let a dropped term, a wrong sign, a
wrong index or a transposed operand through would not be pinning anything.
"""
import os
import shutil

import pytest

import oracle
import pins

MUTANTS = {
    "f16_exponent_bias": ("ldexp((double)(1024 + f), e - 25)", "ldexp((double)(1024 + f), e - 24)"),
    "f16_subnormal_scale": ("ldexp((double)f, -24)", "ldexp((double)f, -25)"),
    "f16_sign_dropped": ("    return sign ? -v : v;\n}\n\n/* bfloat16",
                         "    return v;\n}\n\n/* bfloat16"),
    "bf16_exponent_bias": ("ldexp((double)(128 + f), e - 134)", "ldexp((double)(128 + f), e - 133)"),
    "bf16_fraction_width": ("int f = b & 0x7F;", "int f = b & 0x3F;"),
    "int4_threshold": ("code >= 8 ? (int)code - 16", "code > 8 ? (int)code - 16"),
    "int4_unsigned": ("code >= 8 ? (int)code - 16 : (int)code", "(int)code"),
    "q4_nibble_order": ("(k % 2 == 0) ? (byte & 0xF) : (byte >> 4)",
                        "(k % 2 == 0) ? (byte >> 4) : (byte & 0xF)"),
    "q4_scale_block": ("S[i * (K / 32) + k / 32]", "S[i * (K / 32) + k / 64]"),
    "q4_scale_row": ("S[i * (K / 32) + k / 32]", "S[(k / 32) % (K / 32)]"),
    "gemv16_transposed": ("dec16(W[i * K + k], fmt)", "dec16(W[k * M + i], fmt)"),
    "gemv16_drop_last": ("for (int64_t k = 0; k < K; ++k) acc += dec16",
                         "for (int64_t k = 0; k < K - 1; ++k) acc += dec16"),
    "gemv16_sign": ("acc += dec16(W[i * K + k], fmt)", "acc -= dec16(W[i * K + k], fmt)"),
    "gemv16_x_format": ("* dec16(x[k], fmt)", "* ora_f16_to_f64(x[k])"),
    "gemvq4_drop_first": ("for (int64_t k = 0; k < K; ++k) acc += ora_q4_weight",
                          "for (int64_t k = 1; k < K; ++k) acc += ora_q4_weight"),
    "gemvq4_no_scale": ("return (double)q * s;", "return (double)q;"),
    "int8_unsigned": ("byte >= 128 ? (int)byte - 256 : (int)byte", "(int)byte"),
    "int8_threshold": ("byte >= 128 ? (int)byte - 256", "byte > 128 ? (int)byte - 256"),
    "i8_first_row_scale": ("double row_scale = ora_f16_to_f64(S[i]);", "double row_scale = ora_f16_to_f64(S[0]);"),
    "i8_no_scale": ("return (double)q * row_scale;", "return (double)q;"),
    "i8_columns_reversed": ("ora_int8(Wq[i * K + k])", "ora_int8(Wq[i * K + (K - 1 - k)])"),
    "gemvi8_drop_last": ("for (int64_t k = 0; k < K; ++k) acc += ora_i8_weight",
                         "for (int64_t k = 0; k < K - 1; ++k) acc += ora_i8_weight"),
    "probe_drop_last": ("for (int64_t i = 0; i < n; ++i) s += (double)buf[i];",
                        "for (int64_t i = 0; i + 1 < n; ++i) s += (double)buf[i];"),
    "probe_float_accumulate": ("double s = 0.0;\n    for (int64_t i = 0; i < n; ++i) s += (double)buf[i];",
                               "float s = 0.0f;\n    for (int64_t i = 0; i < n; ++i) s += buf[i];"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    find, repl = MUTANTS[name]
    src = open(oracle.SRC_PATH).read()
    assert src.count(find) == 1, f"mutation site for {name} not found exactly once"
    mpath = tmp_path / "oracle_mut.c"
    mpath.write_text(src.replace(find, repl))
    lib = oracle.build(str(mpath), str(tmp_path / f"liboracle_{name}.so"))
    ora = oracle.Oracle(lib)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(ora)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin caught mutant {name}"
