"""Planted mistakes in the oracle are caught by its pins (CPU only).

Each case copies ``oracle/nuna_oracle.c``, applies one plausible mistake by
text substitution (a dropped term, a wrong sign, a wrong index, a transposed
layout, a wrong rounding rule, a wrong routing rule, a wrong order), builds the
copy with gcc into a temporary directory and runs the pin battery of
``tests/oracle_pins.py`` against it.  The test passes only if at least one pin
fails for every mutant -- i.e. the pins are strong enough to catch it.
"""
import os

import pytest

import oracle
from oracle import build as obuild
import oracle_pins

MUTANTS = {
    "drop_last_rank": ("for (int r = 1; r < P; ++r) acc = acc + orc_load(in[r], dtype, i);",
                       "for (int r = 1; r < P - 1; ++r) acc = acc + orc_load(in[r], dtype, i);"),
    "wrong_sign": ("acc = acc + orc_load(in[r], dtype, i);", "acc = acc - orc_load(in[r], dtype, i);"),
    "descending_order": (
        "float acc = orc_load(in[0], dtype, i);\n    for (int r = 1; r < P; ++r) acc = acc + orc_load(in[r], dtype, i);",
        "float acc = orc_load(in[P - 1], dtype, i);\n    for (int r = P - 2; r >= 0; --r) acc = acc + orc_load(in[r], dtype, i);"),
    "start_from_plus_zero": (
        "float acc = orc_load(in[0], dtype, i);\n    for (int r = 1; r < P; ++r)",
        "float acc = 0.0f;\n    for (int r = 0; r < P; ++r)"),
    "ties_away_from_zero": ("if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u)))",
                            "if (lower >= 0x8000u)"),
    "truncate_not_round": ("if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u)))", "if (0)"),
    "nan_becomes_inf": ("return (uint16_t)((u >> 16) | 0x0040u);", "return (uint16_t)((u >> 16) & 0xff80u);"),
    "rs_strided_shards": ("size_t i = (size_t)r * m + j;", "size_t i = j * (size_t)P + (size_t)r;"),
    "rs_wrong_owner": ("orc_store(out[r], dtype, j, acc);", "orc_store(out[(r + 1) % P], dtype, j, acc);"),
    "ag_dest_offset": ("unsigned char* dst = (unsigned char*)out[d] + (size_t)r * m * es;",
                       "unsigned char* dst = (unsigned char*)out[d] + (size_t)((r + d) % P) * m * es;"),
    "ag_float_roundtrip": ("for (size_t b = 0; b < es; ++b) dst[j * es + b] = src[j * es + b];",
                           "if (es == 2) ((uint16_t*)dst)[j] = orc_f32_to_bf16(orc_bf16_to_f32(((const uint16_t*)src)[j])); else ((float*)dst)[j] = ((const float*)src)[j] * 1.0f;"),
    "a2a_modulo_owner": ("if (ex[j] / per == d) return 1;", "if (ex[j] % P == d) return 1;"),
    "a2a_first_expert_only": ("for (int j = 0; j < k; ++j)\n        if (ex[j] / per == d) return 1;",
                              "for (int j = 0; j < 1; ++j)\n        if (ex[j] / per == d) return 1;"),
    "a2a_token_major_order": (
        "int64_t j = 0;\n    for (int s = 0; s < P; ++s)\n        for (int t = 0; t < T; ++t)\n            if (orc_token_goes_to(topk, P, T, k, E, s, t, d)) {\n                src_rank[j] = s;",
        "int64_t j = 0;\n    for (int t = 0; t < T; ++t)\n        for (int s = 0; s < P; ++s)\n            if (orc_token_goes_to(topk, P, T, k, E, s, t, d)) {\n                src_rank[j] = s;"),
    "combine_descending_ranks": ("for (int d = 0; d < P; ++d) {\n                    int64_t j = pos[",
                                 "for (int d = P - 1; d >= 0; --d) {\n                    int64_t j = pos["),
    "combine_drops_last_rank": ("for (int d = 0; d < P; ++d) {\n                    int64_t j = pos[",
                                "for (int d = 0; d < P - 1; ++d) {\n                    int64_t j = pos["),
    "combine_wrong_row": ("float v = orc_load(y[d], dtype, (size_t)j * row_elems + h);",
                          "float v = orc_load(y[d], dtype, (size_t)(j > 0 ? j - 1 : 0) * row_elems + h);"),
    "combine_weight_transposed": ("if (weights) v = weights[((size_t)s * T + t) * P + d] * v;",
                                  "if (weights) v = weights[((size_t)d * T + t) * P + s] * v;"),
    "combine_weight_ignored": ("if (weights) v = weights[((size_t)s * T + t) * P + d] * v;",
                               "if (weights) v = v;"),
    "a2a_row_offset": ("unsigned char* dst = (unsigned char*)recv[d] + (size_t)j * row_bytes;",
                       "unsigned char* dst = (unsigned char*)recv[d] + (size_t)(j > 0 ? j - 1 : 0) * row_bytes;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    src = open(obuild.SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) >= 1, f"mutation anchor for {name} not found in the oracle source"
    mutated = src.replace(old, new, 1)
    csrc = tmp_path / "mutant.c"
    csrc.write_text(mutated)
    lib = str(tmp_path / "libmutant.so")
    import subprocess
    subprocess.run(["gcc", *obuild.CFLAGS, "-w", str(csrc), "-o", lib], check=True)
    orc = oracle.Oracle(lib)
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(orc)
        except AssertionError:
            caught.append(pin.__name__)
            break
    assert caught, f"mutant {name} passed every pin"


def test_unmutated_oracle_passes_the_same_battery():
    orc = oracle.Oracle(obuild.LIB if os.path.exists(obuild.LIB) else obuild.build())
    for pin in oracle_pins.ALL_PINS:
        pin(orc)
