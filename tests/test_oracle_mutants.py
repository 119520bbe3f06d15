"""Planted mistakes in the oracle (on the CPU) must fail at least one pin.

Each mutant is oracle.c with one plausible slip -- a dropped term, a wrong sign
or index, an operand swapped, a comparison flipped -- compiled into a temporary
library and run through the pins of oracle_pins.py.  A mutant that passes every
pin would show a blind spot in the pins.
"""
import os

import pytest

import oracle
from oracle import build as obuild
import oracle_pins as P

MUTANTS = {
    "inclusive_i32_off_by_one": (
        "        acc += (uint32_t)x[i];\n        y[i] = acc;\n    }\n}\n\n/* ---- Appendix \"Exclusive",
        "        y[i] = acc;\n        acc += (uint32_t)x[i];\n    }\n}\n\n/* ---- Appendix \"Exclusive"),
    "exclusive_i32_wrong_index": (
        "        y[i] = acc;\n        acc += (uint32_t)x[i];\n    }\n}\n\nvoid oracle_scan_inclusive_f32",
        "        y[i] = acc;\n        acc += (uint32_t)x[i > 0 ? i - 1 : 0];\n    }\n}\n\nvoid oracle_scan_inclusive_f32"),
    "inclusive_f32_sign": (
        "        acc += (double)x[i];\n        aacc += fabs((double)x[i]);\n        y[i] = acc;",
        "        acc -= (double)x[i];\n        aacc += fabs((double)x[i]);\n        y[i] = acc;"),
    "inclusive_f32_float_accumulator": (
        "        acc += (double)x[i];\n        aacc += fabs((double)x[i]);\n        y[i] = acc;",
        "        acc = (float)(acc + (double)x[i]);\n        aacc += fabs((double)x[i]);\n        y[i] = acc;"),
    "abs_prefix_dropped_fabs": (
        "        acc += (double)x[i];\n        aacc += fabs((double)x[i]);\n        y[i] = acc;",
        "        acc += (double)x[i];\n        aacc += (double)x[i];\n        y[i] = acc;"),
    "exclusive_f32_inclusive_order": (
        "        y[i] = acc;\n        if (a) a[i] = aacc;\n        acc += (double)x[i];",
        "        acc += (double)x[i];\n        y[i] = acc;\n        if (a) a[i] = aacc;"),
    "half_exponent_bias": ("(1024 + f), e - 25)", "(1024 + f), e - 24)"),
    "half_subnormal_scale": ("ldexp((double)f, -24)", "ldexp((double)f, -25)"),
    "inclusive_f16_dropped_term": (
        "        const double v = oracle_half_to_double(x[i]);\n        acc += v;",
        "        const double v = oracle_half_to_double(x[i]);\n        acc += (i > 0) ? v : 0.0;"),
    "u8_signed_bytes": (
        "        y[i] = acc;\n        acc += (uint32_t)x[i];\n    }\n    if (total)",
        "        y[i] = acc;\n        acc += (uint32_t)(int8_t)x[i];\n    }\n    if (total)"),
    "rows_wrong_input_offset": (
        "oracle_scan_inclusive_i32(x + r * len, y + r * len, len);",
        "oracle_scan_inclusive_i32(x + r, y + r * len, len);"),
    "compact_only_ones": ("if (mask[i] != 0) {", "if (mask[i] == 1) {"),
    "split_unstable_second_part": (
        "for (int64_t i = 0; i < n; ++i) { /* second pass",
        "for (int64_t i = n - 1; i >= 0; --i) { /* second pass"),
    "split_ignores_idx_in": (
        "            if (idx_out) idx_out[c] = idx_in ? idx_in[i] : (int32_t)i;\n            ++c;\n        }\n    }\n    const int64_t",
        "            if (idx_out) idx_out[c] = (int32_t)i;\n            ++c;\n        }\n    }\n    const int64_t"),
    "sort_descending": ("return a->key < b->key ? -1 : 1;", "return a->key < b->key ? 1 : -1;"),
    "sort_ties_reversed": ("return a->index < b->index ? -1 : (a->index > b->index ? 1 : 0);",
                           "return a->index < b->index ? 1 : (a->index > b->index ? -1 : 0);"),
    "typed_sort_zeros_unordered": ("if (sx != sy) return sx ? -1 : 1; /* -0 before +0 */",
                                   "if (sx != sy) return 0; /* -0 before +0 */"),
    "typed_sort_nan_sign_flipped": ("    if (nanx) return sx ? -1 : 1;\n    return sy ? 1 : -1;",
                                    "    if (nanx) return sx ? 1 : -1;\n    return sy ? -1 : 1;"),
    "typed_sort_nan_payload_order": ("return ((payx < payy) != (sx != 0)) ? -1 : 1;",
                                     "return ((payx < payy) == (sx != 0)) ? -1 : 1;"),
    "typed_sort_desc_reverses_ties": ("    if (oracle_kdesc) c = -c;\n    if (c != 0) return c;\n    return (a->index > b->index) - (a->index < b->index);",
                                      "    if (oracle_kdesc) c = -c;\n    if (c != 0) return c;\n    return oracle_kdesc ? (a->index < b->index) - (a->index > b->index) : (a->index > b->index) - (a->index < b->index);"),
    "typed_sort_i32_unsigned": ("const int32_t x = (int32_t)(uint32_t)a, y = (int32_t)(uint32_t)b;",
                                "const uint32_t x = (uint32_t)a, y = (uint32_t)b;"),
    "weighted_sample_ge": ("        if (acc > u) return i;", "        if (acc >= u) return i;"),
    "topp_sample_ascending": ("rc = oracle_sort_f32((const uint32_t*)(probs + r * len), sorted, idx, len, 1);",
                              "rc = oracle_sort_f32((const uint32_t*)(probs + r * len), sorted, idx, len, 0);"),
    "topp_sample_whole_row_mass": ("for (int64_t i = 0; i <= k; ++i) ck += (double)s[i];",
                                   "for (int64_t i = 0; i < len; ++i) ck += (double)s[i];"),
    "topp_sample_sorted_position": ("        token_out[r] = idx[j];", "        token_out[r] = (int32_t)j;"),
    "topk_direction_flipped": ("rc = oracle_sort_f32(x + r * len, sorted, idx, len, largest != 0);",
                               "rc = oracle_sort_f32(x + r * len, sorted, idx, len, largest == 0);"),
    "topk_wrong_row": ("rc = oracle_sort_f32(x + r * len, sorted, idx, len, largest != 0);",
                       "rc = oracle_sort_f32(x + r * k, sorted, idx, len, largest != 0);"),
    "topk_sorted_position": ("            idx_out[r * k + i] = idx[i];",
                             "            idx_out[r * k + i] = (int32_t)i;"),
    "topp_strict_comparison": ("if (c >= pd) {", "if (c > pd) {"),
    "topp_default_len": ("int64_t k = len - 1;", "int64_t k = len;"),
    "topp_exclusive_sum": ("            c += (double)row[i];\n            if (c >= pd) {",
                           "            if (c >= pd) {\n                k = i;\n                break;\n"
                           "            }\n            c += (double)row[i];\n            if (0) {"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(obuild.SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique/found"
    mutated = tmp_path / "oracle_mutant.c"
    mutated.write_text(src.replace(old, new))
    lib = obuild.compile_source(str(mutated), str(tmp_path / "liboracle_mutant.so"))
    o = oracle.Oracle(lib)
    failed = []
    for check in P.ALL_CHECKS:
        try:
            check(o)
        except AssertionError:
            failed.append(check.__name__)
    assert failed, f"mutant {name} passed every pin"
