"""Planted mistakes in the oracle (CPU only): each variant of gc_oracle.c below
carries one plausible slip — a dropped term, a wrong sign or index, a swapped
layout — and the pins must reject every one of them. This shows the pins are
tight enough to trust the oracle they accept."""
import os

import pytest

import oracle
import pins
from oracle.build import SOURCE, build_oracle

MUTANTS = {
    "causal_boundary_exclusive": (
        "int64_t nkeys = (int64_t)prefix_lens[r] + i + 1;",
        "int64_t nkeys = (int64_t)prefix_lens[r] + i;"),
    "causal_one_key_too_many": (
        "int64_t nkeys = (int64_t)prefix_lens[r] + i + 1;",
        "int64_t nkeys = (int64_t)prefix_lens[r] + i + 2;"),
    "prefix_not_visible": (
        "for (int64_t j = 0; j < nkeys; ++j) {\n            int64_t blk = block_of(block_tables, max_blocks, num_blocks, r, j, page);\n            if (blk < 0)",
        "for (int64_t j = 0; j < nkeys; ++j) {\n            int64_t blk = block_of(block_tables, max_blocks, num_blocks, r, j, page);\n            if (j < prefix_lens[r]) { x[j] = -1e300; continue; }\n            if (blk < 0)"),
    "head_mapping_modulo": (
        "int kvh = h / group;",
        "int kvh = h % num_kv_heads;"),
    "scale_dropped": (
        "x[j] = scale * dot;",
        "x[j] = dot;"),
    "scale_squared": (
        "x[j] = scale * dot;",
        "x[j] = scale * scale * dot;"),
    "normalisation_dropped": (
        "double p = x[j] / l;",
        "double p = x[j];"),
    "exponent_sign_flipped": (
        "x[j] = exp(x[j] - m);",
        "x[j] = exp(m - x[j]);"),
    "last_weight_dropped_from_sum": (
        "l += x[j];",
        "if (j + 1 < nkeys) l += x[j];"),
    "lse_without_max": (
        "if (lse) lse[k] = m + log(l);",
        "if (lse) lse[k] = log(l);"),
    "value_page_read_untransposed": (
        "o[c] += p * kv_elem(v_pool, kv8, v_scale, ((blk * num_kv_heads + kvh) * head_dim + c) * page + j % page);",
        "o[c] += p * kv_elem(v_pool, kv8, v_scale, ((blk * num_kv_heads + kvh) * page + j % page) * head_dim + c);"),
    "key_slot_off_by_one": (
        "int64_t krow = ((blk * num_kv_heads + kvh) * page + j % page) * head_dim;",
        "int64_t krow = ((blk * num_kv_heads + kvh) * page + (j + 1) % page) * head_dim;"),
    "value_read_from_key_pool": (
        "o[c] += p * kv_elem(v_pool, kv8, v_scale, ((blk * num_kv_heads + kvh) * head_dim + c) * page + j % page);",
        "o[c] += p * kv_elem(k_pool, kv8, v_scale, ((blk * num_kv_heads + kvh) * page + j % page) * head_dim + c);"),
    "append_position_off_by_one": (
        "int64_t pos = (int64_t)prefix_lens[r] + i;",
        "int64_t pos = (int64_t)prefix_lens[r] + i + 1;"),
    "append_value_untransposed": (
        "int64_t vidx = ((blk * num_kv_heads + h) * head_dim + c) * page + off;",
        "int64_t vidx = ((blk * num_kv_heads + h) * page + off) * head_dim + c;"),
    # 8-bit pools
    "e4m3_exponent_bias_8": (
        "mag = ldexp(1.0 + (double)m / 8.0, e - 7);",
        "mag = ldexp(1.0 + (double)m / 8.0, e - 8);"),
    "e4m3_subnormals_with_hidden_bit": (
        "mag = ldexp((double)m / 8.0, -6);",
        "mag = ldexp((double)m / 8.0, -7);"),
    "e4m3_nan_code_finite": (
        "if (e == 15 && m == 7) return NAN;",
        "if (e == 16) return NAN;"),
    "e4m3_ties_to_odd": (
        "if (d < best_d || (d == best_d && (c & 1) == 0)) {",
        "if (d < best_d || (d == best_d && (c & 1) == 1)) {"),
    "e4m3_ties_away_from_zero": (
        "if (d < best_d || (d == best_d && (c & 1) == 0)) {",
        "if (d <= best_d) {"),
    "e4m3_negative_zero_dropped": (
        "return (uint8_t)(best | (signbit(v) ? 0x80 : 0));",
        "return (uint8_t)(best | (v < 0 ? 0x80 : 0));"),
    "quantise_divides_by_inverse": (
        "return (float)(widen(x) * (double)inv);",
        "return (float)(widen(x) / (double)inv);"),
    "dequantise_scale_dropped": (
        "if (kv8) return gco_e4m3_value(((const uint8_t*)pool)[idx]) * scale;",
        "if (kv8) return gco_e4m3_value(((const uint8_t*)pool)[idx]);"),
    "values_dequantised_with_key_scale": (
        "o[c] += p * kv_elem(v_pool, kv8, v_scale,",
        "o[c] += p * kv_elem(v_pool, kv8, k_scale,"),
    "append_values_quantised_with_key_scale": (
        "((uint8_t*)v_pool)[vidx] = gco_e4m3_encode(scaled32(vs[c], v_inv));",
        "((uint8_t*)v_pool)[vidx] = gco_e4m3_encode(scaled32(vs[c], k_inv));"),
    "request_lookup_off_by_one": (
        "while (token >= first + new_lens[r]) {",
        "while (token > first + new_lens[r]) {"),
    "query_head_row_stride": (
        "qv[c] = widen(q[(token * num_q_heads + h) * head_dim + c]);",
        "qv[c] = widen(q[(token * num_q_heads + kvh) * head_dim + c]);"),
}


@pytest.fixture(scope="module")
def source_text():
    with open(SOURCE) as f:
        return f.read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_planted_mistake(name, source_text, tmp_path):
    old, new = MUTANTS[name]
    assert source_text.count(old) == 1, f"mutation site for {name} not found exactly once"
    src = tmp_path / f"{name}.c"
    src.write_text(source_text.replace(old, new))
    lib_path = build_oracle(str(src), str(tmp_path / f"lib{name}.so"), extra=["-w"])
    lib = oracle.load(lib_path)
    failures = pins.run_all(lib)
    assert failures, f"planted mistake '{name}' passed every pin"


def test_unmodified_oracle_passes_every_pin(oracle_lib):
    assert pins.run_all(oracle_lib) == []
