"""The fp64 oracle against pins that do not come from its own code (CPU only)."""
import numpy as np
import pytest

import oracle
import pins
from paper_2505_23970_amd import workloads as W


def test_hand_examples(oracle_lib):
    assert pins.check_hand_examples(oracle_lib) is None


def test_matches_pure_python_bruteforce(oracle_lib):
    assert pins.check_bruteforce(oracle_lib) is None


def test_prefix_reuse_equals_full_recomputation(oracle_lib):
    """§2.2: stitching cached prefix KV with the new tokens' KV gives the same
    rows as recomputing attention over the whole sequence (torch SDPA, fp64)."""
    assert pins.check_prefix_reuse_equals_recompute(oracle_lib) is None


def test_softmax_rows_sum_to_one(oracle_lib):
    assert pins.check_rows_sum_to_one(oracle_lib) is None


def test_position_coded_window(oracle_lib):
    assert pins.check_position_code(oracle_lib) is None


def test_tiny_config_matches_sdpa(oracle_lib):
    w = W.make_config(1)
    _, _, out, _ = oracle.run_workload(w, lib=oracle_lib)
    np.testing.assert_allclose(out, pins.dense_sdpa(w), rtol=0, atol=1e-12)


def test_append_bit_exact_and_poison_kept(oracle_lib):
    w = W.build([21, 0, 9], [13, 4, 30], 4, 2, 8, seed=41)
    kp, vp = oracle.kv_append(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks,
                              w.k_new, w.v_new, w.k_pool, w.v_pool, lib=oracle_lib)
    changed = int((kp != w.k_pool).sum() + (vp != w.v_pool).sum())
    # every appended element lands on a NaN-poisoned slot, so all of them change
    assert changed == 2 * w.total_new * w.num_kv_heads * w.head_dim
    # untouched slots keep their poison and the prefix keeps its bits
    assert int(np.isnan(W.bf16_bits_to_f32(kp)).sum()) == int(
        np.isnan(W.bf16_bits_to_f32(w.k_pool)).sum()) - w.total_new * w.num_kv_heads * w.head_dim


def test_append_rejects_short_table(oracle_lib):
    w = W.build([30], [5], 2, 1, 8, seed=42, extra_table_slots=0)
    bt = w.block_tables[:, :2]  # needs 3 pages
    with pytest.raises(oracle.OracleError):
        oracle.kv_append(w.prefix_lens, w.new_lens, bt, w.num_blocks, w.k_new, w.v_new,
                         w.k_pool, w.v_pool, lib=oracle_lib)


def test_chunked_turns_equal_one_call(oracle_lib):
    """Multi-turn reuse (§2.2): appending n1 tokens and attending, then appending
    n2 more with prefix P + n1, gives the rows of a single call with n1 + n2."""
    w = W.build([27], [19], 4, 2, 16, seed=43, values="unit")
    n1 = 8
    _, _, full, _ = oracle.run_workload(w, lib=oracle_lib)
    kp1, vp1 = oracle.kv_append(w.prefix_lens, [n1], w.block_tables, w.num_blocks,
                                w.k_new[:n1], w.v_new[:n1], w.k_pool, w.v_pool, lib=oracle_lib)
    o1, _ = oracle.attention(w.prefix_lens, [n1], w.block_tables, w.num_blocks, w.q[:n1],
                             kp1, vp1, w.scale, lib=oracle_lib)
    P2 = w.prefix_lens + n1
    kp2, vp2 = oracle.kv_append(P2, [19 - n1], w.block_tables, w.num_blocks, w.k_new[n1:],
                                w.v_new[n1:], kp1, vp1, lib=oracle_lib)
    o2, _ = oracle.attention(P2, [19 - n1], w.block_tables, w.num_blocks, w.q[n1:], kp2, vp2,
                             w.scale, lib=oracle_lib)
    assert np.array_equal(np.concatenate([o1, o2]), full)


def test_block_relabelling_invariance(oracle_lib):
    w = W.build([45, 3], [10, 20], 4, 1, 8, seed=44, values="unit")
    _, _, out, lse = oracle.run_workload(w, lib=oracle_lib)
    rng = np.random.default_rng(7)
    perm = rng.permutation(w.num_blocks)           # new id of old block b is perm[b]
    kp = np.empty_like(w.k_pool)
    vp = np.empty_like(w.v_pool)
    kp[perm] = w.k_pool
    vp[perm] = w.v_pool
    bt = perm[w.block_tables].astype(np.int32)
    kp2, vp2 = oracle.kv_append(w.prefix_lens, w.new_lens, bt, w.num_blocks, w.k_new, w.v_new,
                                kp, vp, lib=oracle_lib)
    out2, lse2 = oracle.attention(w.prefix_lens, w.new_lens, bt, w.num_blocks, w.q, kp2, vp2,
                                  w.scale, lib=oracle_lib)
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2)


def test_mha_equals_gqa_with_repeated_kv(oracle_lib):
    g = W.build([13], [6], 8, 2, 8, seed=45, values="unit")
    _, _, out_g, _ = oracle.run_workload(g, lib=oracle_lib)
    rep = lambda a: np.repeat(a, 4, axis=1)  # noqa: E731  kv head h // 4 for query head h
    m = W.Workload(name="mha", seed=0, num_q_heads=8, num_kv_heads=8, head_dim=8, page_size=16,
                   prefix_lens=g.prefix_lens, new_lens=g.new_lens, block_tables=g.block_tables,
                   num_blocks=g.num_blocks, q=g.q, k_new=rep(g.k_new), v_new=rep(g.v_new),
                   k_prefix=rep(g.k_prefix), v_prefix=rep(g.v_prefix), k_pool=None, v_pool=None,
                   scale=g.scale).finish()
    _, _, out_m, _ = oracle.run_workload(m, lib=oracle_lib)
    assert np.array_equal(out_g, out_m)


def test_row_subset_matches_full(oracle_lib):
    w = W.build([50, 7], [11, 25], 4, 2, 16, seed=46)
    _, _, full, full_lse = oracle.run_workload(w, lib=oracle_lib)
    rows = np.array([0, 5, 43, 44, 100, 143], np.int64)
    _, _, sub, sub_lse = oracle.run_workload(w, rows=rows, lib=oracle_lib)
    assert np.array_equal(sub, full[rows]) and np.array_equal(sub_lse, full_lse[rows])


def test_bf16_widening_is_exact(oracle_lib):
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.widen_bf16(bits, lib=oracle_lib)
    ref = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # and the encoder used by the generator rounds to nearest even
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.0e-39], np.float32)
    assert W.f32_to_bf16_bits(x).tolist() == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x0021]


def test_e4m3_code_values_from_the_ocp_table(oracle_lib):
    assert pins.check_e4m3_spec_values(oracle_lib) is None


def test_e4m3_rounding_nearest_even_and_saturating(oracle_lib):
    assert pins.check_e4m3_rounding(oracle_lib) is None


def test_e4m3_quantiser_uses_the_fp32_product(oracle_lib):
    assert pins.check_e4m3_quantize_product(oracle_lib) is None


def test_8bit_pools_match_bf16_oracle_on_power_of_two_scales(oracle_lib):
    assert pins.check_e4m3_pools_match_bf16_oracle(oracle_lib) is None


def test_8bit_scales_enter_linearly(oracle_lib):
    """Dequantising first means the key scale multiplies every score and the value
    scale multiplies the output: the result for scales (ks, vs) equals the result
    for (1, 1) with softmax scale `scale * ks`, times vs."""
    w = W.build([33, 5], [9, 17], 8, 2, 16, seed=63)
    k8, v8 = W.e4m3_pools(w)
    k8, v8 = oracle.kv_append_e4m3(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks,
                                   w.k_new, w.v_new, k8, v8, 0.011, 0.023, lib=oracle_lib)
    out, lse = oracle.attention_e4m3(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks, w.q,
                                     k8, v8, 0.011, 0.023, w.scale, lib=oracle_lib)
    out1, lse1 = oracle.attention_e4m3(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks,
                                       w.q, k8, v8, 1.0, 1.0, w.scale * 0.011, lib=oracle_lib)
    np.testing.assert_allclose(out, out1 * 0.023, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(lse, lse1, rtol=1e-12, atol=1e-12)
