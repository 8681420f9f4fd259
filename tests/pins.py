"""Pins for the fp64 oracle: checks against what the paper and mathematics fix,
written so they can run against the oracle or against a planted-mistake copy.

Each check returns None when it holds and a short failure string otherwise.
Sources of truth (none of them is the oracle's own code):
  * hand-worked closed forms (tests/golden/hand_examples.json);
  * an independent pure-Python brute force (oracle/bruteforce.py);
  * torch's scaled_dot_product_attention in float64 on the CPU, applied to the
    dense concatenated sequence (prefix ‖ new) — the paper's defining claim
    that reused prefix KV gives the same result as recomputation (§2.2);
  * invariants: softmax weights sum to 1, block relabelling, chunked turns;
  * for the 8-bit pools: the code values the OCP 8-bit floating-point
    specification prints (tests/golden/e4m3_codes.json), round-to-nearest-even
    and saturation properties, numpy's float32 product for the quantisation
    step, and the (independently pinned) bf16 oracle on pools holding the
    dequantised values.
"""
from __future__ import annotations

import json
import math
import os
from fractions import Fraction

import numpy as np

import oracle
from oracle import bruteforce
from paper_2505_23970_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")
E4M3_GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e4m3_codes.json")


def _value(x):
    if isinstance(x, str):
        if x.startswith("ln"):
            return math.log(float(Fraction(x[2:])))
        return float(Fraction(x))
    return float(x)


def golden_cases():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


def workload_from_case(c) -> W.Workload:
    bits = lambda a: W.f32_to_bf16_bits(np.asarray(a, np.float32))  # noqa: E731
    P = np.asarray(c["prefix_lens"], np.int32)
    n = np.asarray(c["new_lens"], np.int32)
    w = W.Workload(name=c["name"], seed=0, num_q_heads=c["num_q_heads"],
                   num_kv_heads=c["num_kv_heads"], head_dim=c["head_dim"],
                   page_size=c["page_size"], prefix_lens=P, new_lens=n,
                   block_tables=np.asarray(c["block_tables"], np.int32),
                   num_blocks=c["num_blocks"], q=bits(c["q"]), k_new=bits(c["k_new"]),
                   v_new=bits(c["v_new"]), k_prefix=bits(c["k_prefix"]),
                   v_prefix=bits(c["v_prefix"]), k_pool=None, v_pool=None,
                   scale=_value(c["scale"]))
    return w.finish()


# ------------------------------------------------------------------ individual pins

def check_hand_examples(lib):
    for c in golden_cases():
        w = workload_from_case(c)
        _, _, out, lse = oracle.run_workload(w, lib=lib)
        T, Hq, D = w.q.shape
        exp_out = np.array([[[_value(v) for v in head] for head in tok] for tok in c["expected_out"]])
        exp_lse = np.array([[_value(v) for v in tok] for tok in c["expected_lse"]])
        if not np.allclose(out.reshape(T, Hq, D), exp_out, rtol=0, atol=1e-12):
            return f"hand example {c['name']}: out {out.reshape(T, Hq, D).tolist()}"
        if not np.allclose(lse.reshape(T, Hq), exp_lse, rtol=0, atol=1e-12):
            return f"hand example {c['name']}: lse {lse.tolist()}"
    return None


TINY_CASES = [
    # (prefix_lens, new_lens, Hq, Hkv, D, page, values, seed)
    ([5], [3], 2, 1, 2, 4, "unit", 11),
    ([0], [7], 4, 2, 8, 16, "unit", 12),
    ([17], [1], 3, 3, 8, 16, "unit", 13),
    ([3, 0, 20], [4, 5, 2], 4, 1, 8, 4, "unit", 14),
    ([31], [9], 2, 2, 64, 16, "normal", 15),
    ([16, 15], [16, 1], 4, 2, 8, 16, "peaked", 16),
]


def tiny_workloads():
    for P, n, Hq, Hkv, D, S, values, seed in TINY_CASES:
        yield W.build(P, n, Hq, Hkv, D, seed=seed, page_size=S, values=values,
                      name=f"tiny{seed}")


def check_bruteforce(lib):
    for w in tiny_workloads():
        kp, vp, out, lse = oracle.run_workload(w, lib=lib)
        bkp, bvp = bruteforce.kv_append(w.prefix_lens, w.new_lens, w.block_tables, w.k_new,
                                        w.v_new, w.k_pool.tolist(), w.v_pool.tolist(),
                                        w.num_kv_heads, w.head_dim, w.page_size)
        if not (np.array_equal(kp, np.array(bkp, np.uint16))
                and np.array_equal(vp, np.array(bvp, np.uint16))):
            return f"append differs from brute force ({w.name})"
        bo, bl = bruteforce.attention(w.prefix_lens, w.new_lens, w.block_tables, w.q.tolist(),
                                      bkp, bvp, w.num_q_heads, w.num_kv_heads, w.head_dim,
                                      w.page_size, w.scale)
        T, Hq, D = w.q.shape
        bo = np.array(bo, np.float64).reshape(T * Hq, D)
        bl = np.array(bl, np.float64).reshape(T * Hq)
        if not np.allclose(out, bo, rtol=0, atol=1e-12):
            return f"attention differs from brute force ({w.name}): {np.abs(out - bo).max()}"
        if not np.allclose(lse, bl, rtol=0, atol=1e-12):
            return f"lse differs from brute force ({w.name})"
    return None


def dense_sdpa(w: W.Workload, rng_seed=0):
    """Full causal recomputation over the dense sequence prefix ‖ new with torch's
    float64 scaled_dot_product_attention; returns rows [P_r, L_r) as [T*Hq][D]."""
    import torch
    import torch.nn.functional as F
    f = W.bf16_bits_to_f32
    outs = []
    g = w.num_q_heads // w.num_kv_heads
    cup, cun = w.cu_prefix_lens, w.cu_new_lens
    rng = np.random.default_rng(rng_seed)
    for r in range(w.batch):
        P, n = int(w.prefix_lens[r]), int(w.new_lens[r])
        if n == 0:
            continue
        k = np.concatenate([f(w.k_prefix[cup[r]:cup[r + 1]]), f(w.k_new[cun[r]:cun[r + 1]])])
        v = np.concatenate([f(w.v_prefix[cup[r]:cup[r + 1]]), f(w.v_new[cun[r]:cun[r + 1]])])
        q_new = f(w.q[cun[r]:cun[r + 1]])
        # queries at prefix positions do not matter for the new rows; fill them randomly
        q_pre = rng.standard_normal((P, w.num_q_heads, w.head_dim))
        q = np.concatenate([q_pre, q_new])
        qt = torch.from_numpy(q.astype(np.float64)).permute(1, 0, 2)          # [Hq][L][D]
        kt = torch.from_numpy(k.astype(np.float64)).permute(1, 0, 2).repeat_interleave(g, 0)
        vt = torch.from_numpy(v.astype(np.float64)).permute(1, 0, 2).repeat_interleave(g, 0)
        o = F.scaled_dot_product_attention(qt, kt, vt, is_causal=True, scale=w.scale)
        outs.append(o.permute(1, 0, 2)[P:].reshape(n * w.num_q_heads, w.head_dim).numpy())
    return np.concatenate(outs) if outs else np.zeros((0, w.head_dim))


SDPA_CASES = [
    ([37], [21], 8, 2, 16, "unit", 21),
    ([0], [33], 4, 4, 32, "unit", 22),             # cache miss: plain causal prefill
    ([64, 5, 0], [1, 40, 3], 8, 1, 16, "peaked", 23),
    ([150], [1], 4, 2, 64, "normal", 24),          # one new token: decode-shaped
]


def check_prefix_reuse_equals_recompute(lib):
    for P, n, Hq, Hkv, D, values, seed in SDPA_CASES:
        w = W.build(P, n, Hq, Hkv, D, seed=seed, values=values)
        _, _, out, _ = oracle.run_workload(w, lib=lib)
        ref = dense_sdpa(w)
        if not np.allclose(out, ref, rtol=0, atol=1e-12):
            return f"pool path != dense recomputation (seed {seed}): {np.abs(out - ref).max()}"
    return None


def check_rows_sum_to_one(lib):
    w = W.set_values_one(W.build([40, 0], [9, 30], 4, 2, 8, seed=31, values="unit"))
    _, _, out, _ = oracle.run_workload(w, lib=lib)
    if not np.allclose(out, 1.0, rtol=0, atol=1e-14):
        return f"V = 1 gives {out.min()}..{out.max()}"
    return None


def check_position_code(lib):
    """Q = 0 makes every visible key weigh the same, so with V_j[0] = j the output's
    element 0 is the mean of 0..P+i, i.e. (P+i)/2 exactly."""
    w = W.set_position_code(W.build([37, 0], [12, 20], 4, 2, 8, seed=32))
    _, _, out, _ = oracle.run_workload(w, lib=lib)
    expect = []
    for r in range(w.batch):
        for i in range(int(w.new_lens[r])):
            expect += [(int(w.prefix_lens[r]) + i) / 2.0] * w.num_q_heads
    if not np.allclose(out[:, 0], expect, rtol=0, atol=1e-12):
        return "position-coded V: window or offset wrong"
    return None


# ------------------------------------------------------------------ 8-bit pools

def check_e4m3_spec_values(lib):
    with open(E4M3_GOLDEN) as f:
        g = json.load(f)
    for code, val in g["values"].items():
        got = oracle.e4m3_value(int(code, 16), lib=lib)
        want = -0.0 if val == "-0" else float(Fraction(val))
        if got != want or math.copysign(1.0, got) != math.copysign(1.0, want):
            return f"code {code}: {got} != {want}"
    for code in g["nan_codes"]:
        if not math.isnan(oracle.e4m3_value(int(code, 16), lib=lib)):
            return f"code {code} is not NaN"
    vals = [oracle.e4m3_value(c, lib=lib) for c in range(127)]
    if any(not math.isfinite(v) for v in vals) or any(b <= a for a, b in zip(vals, vals[1:])):
        return "codes 0x00..0x7e are not finite and strictly increasing"
    for c in range(127):
        if oracle.e4m3_value(c | 0x80, lib=lib) != -vals[c]:
            return f"code {c | 0x80:#x} is not the negation of {c:#x}"
    return None


def check_e4m3_rounding(lib):
    f32 = np.float32
    vals = [oracle.e4m3_value(c, lib=lib) for c in range(127)]
    enc = lambda v: oracle.e4m3_encode(v, lib=lib)  # noqa: E731
    for c in range(127):
        if enc(vals[c]) != c or enc(-vals[c]) != (c | 0x80):
            return f"code {c:#x} does not round-trip"
    for c in range(126):
        mid = f32((vals[c] + vals[c + 1]) / 2)  # exact: at most 5 significant bits
        even = c if c % 2 == 0 else c + 1
        if enc(mid) != even:
            return f"tie between {c:#x} and {c + 1:#x} went to {enc(mid):#x}"
        if enc(np.nextafter(mid, f32(np.inf))) != c + 1 or enc(np.nextafter(mid, f32(-np.inf))) != c:
            return f"values next to the midpoint of {c:#x} and {c + 1:#x} round the wrong way"
    for v, want in ((464.0, 0x7E), (1e38, 0x7E), (float("inf"), 0x7E), (-float("inf"), 0xFE),
                    (-500.0, 0xFE), (2.0 ** -10, 0x00), (-(2.0 ** -10), 0x80),
                    (float(np.nextafter(f32(2.0 ** -10), f32(1))), 0x01)):
        if enc(v) != want:
            return f"encode({v}) = {enc(v):#x}, want {want:#x}"
    return None


def check_e4m3_quantize_product(lib):
    """The bulk quantiser stores encode(fl32(x * fl32(1 / scale))), the product taken
    by numpy in float32."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    x = W.bf16_bits_to_f32(bits)
    bits = bits[np.isfinite(x)]
    x = x[np.isfinite(x)]
    for scale in (1.0, 0.37, 2.0 ** -7, 3.1 / 448.0):
        inv = oracle.inv_scale(scale)
        got = oracle.quantize_e4m3(bits, scale, lib=lib)
        with np.errstate(over="ignore"):
            prod = (x * inv).astype(np.float32)
        idx = np.random.default_rng(5).choice(bits.size, 1500, replace=False)
        for i in idx:
            if got[i] != oracle.e4m3_encode(prod[i], lib=lib):
                return f"scale {scale}: bf16 {bits[i]:#x} quantised to {got[i]:#x}"
    return None


def _dequantised_bf16(codes, scale, lib):
    table = np.array([oracle.e4m3_value(c, lib=lib) for c in range(256)], np.float64) * scale
    return W.f32_to_bf16_bits(table[codes].astype(np.float32))


def check_e4m3_pools_match_bf16_oracle(lib):
    """With power-of-two scales every dequantised element is a bf16 value, so the
    8-bit append and attention must give exactly what the bf16 oracle gives on
    pools holding those values; different key and value scales catch a swap."""
    ks, vs = 2.0 ** -6, 2.0 ** -4
    for P, n, Hq, Hkv, D, seed in (([21, 0, 9], [13, 4, 30], 4, 2, 8, 61),
                                   ([40], [7], 8, 2, 16, 62)):
        w = W.build(P, n, Hq, Hkv, D, seed=seed)
        k8, v8 = W.e4m3_pools(w)
        kp8, vp8 = oracle.kv_append_e4m3(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks,
                                         w.k_new, w.v_new, k8, v8, ks, vs, lib=lib)
        # the append wrote exactly the quantised new tokens and nothing else
        changed = int((kp8 != k8).sum() + (vp8 != v8).sum())
        want_k = oracle.quantize_e4m3(w.k_new, ks, lib=lib)
        want_v = oracle.quantize_e4m3(w.v_new, vs, lib=lib)
        if changed > 2 * w.total_new * Hkv * D:
            return "8-bit append changed slots it does not own"
        cu = w.cu_new_lens
        for r in range(w.batch):
            for i in range(int(w.new_lens[r])):
                pos = int(w.prefix_lens[r]) + i
                blk, off = int(w.block_tables[r, pos // 16]), pos % 16
                t = int(cu[r]) + i
                if not (np.array_equal(kp8[blk, :, off, :], want_k[t])
                        and np.array_equal(vp8[blk, :, :, off], want_v[t])):
                    return f"8-bit append slot of request {r} token {i} holds other codes"
        out8, lse8 = oracle.attention_e4m3(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks,
                                           w.q, kp8, vp8, ks, vs, w.scale, lib=lib)
        out, lse = oracle.attention(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks, w.q,
                                    _dequantised_bf16(kp8, ks, lib), _dequantised_bf16(vp8, vs, lib),
                                    w.scale, lib=lib)
        if not (np.array_equal(out8, out) and np.array_equal(lse8, lse)):
            return f"8-bit attention differs from the bf16 oracle on dequantised pools ({seed})"
    return None


ALL_CHECKS = [check_hand_examples, check_bruteforce, check_prefix_reuse_equals_recompute,
              check_rows_sum_to_one, check_position_code, check_e4m3_spec_values,
              check_e4m3_rounding, check_e4m3_quantize_product, check_e4m3_pools_match_bf16_oracle]


def run_all(lib):
    failures = []
    for chk in ALL_CHECKS:
        try:
            msg = chk(lib)
        except Exception as e:  # a planted mistake may also crash a check
            msg = f"{chk.__name__} raised {type(e).__name__}: {e}"
        if msg:
            failures.append(f"{chk.__name__}: {msg}")
    return failures
