"""Pins for the fp64 oracle: checks against what the paper and mathematics fix,
written so they can run against the oracle or against a planted-mistake copy.

Each check returns None when it holds and a short failure string otherwise.
Sources of truth (none of them is the oracle's own code):
  * hand-worked closed forms (tests/golden/hand_examples.json);
  * an independent pure-Python brute force (oracle/bruteforce.py);
  * torch's scaled_dot_product_attention in float64 on the CPU, applied to the
    dense concatenated sequence (prefix ‖ new) — the paper's defining claim
    that reused prefix KV gives the same result as recomputation (§2.2);
  * invariants: softmax weights sum to 1, block relabelling, chunked turns.
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


ALL_CHECKS = [check_hand_examples, check_bruteforce, check_prefix_reuse_equals_recompute,
              check_rows_sum_to_one, check_position_code]


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
