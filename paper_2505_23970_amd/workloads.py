"""Seeded synthetic inputs for prefix-cached prefill attention.

This module only *draws inputs*: request lengths, block tables, bf16 bit
patterns for the queries and the new tokens' K/V, and the initial state of the
paged KV pool (the cached prefix pages already resident, as if restored from
the context cache; every other slot NaN-poisoned). It holds none of the
method's arithmetic: the KV append and the attention live in the HIP library
and, separately, in the oracle. Both receive the same arrays from here.

The paper evaluates on ShareGPT multi-turn chats and TriviaQA documents with
Llama-3 8B/70B (§6.1 Methodology); neither the datasets nor the weights are
available, so the recipes below draw random values with the attention shapes
of those models and length distributions shaped like those workloads (77.2 %
of ShareGPT prompts carry more than 1000 context tokens, §3.1.1).

Pool layout (also stated in include/greencache.h):
  k_pool  bf16 [num_blocks][num_kv_heads][page_size][head_dim]
  v_pool  bf16 [num_blocks][num_kv_heads][head_dim][page_size]
Logical page p of request r lives in physical block block_tables[r][p].
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

BF16_NAN = np.uint16(0x7FC0)
BF16_ONE = np.uint16(0x3F80)
E4M3_NAN = np.uint8(0x7F)  # the 8-bit pools' poison (an E4M3 NaN code)
SEED_BASE = 2505239700

CONFIG_NAMES = {
    1: "tiny",
    2: "llama3_8b",
    3: "llama3_70b_chat",
    4: "long_reuse_70b",
    5: "mixed_hit_miss_70b",
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Encode finite float32 values as bfloat16 bit patterns (round to nearest even)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Decode bfloat16 bit patterns to float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass
class Workload:
    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    prefix_lens: np.ndarray      # int32 [B]
    new_lens: np.ndarray         # int32 [B]
    block_tables: np.ndarray     # int32 [B][max_blocks_per_seq]
    num_blocks: int
    q: np.ndarray                # uint16 [T][Hq][D]
    k_new: np.ndarray            # uint16 [T][Hkv][D]
    v_new: np.ndarray            # uint16 [T][Hkv][D]
    k_prefix: np.ndarray         # uint16 [sum P][Hkv][D], request-major (logical order)
    v_prefix: np.ndarray         # uint16 [sum P][Hkv][D]
    k_pool: np.ndarray           # uint16 [NB][Hkv][S][D]  initial pool (prefix resident)
    v_pool: np.ndarray           # uint16 [NB][Hkv][D][S]
    scale: float

    @property
    def batch(self) -> int:
        return int(self.prefix_lens.shape[0])

    @property
    def max_blocks_per_seq(self) -> int:
        return int(self.block_tables.shape[1])

    @property
    def total_new(self) -> int:
        return int(self.new_lens.sum())

    @property
    def cu_new_lens(self) -> np.ndarray:
        cu = np.zeros(self.batch + 1, dtype=np.int32)
        np.cumsum(self.new_lens, out=cu[1:])
        return cu

    @property
    def cu_prefix_lens(self) -> np.ndarray:
        cu = np.zeros(self.batch + 1, dtype=np.int64)
        np.cumsum(self.prefix_lens, out=cu[1:])
        return cu

    def flops(self) -> float:
        """Algorithmic exact-causal FLOPs of QK^T and PV over the attended pairs."""
        P = self.prefix_lens.astype(np.float64)
        n = self.new_lens.astype(np.float64)
        pairs = float(np.sum(n * P + n * (n + 1) / 2))
        return 4.0 * self.head_dim * self.num_q_heads * pairs

    def attn_bytes(self, kv_elem_bytes: int = 2) -> float:
        """Algorithmic HBM bytes of the attention kernel: K and V of every key read
        once per KV head (kv_elem_bytes per element: 2 for bf16 pools, 1 for 8-bit
        pools), Q read once and O written once (bf16)."""
        L = (self.prefix_lens + self.new_lens).astype(np.float64)
        n = self.new_lens.astype(np.float64)
        D, Hq, Hkv = self.head_dim, self.num_q_heads, self.num_kv_heads
        return float(np.sum(2.0 * kv_elem_bytes * Hkv * D * L + 4.0 * Hq * D * n))

    def append_bytes(self) -> float:
        """Algorithmic bytes of the KV append: read new K/V, write them into the pool."""
        return 8.0 * self.num_kv_heads * self.head_dim * self.total_new

    def finish(self) -> "Workload":
        """(Re)build the initial pool from the logical prefix arrays: every slot is
        NaN-poisoned, then each cached prefix page is filled, page by page."""
        S, D, Hkv, NB = self.page_size, self.head_dim, self.num_kv_heads, self.num_blocks
        kp = np.full((NB, Hkv, S, D), BF16_NAN, np.uint16)
        vp = np.full((NB, Hkv, D, S), BF16_NAN, np.uint16)
        cup = self.cu_prefix_lens
        for r in range(self.batch):
            Pr = int(self.prefix_lens[r])
            base = int(cup[r])
            for p in range((Pr + S - 1) // S):
                blk = int(self.block_tables[r, p])
                cnt = min(S, Pr - p * S)
                src_k = self.k_prefix[base + p * S: base + p * S + cnt]  # [cnt][Hkv][D]
                src_v = self.v_prefix[base + p * S: base + p * S + cnt]
                kp[blk, :, :cnt, :] = src_k.transpose(1, 0, 2)
                vp[blk, :, :, :cnt] = src_v.transpose(1, 2, 0)
        self.k_pool, self.v_pool = kp, vp
        return self

    def describe(self) -> dict:
        return {
            "workload": self.name,
            "seed": self.seed,
            "batch": self.batch,
            "num_q_heads": self.num_q_heads,
            "num_kv_heads": self.num_kv_heads,
            "head_dim": self.head_dim,
            "page_size": self.page_size,
            "total_new_tokens": self.total_new,
            "total_prefix_tokens": int(self.prefix_lens.sum()),
            "num_blocks": self.num_blocks,
        }


# --------------------------------------------------------------------------- lengths

def _lengths_for_config(k: int, rng: np.random.Generator):
    if k == 1:
        return np.array([128], np.int64), np.array([32], np.int64)
    if k == 2:
        P = rng.integers(1024, 4096, size=8, endpoint=True)
        n = rng.integers(64, 512, size=8, endpoint=True)
        return P, n
    if k == 3:
        z = rng.standard_normal(16)
        zp = rng.standard_normal(16)
        P = np.clip(np.rint(np.exp(math.log(2048.0) + 0.96 * z)), 1, 8192).astype(np.int64)
        n = np.clip(np.rint(np.exp(math.log(200.0) + 1.0 * zp)), 1, 1024).astype(np.int64)
        return P, n
    if k == 4:
        return np.full(4, 32768, np.int64), np.full(4, 128, np.int64)
    if k == 5:
        miss_n = rng.integers(512, 4096, size=16, endpoint=True)
        hit_P = rng.integers(4096, 16384, size=16, endpoint=True)
        hit_n = rng.integers(32, 256, size=16, endpoint=True)
        P = np.concatenate([np.zeros(16, np.int64), hit_P])
        n = np.concatenate([miss_n, hit_n])
        order = rng.permutation(32)
        return P[order], n[order]
    raise ValueError(f"unknown config {k}")


CONFIG_HEADS = {1: (4, 1, 64), 2: (32, 8, 128), 3: (64, 8, 128), 4: (64, 8, 128), 5: (64, 8, 128)}


# --------------------------------------------------------------------------- builder

def _draw(rng, shape, std):
    return f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32) * np.float32(std))


def build(prefix_lens, new_lens, num_q_heads, num_kv_heads, head_dim, *, seed,
          page_size=16, values="normal", name="custom", rng=None,
          extra_table_slots=1, pool_factor=2):
    """Draw one ragged batch.

    values: "normal" — Q, K, V ~ N(0,1)/sqrt(D) (the configs' recipe);
            "unit"   — Q, K, V ~ N(0,1);
            "peaked" — Q ~ 4 N(0,1), K ~ N(0,1), V ~ N(0,1)/4.
    Draw order: (lengths, drawn by the caller) → block permutation → Q → K_new →
    V_new → K_prefix → V_prefix, each request-major.
    """
    if rng is None:
        rng = np.random.default_rng(seed)
    P = np.asarray(prefix_lens, dtype=np.int64)
    n = np.asarray(new_lens, dtype=np.int64)
    B = int(P.shape[0])
    S, D, Hq, Hkv = int(page_size), int(head_dim), int(num_q_heads), int(num_kv_heads)
    L = P + n
    pages = (L + S - 1) // S
    used = int(pages.sum())
    NB = max(1, pool_factor * used)
    perm = rng.permutation(NB).astype(np.int32)
    maxb = int(pages.max()) + extra_table_slots if B > 0 else 1
    maxb = max(maxb, 1)
    unused = perm[used:] if NB > used else perm[:1]
    bt = np.empty((B, maxb), np.int32)
    off = 0
    for r in range(B):
        k = int(pages[r])
        bt[r, :k] = perm[off:off + k]
        tail = maxb - k
        if tail > 0:  # entries past the sequence point at blocks nobody owns
            bt[r, k:] = unused[np.arange(tail) % unused.shape[0]]
        off += k

    if values == "normal":
        sq = sk = sv = 1.0 / math.sqrt(D)
    elif values == "unit":
        sq = sk = sv = 1.0
    elif values == "peaked":
        sq, sk, sv = 4.0, 1.0, 0.25
    else:
        raise ValueError(values)
    T = int(n.sum())
    SP = int(P.sum())
    q = _draw(rng, (T, Hq, D), sq)
    k_new = _draw(rng, (T, Hkv, D), sk)
    v_new = _draw(rng, (T, Hkv, D), sv)
    k_prefix = _draw(rng, (SP, Hkv, D), sk)
    v_prefix = _draw(rng, (SP, Hkv, D), sv)
    return Workload(name=name, seed=int(seed), num_q_heads=Hq, num_kv_heads=Hkv,
                    head_dim=D, page_size=S, prefix_lens=P.astype(np.int32),
                    new_lens=n.astype(np.int32), block_tables=bt, num_blocks=NB,
                    q=q, k_new=k_new, v_new=v_new, k_prefix=k_prefix, v_prefix=v_prefix,
                    k_pool=None, v_pool=None, scale=1.0 / math.sqrt(D)).finish()




def e4m3_pools(w: Workload, seed: int | None = None):
    """Initial 8-bit pools for w (same shapes and slots as w.k_pool / w.v_pool,
    one byte per element): every cached prefix slot holds a random finite E4M3
    code (sign uniform, exponent field uniform in 2..10, mantissa uniform, so
    magnitudes 2^-5 .. 15 before the pool scale), every other slot the NaN
    code. Random codes rather than quantised prefix values keep the method's
    arithmetic out of this module; the new tokens' K/V stay bf16 and are
    quantised by the append under test."""
    rng = np.random.default_rng(w.seed + 8 if seed is None else seed)
    S, D, Hkv, NB = w.page_size, w.head_dim, w.num_kv_heads, w.num_blocks
    total_p = int(w.prefix_lens.sum())

    def codes():
        sign = rng.integers(0, 2, (total_p, Hkv, D)) << 7
        expo = rng.integers(2, 11, (total_p, Hkv, D)) << 3
        mant = rng.integers(0, 8, (total_p, Hkv, D))
        return (sign | expo | mant).astype(np.uint8)

    kc, vc = codes(), codes()
    kp = np.full((NB, Hkv, S, D), E4M3_NAN, np.uint8)
    vp = np.full((NB, Hkv, D, S), E4M3_NAN, np.uint8)
    cup = w.cu_prefix_lens
    for r in range(w.batch):
        Pr = int(w.prefix_lens[r])
        base = int(cup[r])
        for p in range((Pr + S - 1) // S):
            blk = int(w.block_tables[r, p])
            cnt = min(S, Pr - p * S)
            kp[blk, :, :cnt, :] = kc[base + p * S: base + p * S + cnt].transpose(1, 0, 2)
            vp[blk, :, :, :cnt] = vc[base + p * S: base + p * S + cnt].transpose(1, 2, 0)
    return kp, vp


def make_config(k: int, seed: int | None = None, values: str = "normal") -> Workload:
    """Config k (1..5): the five benchmark shapes, drawn from seed 2505239700 + k."""
    if seed is None:
        seed = SEED_BASE + k
    rng = np.random.default_rng(seed)
    P, n = _lengths_for_config(k, rng)
    Hq, Hkv, D = CONFIG_HEADS[k]
    return build(P, n, Hq, Hkv, D, seed=seed, values=values, name=CONFIG_NAMES[k], rng=rng)


def short_suffix_variant(seed: int | None = None, new_tokens: int = 16) -> Workload:
    """Long-reuse shape with a very short suffix (KV-read bound: flop/byte below the ridge)."""
    if seed is None:
        seed = SEED_BASE + 40
    return build(np.full(4, 32768), np.full(4, new_tokens), 64, 8, 128, seed=seed,
                 name=f"long_reuse_70b_n{new_tokens}")


def decode_variant(seed: int | None = None, batch: int = 32) -> Workload:
    """Decode step at the 70B shape: one new token per request over a cached context
    (prefix lengths lognormal around 4096, clipped to [256, 32768]); K/V-read bound."""
    if seed is None:
        seed = SEED_BASE + 50
    rng = np.random.default_rng(seed)
    P = np.clip(np.round(np.exp(math.log(4096) + 0.8 * rng.standard_normal(batch))), 256, 32768)
    return build(P.astype(np.int64), np.ones(batch, np.int64), 64, 8, 128, seed=seed, rng=rng,
                 name="decode_70b")


# --------------------------------------------------------------------------- structured suites
# Each modifies the logical arrays and rebuilds the pool; none computes attention.

def _logical_k(w: Workload, r: int, j: int):
    """View of logical key j of request r (prefix array or new-token array)."""
    P = int(w.prefix_lens[r])
    if j < P:
        return w.k_prefix, int(w.cu_prefix_lens[r]) + j
    return w.k_new, int(w.cu_new_lens[r]) + (j - P)


def _logical_v(w: Workload, r: int, j: int):
    P = int(w.prefix_lens[r])
    if j < P:
        return w.v_prefix, int(w.cu_prefix_lens[r]) + j
    return w.v_new, int(w.cu_new_lens[r]) + (j - P)


def plant_needles(w: Workload, positions) -> Workload:
    """Needle suite: every query gets element 0 = 16, every key element 0 = 0,
    and for each (request r, logical key j*) the key becomes (16, 0, ..., 0)."""
    w.q[:, :, 0] = f32_to_bf16_bits(np.float32(16.0))
    w.k_new[:, :, 0] = 0
    w.k_prefix[:, :, 0] = 0
    for r, j in positions:
        arr, idx = _logical_k(w, r, j)
        arr[idx, :, :] = 0
        arr[idx, :, 0] = f32_to_bf16_bits(np.float32(16.0))
    return w.finish()


def set_values_one(w: Workload) -> Workload:
    """V ≡ 1 suite."""
    w.v_new[...] = BF16_ONE
    w.v_prefix[...] = BF16_ONE
    return w.finish()


def set_position_code(w: Workload) -> Workload:
    """Q ≡ 0 and V_j[0] = j (logical key position) suite; needs L <= 256 so that
    j and j/2 are exact in bf16."""
    assert int((w.prefix_lens + w.new_lens).max(initial=0)) <= 256
    w.q[...] = 0
    for r in range(w.batch):
        L = int(w.prefix_lens[r] + w.new_lens[r])
        for j in range(L):
            arr, idx = _logical_v(w, r, j)
            arr[idx, :, 0] = f32_to_bf16_bits(np.float32(j))
    return w.finish()


# ----------------------------------------------------------------- request traces (control plane)
# Synthetic stand-ins for the paper's ShareGPT multi-turn chats and TriviaQA
# document questions (§6.1), which are not available. Each request is
# (key, context_tokens, prompt_tokens, total_tokens, turn, time) as the cache
# model of include/greencache_ctl.h defines them.

TRACE_DTYPE = np.dtype([("key", "<i8"), ("context_tokens", "<i8"), ("prompt_tokens", "<i8"),
                        ("total_tokens", "<i8"), ("turn", "<i4"), ("reserved", "<i4"), ("time", "<f8")])

# KV bytes per token of Llama-3-70B (80 layers, 8 KV heads, head_dim 128, K and V, bf16)
LLAMA3_70B_KV_BYTES_PER_TOKEN = 2 * 80 * 8 * 128 * 2


def _lognormal_int(rng, median, sigma, lo, hi, size):
    return np.clip(np.rint(median * np.exp(sigma * rng.standard_normal(size))), lo, hi).astype(np.int64)


def chat_trace(seed: int = SEED_BASE + 60, hours: float = 24.0, sessions_per_s: float = 0.4,
               mean_turns: float = 4.0, window: int = 8192, think_s: float = 3600.0) -> np.ndarray:
    """Multi-turn conversations: sessions arrive as a Poisson process; each has
    1 + Geometric turns (mean `mean_turns`); a turn adds a user prompt (lognormal,
    median 60 tokens) and a response (median 200 tokens); think time between turns
    is exponential with mean `think_s` (1 h: the conversations of a day-long trace
    are resumed later, not answered back to back). Turn k's context is everything before it; a
    session ends once its context would exceed the model's `window` (8k, §6.1)."""
    rng = np.random.default_rng(seed)
    horizon = hours * 3600.0
    n_sessions = int(rng.poisson(sessions_per_s * horizon))
    starts = np.sort(rng.uniform(0.0, horizon, n_sessions))
    rows = []
    for sid, t0 in enumerate(starts):
        turns = int(rng.geometric(1.0 / mean_turns))  # >= 1, mean `mean_turns`
        user = _lognormal_int(rng, 60, 1.0, 4, 2048, turns)
        resp = _lognormal_int(rng, 200, 0.8, 8, 2048, turns)
        gaps = rng.exponential(think_s, turns)
        ctx, t = 0, float(t0)
        for k in range(turns):
            prompt = ctx + int(user[k])
            total = prompt + int(resp[k])
            if total > window or t >= horizon:
                break
            rows.append((sid, ctx, prompt, total, k + 1, 0, t))
            ctx = total
            t += float(gaps[k])
    tr = np.array(rows, dtype=TRACE_DTYPE)
    return tr[np.argsort(tr["time"], kind="stable")]


def document_trace(seed: int = SEED_BASE + 61, hours: float = 24.0, questions_per_s: float = 1.5,
                   documents: int = 20000, alpha: float = 0.7, window: int = 8192) -> np.ndarray:
    """Document questions: `documents` documents with lognormal lengths (median
    4000 tokens, clipped to the 8k window); questions arrive as a Poisson process
    and pick a document with Zipf(alpha) popularity (the paper's alpha 0.4 and
    0.7, §6.1); the cached entry is the document (context = document length),
    the question (median 20 tokens) is not reused."""
    rng = np.random.default_rng(seed)
    horizon = hours * 3600.0
    lengths = _lognormal_int(rng, 4000, 0.5, 500, window - 64, documents)
    p = 1.0 / np.arange(1, documents + 1, dtype=np.float64) ** alpha
    p /= p.sum()
    n = int(rng.poisson(questions_per_s * horizon))
    times = np.sort(rng.uniform(0.0, horizon, n))
    docs = rng.choice(documents, size=n, p=p)
    q = _lognormal_int(rng, 20, 0.5, 4, 64, n)
    turn = np.zeros(documents, np.int64)
    tr = np.zeros(n, dtype=TRACE_DTYPE)
    for i in range(n):
        d = int(docs[i])
        turn[d] += 1
        tr[i] = (d, lengths[d], lengths[d] + q[i], lengths[d] + q[i], turn[d], 0, times[i])
    return tr


def ilp_profile(seed: int = SEED_BASE + 62, steps: int = 24, sizes_tb=tuple(range(17)),
                slo_ttft_s: float = 2.5):
    """A synthetic profile for the cache-size ILP (§5.2-5.4): per hour t, a
    request count (diurnal) and a grid carbon intensity (diurnal, gCO2e/kWh); per
    (t, size) a mean TTFT that falls with the cache's token hit rate (which grows
    with size and saturates) and rises with load, a mean power, and the numbers
    of requests meeting the TTFT and TPOT SLOs (2.5 s / 0.2 s for the 70B chat
    task, §6.1). Returns a dict of numpy arrays."""
    rng = np.random.default_rng(seed)
    t = np.arange(steps)
    rate = 1.0 + 0.8 * np.sin(2 * np.pi * (t - 8) / 24.0) + 0.1 * rng.standard_normal(steps)
    rate = np.clip(rate, 0.2, None)                                   # requests/s
    n = np.rint(rate * 3600.0).astype(np.int64)
    ci = 120.0 + 80.0 * np.cos(2 * np.pi * (t - 13) / 24.0) + 10 * rng.standard_normal(steps)
    ci = np.clip(ci, 20.0, None)
    S = np.asarray(sizes_tb, np.float64)
    hit = 0.7 * (1.0 - np.exp(-S / 6.0))                             # token hit rate vs size
    load = rate[:, None] / 1.8
    ttft = (1.2 + 2.0 * load ** 2) * (1.0 - 0.8 * hit[None, :])      # seconds
    tpot = 0.10 + 0.08 * load * (1.0 - 0.5 * hit[None, :])
    power = 1200.0 + 400.0 * load * (1.0 - 0.3 * hit[None, :])        # watts
    spread_ttft = 0.35 * ttft
    z_ttft = (slo_ttft_s - ttft) / spread_ttft
    z_tpot = (0.2 - tpot) / (0.25 * tpot)
    from math import erf
    cdf = np.vectorize(lambda z: 0.5 * (1.0 + erf(z / np.sqrt(2.0))))
    ok_ttft = np.rint(n[:, None] * cdf(z_ttft)).astype(np.int64)
    ok_tpot = np.rint(n[:, None] * cdf(z_tpot)).astype(np.int64)
    return dict(n=n, ci=ci, sizes_tb=S, ttft=ttft, power=power, ok_ttft=ok_ttft, ok_tpot=ok_tpot)
