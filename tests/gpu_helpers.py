"""Helpers of the GPU parity tests: upload a seeded workload, run the HIP path
through the C ABI, and compare with the fp64 oracle."""
from __future__ import annotations

import numpy as np

import oracle
from paper_2505_23970_amd import workloads as W

# Contract bounds on attention outputs (bf16 inputs, fp32 accumulation).
CONTRACT_MAX_ABS = 1e-2
CONTRACT_MEAN_ABS = 1e-3


def derived_bound(ref, vmax):
    """Per-element bound derived from the kernel's arithmetic: the probabilities
    enter the PV product rounded to bf16 (unit roundoff 2^-8, so at most
    2^-8 * max|v| on the output) and the output is rounded to bf16 (<= 2^-8 |o|);
    fp32 accumulation adds far less. Allow twice the sum."""
    return 2.0 ** -7 * (vmax + np.abs(ref)) + 1e-6


def to_dev_bf16(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to("cuda")


def from_dev_bits(t):
    import torch
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def from_dev_f32(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


class DeviceRun:
    """HIP path of one workload: append, then attention. Keeps device tensors."""

    def __init__(self, w: W.Workload):
        import paper_2505_23970_amd as gc
        self.w = w
        self.batch = gc.PagedBatch(w.prefix_lens, w.new_lens, w.block_tables)
        self.q = to_dev_bf16(w.q)
        self.k_new = to_dev_bf16(w.k_new)
        self.v_new = to_dev_bf16(w.v_new)
        self.k_pool = to_dev_bf16(w.k_pool)
        self.v_pool = to_dev_bf16(w.v_pool)

    def append(self):
        import paper_2505_23970_amd as gc
        gc.kv_append(self.k_new, self.v_new, self.k_pool, self.v_pool, self.batch)

    def attention(self, kv_split_tiles=None, with_lse=True, tiling=None):
        import torch
        import paper_2505_23970_amd as gc
        T, Hq, D = self.w.q.shape
        lse = torch.full((T, Hq), float("nan"), dtype=torch.float32, device="cuda") if with_lse else None
        out = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        gc.prefix_prefill_attention(self.q, self.k_pool, self.v_pool, self.batch, self.w.scale,
                                    out=out, lse=lse, kv_split_tiles=kv_split_tiles, tiling=tiling)
        torch.cuda.synchronize()
        return out, lse


def sample_rows(w: W.Workload, tokens_per_request=6, heads_per_kv=2, seed=0):
    """Rows (token * Hq + head) for a sampled oracle check: the first, second,
    middle and last two tokens of every request plus a random one, with
    `heads_per_kv` query heads of every KV head."""
    rng = np.random.default_rng(seed)
    g = w.num_q_heads // w.num_kv_heads
    cu = w.cu_new_lens
    rows = []
    for r in range(w.batch):
        n = int(w.new_lens[r])
        if n == 0:
            continue
        toks = {0, 1, n // 2, n - 2, n - 1, int(rng.integers(0, n))}
        toks = sorted(t for t in toks if 0 <= t < n)[:max(tokens_per_request, 1)]
        for t in toks:
            for kvh in range(w.num_kv_heads):
                hs = rng.choice(g, size=min(heads_per_kv, g), replace=False)
                for h in sorted(hs):
                    rows.append((int(cu[r]) + t) * w.num_q_heads + kvh * g + int(h))
    return np.array(sorted(set(rows)), np.int64)


def compare_attention(w: W.Workload, out_dev, lse_dev, ref_out, ref_lse, rows=None,
                      contract=True, vmax=None):
    """Compare GPU rows with oracle rows; returns a dict of error figures. `vmax`
    (largest value magnitude) defaults to that of the bf16 values of w."""
    T, Hq, D = w.q.shape
    got = from_dev_f32(out_dev).reshape(T * Hq, D)
    got_lse = from_dev_f32(lse_dev).reshape(T * Hq) if lse_dev is not None else None
    if rows is not None:
        got = got[rows]
        got_lse = got_lse[rows] if got_lse is not None else None
    assert not np.isnan(got).any(), "NaN in the output"
    err = np.abs(got - ref_out)
    if vmax is None:
        vmax = float(np.abs(W.bf16_bits_to_f32(np.concatenate(
            [w.v_new.ravel(), w.v_prefix.ravel()]))).max(initial=0.0))
    bound = derived_bound(ref_out, vmax)
    worst = np.unravel_index(np.argmax(err - bound), err.shape) if err.size else None
    info = {"max_abs": float(err.max(initial=0.0)), "mean_abs": float(err.mean()) if err.size else 0.0,
            "ref_max": float(np.abs(ref_out).max(initial=0.0)), "vmax": vmax}
    assert np.all(err <= bound), (
        f"derived bound exceeded at {worst}: got {got[worst]}, ref {ref_out[worst]}, info {info}")
    if contract:
        assert info["max_abs"] <= CONTRACT_MAX_ABS and info["mean_abs"] <= CONTRACT_MEAN_ABS, info
    if got_lse is not None and ref_lse is not None:
        # the kernel's normaliser is the sum of the bf16-rounded weights (the same
        # weights that enter the PV product), within a factor 1 +- 2^-8 of the exact
        # sum, so ln of it is within 2^-8; fp32 terms add ~1e-5 relative
        lerr = np.abs(got_lse - ref_lse)
        assert np.all(lerr <= 2.0 ** -8 + 1e-5 * np.abs(ref_lse)), f"lse error {lerr.max()}"
        info["lse_max_abs"] = float(lerr.max(initial=0.0))
    return info


def oracle_pools(w: W.Workload):
    return oracle.kv_append(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks,
                            w.k_new, w.v_new, w.k_pool, w.v_pool)


def oracle_rows(w: W.Workload, kp, vp, rows=None):
    return oracle.attention(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks, w.q, kp, vp,
                            w.scale, rows=rows)


# ----------------------------------------------------------------- 8-bit pools

def to_dev_u8(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, np.uint8)).to("cuda")


class DeviceRunFp8:
    """HIP path over 8-bit pools: the initial pools come from W.e4m3_pools(w)."""

    def __init__(self, w: W.Workload, k_scale, v_scale):
        import paper_2505_23970_amd as gc
        self.w, self.ks, self.vs = w, k_scale, v_scale
        self.batch = gc.PagedBatch(w.prefix_lens, w.new_lens, w.block_tables)
        self.k8_init, self.v8_init = W.e4m3_pools(w)
        self.q = to_dev_bf16(w.q)
        self.k_new = to_dev_bf16(w.k_new)
        self.v_new = to_dev_bf16(w.v_new)
        self.k_pool = to_dev_u8(self.k8_init)
        self.v_pool = to_dev_u8(self.v8_init)

    def append(self):
        import paper_2505_23970_amd as gc
        gc.kv_append_fp8(self.k_new, self.v_new, self.k_pool, self.v_pool, self.batch, self.ks, self.vs)

    def pools(self):
        return self.k_pool.cpu().numpy(), self.v_pool.cpu().numpy()

    def attention(self, kv_split_tiles=None, tiling=None):
        import torch
        import paper_2505_23970_amd as gc
        T, Hq, D = self.w.q.shape
        lse = torch.full((T, Hq), float("nan"), dtype=torch.float32, device="cuda")
        out = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        gc.prefix_prefill_attention_fp8(self.q, self.k_pool, self.v_pool, self.batch, self.w.scale,
                                        self.ks, self.vs, out=out, lse=lse,
                                        kv_split_tiles=kv_split_tiles, tiling=tiling)
        torch.cuda.synchronize()
        return out, lse


def oracle_pools_fp8(run: DeviceRunFp8):
    w = run.w
    return oracle.kv_append_e4m3(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks,
                                 w.k_new, w.v_new, run.k8_init, run.v8_init, run.ks, run.vs)


def oracle_rows_fp8(run: DeviceRunFp8, kp8, vp8, rows=None):
    w = run.w
    return oracle.attention_e4m3(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks, w.q,
                                 kp8, vp8, run.ks, run.vs, w.scale, rows=rows)


def e4m3_vmax(codes, scale):
    """Largest finite dequantised magnitude among `codes`."""
    table = np.array([abs(oracle.e4m3_value(c)) for c in range(256)], np.float64)
    vals = table[np.unique(codes)]
    return float(np.nanmax(vals)) * scale
