#!/usr/bin/env python3
"""Benchmark of the prefix-cached prefill path on one MI355X.

One step = the whole hot path over one batch already resident in HBM:
KV append of the new tokens and work-list planning in one launch
(gc_prefix_prefill_prepare), then the attention (gc_prefix_prefill_run). With
--kv fp8 the pools hold 8-bit E4M3 codes (gc_prefix_prefill_prepare_fp8 and
gc_prefix_prefill_run_fp8; products still bf16 x bf16 -> fp32). The default
workload is the largest single-GPU one: the mixed hit/miss batch at the
Llama-3-70B attention shape (64 query / 8 KV heads, head_dim 128, 32 requests:
16 misses with 512-4096 new tokens and no cached prefix, 16 hits with
4096-16384 cached tokens and 32-256 new tokens, page 16, random block
permutation), drawn from a fixed seed. The 32k-token reuse workload is timed
after it and reported under "extra".

Prints one JSON line: throughput (attention TFLOP/s over the step, and new
tokens/s), the dominant kernel's roofline figures measured with HIP events on
the launch stream, and the fp64 CPU oracle timed on a bounded sample of the
same workload on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prefix-cached prefill attn TFLOP/s + new tokens/s; % of bf16 MFMA/HBM roof"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
SAMPLE_EVERY = 5            # timed steps per step that carries timing events
COLD_STEPS = 10             # steps of the cold-cache pass after the timed region
COLD_FLUSH_MIB = 512        # scratch overwritten before each of them

# the largest single-GPU workload: 32 requests at the Llama-3-70B attention shape,
# 16 cache misses (full causal prefill of 512-4096 tokens) and 16 hits (4096-16384
# cached tokens + 32-256 new ones)
DEFAULT_WORKLOAD = "mixed_hit_miss_70b"

WORKLOADS = {
    "tiny": lambda: _cfg(1),
    "llama3_8b": lambda: _cfg(2),
    "llama3_70b_chat": lambda: _cfg(3),
    "long_reuse_70b": lambda: _cfg(4),
    "mixed_hit_miss_70b": lambda: _cfg(5),
    "long_reuse_70b_n16": lambda: _short(),
    "decode_70b": lambda: _decode(),
}


def _cfg(k):
    from paper_2505_23970_amd import workloads as W
    return W.make_config(k)


def _short():
    from paper_2505_23970_amd import workloads as W
    return W.short_suffix_variant()


def _decode():
    from paper_2505_23970_amd import workloads as W
    return W.decode_variant()


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    # The GPU raises its clocks over the first ~40 ms of sustained work after idling
    # (the 70B chat attention runs at 520 us per call cold and 355 us warm), so the
    # default warm-up is long enough to time the steady state of a serving loop.
    ap.add_argument("--warmup", type=int, default=400)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(WORKLOADS))
    ap.add_argument("--no-extra", dest="extra", action="store_false",
                    help="skip the 32k-reuse figure reported beside the default workload")
    ap.add_argument("--kv", default="bf16", choices=["bf16", "fp8"],
                    help="KV pool element type: bf16, or 8-bit E4M3 codes with one scale per pool")
    ap.add_argument("--kv-split-tiles", type=int, default=None,
                    help="override the automatic split policy (0 auto, <0 never, >0 tiles)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target duration of the CPU-oracle sample (0 disables it)")
    ap.add_argument("--restore", action="store_true",
                    help="instead of the benchmark, time restoring the workload's cached prefixes "
                         "from pinned host memory into the pool (the cache's host tier, over PCIe)")
    ap.add_argument("--control", action="store_true",
                    help="benchmark the CPU control plane instead (replacement model, ILP); no GPU")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="instead of the benchmark, run 5 plain device-to-device copies of this "
                         "many MiB (reference point that scales hardware byte counters)")
    return ap.parse_args()


def copy_reference(mib):
    import torch
    n = mib * (1 << 20)
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 5}), flush=True)


PEAK_PCIE_GBS = 64.0  # PCIe Gen5 x16, one direction, nominal


def restore_benchmark(w, steps, warmup):
    """Restore every cached prefix of the workload from pinned host memory into the pool:
    (a) the append kernel reading the host arrays directly over PCIe, (b) a DMA copy to a
    device staging buffer followed by the same kernel on device memory."""
    import torch
    import paper_2505_23970_amd as gc
    dev = torch.device("cuda")
    batch = gc.PagedBatch(w.prefix_lens, w.new_lens, w.block_tables, device=dev)
    kp = torch.from_numpy(w.k_pool.view(np.int16)).view(torch.bfloat16).to(dev)
    vp = torch.from_numpy(w.v_pool.view(np.int16)).view(torch.bfloat16).to(dev)
    kh = torch.from_numpy(w.k_prefix.view(np.int16)).view(torch.bfloat16).pin_memory()
    vh = torch.from_numpy(w.v_prefix.view(np.int16)).view(torch.bfloat16).pin_memory()
    kd, vd = torch.empty_like(kh, device=dev), torch.empty_like(vh, device=dev)
    nbytes = kh.numel() * 2 + vh.numel() * 2

    def zero_copy():
        gc.kv_restore(kh, vh, kp, vp, batch)

    def staged():
        kd.copy_(kh, non_blocking=True)
        vd.copy_(vh, non_blocking=True)
        gc.kv_restore(kd, vd, kp, vp, batch)

    res = {}
    for name, fn in (("zero_copy", zero_copy), ("dma_staged", staged)):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        res[name] = e0.elapsed_time(e1) * 1e-3 / steps
    best = min(res, key=res.get)
    rec = {"metric": "cached-KV restore GB/s (pinned host memory -> paged pool)",
           "value": nbytes / res[best] / 1e9, "unit": "GB/s", "higher_is_better": True,
           "path": best, "bytes": nbytes, "steps": steps, "warmup": warmup,
           "ms": {k: v * 1e3 for k, v in res.items()},
           "gbs": {k: nbytes / v / 1e9 for k, v in res.items()},
           "roofline": {"bound": "pcie", "achieved": nbytes / res[best] / 1e9, "peak": PEAK_PCIE_GBS,
                        "unit": "GB/s", "frac": nbytes / res[best] / 1e9 / PEAK_PCIE_GBS},
           "config": {"workload": w.name, "total_prefix_tokens": int(w.prefix_lens.sum())},
           "data": "synthetic"}
    print(json.dumps(rec), flush=True)


# Pool scales of the 8-bit runs (the pool generator's codes have magnitudes 2^-5 .. 15).
K_SCALE_FP8 = 2.0 ** -6
V_SCALE_FP8 = 0.0213


def auto_kernel_name(w, cus, fp8):
    """Kernel the library's automatic tiling picks for w, named as in the kernel trace
    (the rule of choose_tiling and resident_workgroups in the C ABI, restated: small
    tiles when every request has n * g <= 16, else wide tiles when 256-row tiles are
    >= 85 % full and their grid is not between one and two per compute unit, run as a
    resident launch from two rounds of work items on, else 128-row tiles)."""
    g = w.num_q_heads // w.num_kv_heads
    D = w.head_dim
    f = "true" if fp8 else "false"
    split = " (+ split merge when the plan splits)"
    if g <= 16 and int(w.new_lens.max()) * g <= 16:
        return f"attention_small_kernel<{D}, {f}>" + split
    tq = 256 // g
    units = int(sum((int(n) + tq - 1) // tq for n in w.new_lens))
    rows = int(w.new_lens.sum()) * g
    grid = units * w.num_kv_heads
    wide = rows * 100 >= units * 256 * 85 and not (cus < grid < 2 * cus)
    if wide and cus % 8 == 0 and wide_items(w, cus) * w.num_kv_heads >= 2 * cus:
        # resident launch: one workgroup per CU taking the items from per-XCD queues
        return f"attention_resident_kernel<{D}, {f}>" + split
    return f"attention_kernel<{D}, {8 if wide else 4}, {f}>" + split


def wide_items(w, cus):
    """Work items per KV head of the wide tiling (query tiles of 256 rows, cut into key
    chunks when they do not fill one workgroup per compute unit: the split rule of
    choose_chunk in the C ABI, restated)."""
    g = w.num_q_heads // w.num_kv_heads
    tq = 256 // g
    tiles = []
    for P, n in zip(w.prefix_lens, w.new_lens):
        for q0 in range(0, int(n), tq):
            ntok = min(tq, int(n) - q0)
            tiles.append((int(P) + q0 + ntok + 63) // 64)
    units = len(tiles) * w.num_kv_heads
    if units == 0 or units >= cus:
        return len(tiles)
    chunk = max((sum(tiles) * w.num_kv_heads + cus - 1) // cus, 512 // 64)
    return sum(1 if kt <= chunk else (kt + chunk - 1) // chunk for kt in tiles)


def measured_read_gbs(mib=4096, reps=5):
    """Sustained HBM read rate on this GPU: the library's streaming-read probe over
    a 4 GiB buffer, timed with HIP events. The nominal 8 TB/s is not reachable by
    a read stream; memory-bound results are also reported against this rate."""
    import torch
    import paper_2505_23970_amd as gc
    x = torch.ones(mib * (1 << 20), dtype=torch.uint8, device="cuda")
    sink = gc.read_bandwidth_probe(x)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        gc.read_bandwidth_probe(x, sink)
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) * 1e-3 / reps
    del x, sink
    return mib * (1 << 20) / t / 1e9


def measured_mfma_tflops(iterations=4000, reps=5):
    """Sustained bf16 MFMA rate on this GPU: the library's matrix-core probe (a
    register-only loop of independent 32x32x16 products on every SIMD), timed with
    HIP events. The nominal 2.5 PFLOP/s assumes the peak clock; compute-bound
    results are also reported against this rate."""
    import torch
    import paper_2505_23970_amd as gc
    sink = gc.mfma_peak_probe(iterations)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        gc.mfma_peak_probe(iterations, sink)
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) * 1e-3 / reps
    flops = iterations * gc.MFMA_PROBE_PRODUCTS_PER_ITERATION * gc.MFMA_PROBE_FLOPS_PER_PRODUCT
    return flops / t / 1e12


def traffic_sources(kernel_source):
    """Sources that decide an attention launch's memory traffic: the file that launches
    the kernel (with the kernel's own file where that is another), the planner that
    orders its work items, the host policy that picks the tiling, key split and order,
    the shared definitions and the build script (its flags)."""
    csrc = "paper_2505_23970_amd/csrc/"
    own = [kernel_source]
    if kernel_source in (csrc + "attention.hip", csrc + "attention_plain.hip"):
        own.append(csrc + "attention_kernels.h")
    return own + [csrc + "plan_body.h", csrc + "api.hip", csrc + "gc_internal.h", "paper_2505_23970_amd/build.py"]


def code_text(text):
    """A C/C++/HIP source without its comments, whitespace runs collapsed to one space
    (string and character literals kept as they are)."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        elif c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def code_sha256_16(paths):
    """First 16 hex digits of the SHA-256 of the files' code (code_text), in order: a
    comment-only edit keeps it, any change to the code changes it."""
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), encoding="utf-8") as f:
            h.update(code_text(f.read()).encode())
        h.update(b"\0")
    return h.hexdigest()[:16]


def profiled_traffic(workload):
    """HBM bytes per attention launch from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    summary of this workload, if it was taken on the current code of the profiled kernel
    and its planner (comments aside); else None."""
    path = os.path.join(ROOT, "profiles", f"attention_{workload}.md")
    if not os.path.exists(path):
        return None
    rec = None
    with open(path) as f:
        for line in f:
            if line.startswith("traffic-json:"):
                rec = json.loads(line.split(":", 1)[1])
    if rec is None or not rec.get("kernel_sources"):
        return None
    srcs = rec["kernel_sources"]
    if not all(os.path.exists(os.path.join(ROOT, p)) for p in srcs):
        return None
    return rec["traffic_bytes"] if rec.get("code_sha256_16") == code_sha256_16(srcs) else None


def cpu_oracle_baseline(w, target_s, fp8=None):
    """Time the fp64 oracle on a bounded sample of the workload's output rows.
    fp8 = (k_pool8, v_pool8, k_scale, v_scale) times the 8-bit-pool oracle."""
    import oracle
    if fp8 is None:
        kp, vp = oracle.kv_append(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks,
                                  w.k_new, w.v_new, w.k_pool, w.v_pool)
    else:
        k8, v8, ks, vs = fp8
        kp, vp = oracle.kv_append_e4m3(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks,
                                       w.k_new, w.v_new, k8, v8, ks, vs)
    T, Hq, D = w.q.shape
    cu = w.cu_new_lens
    req = np.repeat(np.arange(w.batch), w.new_lens)
    pos = w.prefix_lens[req] + (np.arange(T) - cu[req])        # logical position per token
    keys_per_token = pos.astype(np.float64) + 1.0
    rng = np.random.default_rng(12345)
    order = rng.permutation(T * Hq)
    threads = oracle.max_threads()

    def timed(rows):
        t0 = time.perf_counter()
        if fp8 is None:
            oracle.attention(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks, w.q, kp, vp,
                             w.scale, rows=rows)
        else:
            oracle.attention_e4m3(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks, w.q, kp,
                                  vp, fp8[2], fp8[3], w.scale, rows=rows)
        return time.perf_counter() - t0

    # calibrate on a small slice, then size the sample to about target_s seconds
    n_cal = min(len(order), max(64, threads * 8))
    cal = np.sort(order[:n_cal])
    t_cal = max(timed(cal), 1e-6)
    n_rows = int(min(len(order), max(n_cal, n_cal * target_s / t_cal)))
    rows = np.sort(order[:n_rows])
    t = timed(rows)
    flops = float(np.sum(4.0 * D * keys_per_token[rows // Hq]))
    sample = (f"{n_rows} of {T * Hq} output rows (token, query head) drawn uniformly at random; "
              f"fp64 oracle{' over 8-bit pools' if fp8 is not None else ''}, append excluded")
    return {"value": flops / t / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": sample, "seconds": t,
            "new_tokens_per_s_equiv": (n_rows / Hq) / t}


def control_benchmark(cpu_seconds):
    """The cache's control plane on synthetic day-long traces (§6.3.2 replacement
    comparison, §5.4.1 ILP): token hit rates by policy and size, replay throughput
    of the native replacement model, and the hourly cache-size decision."""
    from paper_2505_23970_amd import control as K
    from paper_2505_23970_amd import workloads as W
    bpt = W.LLAMA3_70B_KV_BYTES_PER_TOKEN
    traces = {"chat": W.chat_trace(), "doc_alpha0.4": W.document_trace(alpha=0.4),
              "doc_alpha0.7": W.document_trace(alpha=0.7)}
    sizes = (1, 2, 4, 8, 16)
    table = {}
    for name, tr in traces.items():
        pols = ("fifo", "lru", "lcs", "lcs_multiturn") if name == "chat" else ("fifo", "lru", "lcs")
        table[name] = {p: {str(tb): round(K.token_hit_rate(p, tb * 10**12, bpt, tr), 4) for tb in sizes}
                       for p in pols}
    # what drives LCS below LRU on the chat trace: the think time between turns (mean
    # 60 s .. 1 h) changes how far apart a conversation's turns fall, not the order
    think = {}
    for think_s in (60.0, 300.0, 900.0, 3600.0):
        trt = W.chat_trace(think_s=think_s)
        think[f"{think_s:g}s"] = {p: {str(tb): round(K.token_hit_rate(p, tb * 10**12, bpt, trt), 4)
                                      for tb in (1, 4)} for p in ("lru", "lcs")}
    tr = traces["chat"]
    t0 = time.perf_counter()
    c = K.Cache("lcs", 4 * 10**12, bpt)
    c.replay(tr)
    dt = time.perf_counter() - t0
    value = len(tr) / dt
    base = W.ilp_profile()
    N = int(base["n"].sum())
    ilp = {"steps": int(len(base["n"])), "sizes_tb": [int(x) for x in base["sizes_tb"]], "rho": 0.9}
    # the synthetic grid's intensity as drawn, and scaled to a quarter (a low-carbon grid)
    for attribution, ci_scale in (("ttft", 1.0), ("interval", 1.0), ("interval", 0.25)):
        prof = dict(base, ci=base["ci"] * ci_scale)
        cost = K.profile_costs(prof, cache_attribution=attribution)
        t0 = time.perf_counter()
        best, choice = K.solve_cache_sizes(cost, prof["ok_ttft"], prof["ok_tpot"], N, 0.9)
        t_ilp = time.perf_counter() - t0

        def fixed(s):
            ok = (prof["ok_ttft"][:, s].sum() >= 0.9 * N) and (prof["ok_tpot"][:, s].sum() >= 0.9 * N)
            return float(cost[:, s].sum()), bool(ok)
        full_g, full_ok = fixed(len(prof["sizes_tb"]) - 1)
        none_g, none_ok = fixed(0)
        ilp[f"{attribution}_ci_x{ci_scale:g}"] = {"solve_s": t_ilp,
                            "choice_tb": [int(prof["sizes_tb"][s]) for s in choice] if choice else None,
                            "carbon_g": best, "full_cache_g": full_g, "full_cache_meets_slo": full_ok,
                            "no_cache_g": none_g, "no_cache_meets_slo": none_ok}
    rec = {
        "metric": "control plane: replacement-model requests/s (LCS, 4 TB, chat trace); token hit rates; ILP",
        "value": value, "unit": "requests/s", "n_gpus": 0, "higher_is_better": True,
        "data": "synthetic", "config": {"workload": "chat_trace 24 h (Llama-3-70B KV, 320 KiB/token)",
                                        "requests": int(len(tr)), "policy": "lcs", "capacity_tb": 4},
        "token_hit_rate": table,
        "chat_think_time_sweep": think,
        "ilp": ilp,
    }
    if cpu_seconds > 0:
        import oracle.control as OC
        rows = [(int(r["key"]), int(r["context_tokens"]), int(r["prompt_tokens"]), int(r["total_tokens"]),
                 int(r["turn"]), float(r["time"])) for r in tr]
        oc = OC.Cache(OC.LCS, 4 * 10**12, bpt)
        t0 = time.perf_counter()
        n = 0
        while n < len(rows) and time.perf_counter() - t0 < cpu_seconds:
            oc.access(*rows[n])
            n += 1
        dt = time.perf_counter() - t0
        rec["cpu_baseline"] = {"value": n / dt, "unit": "requests/s", "cores": 1, "kind": "oracle",
                               "sample": f"first {n} of {len(rows)} requests of the same trace and cache"}
    print(json.dumps(rec), flush=True)


def main():
    args = parse()
    if args.control:
        control_benchmark(args.cpu_seconds)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(this path has no multi-GPU mode)", file=sys.stderr)
        sys.exit(2)
    if args.copy_mib > 0:
        copy_reference(args.copy_mib)
        return
    import torch
    import paper_2505_23970_amd as gc

    gc.load_library()
    w = WORKLOADS[args.workload]()
    if args.restore:
        restore_benchmark(w, max(args.steps // 10, 5), min(args.warmup, 5))
        return
    fp8 = args.kv == "fp8"
    m = measure(w, args.steps, args.warmup, fp8, args.kv_split_tiles)
    rec = {
        "metric": METRIC,
        "value": m["value"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": m["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        **{k: v for k, v in m.items() if k not in ("value", "ms_per_step")},
    }
    if args.workload == DEFAULT_WORKLOAD and args.extra:
        # the 32k-token reuse workload (4 requests, 128 new tokens each), the long-prefix
        # case, timed the same way right after; reported beside the headline, not instead
        x = measure(WORKLOADS["long_reuse_70b"](), args.steps, args.warmup, fp8, None)
        rec["extra"] = {"long_reuse_70b": {k: x[k] for k in ("value", "ms_per_step", "config", "new_tokens_per_s",
                                                              "attention_tflops", "kernel_ms", "roofline")}}
    if args.cpu_seconds > 0:
        rec["cpu_baseline"] = cpu_oracle_baseline(
            w, args.cpu_seconds, (m["_k8"], m["_v8"], K_SCALE_FP8, V_SCALE_FP8) if fp8 else None)
    else:
        rec["cpu_baseline"] = None
    rec.pop("_k8", None)
    rec.pop("_v8", None)
    print(json.dumps(rec), flush=True)


def ramp_clocks(seconds=0.25):
    """Untimed: run the matrix-core probe for a fraction of a second before a workload's
    warm-up. An idle GPU (it idles while the host draws and uploads a workload) raises its
    clocks over the first ~40 ms of sustained work, which would otherwise fall into the
    first warm-up steps (all of them, with few warm-up steps of a short workload); a
    serving loop runs in the steady state."""
    import torch
    import paper_2505_23970_amd as gc
    sink = gc.mfma_peak_probe(1)
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        gc.mfma_peak_probe(2000, sink)
        torch.cuda.synchronize()


def measure(w, steps, warmup, fp8, kv_split_tiles):
    """One workload: `warmup` untimed steps, then exactly `steps` timed steps (host clock
    around the stream, synchronised on both sides), attention launches bracketed by HIP
    events on every SAMPLE_EVERY-th step, the append-and-plan launch from a short pass
    after, and a cold-cache pass."""
    import torch
    import paper_2505_23970_amd as gc
    F = w.flops()
    T, Hq, D = w.q.shape
    dev = torch.device("cuda")

    def up(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    batch = gc.PagedBatch(w.prefix_lens, w.new_lens, w.block_tables, device=dev)
    q, k_new, v_new = up(w.q), up(w.k_new), up(w.v_new)
    k8 = v8 = None
    if fp8:
        from paper_2505_23970_amd import workloads as W
        k8, v8 = W.e4m3_pools(w)
        k_pool = torch.from_numpy(k8).to(dev)
        v_pool = torch.from_numpy(v8).to(dev)
    else:
        k_pool, v_pool = up(w.k_pool), up(w.v_pool)
    out = torch.empty_like(q)
    ws = gc.alloc_workspace(Hq, k_pool, v_pool, batch, kv_split_tiles)
    torch.cuda.synchronize()
    # the GPU idled while this workload was drawn and uploaded: bring its clocks back up
    # before the warm-up steps
    ramp_clocks()

    def step(ev=None):
        # append and plan in one launch, then the attention
        if ev is not None and ev[0] is not None:
            ev[0].record()
        if fp8:
            gc.prepare(k_new, v_new, k_pool, v_pool, batch, Hq, ws, kv_split_tiles,
                       k_scale=K_SCALE_FP8, v_scale=V_SCALE_FP8)
        else:
            gc.prepare(k_new, v_new, k_pool, v_pool, batch, Hq, ws, kv_split_tiles)
        if ev is not None:
            ev[1].record()
        if fp8:
            gc.run_fp8(q, k_pool, v_pool, batch, w.scale, K_SCALE_FP8, V_SCALE_FP8, ws, out=out,
                       kv_split_tiles=kv_split_tiles)
        else:
            gc.run(q, k_pool, v_pool, batch, w.scale, ws, out=out, kv_split_tiles=kv_split_tiles)
        if ev is not None:
            ev[2].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()

    # timed region: exactly `steps` steps, host clock around the stream. Every
    # SAMPLE_EVERY-th step brackets its attention launch with two timing events on the
    # launch stream (each event record costs a few microseconds of GPU time, so events
    # on every step would inflate the step time the wall clock measures).
    sampled = list(range(0, steps, SAMPLE_EVERY))
    evs = {i: [None] + [torch.cuda.Event(enable_timing=True) for _ in range(2)] for i in sampled}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(evs.get(i))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / steps
    att = np.array([evs[i][1].elapsed_time(evs[i][2]) for i in sampled])
    # the append-and-plan half, from a short pass after the timed region with events
    # before and after each of the two launches
    pev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(len(sampled))]
    for e in pev:
        step(e)
    torch.cuda.synchronize()
    prep = np.array([e[0].elapsed_time(e[1]) for e in pev])
    # cold caches: before each of a few steps, stream-read a scratch buffer twice the
    # size of the 256 MB infinity cache (and of the L2s), so the step reads K/V from HBM
    # as a layer of a real model would (its K/V evicted by the other layers in between);
    # a read, not a write, so that no dirty lines are written back during the step. The
    # events bracket the attention launch only.
    scratch = torch.ones(COLD_FLUSH_MIB << 20, dtype=torch.uint8, device=dev)
    sink = gc.read_bandwidth_probe(scratch)
    cev = [[None] + [torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(COLD_STEPS)]
    for e in cev:
        gc.read_bandwidth_probe(scratch, sink)
        step(e)
    torch.cuda.synchronize()
    cold = np.array([e[1].elapsed_time(e[2]) for e in cev])
    del scratch, sink
    t_att = float(np.mean(att)) * 1e-3

    achieved = F / t_att / 1e12
    kernel_name = auto_kernel_name(w, torch.cuda.get_device_properties(0).multi_processor_count, fp8)
    A = w.attn_bytes(1 if fp8 else 2)
    # the binding roof follows the workload's arithmetic intensity (flop per algorithmic byte)
    ridge = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
    hbm_bound = F / A < ridge
    if hbm_bound:
        roof = {"bound": "hbm", "achieved": A / t_att / 1e9, "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    if hbm_bound:
        meas = measured_read_gbs()
        roof["measured_read_gbs"] = meas
        roof["frac_of_measured"] = roof["achieved"] / meas
    else:
        meas = measured_mfma_tflops()
        roof["measured_mfma_tflops"] = meas
        roof["frac_of_measured"] = roof["achieved"] / meas
    res = {
        "value": F / (ms_step * 1e-3) / 1e12,
        "ms_per_step": ms_step,
        "config": {"workload": w.name, **{k: v for k, v in w.describe().items() if k != "workload"},
                   "kv_split_tiles": kv_split_tiles,
                   "kv_pool": ({"type": "e4m3", "k_scale": K_SCALE_FP8, "v_scale": V_SCALE_FP8}
                               if fp8 else {"type": "bf16"})},
        "new_tokens_per_s": T / (ms_step * 1e-3),
        "attention_tflops": achieved,
        "kernel_ms": {"sampled_steps": len(sampled),
                      "append_and_plan": float(np.mean(prep)),
                      "attention": float(np.mean(att)),
                      "attention_p10": float(np.percentile(att, 10)),
                      "attention_p90": float(np.percentile(att, 90)),
                      "attention_cold": float(np.mean(cold)),
                      "cold_note": f"attention launch after stream-reading {COLD_FLUSH_MIB} MiB (infinity cache "
                                   f"and L2 evicted), {COLD_STEPS} steps after the timed region"},
        "algorithmic": {"flops": F, "attn_bytes": A, "append_bytes": w.append_bytes()},
        "roofline": {**roof,
                     "traffic": profiled_traffic(w.name + ("_fp8" if fp8 else "")),
                     "kernel": kernel_name,
                     "arithmetic_intensity": F / A,
                     "mfma_frac": achieved / PEAK_BF16_TFLOPS,
                     "cold_tflops": F / (float(np.mean(cold)) * 1e-3) / 1e12,
                     "hbm_gbs_algorithmic": A / t_att / 1e9},
        "_k8": k8, "_v8": v8,
    }
    del q, k_new, v_new, k_pool, v_pool, out, ws, batch
    torch.cuda.empty_cache()
    return res


if __name__ == "__main__":
    main()
