"""Resident attention launch (GPU): wide tiles (bf16 or 8-bit pools) with at least two
rounds of work items per compute unit run as one workgroup per CU taking items from per-XCD
ticket queues in the workspace. The queues must start empty after every plan and be
left empty by every run, whatever the workspace held before."""
import sys

import numpy as np
import pytest

import gpu_helpers as H
from paper_2505_23970_amd import workloads as W

pytestmark = pytest.mark.gpu

QUEUE_BYTES = (64, 64 + 4 * 9)  # byte range of the ticket counters in the workspace


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu_ready():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2505_23970_amd as gc
    gc.load_library()


def resident_batch(seed, D=128):
    # 64 q / 8 kv heads: wide tiles of 32 tokens; 4 misses of 1024 tokens and two hits
    # give 139 work items per KV head, 1112 workgroups: more than two per CU
    return W.build([0, 0, 0, 0, 2000, 3000], [1024, 1024, 1024, 1024, 200, 100], 64, 8, D,
                   seed=seed, name=f"resident_{seed}_d{D}")


@pytest.mark.parametrize("D", [64, 128])
def test_resident_runs_repeat_bitwise_and_match_the_oracle(D):
    import torch
    import paper_2505_23970_amd as gc
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    w = resident_batch(301, D)
    items = sum(-(-int(n) // 32) for n in w.new_lens)
    if cus % 8 != 0 or items * w.num_kv_heads < 2 * cus:
        pytest.skip(f"{items * w.num_kv_heads} workgroups do not make two rounds on {cus} CUs")
    say(f"case {w.name}: {items} items per KV head, {cus} CUs")
    kp_ref, vp_ref = H.oracle_pools(w)
    run = H.DeviceRun(w)
    run.append()
    T, Hq, _ = w.q.shape
    ws = gc.alloc_workspace(Hq, run.k_pool, run.v_pool, run.batch)
    ws[QUEUE_BYTES[0]:QUEUE_BYTES[1]] = 0x7F  # left-over counters: the plan must clear them
    gc.plan(Hq, run.k_pool, run.v_pool, run.batch, ws)
    outs, lses = [], []
    for _ in range(3):
        out = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((T, Hq), float("nan"), dtype=torch.float32, device="cuda")
        gc.run(run.q, run.k_pool, run.v_pool, run.batch, w.scale, ws, out=out, lse=lse)
        torch.cuda.synchronize()
        outs.append(H.from_dev_bits(out))
        lses.append(lse.cpu().numpy())
        assert not ws[QUEUE_BYTES[0]:QUEUE_BYTES[1]].any().item(), "the run left its ticket counters set"
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])
    assert np.array_equal(lses[0].view(np.uint32), lses[2].view(np.uint32))
    rows = H.sample_rows(w, seed=31)
    ref_out, ref_lse = H.oracle_rows(w, kp_ref, vp_ref, rows=rows)
    info = H.compare_attention(w, out, lse, ref_out, ref_lse, rows=rows, contract=True)
    say(f"resident launch, three runs bitwise equal; oracle rows: {info}")


def test_resident_runs_on_two_workspaces_interleaved():
    """Two batches planned into two workspaces and run alternately on one stream: each
    run uses its own workspace's queues and matches the oracle."""
    import torch
    import paper_2505_23970_amd as gc
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    runs = []
    for seed in (302, 303):
        w = resident_batch(seed)
        r = H.DeviceRun(w)
        r.append()
        ws = gc.alloc_workspace(w.num_q_heads, r.k_pool, r.v_pool, r.batch)
        gc.plan(w.num_q_heads, r.k_pool, r.v_pool, r.batch, ws)
        runs.append((w, r, ws))
    items = sum(-(-int(n) // 32) for n in runs[0][0].new_lens)
    if cus % 8 != 0 or items * 8 < 2 * cus:
        pytest.skip("not a resident launch on this GPU")
    outs = {}
    for rep in range(2):
        for k, (w, r, ws) in enumerate(runs):
            T, Hq, D = w.q.shape
            out = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
            gc.run(r.q, r.k_pool, r.v_pool, r.batch, w.scale, ws, out=out)
            torch.cuda.synchronize()
            if rep == 0:
                outs[k] = H.from_dev_bits(out)
            else:
                assert np.array_equal(outs[k], H.from_dev_bits(out))
    for k, (w, r, ws) in enumerate(runs):
        kp_ref, vp_ref = H.oracle_pools(w)
        rows = H.sample_rows(w, seed=40 + k)
        ref_out, ref_lse = H.oracle_rows(w, kp_ref, vp_ref, rows=rows)
        out = torch.from_numpy(outs[k].view(np.int16)).view(torch.bfloat16)
        info = H.compare_attention(w, out, None, ref_out, None, rows=rows, contract=True)
        say(f"workspace {k}: {info}")


@pytest.mark.parametrize("D", [64, 128])
def test_resident_launch_over_8bit_pools(D):
    """The resident launch over 8-bit pools (each head dimension its own kernel
    instance): two runs on one plan bitwise equal, sampled rows against the oracle's
    dequantised attention."""
    import torch
    import paper_2505_23970_amd as gc
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    w = W.build([0, 0, 0, 0, 2000, 3000], [1024, 1024, 1024, 1024, 200, 100], 64, 8, D,
                seed=310 + D, name=f"resident_fp8_d{D}")
    items = sum(-(-int(n) // 32) for n in w.new_lens)
    if cus % 8 != 0 or items * w.num_kv_heads < 2 * cus:
        pytest.skip("not a resident launch on this GPU")
    ks, vs = 2.0 ** -6, 0.0213
    say(f"case {w.name}: 8-bit pools, {items} items per KV head")
    run = H.DeviceRunFp8(w, ks, vs)
    run.append()
    kref, vref = H.oracle_pools_fp8(run)
    T, Hq, _ = w.q.shape
    ws = gc.alloc_workspace(Hq, run.k_pool, run.v_pool, run.batch)
    gc.plan(Hq, run.k_pool, run.v_pool, run.batch, ws)
    outs = []
    for _ in range(2):
        out = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((T, Hq), float("nan"), dtype=torch.float32, device="cuda")
        gc.run_fp8(run.q, run.k_pool, run.v_pool, run.batch, w.scale, ks, vs, ws, out=out, lse=lse)
        torch.cuda.synchronize()
        outs.append(H.from_dev_bits(out))
        assert not ws[QUEUE_BYTES[0]:QUEUE_BYTES[1]].any().item()
    assert np.array_equal(outs[0], outs[1])
    rows = H.sample_rows(w, seed=50 + D)
    ref_out, ref_lse = H.oracle_rows_fp8(run, kref, vref, rows=rows)
    info = H.compare_attention(w, out, lse, ref_out, ref_lse, rows=rows, contract=True,
                               vmax=H.e4m3_vmax(vref, vs))
    say(f"8-bit resident launch, d {D}: {info}")
