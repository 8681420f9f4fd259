"""The no-allocation entry point (gc_prefix_prefill_attention_noalloc) through the C
ABI against gc_prefix_prefill_attention with a caller workspace (GPU): two calls in a
row on the library's static scratch, the second with a smaller batch, each bitwise
equal to the workspace call (same kernels and plan, results independent of the
scratch's earlier contents) and within the derived bound of the fp64 oracle."""
import sys

import numpy as np
import pytest

import gpu_helpers as H
from paper_2505_23970_amd import workloads as W

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def bits(t):
    import torch
    return t.view(torch.int16 if t.element_size() == 2 else torch.int32).cpu().numpy()


def one_case(w, split, rows=None):
    import torch
    import paper_2505_23970_amd as gc
    say(f"no-alloc case {w.name}: B={w.batch} T={w.total_new} split={split}")
    run = H.DeviceRun(w)
    run.append()
    T, Hq, D = w.q.shape
    out_a, lse_a = run.attention(kv_split_tiles=split)
    out_b = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse_b = torch.full((T, Hq), float("nan"), dtype=torch.float32, device="cuda")
    ws_bytes = gc.workspace_size(Hq, run.k_pool, run.v_pool, run.batch, kv_split_tiles=split)
    assert ws_bytes <= gc.NOALLOC_SCRATCH_BYTES
    gc.prefix_prefill_attention_noalloc(run.q, run.k_pool, run.v_pool, run.batch, w.scale, out=out_b, lse=lse_b,
                                        kv_split_tiles=split)
    torch.cuda.synchronize()
    assert np.array_equal(bits(out_a), bits(out_b))
    assert np.array_equal(bits(lse_a), bits(lse_b))
    kp, vp = H.oracle_pools(w)
    ref, ref_lse = H.oracle_rows(w, kp, vp, rows=rows)
    H.compare_attention(w, out_b, lse_b, ref, ref_lse, rows=rows)


@pytest.mark.parametrize("split", [None, 2])
def test_noalloc_two_calls_second_smaller(split):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    big = W.build([300, 1000, 33, 0, 517], [77, 20, 130, 45, 260], 16, 2, 128, seed=400, name="noalloc_big")
    small = W.build([40, 7], [9, 30], 16, 2, 128, seed=401, name="noalloc_small")
    one_case(big, split)
    one_case(small, split)


def test_noalloc_resident_launch_two_calls_second_smaller():
    """Batches large enough for the resident wide-tile launch (its work queues live in
    the static scratch too): two calls, the second smaller, each bitwise equal to the
    workspace call; sampled rows against the oracle."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    big = W.build([0, 0, 0, 0, 2000, 3000], [1024, 1024, 1024, 1024, 200, 100], 64, 8, 128, seed=403,
                  name="noalloc_resident_big")
    small = W.build([0, 0, 0, 1500], [1024, 1024, 1024, 100], 64, 8, 128, seed=404, name="noalloc_resident_small")
    one_case(big, None, rows=H.sample_rows(big, seed=61))
    one_case(small, None, rows=H.sample_rows(small, seed=62))


def test_noalloc_rejects_a_batch_beyond_its_scratch():
    """A plan whose workspace exceeds the static scratch is refused before anything is
    enqueued (the output keeps its sentinels)."""
    import torch
    import paper_2505_23970_amd as gc
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    # one 128-row query tile split into 1-tile chunks over a 300k-key prefix: ~4700
    # partial slots of 64 KiB per KV head, far above the scratch
    w = W.build([300_000], [16], 8, 1, 128, seed=402, name="noalloc_too_big")
    run = H.DeviceRun(w)
    need = gc.workspace_size(8, run.k_pool, run.v_pool, run.batch, kv_split_tiles=1)
    assert need > gc.NOALLOC_SCRATCH_BYTES
    out = torch.full(tuple(w.q.shape), float("nan"), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(gc.GcError) as e:
        gc.prefix_prefill_attention_noalloc(run.q, run.k_pool, run.v_pool, run.batch, w.scale, out=out,
                                            kv_split_tiles=1)
    assert e.value.status == -5
    torch.cuda.synchronize()
    assert torch.isnan(out.float()).all().item()
