"""HIP path vs. the fp64 oracle, element by element, through the C ABI (GPU)."""
import sys

import numpy as np
import pytest

import gpu_helpers as H
from paper_2505_23970_amd import workloads as W

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu_ready():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2505_23970_amd as gc
    gc.load_library()  # raises if the HIP library is missing: there is no other path


def check_pool(run: H.DeviceRun, kp_ref, vp_ref):
    kp = H.from_dev_bits(run.k_pool)
    vp = H.from_dev_bits(run.v_pool)
    assert np.array_equal(kp, kp_ref), f"k_pool differs at {np.argwhere(kp != kp_ref)[:5]}"
    assert np.array_equal(vp, vp_ref), f"v_pool differs at {np.argwhere(vp != vp_ref)[:5]}"


def full_check(w, kv_split_tiles=None, rows=None, contract=False, tiling=None):
    """Append + attention on the GPU vs. the oracle. `contract` adds the fixed
    max/mean absolute bounds, which are stated for the configs' value scale."""
    say(f"case {w.name}: B={w.batch} Hq={w.num_q_heads} Hkv={w.num_kv_heads} D={w.head_dim} "
        f"T={w.total_new} split={kv_split_tiles} tiling={tiling}")
    kp_ref, vp_ref = H.oracle_pools(w)
    run = H.DeviceRun(w)
    run.append()
    check_pool(run, kp_ref, vp_ref)
    out, lse = run.attention(kv_split_tiles=kv_split_tiles, tiling=tiling)
    ref_out, ref_lse = H.oracle_rows(w, kp_ref, vp_ref, rows=rows)
    return H.compare_attention(w, out, lse, ref_out, ref_lse, rows=rows, contract=contract), run, out


# ----------------------------------------------------------------- the five workloads

@pytest.mark.timeout(900)
@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_config_all_rows(k):
    """Every output row of the five workloads (and the whole pool after the append)
    against the fp64 oracle, in the tiling and split the automatic plan picks, which
    is what the benchmark times."""
    w = W.make_config(k)
    info, _, _ = full_check(w, contract=True)
    say(f"config {k}: {w.total_new * w.num_q_heads} rows {info}")


def test_decode_workload_sampled():
    w = W.decode_variant()
    info, _, _ = full_check(w, rows=H.sample_rows(w, seed=50), contract=True)
    say(f"decode, 32 requests: {info}")


def test_short_suffix_variant_sampled():
    w = W.short_suffix_variant()
    info, _, _ = full_check(w, rows=H.sample_rows(w, seed=40), contract=True)
    say(f"long reuse, 16 new tokens: {info}")


# ----------------------------------------------------------------- supplementary suites

SUITE_SHAPE = dict(prefix_lens=[300, 1000, 33, 0], new_lens=[77, 20, 130, 45],
                   num_q_heads=16, num_kv_heads=2, head_dim=128)


@pytest.mark.parametrize("values", ["unit", "peaked"])
@pytest.mark.parametrize("split", [None, 2])
def test_value_scales(values, split):
    w = W.build(seed=100, values=values, name=f"suite_{values}", **SUITE_SHAPE)
    full_check(w, kv_split_tiles=split)


@pytest.mark.parametrize("values", ["unit", "peaked"])
@pytest.mark.parametrize("split", [None, 2])
def test_wide_tiles(values, split):
    """256-row work items (8 wavefronts per workgroup) on the supplementary suite."""
    import paper_2505_23970_amd as gc
    w = W.build(seed=102, values=values, name=f"wide_{values}", **SUITE_SHAPE)
    full_check(w, kv_split_tiles=split, tiling=gc.TILES_WIDE)


@pytest.mark.parametrize("values", ["unit", "peaked"])
@pytest.mark.parametrize("split", [None, 3])
def test_small_tiles_on_multi_token_requests(values, split):
    """The small-tile path forced on requests with up to 130 new tokens: many
    2-token query tiles per request, causal masking inside each."""
    import paper_2505_23970_amd as gc
    w = W.build(seed=101, values=values, name=f"small_{values}", **SUITE_SHAPE)
    full_check(w, kv_split_tiles=split, tiling=gc.TILES_SMALL)


@pytest.mark.parametrize("split", [None, 1])
def test_needle_in_prefix_and_in_new_tokens(split):
    w = W.build(seed=101, name="needles", **SUITE_SHAPE)
    # request 0: needle in a random prefix page; request 2: needle among the new
    # tokens at position P + 50 (rows before it must not see it)
    W.plant_needles(w, [(0, 137), (1, 999), (2, 33 + 50)])
    info, run, out = full_check(w, kv_split_tiles=split)
    got = H.from_dev_f32(out)
    vn = W.bf16_bits_to_f32(w.v_new).astype(np.float64)
    vpre = W.bf16_bits_to_f32(w.v_prefix).astype(np.float64)
    cu, cup = w.cu_new_lens, w.cu_prefix_lens
    g = w.num_q_heads // w.num_kv_heads
    # request 0 rows all return the needle's value (weight >= 1 - 3e-6)
    for t in range(int(cu[0]), int(cu[1])):
        for h in range(w.num_q_heads):
            np.testing.assert_allclose(got[t, h], vpre[cup[0] + 137, h // g], atol=2e-2)
    # request 2: rows i >= 50 see V[needle], rows i < 50 do not
    needle_v = vn[cu[2] + 50]
    for i in range(int(w.new_lens[2])):
        t = int(cu[2]) + i
        for h in range(0, w.num_q_heads, 5):
            close = np.allclose(got[t, h], needle_v[h // g], atol=2e-2)
            assert close == (i >= 50), (i, h)


@pytest.mark.parametrize("split", [None, 1])
def test_values_one_normalises(split):
    """V = 1: the output is the sum of the weights over the normaliser. The
    probabilities enter the PV product rounded to bf16 and the normaliser sums the
    same bf16-rounded weights, so the quotient is 1 up to fp32 summation order
    (chunk merges and the two partial sums of a row) and rounds to 1.0 in bf16;
    the bound allows 2^-8 and nearly every row lands exactly on 1.0."""
    w = W.set_values_one(W.build(seed=102, values="unit", name="v_one", **SUITE_SHAPE))
    _, _, out = full_check(w, kv_split_tiles=split)
    got = H.from_dev_f32(out)
    assert np.all(np.abs(got - 1.0) <= 2.0 ** -8)
    assert np.mean(got == 1.0) >= 0.99


@pytest.mark.parametrize("split", [None, 1])
def test_position_code_window(split):
    w = W.set_position_code(W.build([0, 17, 64, 200, 15], [100, 60, 1, 56, 241], 8, 2, 64,
                                    seed=103, name="poscode"))
    _, _, out = full_check(w, kv_split_tiles=split)
    got = H.from_dev_f32(out)[:, :, 0]
    cu = w.cu_new_lens
    for r in range(w.batch):
        for i in range(int(w.new_lens[r])):
            expect = (int(w.prefix_lens[r]) + i) / 2.0
            assert np.all(got[cu[r] + i] == expect), (r, i, got[cu[r] + i], expect)


@pytest.mark.parametrize("split", [None, 1])
def test_score_jump_beyond_offset_slack(split):
    """A key whose score exceeds the earlier ones by ~130 in log2 units. The prefill
    tiles keep the exponent offset of a row's first tile and run the work item again
    with exact running maxima when a row's weight sum overflows; the small tiles
    rescale when a tile's maximum exceeds the offset by more than 2^8. Either way this
    jump must be absorbed (weights of exp2(130) would overflow fp32: NaN or Inf)."""
    w = W.build([300, 70], [40, 9], 8, 1, 128, seed=104, name="score_jump")
    w.q[:, :, 0] = W.f32_to_bf16_bits(np.float32(8.0))
    w.k_prefix[250, :, 0] = W.f32_to_bf16_bits(np.float32(128.0))  # request 0, position 250
    w.finish()
    _, _, out = full_check(w, kv_split_tiles=split)
    vpre = W.bf16_bits_to_f32(w.v_prefix).astype(np.float64)
    got = H.from_dev_f32(out)
    np.testing.assert_allclose(got[:40, 0], np.broadcast_to(vpre[250, 0], (40, 128)), atol=2e-2)


# ----------------------------------------------------------------- edge cases

EDGES = [
    ("miss_only", [0], [1], 8, 1, 128),
    ("single_token_decode_shape", [777], [1], 32, 8, 128),
    ("page_boundaries", [16, 1, 15, 32, 0], [16, 15, 17, 1, 16], 8, 2, 128),
    ("mha", [100, 50], [30, 70], 4, 4, 64),
    ("group3_odd_tile", [40, 130], [100, 9], 6, 2, 128),
    ("group16", [500], [40], 32, 2, 128),
    ("group128_one_token_tiles", [300], [5], 128, 1, 64),
    ("zero_length_requests", [10, 5, 0, 70], [0, 20, 0, 33], 8, 8, 128),
    ("batch32_short", list(range(0, 320, 10)), [3] * 16 + [65] * 16, 8, 1, 128),
    ("tile_multiple_suffix", [64], [128], 8, 1, 128),
]


@pytest.mark.parametrize("name,P,n,Hq,Hkv,D", EDGES, ids=[e[0] for e in EDGES])
def test_edge_cases(name, P, n, Hq, Hkv, D):
    import paper_2505_23970_amd as gc
    w = W.build(P, n, Hq, Hkv, D, seed=200 + EDGES.index((name, P, n, Hq, Hkv, D)),
                values="unit", name=name)
    full_check(w)
    full_check(w, kv_split_tiles=1)
    full_check(w, tiling=gc.TILES_PREFILL)
    full_check(w, tiling=gc.TILES_WIDE)
    full_check(w, kv_split_tiles=1, tiling=gc.TILES_WIDE)
    if Hq // Hkv <= 16:
        full_check(w, tiling=gc.TILES_SMALL)
        full_check(w, kv_split_tiles=1, tiling=gc.TILES_SMALL)


@pytest.mark.parametrize("split", [None, 1, 2, 3, 7])
def test_below_ridge_on_prefill_tiles(split):
    """Batches below the ridge (few new tokens, long prefixes) on 128-row tiles: work
    items of 1 to 60 key tiles, page tails, a miss and a one-token request, with and
    without key splits, at both head dimensions."""
    import paper_2505_23970_amd as gc
    w = W.build([0, 50, 130, 190, 3000, 1, 700], [9, 3, 1, 16, 12, 5, 2], 16, 2, 128, seed=270,
                values="unit", name="below_ridge")
    full_check(w, kv_split_tiles=split, tiling=gc.TILES_PREFILL)
    w64 = W.build([64, 1234, 5], [16, 4, 40], 8, 1, 64, seed=271, values="peaked", name="below_ridge_d64")
    full_check(w64, kv_split_tiles=split, tiling=gc.TILES_PREFILL)


def test_batch_beyond_lds_plan_limit():
    """More requests than the planner keeps in LDS (2048): the work list is built
    from the global length arrays instead."""
    rng = np.random.default_rng(7)
    P = rng.integers(0, 48, 2100).tolist()
    n = rng.integers(0, 4, 2100).tolist()
    w = W.build(P, n, 4, 1, 64, seed=260, values="unit", name="batch2100")
    full_check(w)
    full_check(w, kv_split_tiles=1)


def test_longest_prefix_sampled():
    w = W.build([200_000], [40], 8, 1, 128, seed=250, name="longest")
    rows = np.array([0, 7, 8 * 20 + 3, 8 * 39, 8 * 39 + 7], np.int64)
    full_check(w, rows=rows)


# ----------------------------------------------------------------- determinism and invariants

def test_split_is_deterministic_and_close_to_unsplit():
    w = W.build([3000, 100], [50, 200], 16, 2, 128, seed=300, values="unit")
    run = H.DeviceRun(w)
    run.append()
    a, _ = run.attention(kv_split_tiles=3)
    b, _ = run.attention(kv_split_tiles=3)
    c, _ = run.attention(kv_split_tiles=-1)
    assert np.array_equal(H.from_dev_bits(a), H.from_dev_bits(b))
    d1 = H.from_dev_f32(a) - H.from_dev_f32(c)
    assert np.abs(d1).max() <= 2 ** -6


def test_block_relabelling_is_bitwise_invisible():
    w = W.build([123, 45], [40, 90], 8, 2, 128, seed=301, values="unit")
    run1 = H.DeviceRun(w)
    run1.append()
    o1, l1 = run1.attention()
    perm = np.random.default_rng(3).permutation(w.num_blocks)
    w2 = W.Workload(**{f.name: getattr(w, f.name) for f in W.dataclasses.fields(W.Workload)})
    w2.block_tables = perm[w.block_tables].astype(np.int32)
    w2.finish()
    run2 = H.DeviceRun(w2)
    run2.append()
    o2, l2 = run2.attention()
    assert np.array_equal(H.from_dev_bits(o1), H.from_dev_bits(o2))
    assert np.array_equal(H.from_dev_f32(l1), H.from_dev_f32(l2))


@pytest.mark.parametrize("kv,tiling", [("bf16", "prefill"), ("bf16", "wide"), ("bf16", "small"),
                                       ("bf16", "fused"), ("fp8", "prefill"), ("fp8", "small")])
def test_pool_beyond_4_gib(kv, tiling):
    """Block ids whose byte offsets exceed 2^32: the same batch run on its own pool and
    with every block id shifted past 4 GiB inside a larger pool gives bitwise the same
    output, LSE and appended pages ("fused": the shifted run appends inside the
    attention launch). The blocks that a 32-bit wraparound of those offsets would
    land on hold NaN, so a truncated offset shows up."""
    import torch
    import paper_2505_23970_amd as gc
    til = {"prefill": gc.TILES_PREFILL, "wide": gc.TILES_WIDE, "small": gc.TILES_SMALL,
           "fused": gc.TILES_PREFILL}[tiling]
    w = W.build([300, 17, 96], [37, 5, 64], 16, 2, 128, seed=330, values="unit")
    say(f"case pool beyond 4 GiB: kv={kv} tiling={tiling}")
    fp8 = kv == "fp8"
    ks, vs = 2.0 ** -6, 0.0213
    ref = H.DeviceRunFp8(w, ks, vs) if fp8 else H.DeviceRun(w)
    ref.append()
    o1, l1 = ref.attention(tiling=til)
    NB = w.num_blocks
    page_bytes = w.num_kv_heads * 16 * w.head_dim * (1 if fp8 else 2)
    shift = (1 << 32) // page_bytes
    dtype = torch.uint8 if fp8 else torch.bfloat16
    nan = 0x7F if fp8 else int(W.BF16_NAN)
    pools = []
    for small in (ref.k_pool, ref.v_pool):
        big = torch.empty((shift + NB,) + tuple(small.shape[1:]), dtype=dtype, device="cuda")
        (big[:NB] if fp8 else big[:NB].view(torch.int16)).fill_(nan)
        pools.append(big)
    init_k = H.to_dev_u8(ref.k8_init) if fp8 else H.to_dev_bf16(w.k_pool)
    init_v = H.to_dev_u8(ref.v8_init) if fp8 else H.to_dev_bf16(w.v_pool)
    pools[0][shift:] = init_k
    pools[1][shift:] = init_v
    batch = gc.PagedBatch(w.prefix_lens, w.new_lens, (w.block_tables + shift).astype(np.int32))
    T, Hq, D = w.q.shape
    o2 = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    l2 = torch.full((T, Hq), float("nan"), dtype=torch.float32, device="cuda")
    if fp8:
        gc.kv_append_fp8(ref.k_new, ref.v_new, pools[0], pools[1], batch, ks, vs)
        gc.prefix_prefill_attention_fp8(ref.q, pools[0], pools[1], batch, w.scale, ks, vs, out=o2, lse=l2,
                                        tiling=til)
    elif tiling == "fused":
        shifted = H.DeviceRun.__new__(H.DeviceRun)
        shifted.w, shifted.batch, shifted.k_pool, shifted.v_pool = w, batch, pools[0], pools[1]
        shifted.q, shifted.k_new, shifted.v_new = ref.q, ref.k_new, ref.v_new
        o2, l2 = fused_run(shifted, tiling=til)
    else:
        gc.kv_append(ref.k_new, ref.v_new, pools[0], pools[1], batch)
        gc.prefix_prefill_attention(ref.q, pools[0], pools[1], batch, w.scale, out=o2, lse=l2, tiling=til)
    torch.cuda.synchronize()
    assert np.array_equal(H.from_dev_bits(o1), H.from_dev_bits(o2))
    assert np.array_equal(H.from_dev_f32(l1), H.from_dev_f32(l2))
    for big, small in zip(pools, (ref.k_pool, ref.v_pool)):
        assert torch.equal(big[shift:].view(torch.uint8), small.view(torch.uint8))
    del pools
    torch.cuda.empty_cache()


@pytest.mark.parametrize("split", [None, 1])
@pytest.mark.parametrize("case", ["agree", "device_total_longer", "negative_prefix", "table_too_short"])
def test_plan_status_reports_disagreeing_lengths(case, split):
    """The planner checks the device lengths against the host's: when they disagree the
    plan status is GC_ERR_LENGTHS and a run on that plan leaves out and lse untouched
    (NaN sentinels); when they agree the status is GC_OK and the output is the oracle's."""
    import torch
    import paper_2505_23970_amd as gc
    w = W.build([300, 17, 96], [37, 5, 64], 16, 2, 128, seed=340, values="unit", name="plan_status")
    say(f"case plan status: {case} split={split}")
    run = H.DeviceRun(w)
    run.append()
    batch = gc.PagedBatch(w.prefix_lens, w.new_lens, w.block_tables)
    if case == "device_total_longer":      # request 1 has 3 more new tokens on the device
        batch.cu_new_lens_dev[2:] += 3
    elif case == "negative_prefix":
        batch.prefix_lens_dev[1] = -40
    elif case == "table_too_short":        # request 0's keys run past its table row
        batch.prefix_lens_dev[0] = 16 * w.block_tables.shape[1]
    T, Hq, D = w.q.shape
    ws = gc.alloc_workspace(Hq, run.k_pool, run.v_pool, batch, kv_split_tiles=split)
    gc.plan(Hq, run.k_pool, run.v_pool, batch, ws, kv_split_tiles=split)
    status = gc.plan_status(ws)
    out = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((T, Hq), float("nan"), dtype=torch.float32, device="cuda")
    gc.run(run.q, run.k_pool, run.v_pool, batch, w.scale, ws, out=out, lse=lse, kv_split_tiles=split)
    torch.cuda.synchronize()
    if case == "agree":
        assert status == gc.GC_OK
        kp, vp = H.oracle_pools(w)
        ref, ref_lse = H.oracle_rows(w, kp, vp)
        H.compare_attention(w, out, lse, ref, ref_lse)
    else:
        assert status == gc.GC_ERR_LENGTHS
        assert torch.isnan(out.float()).all().item() and torch.isnan(lse).all().item()


def test_plan_once_run_twice():
    import torch
    import paper_2505_23970_amd as gc
    w = W.build([500, 20], [70, 33], 16, 2, 128, seed=302)
    run = H.DeviceRun(w)
    run.append()
    ws = gc.alloc_workspace(w.num_q_heads, run.k_pool, run.v_pool, run.batch, kv_split_tiles=2)
    gc.plan(w.num_q_heads, run.k_pool, run.v_pool, run.batch, ws, kv_split_tiles=2)
    o1 = gc.run(run.q, run.k_pool, run.v_pool, run.batch, w.scale, ws, kv_split_tiles=2)
    o2 = gc.run(run.q, run.k_pool, run.v_pool, run.batch, w.scale, ws, kv_split_tiles=2)
    torch.cuda.synchronize()
    assert np.array_equal(H.from_dev_bits(o1), H.from_dev_bits(o2))
    kp, vp = H.oracle_pools(w)
    ref, _ = H.oracle_rows(w, kp, vp)
    H.compare_attention(w, o1, None, ref, None)


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_small_tile_splits_repeat_on_one_workspace(kv):
    """Small tiles with key splits (partials and their merge in the workspace), one
    plan and three runs (q, -q, q) on the same workspace: every run matches the
    oracle (nothing a run leaves in the workspace leaks into the next), and the
    first and third are bitwise equal."""
    import copy
    import torch
    import paper_2505_23970_amd as gc
    w = W.build([3000, 700, 40, 1500, 2047], [1, 2, 1, 3, 1], 16, 2, 128, seed=304)
    wn = copy.copy(w)
    wn.q = (w.q.view(np.uint16) ^ np.uint16(0x8000)).view(w.q.dtype)  # exact negation of bf16
    til, split = gc.TILES_SMALL, 4
    T, Hq, D = w.q.shape
    if kv == "bf16":
        run = H.DeviceRun(w)
        run.append()
        kp, vp = H.oracle_pools(w)
        refs = [H.oracle_rows(x, kp, vp) for x in (w, wn)]
        go = gc.run
        extra = {}
    else:
        ks, vs = 0.02, 0.015
        run = H.DeviceRunFp8(w, ks, vs)
        run.append()
        kp8, vp8 = H.oracle_pools_fp8(run)
        refs = [H.oracle.attention_e4m3(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks, x.q,
                                        kp8, vp8, ks, vs, w.scale) for x in (w, wn)]
        go = gc.run_fp8
        extra = {"k_scale": ks, "v_scale": vs}
    say(f"small-tile splits repeat kv={kv} lens={list(w.prefix_lens)}/{list(w.new_lens)} split={split}")
    ws = gc.alloc_workspace(w.num_q_heads, run.k_pool, run.v_pool, run.batch, kv_split_tiles=split, tiling=til)
    gc.plan(w.num_q_heads, run.k_pool, run.v_pool, run.batch, ws, kv_split_tiles=split, tiling=til)
    qn = H.to_dev_bf16(wn.q)
    outs = []
    for q, ref in ((run.q, refs[0]), (qn, refs[1]), (run.q, refs[0])):
        out = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((T, Hq), float("nan"), dtype=torch.float32, device="cuda")
        go(q, run.k_pool, run.v_pool, run.batch, w.scale, workspace=ws, out=out, lse=lse,
           kv_split_tiles=split, tiling=til, **extra)
        torch.cuda.synchronize()
        H.compare_attention(w, out, lse, ref[0], ref[1],
                            vmax=None if kv == "bf16" else H.e4m3_vmax(vp8, vs))
        outs.append((H.from_dev_bits(out), H.from_dev_f32(lse)))
    assert np.array_equal(outs[0][0], outs[2][0]) and np.array_equal(outs[0][1], outs[2][1])



def test_two_turns_equal_one_call():
    """Multi-turn reuse: turn 1 appends n1 tokens and attends; turn 2 treats them as
    cached prefix. The rows match a single call over n1 + n2 new tokens."""
    import torch
    import paper_2505_23970_amd as gc
    w = W.build([200], [90], 8, 2, 128, seed=303, values="unit")
    one = H.DeviceRun(w)
    one.append()
    full, _ = one.attention()
    n1 = 37
    dev = H.DeviceRun(w)
    b1 = gc.PagedBatch(w.prefix_lens, [n1], w.block_tables)
    gc.kv_append(dev.k_new[:n1].contiguous(), dev.v_new[:n1].contiguous(), dev.k_pool, dev.v_pool, b1)
    o1 = gc.prefix_prefill_attention(dev.q[:n1].contiguous(), dev.k_pool, dev.v_pool, b1, w.scale)
    b2 = gc.PagedBatch(w.prefix_lens + n1, [90 - n1], w.block_tables)
    gc.kv_append(dev.k_new[n1:].contiguous(), dev.v_new[n1:].contiguous(), dev.k_pool, dev.v_pool, b2)
    o2 = gc.prefix_prefill_attention(dev.q[n1:].contiguous(), dev.k_pool, dev.v_pool, b2, w.scale)
    torch.cuda.synchronize()
    got = np.concatenate([H.from_dev_f32(o1), H.from_dev_f32(o2)])
    assert np.abs(got - H.from_dev_f32(full)).max() <= 2 ** -7


def test_append_leaves_other_slots_alone_with_bad_block_ids():
    """Table entries outside the pool are skipped by the append kernel; every
    other slot is written exactly as the oracle writes it."""
    w = W.build([20, 3], [30, 40], 8, 2, 128, seed=304)
    bad = w.block_tables.copy()
    bad[1, 2] = w.num_blocks + 5   # page 2 of request 1 (positions 32..47)
    run = H.DeviceRun(w)
    run.batch = __import__("paper_2505_23970_amd").PagedBatch(w.prefix_lens, w.new_lens, bad)
    run.append()
    import torch
    torch.cuda.synchronize()
    kp_ref, vp_ref = H.oracle_pools(w)
    kp = H.from_dev_bits(run.k_pool)
    vp = H.from_dev_bits(run.v_pool)
    skipped = int(w.block_tables[1, 2])
    keep = np.ones(w.num_blocks, bool)
    keep[skipped] = False
    assert np.array_equal(kp[keep], kp_ref[keep]) and np.array_equal(vp[keep], vp_ref[keep])
    assert np.array_equal(kp[skipped], w.k_pool[skipped])   # untouched


def test_read_probe_reads_every_word():
    """The calibration probe XOR-reduces each thread's 16-byte words: a buffer with one
    non-zero word leaves exactly that word's bits in one sink entry."""
    import torch
    import paper_2505_23970_amd as gc
    buf = torch.zeros(1 << 20, dtype=torch.int32, device="cuda")
    buf[12345] = 0x5A5A
    sink = gc.read_bandwidth_probe(buf)
    torch.cuda.synchronize()
    nz = torch.nonzero(sink).flatten().tolist()
    assert len(nz) == 1 and int(sink[nz[0]].item()) == 0x5A5A


def test_mfma_probe_runs_every_product():
    """The matrix-core calibration loop multiplies all-ones operands: every product adds
    16 to each of a thread's 4 x 16 accumulator elements, 4 products per accumulator
    per iteration, so every sink entry is exactly 4096 * iterations; a dropped or
    duplicated product changes it."""
    import torch
    import paper_2505_23970_amd as gc
    for it in (1, 37, 100):
        sink = gc.mfma_peak_probe(it)
        torch.cuda.synchronize()
        assert torch.all(sink == 4096.0 * it).item()


@pytest.mark.parametrize("source", ["pinned_host", "device"])
def test_restore_prefix_from_host_tier(source):
    """Restoring every cached prefix into an all-NaN pool (positions 0 .. P_r - 1 written
    through the append path, sources read over PCIe from pinned host memory) reproduces
    the oracle's initial pool bit for bit; the new tokens' slots stay NaN."""
    import torch
    import paper_2505_23970_amd as gc
    w = W.build([300, 0, 33, 1000, 16], [5, 7, 1, 2, 3], 16, 2, 128, seed=320, name="restore")
    run = H.DeviceRun(w)
    nan = np.full_like(w.k_pool, W.BF16_NAN)
    kp = H.to_dev_bf16(nan)
    vp = H.to_dev_bf16(np.full_like(w.v_pool, W.BF16_NAN))
    ks = torch.from_numpy(w.k_prefix.view(np.int16)).view(torch.bfloat16)
    vs = torch.from_numpy(w.v_prefix.view(np.int16)).view(torch.bfloat16)
    if source == "pinned_host":
        ks, vs = ks.pin_memory(), vs.pin_memory()
    else:
        ks, vs = ks.cuda(), vs.cuda()
    gc.kv_restore(ks, vs, kp, vp, run.batch)
    torch.cuda.synchronize()
    # expected image: the oracle's append of the prefixes (prefix lengths 0, new
    # lengths P_r) into the same all-NaN pools
    zero = np.zeros_like(w.prefix_lens)
    kref, vref = H.oracle.kv_append(zero, w.prefix_lens, w.block_tables, w.num_blocks,
                                    w.k_prefix, w.v_prefix, nan, np.full_like(w.v_pool, W.BF16_NAN))
    assert np.array_equal(H.from_dev_bits(kp), kref)
    assert np.array_equal(H.from_dev_bits(vp), vref)


def test_restore_refuses_pageable_host_memory():
    import torch
    import paper_2505_23970_amd as gc
    w = W.build([40], [2], 8, 2, 64, seed=321, name="restore_pageable")
    run = H.DeviceRun(w)
    ks = torch.from_numpy(w.k_prefix.view(np.int16)).view(torch.bfloat16)
    with pytest.raises(ValueError):
        gc.kv_restore(ks, ks, run.k_pool, run.v_pool, run.batch)


# ----------------------------------------------------------------- 8-bit (E4M3) pools

E4M3_NAN_CODES = (0x7F, 0xFF)


@pytest.mark.parametrize("ks,vs", [(1.0, 1.0), (0.37, 0.0113), (2.0 ** -7, 3.1 / 448.0)])
def test_fp8_append_quantises_every_bf16_value_like_the_oracle(ks, vs):
    """Every bf16 bit pattern goes through the 8-bit append (keys in order, values
    shuffled); codes must equal the oracle's bit for bit, except that a NaN input
    may become either NaN code."""
    w = W.build([5, 0], [200, 56], 4, 2, 128, seed=120, name="e4m3_all_bf16")
    allbits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    w.k_new = allbits.reshape(256, 2, 128).copy()
    w.v_new = np.random.default_rng(121).permutation(allbits).reshape(256, 2, 128)
    say(f"case {w.name}: scales {ks} {vs}")
    run = H.DeviceRunFp8(w, ks, vs)
    run.append()
    kp, vp = run.pools()
    kref, vref = H.oracle_pools_fp8(run)
    for got, ref, name in ((kp, kref, "k"), (vp, vref, "v")):
        diff = got != ref
        if diff.any():
            assert np.isin(got[diff], E4M3_NAN_CODES).all() and np.isin(ref[diff], E4M3_NAN_CODES).all(), (
                f"{name}_pool differs at {np.argwhere(diff)[:5]}: got {got[diff][:5]}, ref {ref[diff][:5]}")
        n_nan_inputs = int(np.isnan(W.bf16_bits_to_f32(allbits)).sum())
        assert int(diff.sum()) <= n_nan_inputs


def fp8_check(w, ks, vs, kv_split_tiles=None, tiling=None, rows=None, contract=True):
    say(f"case {w.name} (8-bit pools, scales {ks} {vs}): B={w.batch} Hq={w.num_q_heads} "
        f"Hkv={w.num_kv_heads} D={w.head_dim} T={w.total_new} split={kv_split_tiles} tiling={tiling}")
    run = H.DeviceRunFp8(w, ks, vs)
    run.append()
    kref, vref = H.oracle_pools_fp8(run)
    kp, vp = run.pools()
    assert np.array_equal(kp, kref), f"k_pool differs at {np.argwhere(kp != kref)[:5]}"
    assert np.array_equal(vp, vref), f"v_pool differs at {np.argwhere(vp != vref)[:5]}"
    out, lse = run.attention(kv_split_tiles=kv_split_tiles, tiling=tiling)
    ref_out, ref_lse = H.oracle_rows_fp8(run, kref, vref, rows=rows)
    vmax = H.e4m3_vmax(vref, vs)
    return H.compare_attention(w, out, lse, ref_out, ref_lse, rows=rows, contract=contract, vmax=vmax)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("split", [None, 2])
@pytest.mark.parametrize("tiling", ["prefill", "wide", "small"])
def test_fp8_pools_every_tiling(tiling, split, D):
    """Every tiling over 8-bit pools, with and without key splits, at both head
    dimensions (each (tiling, D) pair is its own kernel instance)."""
    import paper_2505_23970_amd as gc
    t = {"prefill": gc.TILES_PREFILL, "wide": gc.TILES_WIDE, "small": gc.TILES_SMALL}[tiling]
    shape = dict(SUITE_SHAPE, head_dim=D)
    w = W.build(seed=110 + D, name=f"fp8_{tiling}_d{D}", **shape)
    info = fp8_check(w, 0.0113, 0.0271, kv_split_tiles=split, tiling=t)
    say(f"8-bit {tiling} D={D} split {split}: {info}")


@pytest.mark.parametrize("D", [64, 128])
def test_fp8_pools_ragged_edges(D):
    """Empty suffixes and prefixes, one-token requests and page-straddling lengths,
    automatic tiling."""
    w = W.build([0, 17, 1, 250, 0], [33, 1, 70, 0, 5], 8, 2, D, seed=111, name=f"fp8_edges_d{D}")
    info = fp8_check(w, 0.02, 0.015)
    say(f"8-bit edges D={D}: {info}")


def test_fp8_config2_all_rows():
    w = W.make_config(2)
    info = fp8_check(w, 2.0 ** -6, 0.0213)
    say(f"8-bit config 2: {info}")


@pytest.mark.timeout(600)
def test_fp8_long_reuse_sampled():
    """The 32k-prefix workload over 8-bit pools (automatic plan: key splits), sampled rows."""
    w = W.make_config(4)
    info = fp8_check(w, 2.0 ** -6, 0.0213, rows=H.sample_rows(w, seed=44))
    say(f"8-bit config 4: {info}")


@pytest.mark.parametrize("split", [None, 1, 2, 3, 4, 5, 7])
def test_fp8_below_ridge_on_prefill_tiles(split):
    """8-bit pools, batches below the ridge on 128-row tiles: work items of 1 to 60 key
    tiles, page tails, a miss and a one-token request, with and without key splits, at
    both head dimensions."""
    import paper_2505_23970_amd as gc
    w = W.build([0, 50, 130, 190, 3000, 1, 700], [9, 3, 1, 16, 12, 5, 2], 16, 2, 128, seed=272,
                name="fp8_below_ridge")
    info = fp8_check(w, 0.02, 0.015, kv_split_tiles=split, tiling=gc.TILES_PREFILL)
    say(f"8-bit below ridge split {split}: {info}")
    w64 = W.build([64, 1234, 5], [16, 4, 40], 8, 1, 64, seed=273, name="fp8_below_ridge_d64")
    fp8_check(w64, 0.0113, 0.0271, kv_split_tiles=split, tiling=gc.TILES_PREFILL)


def test_fp8_short_suffix_variant_sampled():
    """The 32k-prefix workload with 16 new tokens per request over 8-bit pools (automatic
    key splits), sampled rows."""
    w = W.short_suffix_variant()
    info = fp8_check(w, 2.0 ** -6, 0.0213, rows=H.sample_rows(w, seed=41))
    say(f"8-bit long reuse, 16 new tokens: {info}")


def test_fp8_decode_workload_sampled():
    w = W.decode_variant()
    info = fp8_check(w, 2.0 ** -6, 0.0213, rows=H.sample_rows(w, seed=51))
    say(f"8-bit decode, 32 requests: {info}")


# ----------------------------------------------------------------- append and plan in one launch

@pytest.mark.parametrize("kv", ["bf16", "fp8"])
@pytest.mark.parametrize("split", [None, 2])
def test_prepare_equals_append_then_plan(kv, split):
    """gc_prefix_prefill_prepare (append and plan in one launch) followed by run gives
    the separate calls' pools and outputs bit for bit."""
    import torch
    import paper_2505_23970_amd as gc
    w = W.build(seed=112, name=f"prepare_{kv}", **SUITE_SHAPE)
    say(f"case {w.name}: split {split}")
    if kv == "fp8":
        a, b = H.DeviceRunFp8(w, 0.0113, 0.0271), H.DeviceRunFp8(w, 0.0113, 0.0271)
        extra = dict(k_scale=a.ks, v_scale=a.vs)
    else:
        a, b = H.DeviceRun(w), H.DeviceRun(w)
        extra = {}
    a.append()
    out_a, lse_a = a.attention(kv_split_tiles=split)
    T, Hq, D = w.q.shape
    ws = gc.alloc_workspace(Hq, b.k_pool, b.v_pool, b.batch, split)
    gc.prepare(b.k_new, b.v_new, b.k_pool, b.v_pool, b.batch, Hq, ws, kv_split_tiles=split, **extra)
    lse_b = torch.full((T, Hq), float("nan"), dtype=torch.float32, device="cuda")
    out_b = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    if kv == "fp8":
        gc.run_fp8(b.q, b.k_pool, b.v_pool, b.batch, w.scale, b.ks, b.vs, ws, out=out_b, lse=lse_b,
                   kv_split_tiles=split)
    else:
        gc.run(b.q, b.k_pool, b.v_pool, b.batch, w.scale, ws, out=out_b, lse=lse_b, kv_split_tiles=split)
    torch.cuda.synchronize()
    # Unused pool slots hold NaN sentinels, so every comparison is on the bits.
    bits = {1: torch.uint8, 2: torch.int16, 4: torch.int32}
    same = lambda x, y: torch.equal(x.view(bits[x.element_size()]), y.view(bits[y.element_size()]))
    assert same(a.k_pool, b.k_pool) and same(a.v_pool, b.v_pool)
    assert same(out_a, out_b)
    assert same(lse_a, lse_b)


# ----------------------------------------------------------------- append fused into the attention launch

def same_bits(x, y):
    """Bitwise equality of two device tensors (unused pool slots hold NaN sentinels)."""
    import torch
    bits = {1: torch.uint8, 2: torch.int16, 4: torch.int32}
    return torch.equal(x.view(bits[x.element_size()]), y.view(bits[y.element_size()]))


def fused_run(run: H.DeviceRun, kv_split_tiles=None, tiling=None):
    """gc_prefix_prefill_plan, then gc_prefix_prefill_run_with_append on `run`'s
    initial pools; returns out and lse."""
    import torch
    import paper_2505_23970_amd as gc
    w = run.w
    T, Hq, D = w.q.shape
    ws = gc.alloc_workspace(Hq, run.k_pool, run.v_pool, run.batch, kv_split_tiles, tiling)
    gc.plan(Hq, run.k_pool, run.v_pool, run.batch, ws, kv_split_tiles=kv_split_tiles, tiling=tiling)
    lse = torch.full((T, Hq), float("nan"), dtype=torch.float32, device="cuda")
    out = torch.full((T, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    gc.run_with_append(run.q, run.k_new, run.v_new, run.k_pool, run.v_pool, run.batch, w.scale, ws, out=out,
                       lse=lse, kv_split_tiles=kv_split_tiles, tiling=tiling)
    torch.cuda.synchronize()
    return out, lse


def fused_equals_separate(w, kv_split_tiles=None, tiling=None):
    """The fused launch gives the separate append + run's pools, output and LSE bit for bit."""
    import torch
    say(f"case {w.name}: fused append, B={w.batch} Hq={w.num_q_heads} Hkv={w.num_kv_heads} "
        f"D={w.head_dim} T={w.total_new} split={kv_split_tiles} tiling={tiling}")
    a, b = H.DeviceRun(w), H.DeviceRun(w)
    a.append()
    out_a, lse_a = a.attention(kv_split_tiles=kv_split_tiles, tiling=tiling)
    out_b, lse_b = fused_run(b, kv_split_tiles, tiling)
    assert same_bits(a.k_pool, b.k_pool) and same_bits(a.v_pool, b.v_pool)
    if not same_bits(out_a, out_b):
        bad = torch.nonzero(out_a.view(torch.int16) != out_b.view(torch.int16))[:5].tolist()
        raise AssertionError(f"outputs differ at {bad}")
    assert same_bits(lse_a, lse_b)


@pytest.mark.parametrize("split", [None, 2])
@pytest.mark.parametrize("tiling", [None, 1, 3, 2], ids=["auto", "prefill", "wide", "small"])
def test_fused_append_every_tiling(tiling, split):
    w = W.build(seed=120, name="fused_suite", values="unit", **SUITE_SHAPE)
    fused_equals_separate(w, split, tiling)


@pytest.mark.parametrize("name,P,n,Hq,Hkv,D", EDGES, ids=[e[0] for e in EDGES])
def test_fused_append_edge_cases(name, P, n, Hq, Hkv, D):
    import paper_2505_23970_amd as gc
    w = W.build(P, n, Hq, Hkv, D, seed=300 + EDGES.index((name, P, n, Hq, Hkv, D)), values="unit",
                name=name)
    fused_equals_separate(w)
    fused_equals_separate(w, kv_split_tiles=1)
    fused_equals_separate(w, tiling=gc.TILES_WIDE)
    fused_equals_separate(w, kv_split_tiles=1, tiling=gc.TILES_PREFILL)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_fused_append_configs(k):
    fused_equals_separate(W.make_config(k))


def test_fused_append_decode_workload():
    # small tiles: the append is its own launch ahead of the attention
    fused_equals_separate(W.decode_variant())


@pytest.mark.parametrize("split", [None, 3])
def test_fused_append_against_the_oracle(split):
    """Pools and every output row of the fused launch against the oracle directly."""
    w = W.build([130, 0, 64, 1500, 17], [200, 70, 64, 1, 95], 16, 2, 128, seed=125, name="fused_oracle")
    say(f"case {w.name}: fused append vs oracle, split {split}")
    kp_ref, vp_ref = H.oracle_pools(w)
    run = H.DeviceRun(w)
    out, lse = fused_run(run, kv_split_tiles=split)
    check_pool(run, kp_ref, vp_ref)
    ref_out, ref_lse = H.oracle_rows(w, kp_ref, vp_ref)
    info = H.compare_attention(w, out, lse, ref_out, ref_lse, contract=True)
    say(f"fused vs oracle: {info}")


def test_bench_line_keeps_the_contract():
    """bench.py on the tiny workload prints one JSON line with the contract's fields, the
    roofline object (measured live) and the CPU-oracle baseline."""
    import json
    import os
    import subprocess
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    res = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--workload", "tiny", "--steps", "5",
                          "--warmup", "5", "--cpu-seconds", "0.5"], capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stderr[-2000:]
    lines = [l for l in res.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 5 and d["warmup"] == 5 and d["config"]["workload"] == "tiny"
    assert d["value"] > 0 and d["ms_per_step"] > 0 and d["kernel_ms"]["attention_cold"] > 0
    r = d["roofline"]
    assert r["bound"] in ("mfma", "hbm") and r["peak"] in (2500.0, 8000.0)
    assert abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-9 and r["frac_of_measured"] > 0
    c = d["cpu_baseline"]
    assert c["kind"] == "oracle" and c["value"] > 0 and c["cores"] >= 1 and c["sample"]
