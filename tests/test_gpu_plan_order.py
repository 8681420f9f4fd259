"""Order of the planner's work list (white box, GPU).

The library keeps the work list in the workspace from byte offset 256, as records
of eight int32: request, first new token, first and end key tile, partial slot
(-1: the item writes its rows directly), and the request's prefix length, first
new row and new-token count. These tests plan several batches and tilings and read
the list back:
  * every (query tile, key chunk) of the batch appears exactly once, with its
    request's lengths, and split tiles own distinct partial slots;
  * the order is the one the launch is built on. The lightest items, two rounds of
    the resident workgroup slots, come last, by cost (key tiles), heaviest first,
    so that the launch ends on its lightest items. Before them the items are
    sorted by the key tiles of their request, longest request first, so that the
    query tiles of one request, which read nearly the same keys, run side by side.
The attention results do not depend on this order (the parity tests cover them);
the launch's balance and its L2 reuse do.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

ITEMS_OFFSET = 256
RECORD = 8
BUCKETS = 2048  # the planner's counting-sort buckets: costs clamp at 2047


@pytest.fixture(scope="module", autouse=True)
def gpu_ready():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2505_23970_amd as gc
    gc.load_library()


def cdiv(a, b):
    return -(-a // b)


def tile_shape(tiling, group):
    """(new tokens per query tile, keys per key tile, resident slots per CU)."""
    import paper_2505_23970_amd as gc
    if tiling == gc.TILES_SMALL:
        return 16 // group, 32, 4
    if tiling == gc.TILES_WIDE:
        return 256 // group, 64, 1
    return 128 // group, 64, 2


def expected_items(P, n, tq, bn, chunk):
    """(r, q0, kt_begin, kt_end, ns) of every item, from the tiling rules: query
    tiles of tq new tokens, key tiles of bn keys up to the tile's last row, keys cut
    into ceil(kt / chunk) balanced chunks when kt > chunk (chunk <= 0: never)."""
    out = []
    for r in range(len(P)):
        for q0 in range(0, int(n[r]), tq):
            ntok = min(tq, int(n[r]) - q0)
            kt = cdiv(int(P[r]) + q0 + ntok, bn)
            ns = 1 if chunk <= 0 or kt <= chunk else cdiv(kt, chunk)
            for s in range(ns):
                out.append((r, q0, s * kt // ns, (s + 1) * kt // ns, ns))
    return out


def threshold(costs, tail):
    """Smallest cost c such that the items of cost < c number at least `tail`;
    BUCKETS when the list is not longer than the tail (nothing is grouped)."""
    if len(costs) <= tail:
        return BUCKETS
    hist = np.bincount(np.minimum(costs, BUCKETS - 1), minlength=BUCKETS)
    below, c = 0, 0
    while c < BUCKETS and below < tail:
        below += hist[c]
        c += 1
    return c


def plan_and_read(P, n, Hq, Hkv, D, tiling, split):
    import torch
    import paper_2505_23970_amd as gc
    pages = [cdiv(int(p) + int(m), 16) for p, m in zip(P, n)]
    mb = max(pages)
    bt = np.zeros((len(P), mb), np.int32)
    nxt = 0
    for r, k in enumerate(pages):
        bt[r, :k] = np.arange(nxt, nxt + k)
        nxt += k
    batch = gc.PagedBatch(P, n, bt)
    k_pool = torch.empty((nxt, Hkv, 16, D), dtype=torch.bfloat16, device="cuda")
    v_pool = torch.empty((nxt, Hkv, D, 16), dtype=torch.bfloat16, device="cuda")
    ws = gc.alloc_workspace(Hq, k_pool, v_pool, batch, split, tiling=tiling)
    ws.fill_(0xEE)
    gc.plan(Hq, k_pool, v_pool, batch, ws, kv_split_tiles=split, tiling=tiling)
    assert gc.plan_status(ws) == 0
    return ws, batch


CASES = {
    # misses of distinct lengths (tiles of every cost) and hits (prefix-heavy)
    "misses_hits_prefill": ([0] * 8 + [3000 + 100 * i for i in range(8)],
                            [1024 + 64 * i for i in range(8)] + [100 + 5 * i for i in range(8)],
                            32, 8, 64, "prefill", -1),
    "misses_hits_wide": ([0] * 8 + [3000 + 100 * i for i in range(8)],
                         [1024 + 64 * i for i in range(8)] + [100 + 5 * i for i in range(8)],
                         64, 8, 128, "wide", -1),
    "split_chunks_prefill": ([0, 0, 5000, 7000, 9000, 200], [900, 700, 300, 260, 64, 1500],
                             32, 8, 64, "prefill", 6),
    "misses_small": ([0, 0, 0, 0, 40], [1024, 960, 896, 832, 33], 32, 8, 128, "small", -1),
    "short_list_plain": ([1024, 2048, 4000], [100, 64, 300], 32, 8, 128, "prefill", -1),
    # more requests than the planner keeps in LDS: lengths read from global memory; four
    # requests at a time share a length in key tiles, so only the order itself is checked
    "many_requests_global_lens": ([16 * i for i in range(600)], [64] * 600, 32, 8, 64, "prefill", -1),
}
SHARED_LENGTHS = {"many_requests_global_lens"}


@pytest.mark.parametrize("name", sorted(CASES))
def test_work_list_is_complete_and_in_order(name):
    import torch
    import paper_2505_23970_amd as gc
    P, n, Hq, Hkv, D, til, split = CASES[name]
    tiling = {"prefill": gc.TILES_PREFILL, "wide": gc.TILES_WIDE, "small": gc.TILES_SMALL}[til]
    P = np.array(P, np.int32)
    n = np.array(n, np.int32)
    tq, bn, per_cu = tile_shape(tiling, Hq // Hkv)
    want = expected_items(P, n, tq, bn, split)
    ws, batch = plan_and_read(P, n, Hq, Hkv, D, tiling, split)
    recs = ws[ITEMS_OFFSET:ITEMS_OFFSET + 4 * RECORD * len(want)].cpu().numpy().view(np.int32).reshape(-1, RECORD)
    cu = batch.cu_new_lens
    print(f"case {name}: {len(want)} items per KV head, tiling {til}, split {split}", flush=True)

    # complete: the same multiset of (r, q0, kt_begin, kt_end), with the request's lengths
    got = sorted(tuple(int(x) for x in rec[:4]) for rec in recs)
    assert got == sorted(w[:4] for w in want)
    for rec in recs:
        r = int(rec[0])
        assert (rec[5], rec[6], rec[7]) == (P[r], cu[r], cu[r + 1] - cu[r])
    ns_of = {w[:4]: w[4] for w in want}
    parts = [int(rec[4]) for rec in recs]
    for rec, part in zip(recs, parts):
        assert (part == -1) == (ns_of[tuple(int(x) for x in rec[:4])] == 1)
    split_parts = [p for p in parts if p >= 0]
    assert len(set(split_parts)) == len(split_parts)
    assert all(0 <= p < len(split_parts) for p in split_parts)

    # order
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    tail = cdiv(2 * per_cu * cus, Hkv)
    costs = np.array([int(rec[3] - rec[2]) for rec in recs])
    req_tiles = np.array([cdiv(int(P[r]) + int(n[r]), bn) for r in recs[:, 0]])
    c_star = threshold(costs, tail)
    cc = np.minimum(costs, BUCKETS - 1)
    key = np.where(cc >= c_star, np.minimum(req_tiles, BUCKETS - 1), cc)
    assert np.all(key[:-1] >= key[1:]), f"order broken at {np.argwhere(key[:-1] < key[1:])[:5].ravel()}"
    grouped = cc >= c_star
    if name == "short_list_plain":
        assert not grouped.any()
    else:
        assert grouped.sum() > len(recs) // 2, "the case should exercise the grouped order"
        # every request's grouped items are contiguous where request lengths are distinct
        if name not in SHARED_LENGTHS:
            rs = recs[grouped, 0]
            change = np.flatnonzero(rs[1:] != rs[:-1])
            assert len(change) == len(set(rs.tolist())) - 1
        # and the tail holds the lightest items, at least two rounds of the slots
        assert (~grouped).sum() >= min(tail, len(recs))
        if (~grouped).any():
            assert costs[~grouped].max() < costs[grouped].min()
