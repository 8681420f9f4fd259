"""Pure-Python brute force of the oracle's definition, for tiny inputs only.

Test infrastructure. A second, independent code base (no numpy, no C) for
the same plain definition the C oracle follows (GreenCache §2.2, Fig. 1a:
cached prefix KV and the new tokens' KV processed together; §2.1 prefill):
causal scaled-dot-product attention of new token i over logical keys
0 .. P + i, with query head h reading KV head h // (Hq // Hkv).
It walks the pool through the block table itself.
"""
from __future__ import annotations

import math
import struct


def bf16_to_float(bits: int) -> float:
    return struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]


def attention(prefix_lens, new_lens, block_tables, q, k_pool, v_pool, Hq, Hkv, D, S, scale):
    """Returns (out, lse): out[token][head] = list of D floats, lse[token][head].

    q: nested lists / arrays indexable as q[token][head][c] (bf16 bits);
    k_pool[blk][kvh][slot][c], v_pool[blk][kvh][c][slot] (bf16 bits).
    """
    g = Hq // Hkv
    out, lse = [], []
    token = 0
    for r in range(len(prefix_lens)):
        P = int(prefix_lens[r])
        for i in range(int(new_lens[r])):
            orow, lrow = [], []
            for h in range(Hq):
                kvh = h // g
                qv = [bf16_to_float(q[token][h][c]) for c in range(D)]
                logits = []
                for j in range(P + i + 1):
                    blk = int(block_tables[r][j // S])
                    kv = k_pool[blk][kvh][j % S]
                    logits.append(scale * math.fsum(qv[c] * bf16_to_float(kv[c]) for c in range(D)))
                top = max(logits)
                weights = [math.exp(x - top) for x in logits]
                total = math.fsum(weights)
                o = []
                for c in range(D):
                    acc = []
                    for j, w in enumerate(weights):
                        blk = int(block_tables[r][j // S])
                        acc.append(w / total * bf16_to_float(v_pool[blk][kvh][c][j % S]))
                    o.append(math.fsum(acc))
                orow.append(o)
                lrow.append(top + math.log(total))
            out.append(orow)
            lse.append(lrow)
            token += 1
    return out, lse


def kv_append(prefix_lens, new_lens, block_tables, k_new, v_new, k_pool, v_pool, Hkv, D, S):
    """Scatter, element by element, into copies of the pools (nested lists)."""
    k_pool = [[[list(row) for row in head] for head in blk] for blk in k_pool]
    v_pool = [[[list(row) for row in head] for head in blk] for blk in v_pool]
    token = 0
    for r in range(len(prefix_lens)):
        for i in range(int(new_lens[r])):
            pos = int(prefix_lens[r]) + i
            blk = int(block_tables[r][pos // S])
            slot = pos % S
            for kvh in range(Hkv):
                for c in range(D):
                    k_pool[blk][kvh][slot][c] = int(k_new[token][kvh][c])
                    v_pool[blk][kvh][c][slot] = int(v_new[token][kvh][c])
            token += 1
    return k_pool, v_pool
