"""bench.py on the CPU: the one-GPU refusal, the algorithmic FLOP and byte counts
its roofline figures divide by, and the lookup of profiled HBM traffic."""
import hashlib
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2505_23970_amd import workloads as W  # noqa: E402


def test_refuses_more_than_one_gpu():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode != 0
    assert "one GPU" in res.stderr


def test_flops_count_every_visible_query_key_pair():
    """4 d flops (QK^T and PV, multiply and add) per (query head, visible key) pair,
    counted here by walking every new token's causal window."""
    w = W.build([0, 5, 40, 17], [3, 1, 20, 0], 8, 2, 64, seed=1)
    pairs = 0
    for r in range(w.batch):
        P, n = int(w.prefix_lens[r]), int(w.new_lens[r])
        for i in range(n):
            pairs += P + i + 1           # keys 0 .. P + i inclusive
    assert w.flops() == 4 * w.head_dim * w.num_q_heads * pairs


def test_attention_bytes_read_kv_once_and_q_o_once():
    w = W.build([0, 5, 40], [3, 1, 20], 8, 2, 64, seed=2)
    D, Hq, Hkv = w.head_dim, w.num_q_heads, w.num_kv_heads
    kv = sum(int(P + n) for P, n in zip(w.prefix_lens, w.new_lens)) * Hkv * D * 2 * 2
    qo = w.total_new * Hq * D * 2 * 2
    assert w.attn_bytes(2) == kv + qo
    assert w.attn_bytes(1) == kv // 2 + qo
    assert w.append_bytes() == w.total_new * Hkv * D * 2 * 2 * 2


def test_profiled_traffic_follows_the_committed_profile():
    """The traffic figure comes from the profile's traffic-json line and only while
    the profiled kernel's code (kernel, planner, host policy) is unchanged."""
    path = os.path.join(ROOT, "profiles", "attention_llama3_8b.md")
    rec = None
    for line in open(path):
        if line.startswith("traffic-json:"):
            rec = json.loads(line.split(":", 1)[1])
    assert rec is not None and rec["traffic_bytes"] == rec["fetch_bytes"] + rec["write_bytes"]
    assert rec["kernel_sources"] == bench.traffic_sources(rec["kernel_sources"][0])
    got = bench.profiled_traffic("llama3_8b")
    if bench.code_sha256_16(rec["kernel_sources"]) == rec["code_sha256_16"]:
        assert got == rec["traffic_bytes"]
        # HBM traffic of one launch is at least the bytes the kernel must write (O)
        w = bench.WORKLOADS["llama3_8b"]()
        assert got >= 2 * w.total_new * w.num_q_heads * w.head_dim
    else:
        assert got is None


def test_code_hash_ignores_comments_and_layout_only(tmp_path):
    files = {
        "a.hip": "int f(int x) { return x + 1; } // one\n",
        "b.hip": "/* a header */\nint f(int x)  {\n    return x + 1;  // another\n}\n",
        "c.hip": "int f(int x) { return x + 2; }\n",
        "d.hip": 'const char* p = "// kept"; char q = \'/\';\n',
        "e.hip": 'const char* p = "// changed"; char q = \'/\';\n',
    }
    for name, text in files.items():
        (tmp_path / name).write_text(text)
    h = {name: bench.code_sha256_16([str(tmp_path / name)]) for name in files}
    assert h["a.hip"] == h["b.hip"]
    assert h["a.hip"] != h["c.hip"]
    assert h["d.hip"] != h["e.hip"]  # text inside a string literal is code
    assert bench.code_text(files["d.hip"]) == 'const char* p = "// kept"; char q = \'/\';'
    assert bench.profiled_traffic("no_such_workload") is None


def test_every_bench_workload_is_well_formed():
    for name, make in bench.WORKLOADS.items():
        if name in ("mixed_hit_miss_70b", "long_reuse_70b", "long_reuse_70b_n16"):
            continue  # ~1-2 GB of inputs each; their lengths are covered by the generator tests
        w = make()
        assert w.flops() > 0 and w.attn_bytes() > 0
        assert np.all(w.prefix_lens >= 0) and np.all(w.new_lens >= 0)
        assert w.q.shape == (w.total_new, w.num_q_heads, w.head_dim)


@pytest.mark.parametrize("name,fp8", [("mixed_hit_miss_70b", False), ("llama3_70b_chat", False),
                                      ("long_reuse_70b", False), ("long_reuse_70b_n16", False),
                                      ("llama3_8b", False), ("llama3_8b", True), ("decode_70b", False),
                                      ("decode_70b", True)])
def test_named_kernel_is_the_profiled_one(name, fp8):
    """bench.py names the kernel the library picks by restating its host rules; the
    committed profile of the workload records the kernel the GPU actually ran."""
    path = os.path.join(ROOT, "profiles", f"attention_{name}{'_fp8' if fp8 else ''}.md")
    first = open(path).readline()
    profiled = first[2:].split(" \u2014 ")[0].strip()
    w = bench.WORKLOADS[name]()
    assert bench.auto_kernel_name(w, 256, fp8).startswith(profiled + " "), (profiled, first)
