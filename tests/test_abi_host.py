"""The C ABI on the CPU: the library loads, exports every symbol the header
declares, and rejects invalid calls on the host before any HIP call."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2505_23970_amd as gc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "greencache.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gc_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    return gc.load_library()


def test_header_declares_the_python_surface():
    assert declared_functions() == sorted(gc.EXPORTED)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_read_probe_rejects_bad_arguments(lib):
    assert lib.gc_read_bandwidth_probe(None, 1024, 0x2000, None) == -1
    assert lib.gc_read_bandwidth_probe(0x2000, 1024, None, None) == -1
    assert lib.gc_read_bandwidth_probe(0x2000, 1000, 0x2000, None) == -2   # not a multiple of 16
    assert lib.gc_read_bandwidth_probe(0x2000, 0, 0x2000, None) == 0       # nothing to read, nothing enqueued


def test_mfma_probe_rejects_bad_arguments(lib):
    assert lib.gc_mfma_peak_probe(10, None, None) == -1
    assert lib.gc_mfma_peak_probe(-1, 0x2000, None) == -2
    assert lib.gc_mfma_peak_probe(0, 0x2000, None) == 0       # nothing to run, nothing enqueued


def test_plan_status_rejects_bad_arguments(lib):
    """Checked before the copy of the status word (no HIP call)."""
    assert lib.gc_prefix_prefill_plan_status(None, 256, None) == -1
    assert lib.gc_prefix_prefill_plan_status(0x2000, 3, None) == -5


def test_status_strings(lib):
    for code, name in gc.STATUS_NAMES.items():
        assert lib.gc_status_string(code).decode().startswith(name)
    assert lib.gc_status_string(99).decode() == "unknown gc_status"


class HostBatch:
    """A batch whose device pointers are fake non-NULL values: only host checks
    may run on it (they all return before the first HIP call)."""

    def __init__(self, P, n, fake_dev=True):
        self.P = np.ascontiguousarray(P, np.int32)
        self.n = np.ascontiguousarray(n, np.int32)
        dev = 0x1000 if fake_dev else None
        self.desc = gc.BatchDesc(len(self.P),
                                 self.P.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                 self.n.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                 dev, dev, dev)


def geo(Hq=8, Hkv=2, D=128, S=16, NB=64, maxb=8):
    return gc.Geometry(Hq, Hkv, D, S, NB, maxb)


def append_status(lib, g, b, ptrs=(0x2000, 0x2000, 0x2000, 0x2000)):
    return lib.gc_kv_append(ctypes.byref(g) if g is not None else None,
                            ctypes.byref(b.desc) if b is not None else None, *ptrs, None)


NEVER_SPLIT = gc.PlanOptions(-1)


def run_status(lib, g, b, scale=0.125, ws=0x3000, ws_bytes=1 << 40, opts=NEVER_SPLIT,
               ptrs=(0x2000, 0x2000, 0x2000, 0x2000)):
    q, kp, vp, out = ptrs
    return lib.gc_prefix_prefill_run(ctypes.byref(g), ctypes.byref(b.desc),
                                     ctypes.byref(opts) if opts is not None else None,
                                     q, kp, vp, scale, out, None, ws, ws_bytes, None)


def test_null_arguments(lib):
    b = HostBatch([4], [3])
    assert append_status(lib, None, b) == -1
    assert append_status(lib, geo(), None) == -1
    assert append_status(lib, geo(), b, ptrs=(None, 0x2000, 0x2000, 0x2000)) == -1
    assert append_status(lib, geo(), HostBatch([4], [3], fake_dev=False)) == -1
    assert run_status(lib, geo(), b, ptrs=(0x2000, None, 0x2000, 0x2000)) == -1
    size = ctypes.c_size_t()
    assert lib.gc_prefix_prefill_workspace_size(ctypes.byref(geo()), ctypes.byref(b.desc),
                                                None, None) == -1


def test_bad_shapes(lib):
    b = HostBatch([4], [3])
    assert append_status(lib, geo(Hq=6, Hkv=4), b) == -2      # Hq % Hkv != 0
    assert append_status(lib, geo(Hkv=0), b) == -2
    assert append_status(lib, geo(), HostBatch([-1], [3])) == -2
    assert append_status(lib, geo(), HostBatch([4], [-3])) == -2
    assert append_status(lib, geo(NB=0), b) == -2
    assert run_status(lib, geo(), b, scale=float("nan")) == -2
    assert run_status(lib, geo(), b, scale=0.0) == -2
    bad = gc.PlanOptions(0)
    bad.reserved[3] = 1
    assert run_status(lib, geo(), b, opts=bad) == -2


def test_unsupported(lib):
    b = HostBatch([4], [3])
    assert append_status(lib, geo(D=96), b) == -3
    assert append_status(lib, geo(S=32), b) == -3
    assert append_status(lib, geo(Hq=256, Hkv=1), b) == -3


def test_tiling_option(lib):
    b = HostBatch([40], [3])
    bad = gc.PlanOptions(-1, 7)
    assert run_status(lib, geo(), b, opts=bad) == -2                  # not a gc_tiling value
    small = gc.PlanOptions(-1, gc.TILES_SMALL)
    assert run_status(lib, geo(Hq=32, Hkv=1), b, opts=small) == -3    # 32 heads per KV head
    # forced small tiles on 16 heads per KV head pass the host checks (a NULL pointer then fires)
    nul = (None, 0x2000, 0x2000, 0x2000)
    assert run_status(lib, geo(Hq=16, Hkv=1), b, opts=small, ptrs=nul) == -1
    # the two tilings plan different work lists: 300 tokens at 4 heads per KV head
    # are ten 128-row tiles or seventy-five 16-row tiles
    b = HostBatch([40], [300])
    sizes = {}
    for t in (gc.TILES_PREFILL, gc.TILES_SMALL, gc.TILES_WIDE):
        s = ctypes.c_size_t()
        assert lib.gc_prefix_prefill_workspace_size(ctypes.byref(geo(maxb=30)), ctypes.byref(b.desc),
                                                    ctypes.byref(gc.PlanOptions(-1, t)),
                                                    ctypes.byref(s)) == 0
        sizes[t] = s.value
    assert sizes[gc.TILES_SMALL] > sizes[gc.TILES_PREFILL] >= sizes[gc.TILES_WIDE]


def test_block_table_too_short(lib):
    assert append_status(lib, geo(maxb=2), HostBatch([20], [13])) == -4   # needs 3 pages
    # long enough: the next check (a NULL data pointer) is the one that fires,
    # so nothing is ever launched with the fake device pointers
    nul = (None, 0x2000, 0x2000, 0x2000)
    assert append_status(lib, geo(maxb=3), HostBatch([20], [13]), ptrs=nul) == -1
    # a request without new tokens needs no table entries
    assert append_status(lib, geo(maxb=1), HostBatch([500, 3], [0, 2]), ptrs=nul) == -1


def test_workspace_checks(lib):
    b = HostBatch([40], [9])
    size = ctypes.c_size_t()
    assert lib.gc_prefix_prefill_workspace_size(ctypes.byref(geo()), ctypes.byref(b.desc),
                                                ctypes.byref(NEVER_SPLIT), ctypes.byref(size)) == 0
    assert size.value > 0
    assert run_status(lib, geo(), b, ws=None) == -5
    assert run_status(lib, geo(), b, ws_bytes=size.value - 1) == -5
    assert lib.gc_prefix_prefill_plan(ctypes.byref(geo()), ctypes.byref(b.desc),
                                      ctypes.byref(NEVER_SPLIT), None, 0, None) == -5


def test_empty_batches_are_no_ops(lib):
    empty = HostBatch([], [], fake_dev=False)
    assert append_status(lib, geo(), empty, ptrs=(None, None, None, None)) == 0
    assert run_status(lib, geo(), empty, ptrs=(None, None, None, None), ws=None, ws_bytes=0) == 0
    no_tokens = HostBatch([100, 7], [0, 0], fake_dev=False)
    assert append_status(lib, geo(), no_tokens, ptrs=(None, None, None, None)) == 0
    size = ctypes.c_size_t(123)
    assert lib.gc_prefix_prefill_workspace_size(ctypes.byref(geo()), ctypes.byref(no_tokens.desc),
                                                None, ctypes.byref(size)) == 0
    assert size.value == 0


def test_split_grows_workspace(lib):
    b = HostBatch([4000], [300])
    sizes = []
    for tiles in (-1, 8):
        s = ctypes.c_size_t()
        assert lib.gc_prefix_prefill_workspace_size(ctypes.byref(geo(maxb=300)), ctypes.byref(b.desc),
                                                    ctypes.byref(gc.PlanOptions(tiles)),
                                                    ctypes.byref(s)) == 0
        sizes.append(s.value)
    assert sizes[1] > sizes[0]


def test_binding_refuses_missing_library(tmp_path):
    with pytest.raises(RuntimeError):
        gc.load_library(str(tmp_path / "nope.so"))


def test_fp8_entry_points_check_scales_on_the_host(lib):
    b = HostBatch([4], [3])
    g = geo()
    p = 0x2000

    def app(ks, vs, ptrs=(p, p, p, p)):
        kn, vn, kp, vp = ptrs
        return lib.gc_kv_append_fp8(ctypes.byref(g), ctypes.byref(b.desc), kn, vn, ks, vs, kp, vp, None)

    def run(ks, vs):
        return lib.gc_prefix_prefill_run_fp8(ctypes.byref(g), ctypes.byref(b.desc),
                                             ctypes.byref(NEVER_SPLIT), p, p, p, ks, vs, 0.125, p,
                                             None, 0x3000, 1 << 40, None)

    for ks, vs in ((0.0, 1.0), (1.0, -2.0), (float("nan"), 1.0), (1.0, float("inf")),
                   (1e-45, 1.0)):  # the last one: fl32(1 / scale) overflows
        assert app(ks, vs) == -2, (ks, vs)
        assert run(ks, vs) == -2, (ks, vs)
    assert app(0.5, 0.25, ptrs=(p, None, p, p)) == -1
    assert lib.gc_prefix_prefill_attention_fp8(ctypes.byref(g), ctypes.byref(b.desc), None, p, None, p,
                                               0.5, 0.5, 0.125, p, None, 0x3000, 1 << 40, None) == -1
    # an empty batch is a no-op even for 8-bit pools
    e = HostBatch([], [], fake_dev=False)
    assert lib.gc_kv_append_fp8(ctypes.byref(g), ctypes.byref(e.desc), None, None, 0.5, 0.5, None,
                                None, None) == 0


def test_prepare_entry_points_check_on_the_host(lib):
    b = HostBatch([4], [3])
    g = geo()
    p = 0x2000

    def prep(kn=p, vn=p, kp=p, ws_bytes=1 << 40):
        return lib.gc_prefix_prefill_prepare(ctypes.byref(g), ctypes.byref(b.desc), ctypes.byref(NEVER_SPLIT),
                                             kn, vn, kp, p, 0x3000, ws_bytes, None)

    assert prep(kn=None) == -1
    assert prep(vn=None) == -1
    assert prep(kp=None) == -1
    assert prep(ws_bytes=1) == -5
    assert lib.gc_prefix_prefill_prepare_fp8(ctypes.byref(g), ctypes.byref(b.desc), ctypes.byref(NEVER_SPLIT),
                                             p, p, 0.0, 1.0, p, p, 0x3000, 1 << 40, None) == -2
    e = HostBatch([], [], fake_dev=False)
    assert lib.gc_prefix_prefill_prepare(ctypes.byref(g), ctypes.byref(e.desc), None, None, None, None, None,
                                         None, 0, None) == 0


def test_run_with_append_checks_on_the_host(lib):
    b = HostBatch([4], [3])
    g = geo()
    p = 0x2000

    def call(q=p, kn=p, vn=p, kp=p, scale=0.125, out=p, ws_bytes=1 << 40, batch=b):
        return lib.gc_prefix_prefill_run_with_append(ctypes.byref(g), ctypes.byref(batch.desc),
                                                     ctypes.byref(NEVER_SPLIT), q, kn, vn, kp, p, scale, out,
                                                     None, 0x3000, ws_bytes, None)

    assert call(kn=None) == -1
    assert call(vn=None) == -1
    assert call(q=None) == -1
    assert call(kp=None) == -1
    assert call(out=None) == -1
    assert call(scale=0.0) == -2
    assert call(scale=float("nan")) == -2
    assert call(ws_bytes=1) == -5
    # nothing to do for a batch without new tokens, whatever the pointers
    e = HostBatch([], [], fake_dev=False)
    assert call(q=None, kn=None, vn=None, kp=None, out=None, ws_bytes=0, batch=e) == 0
