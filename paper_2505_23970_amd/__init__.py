"""Prefix-cached prefill attention on MI355X (gfx950): Python binding.

GreenCache (arXiv 2505.23970, §2.2, Fig. 1a) reuses the KV of a request's
cached context: the new tokens' KV is appended to the cache and the new
tokens attend over the cached prefix plus themselves. The work runs in the
HIP library libgreencache.so (C ABI in include/greencache.h); this module
only checks tensors and marshals pointers, shapes and the current stream.
PyTorch provides device memory and streams. There is no fallback path: if
the library is not built, every call raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(_HERE, "libgreencache.so")

GC_OK = 0
STATUS_NAMES = {0: "GC_OK", -1: "GC_ERR_NULL_ARG", -2: "GC_ERR_BAD_SHAPE", -3: "GC_ERR_UNSUPPORTED",
                -4: "GC_ERR_BLOCK_TABLE", -5: "GC_ERR_WORKSPACE", -6: "GC_ERR_HIP", -7: "GC_ERR_LENGTHS"}
GC_ERR_LENGTHS = -7

EXPORTED = ("gc_kv_append", "gc_prefix_prefill_workspace_size", "gc_prefix_prefill_plan",
            "gc_prefix_prefill_run", "gc_prefix_prefill_attention", "gc_kv_append_fp8",
            "gc_prefix_prefill_run_fp8", "gc_prefix_prefill_attention_fp8", "gc_prefix_prefill_prepare",
            "gc_prefix_prefill_prepare_fp8", "gc_prefix_prefill_run_with_append",
            "gc_prefix_prefill_plan_status", "gc_prefix_prefill_attention_noalloc", "gc_read_bandwidth_probe",
            "gc_mfma_peak_probe", "gc_status_string")
READ_PROBE_SINK_WORDS = 2048 * 256
MFMA_PROBE_SINK_FLOATS = 1024 * 256
MFMA_PROBE_PRODUCTS_PER_ITERATION = 1024 * 4 * 16
MFMA_PROBE_FLOPS_PER_PRODUCT = 32 * 32 * 16 * 2


class GcError(RuntimeError):
    def __init__(self, fn, status, lib=None):
        text = STATUS_NAMES.get(status, str(status))
        if lib is not None:
            try:
                text = lib.gc_status_string(status).decode()
            except Exception:
                pass
        super().__init__(f"{fn} failed: {text}")
        self.status = status


class Geometry(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("num_blocks", ctypes.c_int32), ("max_blocks_per_seq", ctypes.c_int32)]


class BatchDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32),
                ("prefix_lens_host", ctypes.POINTER(ctypes.c_int32)),
                ("new_lens_host", ctypes.POINTER(ctypes.c_int32)),
                ("prefix_lens_dev", ctypes.c_void_p),
                ("cu_new_lens_dev", ctypes.c_void_p),
                ("block_tables_dev", ctypes.c_void_p)]


class PlanOptions(ctypes.Structure):
    _fields_ = [("kv_split_tiles", ctypes.c_int32), ("tiling", ctypes.c_int32),
                ("reserved", ctypes.c_int32 * 6)]


# gc_tiling values
TILES_AUTO, TILES_PREFILL, TILES_SMALL, TILES_WIDE = 0, 1, 2, 3


_lib = None


def load_library(path: str | None = None):
    """Load libgreencache.so. Raises if it has not been built: there is no other path."""
    global _lib
    if path is None and _lib is not None:
        return _lib
    p = path or LIBRARY
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2505_23970_amd.build`")
    lib = ctypes.CDLL(p)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    G, Bp, O = ctypes.POINTER(Geometry), ctypes.POINTER(BatchDesc), ctypes.POINTER(PlanOptions)
    lib.gc_kv_append.restype = i32
    lib.gc_kv_append.argtypes = [G, Bp, vp, vp, vp, vp, vp]
    lib.gc_prefix_prefill_workspace_size.restype = i32
    lib.gc_prefix_prefill_workspace_size.argtypes = [G, Bp, O, ctypes.POINTER(ctypes.c_size_t)]
    lib.gc_prefix_prefill_plan.restype = i32
    lib.gc_prefix_prefill_plan.argtypes = [G, Bp, O, vp, ctypes.c_size_t, vp]
    for fn in (lib.gc_prefix_prefill_run, lib.gc_prefix_prefill_attention):
        fn.restype = i32
        fn.argtypes = [G, Bp, O, vp, vp, vp, ctypes.c_float, vp, vp, vp, ctypes.c_size_t, vp]
    f32 = ctypes.c_float
    lib.gc_kv_append_fp8.restype = i32
    lib.gc_kv_append_fp8.argtypes = [G, Bp, vp, vp, f32, f32, vp, vp, vp]
    for fn in (lib.gc_prefix_prefill_run_fp8, lib.gc_prefix_prefill_attention_fp8):
        fn.restype = i32
        fn.argtypes = [G, Bp, O, vp, vp, vp, f32, f32, f32, vp, vp, vp, ctypes.c_size_t, vp]
    lib.gc_prefix_prefill_prepare.restype = i32
    lib.gc_prefix_prefill_prepare.argtypes = [G, Bp, O, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.gc_prefix_prefill_prepare_fp8.restype = i32
    lib.gc_prefix_prefill_prepare_fp8.argtypes = [G, Bp, O, vp, vp, f32, f32, vp, vp, vp, ctypes.c_size_t, vp]
    lib.gc_prefix_prefill_run_with_append.restype = i32
    lib.gc_prefix_prefill_run_with_append.argtypes = [G, Bp, O, vp, vp, vp, vp, vp, f32, vp, vp, vp,
                                                      ctypes.c_size_t, vp]
    lib.gc_prefix_prefill_attention_noalloc.restype = i32
    lib.gc_prefix_prefill_attention_noalloc.argtypes = [G, Bp, O, vp, vp, vp, ctypes.c_float, vp, vp, vp]
    lib.gc_prefix_prefill_plan_status.restype = i32
    lib.gc_prefix_prefill_plan_status.argtypes = [vp, ctypes.c_size_t, vp]
    lib.gc_read_bandwidth_probe.restype = i32
    lib.gc_read_bandwidth_probe.argtypes = [vp, ctypes.c_size_t, vp, vp]
    lib.gc_mfma_peak_probe.restype = i32
    lib.gc_mfma_peak_probe.argtypes = [i32, vp, vp]
    lib.gc_status_string.restype = ctypes.c_char_p
    lib.gc_status_string.argtypes = [i32]
    if path is None:
        _lib = lib
    return lib


def _check(fn, status, lib):
    if status != GC_OK:
        raise GcError(fn, status, lib)


def _stream_handle(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _require(t, dtype, name, device=None):
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on the GPU (got {t.device})")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


class PagedBatch:
    """A ragged batch: host lengths (numpy) plus their device copies (torch).

    prefix_lens[r]: cached tokens of request r already in the pool;
    new_lens[r]: its new tokens; block_tables[r][p]: physical block of logical page p.
    """

    def __init__(self, prefix_lens, new_lens, block_tables, device="cuda"):
        import torch
        self._restore = None
        self.prefix_lens = np.ascontiguousarray(prefix_lens, dtype=np.int32)
        self.new_lens = np.ascontiguousarray(new_lens, dtype=np.int32)
        bt = np.ascontiguousarray(block_tables, dtype=np.int32)
        if bt.ndim != 2 or bt.shape[0] != self.prefix_lens.shape[0]:
            raise ValueError("block_tables must be [batch][max_blocks_per_seq]")
        self.block_tables_host = bt
        cu = np.zeros(self.prefix_lens.shape[0] + 1, np.int32)
        np.cumsum(self.new_lens, out=cu[1:])
        self.cu_new_lens = cu
        self.prefix_lens_dev = torch.from_numpy(self.prefix_lens.copy()).to(device)
        self.device = self.prefix_lens_dev.device  # concrete, e.g. cuda:0
        self.cu_new_lens_dev = torch.from_numpy(cu.copy()).to(self.device)
        self.block_tables_dev = torch.from_numpy(bt.copy()).to(self.device)
        self._desc = BatchDesc(
            int(self.prefix_lens.shape[0]),
            self.prefix_lens.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
            self.new_lens.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
            self.prefix_lens_dev.data_ptr(), self.cu_new_lens_dev.data_ptr(),
            self.block_tables_dev.data_ptr())

    @property
    def batch(self) -> int:
        return int(self.prefix_lens.shape[0])

    @property
    def total_new(self) -> int:
        return int(self.new_lens.sum())

    @property
    def max_blocks_per_seq(self) -> int:
        return int(self.block_tables_host.shape[1])

    def desc(self) -> BatchDesc:
        return self._desc


def geometry(num_q_heads, num_kv_heads, head_dim, num_blocks, max_blocks_per_seq, page_size=16):
    return Geometry(int(num_q_heads), int(num_kv_heads), int(head_dim), int(page_size),
                    int(num_blocks), int(max_blocks_per_seq))


def _geo_from_pools(k_pool, v_pool, q_heads, batch: PagedBatch):
    NB, Hkv, S, D = k_pool.shape
    if tuple(v_pool.shape) != (NB, Hkv, D, S):
        raise ValueError(f"v_pool must be [NB][Hkv][D][S] = {(NB, Hkv, D, S)}, got {tuple(v_pool.shape)}")
    return geometry(q_heads, Hkv, D, NB, batch.max_blocks_per_seq, S)


def _opts(kv_split_tiles, tiling=None):
    if kv_split_tiles is None and tiling is None:
        return None
    o = PlanOptions()
    o.kv_split_tiles = int(kv_split_tiles or 0)
    o.tiling = int(tiling or 0)
    return ctypes.byref(o)


def kv_append(k_new, v_new, k_pool, v_pool, batch: PagedBatch, stream=None):
    """Append the new tokens' K/V ([T][Hkv][D] bf16) into the pools in place."""
    import torch
    lib = load_library()
    for name, t in (("k_new", k_new), ("v_new", v_new), ("k_pool", k_pool), ("v_pool", v_pool)):
        _require(t, torch.bfloat16, name, batch.device)
    geo = _geo_from_pools(k_pool, v_pool, k_pool.shape[1], batch)
    T, Hkv, D = k_new.shape
    if (T, Hkv, D) != (batch.total_new, geo.num_kv_heads, geo.head_dim) or v_new.shape != k_new.shape:
        raise ValueError("k_new/v_new must be [T][Hkv][D] matching the batch and pools")
    st = lib.gc_kv_append(ctypes.byref(geo), ctypes.byref(batch.desc()), k_new.data_ptr(),
                          v_new.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(),
                          _stream_handle(stream))
    _check("gc_kv_append", st, lib)


def kv_restore(k_src, v_src, k_pool, v_pool, batch: PagedBatch, stream=None):
    """Restore the cached prefixes into the pools: positions 0 .. P_r - 1 of every
    request from k_src / v_src ([sum P_r][Hkv][D] bf16, request-major). The sources
    may be pinned host tensors, which the GPU reads directly over PCIe (the cache's
    CPU tier), or device tensors. This is gc_kv_append with prefix lengths 0 and new
    lengths P_r; the restore batch's device arrays are built once per PagedBatch."""
    import torch
    lib = load_library()
    for name, t in (("k_src", k_src), ("v_src", v_src)):
        if t.dtype != torch.bfloat16 or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous bfloat16 tensor")
        if t.device.type == "cpu" and not t.is_pinned():
            raise ValueError(f"{name} is in pageable host memory: the GPU reads only pinned host memory")
        if t.device.type != "cpu" and t.device != batch.device:
            raise ValueError(f"{name} is on {t.device}, the batch on {batch.device}")
    for name, t in (("k_pool", k_pool), ("v_pool", v_pool)):
        _require(t, torch.bfloat16, name, batch.device)
    if getattr(batch, "_restore", None) is None:
        batch._restore = PagedBatch(np.zeros_like(batch.prefix_lens), batch.prefix_lens,
                                    batch.block_tables_host, device=batch.device)
    rb = batch._restore
    geo = _geo_from_pools(k_pool, v_pool, k_pool.shape[1], rb)
    T, Hkv, D = k_src.shape
    if (T, Hkv, D) != (rb.total_new, geo.num_kv_heads, geo.head_dim) or v_src.shape != k_src.shape:
        raise ValueError("k_src/v_src must be [sum of prefix lengths][Hkv][D] matching the batch and pools")
    st = lib.gc_kv_append(ctypes.byref(geo), ctypes.byref(rb.desc()), k_src.data_ptr(), v_src.data_ptr(),
                          k_pool.data_ptr(), v_pool.data_ptr(), _stream_handle(stream))
    _check("gc_kv_append (restore)", st, lib)


def workspace_size(num_q_heads, k_pool, v_pool, batch: PagedBatch, kv_split_tiles=None,
                   tiling=None) -> int:
    lib = load_library()
    geo = _geo_from_pools(k_pool, v_pool, num_q_heads, batch)
    out = ctypes.c_size_t(0)
    st = lib.gc_prefix_prefill_workspace_size(ctypes.byref(geo), ctypes.byref(batch.desc()),
                                              _opts(kv_split_tiles, tiling), ctypes.byref(out))
    _check("gc_prefix_prefill_workspace_size", st, lib)
    return int(out.value)


def alloc_workspace(num_q_heads, k_pool, v_pool, batch: PagedBatch, kv_split_tiles=None, tiling=None):
    import torch
    n = workspace_size(num_q_heads, k_pool, v_pool, batch, kv_split_tiles, tiling)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=batch.device)


def _attn_args(q, k_pool, v_pool, batch, out, lse, workspace, pool_dtype=None):
    import torch
    pool_dtype = pool_dtype or torch.bfloat16
    _require(q, torch.bfloat16, "q", batch.device)
    _require(k_pool, pool_dtype, "k_pool", batch.device)
    _require(v_pool, pool_dtype, "v_pool", batch.device)
    T, Hq, D = q.shape
    geo = _geo_from_pools(k_pool, v_pool, Hq, batch)
    if T != batch.total_new or D != geo.head_dim:
        raise ValueError("q must be [T][Hq][D] matching the batch and pools")
    if out is None:
        out = torch.empty_like(q)
    _require(out, torch.bfloat16, "out", batch.device)
    if tuple(out.shape) != tuple(q.shape):
        raise ValueError("out must have q's shape")
    if lse is not None:
        _require(lse, torch.float32, "lse", batch.device)
        if tuple(lse.shape) != (T, Hq):
            raise ValueError("lse must be [T][Hq] float32")
    if workspace is not None:
        _require(workspace, torch.uint8, "workspace", batch.device)
    return geo, out


def plan(num_q_heads, k_pool, v_pool, batch: PagedBatch, workspace, kv_split_tiles=None, stream=None,
         tiling=None):
    import torch
    lib = load_library()
    _require(workspace, torch.uint8, "workspace", batch.device)
    geo = _geo_from_pools(k_pool, v_pool, num_q_heads, batch)
    st = lib.gc_prefix_prefill_plan(ctypes.byref(geo), ctypes.byref(batch.desc()),
                                    _opts(kv_split_tiles, tiling), workspace.data_ptr(),
                                    workspace.numel(), _stream_handle(stream))
    _check("gc_prefix_prefill_plan", st, lib)


NOALLOC_SCRATCH_BYTES = 64 << 20


def prefix_prefill_attention_noalloc(q, k_pool, v_pool, batch: PagedBatch, scale, out=None, lse=None,
                                     kv_split_tiles=None, stream=None, tiling=None):
    """gc_prefix_prefill_attention_noalloc: plan and attention with the library's own
    static device scratch instead of a caller workspace (for callers that cannot
    allocate). Calls that overlap on one GPU race on that scratch."""
    lib = load_library()
    geo, out = _attn_args(q, k_pool, v_pool, batch, out, lse, None)
    st = lib.gc_prefix_prefill_attention_noalloc(ctypes.byref(geo), ctypes.byref(batch.desc()),
                                                 _opts(kv_split_tiles, tiling), q.data_ptr(), k_pool.data_ptr(),
                                                 v_pool.data_ptr(), float(scale), out.data_ptr(),
                                                 lse.data_ptr() if lse is not None else None,
                                                 _stream_handle(stream))
    _check("gc_prefix_prefill_attention_noalloc", st, lib)
    return out


def plan_status(workspace, stream=None) -> int:
    """Status of the last plan in `workspace` (waits for the stream): GC_OK when the
    device lengths agreed with the host's, GC_ERR_LENGTHS when they did not (the plan
    then holds no work). Other failures raise."""
    import torch
    lib = load_library()
    _require(workspace, torch.uint8, "workspace")
    st = lib.gc_prefix_prefill_plan_status(workspace.data_ptr(), workspace.numel(), _stream_handle(stream))
    if st not in (GC_OK, GC_ERR_LENGTHS):
        _check("gc_prefix_prefill_plan_status", st, lib)
    return int(st)


def run(q, k_pool, v_pool, batch: PagedBatch, scale, workspace, out=None, lse=None,
        kv_split_tiles=None, stream=None, tiling=None):
    lib = load_library()
    geo, out = _attn_args(q, k_pool, v_pool, batch, out, lse, workspace)
    st = lib.gc_prefix_prefill_run(ctypes.byref(geo), ctypes.byref(batch.desc()),
                                   _opts(kv_split_tiles, tiling), q.data_ptr(), k_pool.data_ptr(),
                                   v_pool.data_ptr(), float(scale), out.data_ptr(),
                                   lse.data_ptr() if lse is not None else None,
                                   workspace.data_ptr(), workspace.numel(), _stream_handle(stream))
    _check("gc_prefix_prefill_run", st, lib)
    return out


def run_with_append(q, k_new, v_new, k_pool, v_pool, batch: PagedBatch, scale, workspace, out=None, lse=None,
                    kv_split_tiles=None, stream=None, tiling=None):
    """Append the new tokens' K/V (bf16 [T][Hkv][D]) into the pools and run the attention,
    in one launch with prefill tiles, from a plan already in `workspace`."""
    import torch
    lib = load_library()
    geo, out = _attn_args(q, k_pool, v_pool, batch, out, lse, workspace)
    for name, t in (("k_new", k_new), ("v_new", v_new)):
        _require(t, torch.bfloat16, name, batch.device)
    if tuple(k_new.shape) != (batch.total_new, geo.num_kv_heads, geo.head_dim) or v_new.shape != k_new.shape:
        raise ValueError("k_new/v_new must be [T][Hkv][D] matching the batch and pools")
    st = lib.gc_prefix_prefill_run_with_append(
        ctypes.byref(geo), ctypes.byref(batch.desc()), _opts(kv_split_tiles, tiling), q.data_ptr(),
        k_new.data_ptr(), v_new.data_ptr(), k_pool.data_ptr(), v_pool.data_ptr(), float(scale), out.data_ptr(),
        lse.data_ptr() if lse is not None else None, workspace.data_ptr(), workspace.numel(),
        _stream_handle(stream))
    _check("gc_prefix_prefill_run_with_append", st, lib)
    return out


def read_bandwidth_probe(buf, sink=None, stream=None):
    """Enqueue one streaming read of every byte of `buf` (a device tensor whose size
    is a multiple of 16 bytes); returns the sink tensor it writes."""
    import torch
    lib = load_library()
    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous device tensor")
    if sink is None:
        sink = torch.empty(READ_PROBE_SINK_WORDS, dtype=torch.int32, device=buf.device)
    st = lib.gc_read_bandwidth_probe(buf.data_ptr(), buf.numel() * buf.element_size(), sink.data_ptr(),
                                     _stream_handle(stream))
    _check("gc_read_bandwidth_probe", st, lib)
    return sink


def mfma_peak_probe(iterations, sink=None, device=None, stream=None):
    """Enqueue the matrix-core calibration loop (`iterations` rounds of
    MFMA_PROBE_PRODUCTS_PER_ITERATION bf16 32x32x16 products); returns the sink
    tensor it writes (every entry 4096 * iterations)."""
    import torch
    lib = load_library()
    if sink is None:
        sink = torch.empty(MFMA_PROBE_SINK_FLOATS, dtype=torch.float32, device=device or "cuda")
    _require(sink, torch.float32, "sink")
    if sink.numel() < MFMA_PROBE_SINK_FLOATS:
        raise ValueError(f"sink needs {MFMA_PROBE_SINK_FLOATS} floats")
    st = lib.gc_mfma_peak_probe(int(iterations), sink.data_ptr(), _stream_handle(stream))
    _check("gc_mfma_peak_probe", st, lib)
    return sink


def prefix_prefill_attention(q, k_pool, v_pool, batch: PagedBatch, scale, workspace=None,
                             out=None, lse=None, kv_split_tiles=None, stream=None, tiling=None):
    """Attention of the new tokens (q: [T][Hq][D] bf16) over cached prefix + new keys.

    The pools must already hold the new tokens' K/V (call kv_append first).
    Returns out ([T][Hq][D] bf16); fills lse ([T][Hq] fp32) when given.
    """
    lib = load_library()
    if workspace is None:
        workspace = alloc_workspace(q.shape[1], k_pool, v_pool, batch, kv_split_tiles, tiling)
    geo, out = _attn_args(q, k_pool, v_pool, batch, out, lse, workspace)
    st = lib.gc_prefix_prefill_attention(ctypes.byref(geo), ctypes.byref(batch.desc()),
                                         _opts(kv_split_tiles, tiling), q.data_ptr(), k_pool.data_ptr(),
                                         v_pool.data_ptr(), float(scale), out.data_ptr(),
                                         lse.data_ptr() if lse is not None else None,
                                         workspace.data_ptr(), workspace.numel(),
                                         _stream_handle(stream))
    _check("gc_prefix_prefill_attention", st, lib)
    return out


# ----------------------------------------------------------------- 8-bit (E4M3) pools
# Pools are uint8 tensors of E4M3 codes with the bf16 pools' shapes; each pool has
# one scale (element = code value * scale). See include/greencache.h.

def kv_append_fp8(k_new, v_new, k_pool8, v_pool8, batch: PagedBatch, k_scale, v_scale, stream=None):
    """Quantise the new tokens' K/V ([T][Hkv][D] bf16) into the 8-bit pools in place."""
    import torch
    lib = load_library()
    for name, t in (("k_new", k_new), ("v_new", v_new)):
        _require(t, torch.bfloat16, name, batch.device)
    for name, t in (("k_pool8", k_pool8), ("v_pool8", v_pool8)):
        _require(t, torch.uint8, name, batch.device)
    geo = _geo_from_pools(k_pool8, v_pool8, k_pool8.shape[1], batch)
    T, Hkv, D = k_new.shape
    if (T, Hkv, D) != (batch.total_new, geo.num_kv_heads, geo.head_dim) or v_new.shape != k_new.shape:
        raise ValueError("k_new/v_new must be [T][Hkv][D] matching the batch and pools")
    st = lib.gc_kv_append_fp8(ctypes.byref(geo), ctypes.byref(batch.desc()), k_new.data_ptr(),
                              v_new.data_ptr(), float(k_scale), float(v_scale), k_pool8.data_ptr(),
                              v_pool8.data_ptr(), _stream_handle(stream))
    _check("gc_kv_append_fp8", st, lib)


def run_fp8(q, k_pool8, v_pool8, batch: PagedBatch, scale, k_scale, v_scale, workspace, out=None,
            lse=None, kv_split_tiles=None, stream=None, tiling=None):
    import torch
    lib = load_library()
    geo, out = _attn_args(q, k_pool8, v_pool8, batch, out, lse, workspace, torch.uint8)
    st = lib.gc_prefix_prefill_run_fp8(ctypes.byref(geo), ctypes.byref(batch.desc()),
                                       _opts(kv_split_tiles, tiling), q.data_ptr(), k_pool8.data_ptr(),
                                       v_pool8.data_ptr(), float(k_scale), float(v_scale), float(scale),
                                       out.data_ptr(), lse.data_ptr() if lse is not None else None,
                                       workspace.data_ptr(), workspace.numel(), _stream_handle(stream))
    _check("gc_prefix_prefill_run_fp8", st, lib)
    return out


def prefix_prefill_attention_fp8(q, k_pool8, v_pool8, batch: PagedBatch, scale, k_scale, v_scale,
                                 workspace=None, out=None, lse=None, kv_split_tiles=None,
                                 stream=None, tiling=None):
    """prefix_prefill_attention over 8-bit pools (uint8 E4M3 codes, one scale per pool)."""
    import torch
    lib = load_library()
    if workspace is None:
        workspace = alloc_workspace(q.shape[1], k_pool8, v_pool8, batch, kv_split_tiles, tiling)
    geo, out = _attn_args(q, k_pool8, v_pool8, batch, out, lse, workspace, torch.uint8)
    st = lib.gc_prefix_prefill_attention_fp8(ctypes.byref(geo), ctypes.byref(batch.desc()),
                                             _opts(kv_split_tiles, tiling), q.data_ptr(),
                                             k_pool8.data_ptr(), v_pool8.data_ptr(), float(k_scale),
                                             float(v_scale), float(scale), out.data_ptr(),
                                             lse.data_ptr() if lse is not None else None,
                                             workspace.data_ptr(), workspace.numel(),
                                             _stream_handle(stream))
    _check("gc_prefix_prefill_attention_fp8", st, lib)
    return out


def prepare(k_new, v_new, k_pool, v_pool, batch: PagedBatch, num_q_heads, workspace, kv_split_tiles=None,
            stream=None, tiling=None, k_scale=None, v_scale=None):
    """Append the new tokens' K/V and plan the attention in one launch (then call run
    or run_fp8 with the same options). 8-bit pools (uint8) take k_scale and v_scale."""
    import torch
    lib = load_library()
    fp8 = k_pool.dtype == torch.uint8
    for name, t in (("k_new", k_new), ("v_new", v_new)):
        _require(t, torch.bfloat16, name, batch.device)
    for name, t in (("k_pool", k_pool), ("v_pool", v_pool)):
        _require(t, torch.uint8 if fp8 else torch.bfloat16, name, batch.device)
    _require(workspace, torch.uint8, "workspace", batch.device)
    geo = _geo_from_pools(k_pool, v_pool, num_q_heads, batch)
    T, Hkv, D = k_new.shape
    if (T, Hkv, D) != (batch.total_new, geo.num_kv_heads, geo.head_dim) or v_new.shape != k_new.shape:
        raise ValueError("k_new/v_new must be [T][Hkv][D] matching the batch and pools")
    head = (ctypes.byref(geo), ctypes.byref(batch.desc()), _opts(kv_split_tiles, tiling), k_new.data_ptr(),
            v_new.data_ptr())
    tail = (k_pool.data_ptr(), v_pool.data_ptr(), workspace.data_ptr(), workspace.numel(), _stream_handle(stream))
    if fp8:
        if k_scale is None or v_scale is None:
            raise ValueError("8-bit pools need k_scale and v_scale")
        st = lib.gc_prefix_prefill_prepare_fp8(*head, float(k_scale), float(v_scale), *tail)
        _check("gc_prefix_prefill_prepare_fp8", st, lib)
    else:
        st = lib.gc_prefix_prefill_prepare(*head, *tail)
        _check("gc_prefix_prefill_prepare", st, lib)
