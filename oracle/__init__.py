"""fp64 CPU oracle for prefix-cached prefill attention and the KV append.

TEST INFRASTRUCTURE. Only tests/, the package smoke check and the benchmark's
CPU-baseline leg may import this package. The product path (the HIP library
and its Python binding) shares no code with it and never calls it.

The arithmetic lives in gc_oracle.c (plain loops, double precision, OpenMP
over output rows); this module only marshals numpy arrays through ctypes.
Definition followed: GreenCache §2.2 "Caching for LLM Serving" (Fig. 1a:
cached prefix KV and new tokens' KV processed together, new KV saved) and
§2.1 (Transformer prefill), read as textbook causal scaled-dot-product
attention with grouped KV heads.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .build import LIBRARY, build_oracle

_lib = None


def load(path: str | None = None):
    """Load (building first if needed) the oracle library. A path other than the
    default loads that library instead (used for planted-mistake variants)."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIBRARY):
            build_oracle()
        _lib = _bind(ctypes.CDLL(LIBRARY))
    return _lib


def _bind(lib):
    i32p = ctypes.POINTER(ctypes.c_int32)
    u16p = ctypes.POINTER(ctypes.c_uint16)
    f64p = ctypes.POINTER(ctypes.c_double)
    i64p = ctypes.POINTER(ctypes.c_int64)
    c_int = ctypes.c_int
    lib.gco_kv_append.restype = c_int
    lib.gco_kv_append.argtypes = [c_int, i32p, i32p, i32p, c_int, c_int, c_int, c_int, c_int,
                                  u16p, u16p, u16p, u16p]
    lib.gco_attention.restype = c_int
    lib.gco_attention.argtypes = [c_int, i32p, i32p, i32p, c_int, c_int, c_int, c_int, c_int,
                                  c_int, u16p, u16p, u16p, ctypes.c_double, ctypes.c_int64,
                                  i64p, f64p, f64p, c_int]
    lib.gco_widen_bf16.restype = None
    lib.gco_widen_bf16.argtypes = [ctypes.c_int64, u16p, f64p]
    lib.gco_max_threads.restype = c_int
    lib.gco_max_threads.argtypes = []
    u8p = ctypes.POINTER(ctypes.c_uint8)
    lib.gco_e4m3_value.restype = ctypes.c_double
    lib.gco_e4m3_value.argtypes = [ctypes.c_uint8]
    lib.gco_e4m3_encode.restype = ctypes.c_uint8
    lib.gco_e4m3_encode.argtypes = [ctypes.c_float]
    lib.gco_quantize_e4m3.restype = None
    lib.gco_quantize_e4m3.argtypes = [ctypes.c_int64, u16p, ctypes.c_float, u8p]
    lib.gco_kv_append_e4m3.restype = c_int
    lib.gco_kv_append_e4m3.argtypes = [c_int, i32p, i32p, i32p, c_int, c_int, c_int, c_int, c_int,
                                       u16p, u16p, ctypes.c_float, ctypes.c_float, u8p, u8p]
    lib.gco_attention_e4m3.restype = c_int
    lib.gco_attention_e4m3.argtypes = [c_int, i32p, i32p, i32p, c_int, c_int, c_int, c_int, c_int,
                                       c_int, u16p, u8p, u8p, ctypes.c_double, ctypes.c_double,
                                       ctypes.c_double, ctypes.c_int64, i64p, f64p, f64p, c_int]
    return lib


def _p(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


class OracleError(RuntimeError):
    pass


def kv_append(prefix_lens, new_lens, block_tables, num_blocks, k_new, v_new, k_pool, v_pool,
              lib=None):
    """Return copies of (k_pool, v_pool) after appending the new tokens' K/V.

    k_pool: uint16 [NB][Hkv][S][D]; v_pool: uint16 [NB][Hkv][D][S];
    k_new, v_new: uint16 [T][Hkv][D] (bf16 bit patterns).
    """
    lib = lib or load()
    P = _c(prefix_lens, np.int32)
    n = _c(new_lens, np.int32)
    bt = _c(block_tables, np.int32)
    kp = np.array(k_pool, dtype=np.uint16, copy=True, order="C")
    vp = np.array(v_pool, dtype=np.uint16, copy=True, order="C")
    NB, Hkv, S, D = kp.shape
    assert vp.shape == (NB, Hkv, D, S)
    kn = _c(k_new, np.uint16)
    vn = _c(v_new, np.uint16)
    st = lib.gco_kv_append(int(P.shape[0]), _p(P, ctypes.c_int32), _p(n, ctypes.c_int32),
                           _p(bt, ctypes.c_int32), int(bt.shape[1]) if bt.ndim == 2 else 0,
                           int(num_blocks), int(Hkv), int(D), int(S),
                           _p(kn, ctypes.c_uint16), _p(vn, ctypes.c_uint16),
                           _p(kp, ctypes.c_uint16), _p(vp, ctypes.c_uint16))
    if st != 0:
        raise OracleError(f"gco_kv_append returned {st}")
    return kp, vp


def attention(prefix_lens, new_lens, block_tables, num_blocks, q, k_pool, v_pool, scale,
              rows=None, num_threads=0, lib=None):
    """fp64 attention of the new tokens over (cached prefix + new tokens).

    q: uint16 [T][Hq][D]. rows: optional int64 array of row ids (token*Hq + head);
    returns (out [n_rows][D] float64, lse [n_rows] float64), all rows when rows is None.
    The pools must already hold the new tokens' K/V (call kv_append first).
    """
    lib = lib or load()
    P = _c(prefix_lens, np.int32)
    n = _c(new_lens, np.int32)
    bt = _c(block_tables, np.int32)
    qq = _c(q, np.uint16)
    kp = _c(k_pool, np.uint16)
    vp = _c(v_pool, np.uint16)
    T, Hq, D = qq.shape
    NB, Hkv, S, D2 = kp.shape
    assert D2 == D
    if rows is None:
        nrows = T * Hq
        rows_p = None
    else:
        rows = _c(rows, np.int64)
        nrows = int(rows.shape[0])
        rows_p = _p(rows, ctypes.c_int64)
    out = np.zeros((nrows, D), np.float64)
    lse = np.zeros(nrows, np.float64)
    st = lib.gco_attention(int(P.shape[0]), _p(P, ctypes.c_int32), _p(n, ctypes.c_int32),
                           _p(bt, ctypes.c_int32), int(bt.shape[1]) if bt.ndim == 2 else 0,
                           int(num_blocks), int(Hq), int(Hkv), int(D), int(S),
                           _p(qq, ctypes.c_uint16), _p(kp, ctypes.c_uint16),
                           _p(vp, ctypes.c_uint16), float(scale), nrows, rows_p,
                           _p(out, ctypes.c_double), _p(lse, ctypes.c_double), int(num_threads))
    if st != 0:
        raise OracleError(f"gco_attention returned {st}")
    return out, lse


def inv_scale(scale) -> np.float32:
    """fl32(1 / scale): the factor every stored 8-bit element is quantised with."""
    return np.float32(1.0) / np.float32(scale)


def e4m3_value(code, lib=None) -> float:
    """Value of one E4M3 code (NaN for S.1111.111)."""
    return float((lib or load()).gco_e4m3_value(int(code)))


def e4m3_encode(v, lib=None) -> int:
    """Code stored for the fp32 value v (clamped to +-448, nearest, ties to even)."""
    return int((lib or load()).gco_e4m3_encode(float(np.float32(v))))


def quantize_e4m3(bits, scale, lib=None) -> np.ndarray:
    """Codes for bf16 bit patterns `bits` quantised with fl32(1 / scale)."""
    lib = lib or load()
    b = _c(bits, np.uint16)
    out = np.empty(b.shape, np.uint8)
    lib.gco_quantize_e4m3(int(b.size), _p(b, ctypes.c_uint16), float(inv_scale(scale)),
                          _p(out, ctypes.c_uint8))
    return out


def kv_append_e4m3(prefix_lens, new_lens, block_tables, num_blocks, k_new, v_new, k_pool, v_pool,
                   k_scale, v_scale, lib=None):
    """Return copies of 8-bit (k_pool, v_pool) (uint8, bf16 pool shapes) after
    quantising and appending the new tokens' K/V."""
    lib = lib or load()
    P = _c(prefix_lens, np.int32)
    n = _c(new_lens, np.int32)
    bt = _c(block_tables, np.int32)
    kp = np.array(k_pool, dtype=np.uint8, copy=True, order="C")
    vp = np.array(v_pool, dtype=np.uint8, copy=True, order="C")
    NB, Hkv, S, D = kp.shape
    assert vp.shape == (NB, Hkv, D, S)
    kn = _c(k_new, np.uint16)
    vn = _c(v_new, np.uint16)
    st = lib.gco_kv_append_e4m3(int(P.shape[0]), _p(P, ctypes.c_int32), _p(n, ctypes.c_int32),
                                _p(bt, ctypes.c_int32), int(bt.shape[1]) if bt.ndim == 2 else 0,
                                int(num_blocks), int(Hkv), int(D), int(S),
                                _p(kn, ctypes.c_uint16), _p(vn, ctypes.c_uint16),
                                float(inv_scale(k_scale)), float(inv_scale(v_scale)),
                                _p(kp, ctypes.c_uint8), _p(vp, ctypes.c_uint8))
    if st != 0:
        raise OracleError(f"gco_kv_append_e4m3 returned {st}")
    return kp, vp


def attention_e4m3(prefix_lens, new_lens, block_tables, num_blocks, q, k_pool, v_pool, k_scale,
                   v_scale, scale, rows=None, num_threads=0, lib=None):
    """fp64 attention over 8-bit pools (every element dequantised first); same
    return values as attention()."""
    lib = lib or load()
    P = _c(prefix_lens, np.int32)
    n = _c(new_lens, np.int32)
    bt = _c(block_tables, np.int32)
    qq = _c(q, np.uint16)
    kp = _c(k_pool, np.uint8)
    vp = _c(v_pool, np.uint8)
    T, Hq, D = qq.shape
    NB, Hkv, S, D2 = kp.shape
    assert D2 == D
    if rows is None:
        nrows = T * Hq
        rows_p = None
    else:
        rows = _c(rows, np.int64)
        nrows = int(rows.shape[0])
        rows_p = _p(rows, ctypes.c_int64)
    out = np.zeros((nrows, D), np.float64)
    lse = np.zeros(nrows, np.float64)
    st = lib.gco_attention_e4m3(int(P.shape[0]), _p(P, ctypes.c_int32), _p(n, ctypes.c_int32),
                                _p(bt, ctypes.c_int32), int(bt.shape[1]) if bt.ndim == 2 else 0,
                                int(num_blocks), int(Hq), int(Hkv), int(D), int(S),
                                _p(qq, ctypes.c_uint16), _p(kp, ctypes.c_uint8),
                                _p(vp, ctypes.c_uint8), float(k_scale), float(v_scale), float(scale),
                                nrows, rows_p, _p(out, ctypes.c_double), _p(lse, ctypes.c_double),
                                int(num_threads))
    if st != 0:
        raise OracleError(f"gco_attention_e4m3 returned {st}")
    return out, lse


def widen_bf16(bits, lib=None) -> np.ndarray:
    lib = lib or load()
    b = _c(bits, np.uint16).ravel()
    out = np.empty(b.shape[0], np.float64)
    lib.gco_widen_bf16(int(b.shape[0]), _p(b, ctypes.c_uint16), _p(out, ctypes.c_double))
    return out


def max_threads(lib=None) -> int:
    return int((lib or load()).gco_max_threads())


def run_workload(w, rows=None, num_threads=0, lib=None):
    """Append then attention for a workloads.Workload; returns (k_pool, v_pool, out, lse)."""
    kp, vp = kv_append(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks,
                       w.k_new, w.v_new, w.k_pool, w.v_pool, lib=lib)
    out, lse = attention(w.prefix_lens, w.new_lens, w.block_tables, w.num_blocks, w.q, kp, vp,
                         w.scale, rows=rows, num_threads=num_threads, lib=lib)
    return kp, vp, out, lse
