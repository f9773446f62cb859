"""CPU oracle for session-prefill attention -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the bench's CPU-baseline leg
may import this package.  The product path (``paper_2607_17181_amd``) never
does and has no CPU fallback.

The arithmetic lives in ``sp_attn_oracle.c`` (fp64 on bf16 inputs, plain
two-pass softmax, block-table walk written independently of the HIP
library); this module only marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np

from .build import LIB, build

_libs = {}


def _load(path: Optional[str] = None):
    """Load (once) the oracle library at ``path`` (default: the built oracle)."""
    path = path or LIB
    if path not in _libs:
        if path == LIB and not os.path.exists(LIB):
            build()
        lib = ctypes.CDLL(path)
        p = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        lib.oracle_append_kv.argtypes = [i32, p, p, p, i64, i32, i64, i32, i32, p, p, p, p]
        lib.oracle_gather_kv.argtypes = [i32, p, p, p, i64, i32, i64, i32, i32, p, p, p, p]
        lib.oracle_sp_attention.argtypes = [i32, p, p, p, i64, i32, i64, i32, i32, i32, f64,
                                            p, p, p, i64, p, p, p]
        lib.oracle_attention_contiguous.argtypes = [i32, p, p, i32, i32, i32, f64, p, p, p,
                                                    i64, p, p, p]
        lib.oracle_num_threads.argtypes = []
        for f in (lib.oracle_append_kv, lib.oracle_gather_kv, lib.oracle_sp_attention,
                  lib.oracle_attention_contiguous, lib.oracle_num_threads):
            f.restype = ctypes.c_int
        _libs[path] = lib
    return _libs[path]


def _ptr(a: np.ndarray) -> ctypes.c_void_p:
    return ctypes.c_void_p(a.ctypes.data)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _u16(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.uint16)


def num_threads(lib_path: Optional[str] = None) -> int:
    """OpenMP threads the oracle runs on."""
    return int(_load(lib_path).oracle_num_threads())


def append_kv(prefix_lens, suffix_lens, block_tables, page_size: int,
              k_new: np.ndarray, v_new: np.ndarray, k_pool: np.ndarray,
              v_pool: np.ndarray, lib_path: Optional[str] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Return copies of the pools with every new token's K/V row scattered in."""
    pre, suf, bt = _i32(prefix_lens), _i32(suffix_lens), _i32(block_tables)
    kp, vp = np.array(k_pool, dtype=np.uint16, copy=True), np.array(v_pool, dtype=np.uint16, copy=True)
    kn, vn = _u16(k_new), _u16(v_new)
    Hkv, d = kp.shape[1], kp.shape[3]
    rc = _load(lib_path).oracle_append_kv(pre.shape[0], _ptr(pre), _ptr(suf), _ptr(bt), bt.shape[1],
                                  page_size, kp.shape[0], Hkv, d, _ptr(kn), _ptr(vn),
                                  _ptr(kp), _ptr(vp))
    if rc != 0:
        raise ValueError(f"oracle_append_kv failed ({rc})")
    return kp, vp


def gather_kv(prefix_lens, suffix_lens, block_tables, page_size: int,
              k_pool: np.ndarray, v_pool: np.ndarray,
              lib_path: Optional[str] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Contiguous K/V rows [sum(P+S), Hkv, d] read from the pool through block tables."""
    pre, suf, bt = _i32(prefix_lens), _i32(suffix_lens), _i32(block_tables)
    kp, vp = _u16(k_pool), _u16(v_pool)
    n = int(pre.astype(np.int64).sum() + suf.astype(np.int64).sum())
    Hkv, d = kp.shape[1], kp.shape[3]
    ko = np.empty((n, Hkv, d), dtype=np.uint16)
    vo = np.empty_like(ko)
    rc = _load(lib_path).oracle_gather_kv(pre.shape[0], _ptr(pre), _ptr(suf), _ptr(bt), bt.shape[1],
                                  page_size, kp.shape[0], Hkv, d, _ptr(kp), _ptr(vp),
                                  _ptr(ko), _ptr(vo))
    if rc != 0:
        raise ValueError(f"oracle_gather_kv failed ({rc})")
    return ko, vo


def sp_attention(prefix_lens, suffix_lens, block_tables, page_size: int, q: np.ndarray,
                 k_pool: np.ndarray, v_pool: np.ndarray, rows: Optional[np.ndarray] = None,
                 sm_scale: float = 0.0,
                 lib_path: Optional[str] = None) -> Tuple[np.ndarray, np.ndarray]:
    """fp64 SP attention through block tables.

    ``q`` is [T, Hq, d] bf16 bits; the K pool is [num_pages, Hkv, page_size, d]
    and the V pool [num_pages, Hkv, d, page_size].
    Returns (o [R, d], lse [R]) for the flat rows ``rows`` (token * Hq + head),
    or (o [T, Hq, d], lse [T, Hq]) when ``rows`` is None.
    """
    pre, suf, bt = _i32(prefix_lens), _i32(suffix_lens), _i32(block_tables)
    qb, kp, vp = _u16(q), _u16(k_pool), _u16(v_pool)
    T, Hq, d = qb.shape
    Hkv = kp.shape[1]
    if rows is None:
        o = np.empty((T * Hq, d), dtype=np.float64)
        lse = np.empty(T * Hq, dtype=np.float64)
        rp, nr = None, T * Hq
    else:
        r = np.ascontiguousarray(rows, dtype=np.int64)
        o = np.empty((r.shape[0], d), dtype=np.float64)
        lse = np.empty(r.shape[0], dtype=np.float64)
        rp, nr = _ptr(r), r.shape[0]
    rc = _load(lib_path).oracle_sp_attention(pre.shape[0], _ptr(pre), _ptr(suf), _ptr(bt), bt.shape[1],
                                     page_size, kp.shape[0], Hq, Hkv, d, float(sm_scale),
                                     _ptr(qb), _ptr(kp), _ptr(vp), nr, rp, _ptr(o), _ptr(lse))
    if rc != 0:
        raise ValueError(f"oracle_sp_attention failed ({rc})")
    if rows is None:
        return o.reshape(T, Hq, d), lse.reshape(T, Hq)
    return o, lse


def attention_contiguous(prefix_lens, suffix_lens, q: np.ndarray, k_all: np.ndarray,
                         v_all: np.ndarray, rows: Optional[np.ndarray] = None,
                         sm_scale: float = 0.0,
                         lib_path: Optional[str] = None) -> Tuple[np.ndarray, np.ndarray]:
    """fp64 attention reading K/V from contiguous rows [sum(P+S), Hkv, d]."""
    pre, suf = _i32(prefix_lens), _i32(suffix_lens)
    qb, ka, va = _u16(q), _u16(k_all), _u16(v_all)
    T, Hq, d = qb.shape
    Hkv = ka.shape[1]
    if rows is None:
        o = np.empty((T * Hq, d), dtype=np.float64)
        lse = np.empty(T * Hq, dtype=np.float64)
        rp, nr = None, T * Hq
    else:
        r = np.ascontiguousarray(rows, dtype=np.int64)
        o = np.empty((r.shape[0], d), dtype=np.float64)
        lse = np.empty(r.shape[0], dtype=np.float64)
        rp, nr = _ptr(r), r.shape[0]
    rc = _load(lib_path).oracle_attention_contiguous(pre.shape[0], _ptr(pre), _ptr(suf), Hq, Hkv, d,
                                             float(sm_scale), _ptr(qb), _ptr(ka), _ptr(va), nr,
                                             rp, _ptr(o), _ptr(lse))
    if rc != 0:
        raise ValueError(f"oracle_attention_contiguous failed ({rc})")
    if rows is None:
        return o.reshape(T, Hq, d), lse.reshape(T, Hq)
    return o, lse
