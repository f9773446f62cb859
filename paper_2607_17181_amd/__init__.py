"""Python binding of libtalaria_sp_attn (session-prefill attention on MI355X).

Argument marshalling only: every step of the path (append, page gather,
prefill, combine, decode, page transfer, staging) runs in the HIP library,
and batch selection in its host code.  There is no CPU fallback; if the
library has not been built, every call raises.

The calls mirror the C ABI in ``include/talaria_sp_attn.h``:

    sp = plan(geom, prefix_lens, suffix_lens, max_pages_per_seq)
    check_tables(sp, host_block_tables)                               # opt-in, host only
    append_kv(sp, k_new, v_new, k_pool, v_pool, block_tables)
    prefill(sp, q, k_pool, v_pool, block_tables, out, lse, workspace)
    prefill_noalloc(sp, q, k_pool, v_pool, block_tables, out, lse)     # no workspace
    decode(sp, q, k_pool, v_pool, block_tables, out, lse, workspace)   # S_b <= 1
    gather_kv(sp, k_pool, v_pool, block_tables, k_out, v_out)
    calibrate_xcd(sp, q, k_pool, v_pool, block_tables, out, workspace)  # set-up: XCD order
    set_xcd_order(order) / get_xcd_order()
    hkvr_restore(cache, slab, page_ids, k_cache, v_cache)       # host -> device pages
    hkvr_checkpoint(cache, k_cache, v_cache, page_ids, slab)    # device pages -> host
    stage_mark_dirty(chunks, used_pages, num_pages, page_bytes, dirty)
    stage_gather(chunks, staged, dirty, staging, host_weights, weights)
    sp_select(candidates, cost_model, budget)                    # host only

Device arrays are ``torch`` tensors (bf16 data may also be passed as int16
or uint16 bit patterns); torch provides device memory and the current
stream, nothing else.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# The in-tree build, and only that one.
LIB_PATH = os.path.join(_PKG, "libtalaria_sp_attn.so")

OK, EINVAL, EUNSUPPORTED, ENOSPACE, EHIP = 0, -1, -2, -3, -4
MAX_SEQS = 128
PLAN_WORDS = 448
ITEM_FIELDS = ("seq", "kv_head", "first_token", "num_tokens", "key_begin", "key_end", "split",
               "num_splits")


class TalariaError(RuntimeError):
    """A negative status from the library; ``.status`` holds the code."""

    def __init__(self, status: int, message: str):
        super().__init__(f"[{status}] {message}")
        self.status = status


class Geom(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("num_pages", ctypes.c_int32)]


class KvCache(ctypes.Structure):
    """Geometry of a layer-first device KV cache (talaria_kv_cache)."""
    _fields_ = [("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("num_pages", ctypes.c_int32)]


class CostModel(ctypes.Structure):
    """talaria_sp_cost_model: predicted-cost coefficients of SP selection."""
    _fields_ = [("num_layers", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("attn_flops_per_s", ctypes.c_double),
                ("per_token_s", ctypes.c_double), ("restore_bytes_per_s", ctypes.c_double),
                ("batch_overhead_s", ctypes.c_double)]


class Budget(ctypes.Structure):
    """talaria_sp_budget: what the slot has left after protected decode."""
    _fields_ = [("time_budget_s", ctypes.c_double), ("free_pages", ctypes.c_int64),
                ("max_batch", ctypes.c_int32)]


class _RawPlan(ctypes.Structure):
    _fields_ = [("opaque", ctypes.c_uint64 * PLAN_WORDS)]


_lib = None


def library() -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -c 'import __graft_entry__ as g; g.build()'`")
        lib = ctypes.CDLL(LIB_PATH)
        p, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        lib.talaria_sp_attn_plan.argtypes = [ctypes.POINTER(Geom), i32, p, p, i32, i32,
                                             ctypes.POINTER(sz), ctypes.POINTER(_RawPlan)]
        lib.talaria_sp_attn_append_kv.argtypes = [ctypes.POINTER(_RawPlan), p, p, p, p, p, p]
        lib.talaria_sp_attn_prefill.argtypes = [ctypes.POINTER(_RawPlan), p, p, p, p,
                                                ctypes.c_float, p, p, p, sz, p]
        lib.talaria_sp_attn_prefill_noalloc.argtypes = [ctypes.POINTER(_RawPlan), p, p, p, p,
                                                        ctypes.c_float, p, p, p]
        lib.talaria_sp_attn_prefill_noalloc.restype = ctypes.c_int
        lib.talaria_sp_attn_noalloc_scratch_bytes.argtypes = []
        lib.talaria_sp_attn_noalloc_scratch_bytes.restype = ctypes.c_size_t
        lib.talaria_sp_attn_check_tables.argtypes = [ctypes.POINTER(_RawPlan), p]
        lib.talaria_sp_attn_check_tables.restype = ctypes.c_int
        lib.talaria_sp_attn_gather_kv.argtypes = [ctypes.POINTER(_RawPlan), p, p, p, p, p, p]
        lib.talaria_sp_attn_decode.argtypes = [ctypes.POINTER(_RawPlan), p, p, p, p,
                                               ctypes.c_float, p, p, p, sz, p]
        lib.talaria_sp_attn_decode.restype = ctypes.c_int
        lib.talaria_sp_attn_plan_items.argtypes = [ctypes.POINTER(_RawPlan), p, i32]
        for f in (lib.talaria_sp_attn_plan, lib.talaria_sp_attn_append_kv,
                  lib.talaria_sp_attn_prefill, lib.talaria_sp_attn_gather_kv,
                  lib.talaria_sp_attn_plan_items):
            f.restype = ctypes.c_int
        lib.talaria_hkvr_restore.argtypes = [ctypes.POINTER(KvCache), i32, p, p, p, p, p]
        lib.talaria_hkvr_checkpoint.argtypes = [ctypes.POINTER(KvCache), i32, p, p, p, p, p]
        lib.talaria_hkvr_restore.restype = ctypes.c_int
        lib.talaria_hkvr_checkpoint.restype = ctypes.c_int
        i64 = ctypes.c_int64
        lib.talaria_stage_mark_dirty.argtypes = [p, i32, p, i64, i64, p, p]
        lib.talaria_stage_gather.argtypes = [p, i32, p, p, p, i64, p, p, i64, p]
        lib.talaria_stage_mark_dirty.restype = ctypes.c_int
        lib.talaria_stage_gather.restype = ctypes.c_int
        lib.talaria_sp_select.argtypes = [p, i32, ctypes.POINTER(CostModel),
                                          ctypes.POINTER(Budget), p, p, p,
                                          ctypes.POINTER(ctypes.c_double),
                                          ctypes.POINTER(ctypes.c_int64)]
        lib.talaria_sp_select.restype = ctypes.c_int
        lib.talaria_sp_attn_calibrate_xcd.argtypes = [ctypes.POINTER(_RawPlan), p, p, p, p, p, p,
                                                      sz, p, sz, p, p]
        lib.talaria_sp_set_xcd_order.argtypes = [p]
        lib.talaria_sp_get_xcd_order.argtypes = [p]
        for f in (lib.talaria_sp_attn_calibrate_xcd, lib.talaria_sp_set_xcd_order,
                  lib.talaria_sp_get_xcd_order):
            f.restype = ctypes.c_int
        lib.talaria_sp_last_error.argtypes = []
        lib.talaria_sp_last_error.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def last_error() -> str:
    return library().talaria_sp_last_error().decode()


def _check(status: int) -> int:
    if status < 0:
        raise TalariaError(status, last_error())
    return status


@dataclass
class SpPlan:
    """A plan plus the host-side facts the binding uses for shape checks."""

    raw: _RawPlan
    geom: Geom
    prefix_lens: np.ndarray
    suffix_lens: np.ndarray
    max_pages_per_seq: int
    workspace_bytes: int

    @property
    def total_tokens(self) -> int:
        return int(self.suffix_lens.sum())

    @property
    def total_kv_tokens(self) -> int:
        return int(self.prefix_lens.astype(np.int64).sum() + self.suffix_lens.sum())

    @property
    def num_seqs(self) -> int:
        return int(self.prefix_lens.shape[0])


def make_geom(num_q_heads: int, num_kv_heads: int, head_dim: int, page_size: int,
              num_pages: int) -> Geom:
    return Geom(num_q_heads, num_kv_heads, head_dim, page_size, num_pages)


def plan(geom: Geom, prefix_lens: Sequence[int], suffix_lens: Sequence[int],
         max_pages_per_seq: int, kv_splits: int = 0) -> SpPlan:
    """talaria_sp_attn_plan (host only)."""
    pre = np.ascontiguousarray(prefix_lens, dtype=np.int32)
    suf = np.ascontiguousarray(suffix_lens, dtype=np.int32)
    if pre.shape != suf.shape or pre.ndim != 1:
        raise ValueError("prefix_lens and suffix_lens must be 1-D with equal length")
    raw = _RawPlan()
    ws = ctypes.c_size_t(0)
    _check(library().talaria_sp_attn_plan(ctypes.byref(geom), pre.shape[0],
                                          pre.ctypes.data if pre.size else None,
                                          suf.ctypes.data if suf.size else None,
                                          int(max_pages_per_seq), int(kv_splits),
                                          ctypes.byref(ws), ctypes.byref(raw)))
    return SpPlan(raw, geom, pre.copy(), suf.copy(), int(max_pages_per_seq), int(ws.value))


def check_tables(sp: SpPlan, host_block_tables) -> None:
    """talaria_sp_attn_check_tables: validate a host copy of the block tables
    (ids in range, no page twice in one sequence, appended pages exclusive);
    raises TalariaError(EINVAL) naming the first bad entry."""
    bt = np.ascontiguousarray(host_block_tables, dtype=np.int32)
    if bt.shape != (sp.num_seqs, sp.max_pages_per_seq):
        raise ValueError(f"block tables have shape {bt.shape}, expected "
                         f"{(sp.num_seqs, sp.max_pages_per_seq)}")
    _check(library().talaria_sp_attn_check_tables(ctypes.byref(sp.raw),
                                                  bt.ctypes.data if bt.size else None))


def plan_items(sp: SpPlan) -> np.ndarray:
    """The plan's work list as int32 [num_items, 8] (fields in ITEM_FIELDS)."""
    n = _check(library().talaria_sp_attn_plan_items(ctypes.byref(sp.raw), None, 0))
    out = np.zeros((max(n, 1), 8), dtype=np.int32)
    _check(library().talaria_sp_attn_plan_items(ctypes.byref(sp.raw), out.ctypes.data, n))
    return out[:n]


# ---- device-side calls --------------------------------------------------------------

def _torch():
    import torch
    return torch


_BF16_LIKE = None


def _dev(t, shape, what: str, bits16: bool = True, dtype=None):
    """Validate a device tensor and return its address."""
    torch = _torch()
    global _BF16_LIKE
    if _BF16_LIKE is None:
        _BF16_LIKE = {torch.bfloat16, torch.int16, torch.uint16}
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{what} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{what} must be on a GPU")
    if bits16 and t.dtype not in _BF16_LIKE:
        raise TypeError(f"{what} must be bf16 (or 16-bit bit patterns), got {t.dtype}")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{what} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return _torch().cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _pool_shapes(sp: SpPlan):
    g = sp.geom
    k = (g.num_pages, g.num_kv_heads, g.page_size, g.head_dim)
    v = (g.num_pages, g.num_kv_heads, g.head_dim, g.page_size)
    return k, v


def append_kv(sp: SpPlan, k_new, v_new, k_pool, v_pool, block_tables, stream=None) -> None:
    """talaria_sp_attn_append_kv: scatter the new tokens' K/V into their pages."""
    torch = _torch()
    g = sp.geom
    kshape, vshape = _pool_shapes(sp)
    row = (sp.total_tokens, g.num_kv_heads, g.head_dim)
    args = (_dev(k_new, row, "k_new"), _dev(v_new, row, "v_new"),
            _dev(k_pool, kshape, "k_pool"), _dev(v_pool, vshape, "v_pool"),
            _dev(block_tables, (sp.num_seqs, sp.max_pages_per_seq), "block_tables",
                 bits16=False, dtype=torch.int32))
    _check(library().talaria_sp_attn_append_kv(ctypes.byref(sp.raw), *args, _stream(stream)))


def _attention_call(fn, sp: SpPlan, q, k_pool, v_pool, block_tables, out, lse, workspace,
                    sm_scale, stream) -> None:
    torch = _torch()
    g = sp.geom
    kshape, vshape = _pool_shapes(sp)
    qshape = (sp.total_tokens, g.num_q_heads, g.head_dim)
    lse_ptr = None
    if lse is not None:
        lse_ptr = _dev(lse, (sp.total_tokens, g.num_q_heads), "lse", bits16=False,
                       dtype=torch.float32)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        if not workspace.is_cuda or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous GPU tensor")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    args = (_dev(q, qshape, "q"), _dev(k_pool, kshape, "k_pool"), _dev(v_pool, vshape, "v_pool"),
            _dev(block_tables, (sp.num_seqs, sp.max_pages_per_seq), "block_tables",
                 bits16=False, dtype=torch.int32))
    _check(fn(ctypes.byref(sp.raw), *args, float(sm_scale), _dev(out, qshape, "out"), lse_ptr,
              ws_ptr, ws_bytes, _stream(stream)))


def prefill(sp: SpPlan, q, k_pool, v_pool, block_tables, out, lse=None, workspace=None,
            sm_scale: float = 0.0, stream=None) -> None:
    """talaria_sp_attn_prefill: causal SP attention into ``out`` (and ``lse``)."""
    _attention_call(library().talaria_sp_attn_prefill, sp, q, k_pool, v_pool, block_tables, out,
                    lse, workspace, sm_scale, stream)


def prefill_noalloc(sp: SpPlan, q, k_pool, v_pool, block_tables, out, lse=None,
                    sm_scale: float = 0.0, stream=None) -> None:
    """talaria_sp_attn_prefill_noalloc: prefill with the library's own scratch in
    place of a workspace (allocates nothing; overlapping calls on one GPU race)."""
    torch = _torch()
    g = sp.geom
    kshape, vshape = _pool_shapes(sp)
    qshape = (sp.total_tokens, g.num_q_heads, g.head_dim)
    lse_ptr = None
    if lse is not None:
        lse_ptr = _dev(lse, (sp.total_tokens, g.num_q_heads), "lse", bits16=False,
                       dtype=torch.float32)
    args = (_dev(q, qshape, "q"), _dev(k_pool, kshape, "k_pool"), _dev(v_pool, vshape, "v_pool"),
            _dev(block_tables, (sp.num_seqs, sp.max_pages_per_seq), "block_tables",
                 bits16=False, dtype=torch.int32))
    _check(library().talaria_sp_attn_prefill_noalloc(ctypes.byref(sp.raw), *args,
                                                     float(sm_scale), _dev(out, qshape, "out"),
                                                     lse_ptr, _stream(stream)))


def noalloc_scratch_bytes() -> int:
    """Bytes of per-GPU scratch behind prefill_noalloc."""
    return int(library().talaria_sp_attn_noalloc_scratch_bytes())


def decode(sp: SpPlan, q, k_pool, v_pool, block_tables, out, lse=None, workspace=None,
           sm_scale: float = 0.0, stream=None) -> None:
    """talaria_sp_attn_decode: one new token per sequence (suffix lengths <= 1)."""
    _attention_call(library().talaria_sp_attn_decode, sp, q, k_pool, v_pool, block_tables, out,
                    lse, workspace, sm_scale, stream)


def calibrate_xcd(sp: SpPlan, q, k_pool, v_pool, block_tables, out, workspace=None,
                  stream=None) -> list:
    """talaria_sp_attn_calibrate_xcd: time one prefill of ``sp`` per XCD and set the
    process-wide XCD order (fastest first), which plans made afterwards use for
    placement.  Synchronises the stream; returns the order."""
    torch = _torch()
    g = sp.geom
    kshape, vshape = _pool_shapes(sp)
    qshape = (sp.total_tokens, g.num_q_heads, g.head_dim)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        if not workspace.is_cuda or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous GPU tensor")
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    n = max(int(plan_items(sp).shape[0]), 1)
    stamps = torch.empty(4 * n, dtype=torch.int64, device=q.device)
    order = (ctypes.c_int32 * 8)()
    _check(library().talaria_sp_attn_calibrate_xcd(
        ctypes.byref(sp.raw), _dev(q, qshape, "q"), _dev(k_pool, kshape, "k_pool"),
        _dev(v_pool, vshape, "v_pool"),
        _dev(block_tables, (sp.num_seqs, sp.max_pages_per_seq), "block_tables", bits16=False,
             dtype=torch.int32),
        _dev(out, qshape, "out"), ws_ptr, ws_bytes, stamps.data_ptr(), stamps.numel() * 8,
        order, _stream(stream)))
    return list(order)


def set_xcd_order(order: Optional[Sequence[int]]) -> None:
    """talaria_sp_set_xcd_order: order[g] = XCD that takes the g-th longest block of
    items (a permutation of 0..7); None clears the order."""
    if order is None:
        _check(library().talaria_sp_set_xcd_order(None))
        return
    arr = (ctypes.c_int32 * 8)(*[int(x) for x in order]) if len(order) == 8 else None
    if arr is None:
        raise ValueError("order must have 8 entries")
    _check(library().talaria_sp_set_xcd_order(arr))


def get_xcd_order() -> Optional[list]:
    """talaria_sp_get_xcd_order: the current XCD order, or None when none is set."""
    arr = (ctypes.c_int32 * 8)()
    return list(arr) if _check(library().talaria_sp_get_xcd_order(arr)) == 1 else None


def gather_kv(sp: SpPlan, k_pool, v_pool, block_tables, k_out, v_out, stream=None) -> None:
    """talaria_sp_attn_gather_kv: pages -> contiguous token-major K/V rows."""
    torch = _torch()
    g = sp.geom
    kshape, vshape = _pool_shapes(sp)
    oshape = (sp.total_kv_tokens, g.num_kv_heads, g.head_dim)
    _check(library().talaria_sp_attn_gather_kv(
        ctypes.byref(sp.raw), _dev(k_pool, kshape, "k_pool"), _dev(v_pool, vshape, "v_pool"),
        _dev(block_tables, (sp.num_seqs, sp.max_pages_per_seq), "block_tables", bits16=False,
             dtype=torch.int32),
        _dev(k_out, oshape, "k_out"), _dev(v_out, oshape, "v_out"), _stream(stream)))


def workspace_tensor(sp: SpPlan, device="cuda"):
    """A device byte buffer of the plan's workspace size (None if it needs none)."""
    if sp.workspace_bytes == 0:
        return None
    return _torch().empty(sp.workspace_bytes, dtype=_torch().uint8, device=device)


# ---- HKVR page transfer ---------------------------------------------------------------

def kv_cache(num_layers: int, num_kv_heads: int, head_dim: int, page_size: int,
             num_pages: int) -> KvCache:
    return KvCache(num_layers, num_kv_heads, head_dim, page_size, num_pages)


def _cache_shapes(c: KvCache):
    k = (c.num_layers, c.num_pages, c.num_kv_heads, c.page_size, c.head_dim)
    v = (c.num_layers, c.num_pages, c.num_kv_heads, c.head_dim, c.page_size)
    return k, v


def slab_shape(c: KvCache, num_slab_pages: int):
    """Page-first host slab: [pages][layers][K, V][Hkv * page_size * head_dim]."""
    return (num_slab_pages, c.num_layers, 2, c.num_kv_heads * c.page_size * c.head_dim)


def _slab(t, shape):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or t.is_cuda or not t.is_pinned():
        raise ValueError("slab must be a pinned host tensor (pin_memory=True)")
    if t.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
        raise TypeError(f"slab must be bf16 (or 16-bit bit patterns), got {t.dtype}")
    if not t.is_contiguous() or tuple(t.shape) != tuple(shape):
        raise ValueError(f"slab has shape {tuple(t.shape)}, expected contiguous {tuple(shape)}")
    return t.data_ptr()


def _hkvr_args(c, slab, page_ids, k_cache, v_cache):
    torch = _torch()
    kshape, vshape = _cache_shapes(c)
    n = int(page_ids.shape[0]) if page_ids.dim() == 1 else -1
    if n < 0:
        raise ValueError("page_ids must be 1-D")
    return n, (_slab(slab, slab_shape(c, n)),
               _dev(page_ids, (n,), "page_ids", bits16=False, dtype=torch.int32),
               _dev(k_cache, kshape, "k_cache"), _dev(v_cache, vshape, "v_cache"))


def hkvr_restore(c: KvCache, slab, page_ids, k_cache, v_cache, stream=None) -> None:
    """talaria_hkvr_restore: page-first host slab -> layer-first device pages."""
    n, (sp, ip, kp, vp) = _hkvr_args(c, slab, page_ids, k_cache, v_cache)
    _check(library().talaria_hkvr_restore(ctypes.byref(c), n, sp, ip, kp, vp, _stream(stream)))


def hkvr_checkpoint(c: KvCache, k_cache, v_cache, page_ids, slab, stream=None) -> None:
    """talaria_hkvr_checkpoint: layer-first device pages -> page-first host slab."""
    n, (sp, ip, kp, vp) = _hkvr_args(c, slab, page_ids, k_cache, v_cache)
    _check(library().talaria_hkvr_checkpoint(ctypes.byref(c), n, kp, vp, ip, sp,
                                             _stream(stream)))


# ---- D2D-staged weight switching ------------------------------------------------------

def _words(n_bits: int) -> int:
    return (n_bits + 31) // 32


def _u8dev(t, what):
    torch = _torch()
    return _dev(t, None, what, bits16=False, dtype=torch.uint8)


def stage_mark_dirty(chunks, used_pages, num_pages: int, page_bytes: int, dirty,
                     stream=None) -> None:
    """talaria_stage_mark_dirty.  chunks: device int64 [n, 3] (stage_offset,
    weight_offset, bytes); used_pages / dirty: device int32 bitmaps."""
    torch = _torch()
    n = int(chunks.shape[0])
    cp = _dev(chunks, (n, 3), "chunks", bits16=False, dtype=torch.int64)
    up = _dev(used_pages, (_words(num_pages),), "used_pages", bits16=False, dtype=torch.int32)
    dp = _dev(dirty, (_words(n),), "dirty", bits16=False, dtype=torch.int32)
    _check(library().talaria_stage_mark_dirty(cp, n, up, int(num_pages), int(page_bytes), dp,
                                              _stream(stream)))


def stage_gather(chunks, staged, dirty, staging, host_weights, weights, stream=None) -> None:
    """talaria_stage_gather.  staging / weights: device uint8; host_weights:
    pinned host uint8 with the weights' size."""
    torch = _torch()
    n = int(chunks.shape[0])
    cp = _dev(chunks, (n, 3), "chunks", bits16=False, dtype=torch.int64)
    sp = _dev(staged, (_words(n),), "staged", bits16=False, dtype=torch.int32)
    dp = _dev(dirty, (_words(n),), "dirty", bits16=False, dtype=torch.int32)
    if host_weights.is_cuda or not host_weights.is_pinned() or host_weights.dtype != torch.uint8:
        raise ValueError("host_weights must be a pinned host uint8 tensor")
    if host_weights.numel() != weights.numel() or not host_weights.is_contiguous():
        raise ValueError("host_weights must be contiguous with the weights' size")
    _check(library().talaria_stage_gather(cp, n, sp, dp, _u8dev(staging, "staging"),
                                          staging.numel(), host_weights.data_ptr(),
                                          _u8dev(weights, "weights"), weights.numel(),
                                          _stream(stream)))


# ---- SP batch selection (host) --------------------------------------------------------

def sp_select(candidates, model: CostModel, budget: Budget):
    """talaria_sp_select.  candidates: int32 [n, 3] rows (prefix_len,
    suffix_len, host_resident).  Returns (selected indices, plan prefix
    lengths, plan suffix lengths, predicted seconds, predicted pages)."""
    c = np.ascontiguousarray(candidates, dtype=np.int32).reshape(-1, 3)
    cap = max(int(budget.max_batch), 1)
    sel = np.zeros(cap, np.int32)
    pre = np.zeros(cap, np.int32)
    suf = np.zeros(cap, np.int32)
    secs = ctypes.c_double(0.0)
    pages = ctypes.c_int64(0)
    n = _check(library().talaria_sp_select(
        c.ctypes.data if c.size else None, c.shape[0], ctypes.byref(model), ctypes.byref(budget),
        sel.ctypes.data, pre.ctypes.data, suf.ctypes.data, ctypes.byref(secs),
        ctypes.byref(pages)))
    return sel[:n].copy(), pre[:n].copy(), suf[:n].copy(), secs.value, pages.value
