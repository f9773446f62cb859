"""Argument checks of the page-transfer and staging calls, on the CPU: every
rejected call returns its error code and message before anything is
launched, and empty calls are successful no-ops."""
import ctypes

import pytest

import paper_2607_17181_amd as tsa

NULL = None
BAD = ctypes.c_void_p(0x1001)  # non-NULL, not 16-byte aligned; never dereferenced


def _cache(layers=2, hkv=1, d=128, ps=16, pages=8):
    return tsa.kv_cache(layers, hkv, d, ps, pages)


@pytest.mark.parametrize("cache,code", [
    (None, tsa.EINVAL),
    (_cache(layers=0), tsa.EINVAL),
    (_cache(pages=0), tsa.EINVAL),
    (_cache(d=96), tsa.EUNSUPPORTED),
    (_cache(ps=12), tsa.EUNSUPPORTED),
    (_cache(ps=4), tsa.EUNSUPPORTED),
    (_cache(ps=512), tsa.EUNSUPPORTED),
    (_cache(layers=70000), tsa.EUNSUPPORTED),
])
def test_hkvr_rejects_bad_cache_geometry(cache, code):
    lib = tsa.library()
    ref = ctypes.byref(cache) if cache is not None else None
    assert lib.talaria_hkvr_restore(ref, 1, BAD, BAD, BAD, BAD, NULL) == code
    assert lib.talaria_hkvr_checkpoint(ref, 1, BAD, BAD, BAD, BAD, NULL) == code
    assert tsa.last_error()


def test_hkvr_empty_call_is_a_no_op_and_null_pointers_are_rejected():
    lib = tsa.library()
    c = ctypes.byref(_cache())
    assert lib.talaria_hkvr_restore(c, 0, NULL, NULL, NULL, NULL, NULL) == tsa.OK
    assert lib.talaria_hkvr_restore(c, 3, NULL, BAD, BAD, BAD, NULL) == tsa.EINVAL
    assert lib.talaria_hkvr_checkpoint(c, 3, BAD, BAD, NULL, BAD, NULL) == tsa.EINVAL
    assert lib.talaria_hkvr_restore(c, -1, BAD, BAD, BAD, BAD, NULL) == tsa.EINVAL


def test_stage_mark_dirty_argument_checks():
    lib = tsa.library()
    f = lib.talaria_stage_mark_dirty
    assert f(BAD, -1, BAD, 8, 4096, BAD, NULL) == tsa.EINVAL
    assert f(BAD, 4, BAD, 8, 0, BAD, NULL) == tsa.EINVAL          # page_bytes
    assert f(BAD, 4, BAD, -1, 4096, BAD, NULL) == tsa.EINVAL      # num_pages
    assert f(NULL, 0, NULL, 8, 4096, NULL, NULL) == tsa.OK        # empty
    assert f(NULL, 4, BAD, 8, 4096, BAD, NULL) == tsa.EINVAL      # chunks NULL
    assert f(BAD, 4, NULL, 8, 4096, BAD, NULL) == tsa.EINVAL      # used_pages NULL
    assert f(BAD, 4, BAD, 0, 4096, BAD, NULL) == tsa.EINVAL       # no pages


def test_stage_gather_argument_checks():
    lib = tsa.library()
    f = lib.talaria_stage_gather
    aligned = ctypes.c_void_p(0x10000)  # only ever paired with a rejected argument
    assert f(BAD, -1, BAD, BAD, BAD, 16, BAD, BAD, 16, NULL) == tsa.EINVAL
    assert f(BAD, 2, BAD, BAD, BAD, -16, BAD, BAD, 16, NULL) == tsa.EINVAL
    assert f(NULL, 0, NULL, NULL, NULL, 0, NULL, NULL, 0, NULL) == tsa.OK
    assert f(BAD, 2, NULL, BAD, aligned, 16, aligned, aligned, 16, NULL) == tsa.EINVAL
    assert f(BAD, 2, BAD, BAD, aligned, 16, aligned, NULL, 16, NULL) == tsa.EINVAL
    # misaligned regions are rejected before any launch
    assert f(BAD, 2, BAD, BAD, BAD, 16, aligned, aligned, 16, NULL) == tsa.EINVAL
    assert "aligned" in tsa.last_error()


def test_prefill_noalloc_rejects_plans_beyond_its_scratch():
    """A plan whose workspace exceeds the per-GPU scratch is ENOSPACE before any
    pointer is looked at or anything is launched; a plan that fits passes the
    size check (and then stops at the NULL-pointer check)."""
    lib = tsa.library()
    assert tsa.noalloc_scratch_bytes() == 64 << 20
    geom = tsa.make_geom(8, 1, 128, 16, 2000)
    big = tsa.plan(geom, [20000], [512], 1300, kv_splits=64)  # 16 query tiles x 64 splits
    assert big.workspace_bytes > tsa.noalloc_scratch_bytes()
    f = lib.talaria_sp_attn_prefill_noalloc
    assert f(ctypes.byref(big.raw), BAD, BAD, BAD, BAD, 0.0, BAD, NULL, NULL) == tsa.ENOSPACE
    assert "scratch" in tsa.last_error()
    small = tsa.plan(geom, [5000], [256], 400, kv_splits=4)
    assert 0 < small.workspace_bytes <= tsa.noalloc_scratch_bytes()
    assert f(ctypes.byref(small.raw), NULL, BAD, BAD, BAD, 0.0, BAD, NULL, NULL) == tsa.EINVAL
    assert f(None, BAD, BAD, BAD, BAD, 0.0, BAD, NULL, NULL) == tsa.EINVAL
