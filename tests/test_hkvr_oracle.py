"""Pins of the HKVR page-transfer oracle (CPU).

The oracle is checked against an element-by-element loop written from flat
offsets, against the attention oracle's own page walk (which fixes the order
of elements inside a page block), and against round-trip and no-op
invariants."""
import numpy as np

import oracle
from oracle import hkvr
from workload import BF16_NAN, workload_from_lengths


def _cache(rng, L, P, H, ps, d):
    k = rng.integers(0, 1 << 16, size=(L, P, H, ps, d), dtype=np.uint16)
    v = rng.integers(0, 1 << 16, size=(L, P, H, d, ps), dtype=np.uint16)
    return k, v


def test_restore_matches_flat_offset_loop():
    rng = np.random.default_rng(0)
    L, P, H, ps, d, n = 2, 6, 2, 8, 4, 3
    k, v = _cache(rng, L, P, H, ps, d)
    ids = np.array([4, 0, 2])
    blk = H * ps * d
    slab = rng.integers(0, 1 << 16, size=(n, L, 2, blk), dtype=np.uint16)
    kr, vr = hkvr.restore(slab, ids, k, v)
    kf, vf = k.reshape(-1).copy(), v.reshape(-1).copy()
    sf = slab.reshape(-1)
    for p in range(n):
        for layer in range(L):
            for e in range(blk):
                dev = (layer * P + ids[p]) * blk + e
                kf[dev] = sf[((p * L + layer) * 2 + 0) * blk + e]
                vf[dev] = sf[((p * L + layer) * 2 + 1) * blk + e]
    assert np.array_equal(kr.reshape(-1), kf) and np.array_equal(vr.reshape(-1), vf)


def test_checkpoint_matches_flat_offset_loop():
    rng = np.random.default_rng(1)
    L, P, H, ps, d, n = 3, 5, 1, 8, 8, 4
    k, v = _cache(rng, L, P, H, ps, d)
    ids = np.array([3, 1, 4, 0])
    blk = H * ps * d
    slab = hkvr.checkpoint(k, v, ids, np.zeros((n, L, 2, blk), np.uint16))
    kf, vf, sf = k.reshape(-1), v.reshape(-1), slab.reshape(-1)
    for p in range(n):
        for layer in range(L):
            for e in range(blk):
                dev = (layer * P + ids[p]) * blk + e
                assert sf[((p * L + layer) * 2) * blk + e] == kf[dev]
                assert sf[((p * L + layer) * 2 + 1) * blk + e] == vf[dev]


def test_round_trip_through_other_pages():
    rng = np.random.default_rng(2)
    L, P, H, ps, d, n = 2, 9, 2, 16, 8, 5
    k, v = _cache(rng, L, P, H, ps, d)
    ids_a = np.array([7, 2, 5, 0, 8])
    slab = hkvr.checkpoint(k, v, ids_a, np.zeros((n, L, 2, H * ps * d), np.uint16))
    k2, v2 = _cache(rng, L, P, H, ps, d)
    ids_b = rng.permutation(P)[:n]
    k3, v3 = hkvr.restore(slab, ids_b, k2, v2)
    for p in range(n):
        assert np.array_equal(k3[:, ids_b[p]], k[:, ids_a[p]])
        assert np.array_equal(v3[:, ids_b[p]], v[:, ids_a[p]])
    untouched = np.setdiff1d(np.arange(P), ids_b)
    assert np.array_equal(k3[:, untouched], k2[:, untouched])
    assert np.array_equal(hkvr.checkpoint(k3, v3, ids_b, np.zeros_like(slab)), slab)


def test_out_of_range_ids_move_nothing():
    rng = np.random.default_rng(3)
    L, P, H, ps, d = 2, 4, 1, 8, 8
    k, v = _cache(rng, L, P, H, ps, d)
    slab = rng.integers(0, 1 << 16, size=(3, L, 2, H * ps * d), dtype=np.uint16)
    ids = np.array([-1, 4, 1])
    kr, vr = hkvr.restore(slab, ids, k, v)
    others = [0, 2, 3]
    assert np.array_equal(kr[:, others], k[:, others]) and np.array_equal(vr[:, others], v[:, others])
    s2 = hkvr.checkpoint(k, v, ids, slab)
    assert np.array_equal(s2[:2], slab[:2])


def test_restored_pages_read_back_as_token_rows():
    """The slab's page blocks use the attention pools' element order: after a
    restore, the attention oracle's own page walk (oracle.gather_kv) returns
    the token rows the slab was built from, for every layer."""
    rng = np.random.default_rng(4)
    H, d, ps, L = 2, 16, 8, 3
    wl = workload_from_lengths("hkvr", 9, num_q_heads=4, num_kv_heads=H, head_dim=d, page_size=ps,
                               num_pages=40, prefix_lens=[40], suffix_lens=[0])
    n = 5  # 40 tokens = 5 pages
    ids = wl.block_tables[0, :n].astype(np.int64)
    rows_k = rng.integers(0, 1 << 16, size=(L, n * ps, H, d), dtype=np.uint16)
    rows_v = rng.integers(0, 1 << 16, size=(L, n * ps, H, d), dtype=np.uint16)
    slab = np.empty((n, L, 2, H * ps * d), np.uint16)
    for p in range(n):
        for layer in range(L):
            kb = rows_k[layer, p * ps:(p + 1) * ps]          # [ps][H][d]
            vb = rows_v[layer, p * ps:(p + 1) * ps]
            slab[p, layer, 0] = kb.transpose(1, 0, 2).reshape(-1)  # [H][ps][d]
            slab[p, layer, 1] = vb.transpose(1, 2, 0).reshape(-1)  # [H][d][ps]
    k = np.full((L, wl.num_pages, H, ps, d), BF16_NAN, np.uint16)
    v = np.full((L, wl.num_pages, H, d, ps), BF16_NAN, np.uint16)
    k, v = hkvr.restore(slab, ids, k, v)
    for layer in range(L):
        ko, vo = oracle.gather_kv(wl.prefix_lens, wl.suffix_lens, wl.block_tables, ps,
                                  k[layer], v[layer])
        assert np.array_equal(ko, rows_k[layer]) and np.array_equal(vo, rows_v[layer])
