"""Pins that tie the CPU oracle to facts outside itself.

Each ``pin_*`` function takes an optional oracle library path (so that a
deliberately mutated oracle build can be checked against the same pins) and
raises ``AssertionError`` (or the oracle's ``ValueError``) when the oracle
disagrees with:

* an explicit masked-matrix softmax written with numpy (brute force);
* PyTorch's CPU ``scaled_dot_product_attention`` in float64 with the
  library's own bottom-right causal mask and grouped-query head mapping;
* closed forms (constant V, zero Q, the first token of a cold sequence, a
  dominant logit);
* invariants (paged == contiguous, page permutation, chunked == one-shot,
  identical queries in one GQA group, stale NaN slots);
* a plain numpy scatter / concatenation for append and gather.

The attention definition being pinned is the SP prefill of the paper's
Sections 3.4 and 4.3 (prefill only the new tail of a continuation over its
preserved prefix KV), with the causal alignment, head mapping and softmax
scale readings stated in the oracle's header.
"""
from __future__ import annotations

import math
from typing import Optional, Tuple

import numpy as np

import oracle
from workload import BF16_NAN, bf16_bits_from_f32, f32_from_bf16_bits, workload_from_lengths

TOL = 1e-12


def _case(seed, Hq=4, Hkv=2, d=16, ps=4, pre=(5, 0, 13), suf=(7, 3, 1), num_pages=None,
          chunks=1, q_std=1.0):
    need = sum((p + s + ps - 1) // ps for p, s in zip(pre, suf))
    wl = workload_from_lengths("pin", seed, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d,
                               page_size=ps, num_pages=num_pages or need + 5, prefix_lens=pre,
                               suffix_lens=suf, num_chunks=chunks, q_std=q_std)
    kp, vp = wl.pool_bits(fill=int(BF16_NAN))
    return wl, kp, vp


def _run_oracle(wl, kp, vp, lib=None, sm_scale=0.0, q=None, rows=None):
    """Append (chunk by chunk) then attend; return o [T,Hq,d], lse [T,Hq]."""
    q = wl.q if q is None else q
    o = np.empty(q.shape, dtype=np.float64)
    lse = np.empty(q.shape[:2], dtype=np.float64)
    for pre, suf, tok in wl.chunks:
        kp, vp = oracle.append_kv(pre, suf, wl.block_tables, wl.page_size, wl.k_new[tok],
                                  wl.v_new[tok], kp, vp, lib_path=lib)
        oc, lc = oracle.sp_attention(pre, suf, wl.block_tables, wl.page_size, q[tok], kp, vp,
                                     sm_scale=sm_scale, lib_path=lib)
        o[tok] = oc
        lse[tok] = lc
    return o, lse, kp, vp


def _seq_kv(wl, b):
    """float64 K, V [P_b + S_b, Hkv, d] of sequence b from the generator's rows."""
    poff = int(wl.prefix_lens[:b].sum())
    toff = int(wl.suffix_lens[:b].sum())
    P, S = int(wl.prefix_lens[b]), int(wl.suffix_lens[b])
    K = np.concatenate([wl.prefix_k[poff:poff + P], wl.k_new[toff:toff + S]])
    V = np.concatenate([wl.prefix_v[poff:poff + P], wl.v_new[toff:toff + S]])
    return (f32_from_bf16_bits(K).astype(np.float64), f32_from_bf16_bits(V).astype(np.float64),
            toff, P, S)


def brute_force(wl, sm_scale: Optional[float] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Explicit S x (P+S) masked softmax matrix per (sequence, head)."""
    Hq, Hkv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    G = Hq // Hkv
    sigma = sm_scale if sm_scale else 1.0 / math.sqrt(d)
    qf = f32_from_bf16_bits(wl.q).astype(np.float64)
    o = np.zeros(qf.shape)
    lse = np.zeros(qf.shape[:2])
    for b in range(wl.num_seqs):
        K, V, toff, P, S = _seq_kv(wl, b)
        if S == 0:
            continue
        masked = np.arange(P + S)[None, :] > P + np.arange(S)[:, None]
        for h in range(Hq):
            g = h // G
            sc = sigma * (qf[toff:toff + S, h] @ K[:, g].T)
            sc[masked] = -np.inf
            mx = sc.max(axis=1, keepdims=True)
            w = np.exp(sc - mx)
            lsum = w.sum(axis=1)
            o[toff:toff + S, h] = (w @ V[:, g]) / lsum[:, None]
            lse[toff:toff + S, h] = mx[:, 0] + np.log(lsum)
    return o, lse


def pin_bruteforce(lib=None):
    shapes = [
        dict(Hq=4, Hkv=2, d=16, ps=4, pre=(5, 0, 13), suf=(7, 3, 1)),
        dict(Hq=2, Hkv=1, d=8, ps=1, pre=(3,), suf=(4,)),
        dict(Hq=3, Hkv=3, d=8, ps=16, pre=(17, 40), suf=(20, 9)),
        dict(Hq=8, Hkv=1, d=32, ps=8, pre=(0, 9, 31), suf=(12, 0, 16)),
    ]
    for i, sh in enumerate(shapes):
        wl, kp, vp = _case(100 + i, **sh)
        scale = 0.0 if i % 2 == 0 else 0.37
        o, lse, _, _ = _run_oracle(wl, kp, vp, lib, sm_scale=scale)
        bo, blse = brute_force(wl, sm_scale=scale or None)
        assert np.max(np.abs(o - bo)) <= TOL, f"shape {i}: o differs from brute force"
        assert np.max(np.abs(lse - blse)) <= TOL, f"shape {i}: lse differs from brute force"


def pin_torch_sdpa(lib=None):
    import torch
    from torch.nn.attention.bias import causal_lower_right

    wl, kp, vp = _case(7, Hq=4, Hkv=2, d=16, ps=4, pre=(11, 0), suf=(6, 9))
    o, _, _, _ = _run_oracle(wl, kp, vp, lib)
    qf = torch.from_numpy(f32_from_bf16_bits(wl.q).astype(np.float64))
    for b in range(wl.num_seqs):
        K, V, toff, P, S = _seq_kv(wl, b)
        qb = qf[toff:toff + S].permute(1, 0, 2)[None]
        kb = torch.from_numpy(K).permute(1, 0, 2)[None]
        vb = torch.from_numpy(V).permute(1, 0, 2)[None]
        if P == 0:
            ref = torch.nn.functional.scaled_dot_product_attention(qb, kb, vb, is_causal=True,
                                                                   enable_gqa=True)
        else:
            mask = causal_lower_right(S, P + S)._materialize()
            ref = torch.nn.functional.scaled_dot_product_attention(qb, kb, vb, attn_mask=mask,
                                                                   enable_gqa=True)
        ref = ref[0].permute(1, 0, 2).numpy()
        assert np.max(np.abs(o[toff:toff + S] - ref)) <= TOL, f"seq {b}: differs from torch SDPA"


def pin_constant_v(lib=None):
    wl, kp, vp = _case(8, Hq=2, Hkv=1, d=16, ps=4, pre=(9, 30), suf=(5, 4))
    c = bf16_bits_from_f32(np.linspace(-2.0, 3.0, wl.head_dim, dtype=np.float32))
    wl.v_new[:] = c
    wl.prefix_v[:] = c
    kp, vp = wl.pool_bits(fill=int(BF16_NAN))
    o, _, _, _ = _run_oracle(wl, kp, vp, lib)
    cf = f32_from_bf16_bits(c).astype(np.float64)
    assert np.max(np.abs(o - cf)) <= TOL, "constant V must give V"


def pin_zero_q(lib=None):
    wl, kp, vp = _case(9, Hq=4, Hkv=2, d=8, ps=4, pre=(6, 0), suf=(5, 7))
    q0 = np.zeros_like(wl.q)
    o, lse, _, _ = _run_oracle(wl, kp, vp, lib, q=q0)
    G = wl.num_q_heads // wl.num_kv_heads
    for b in range(wl.num_seqs):
        K, V, toff, P, S = _seq_kv(wl, b)
        csum = np.cumsum(V, axis=0)
        for i in range(S):
            n = P + i + 1
            for h in range(wl.num_q_heads):
                mean = csum[n - 1, h // G] / n
                assert np.max(np.abs(o[toff + i, h] - mean)) <= TOL, "Q=0 must average V"
                assert abs(lse[toff + i, h] - math.log(n)) <= TOL, "Q=0 must give lse = ln n"


def pin_first_token(lib=None):
    wl, kp, vp = _case(10, Hq=2, Hkv=2, d=16, ps=4, pre=(0,), suf=(6,))
    o, lse, _, _ = _run_oracle(wl, kp, vp, lib)
    qf = f32_from_bf16_bits(wl.q).astype(np.float64)
    kf = f32_from_bf16_bits(wl.k_new).astype(np.float64)
    vf = f32_from_bf16_bits(wl.v_new).astype(np.float64)
    for h in range(2):
        assert np.array_equal(o[0, h], vf[0, h]), "first token of a cold sequence must return v_0"
        exact = math.fsum(float(a) * float(b) for a, b in zip(qf[0, h], kf[0, h]))
        assert abs(lse[0, h] - exact / 4.0) <= TOL, "first token lse must be sigma * q.k_0"


def pin_dominant_logit(lib=None):
    wl, kp, vp = _case(11, Hq=1, Hkv=1, d=16, ps=4, pre=(12,), suf=(1,), q_std=0.01)
    # Key 5 of the prefix is aligned with q and scaled up: its logit exceeds
    # every other by >= 40, so softmax weight elsewhere is < 13 * e^-40.
    qf = f32_from_bf16_bits(wl.q[0, 0]).astype(np.float64)
    big = bf16_bits_from_f32((qf / np.linalg.norm(qf) * 256.0).astype(np.float32))
    wl.q[0, 0] = bf16_bits_from_f32((qf / np.linalg.norm(qf) * 4.0).astype(np.float32))
    wl.prefix_k[:] = bf16_bits_from_f32(np.zeros((12, 1, 16), np.float32))
    wl.k_new[:] = bf16_bits_from_f32(np.zeros((1, 1, 16), np.float32))
    wl.prefix_k[5, 0] = big
    kp, vp = wl.pool_bits(fill=int(BF16_NAN))
    o, _, _, _ = _run_oracle(wl, kp, vp, lib)
    v5 = f32_from_bf16_bits(wl.prefix_v[5, 0]).astype(np.float64)
    vmax = np.max(np.abs(f32_from_bf16_bits(wl.prefix_v))) + np.max(np.abs(v5))
    assert np.max(np.abs(o[0, 0] - v5)) <= 13 * math.exp(-40) * vmax + TOL, "dominant key must win"


def pin_paged_equals_contiguous(lib=None):
    wl, kp, vp = _case(12, Hq=4, Hkv=2, d=16, ps=4, pre=(14, 3), suf=(6, 10))
    o, lse, kp2, vp2 = _run_oracle(wl, kp, vp, lib)
    kc, vc = [], []
    for b in range(wl.num_seqs):
        poff = int(wl.prefix_lens[:b].sum())
        toff = int(wl.suffix_lens[:b].sum())
        P, S = int(wl.prefix_lens[b]), int(wl.suffix_lens[b])
        kc += [wl.prefix_k[poff:poff + P], wl.k_new[toff:toff + S]]
        vc += [wl.prefix_v[poff:poff + P], wl.v_new[toff:toff + S]]
    oc, lc = oracle.attention_contiguous(wl.prefix_lens, wl.suffix_lens, wl.q,
                                         np.concatenate(kc), np.concatenate(vc), lib_path=lib)
    assert np.array_equal(o, oc) and np.array_equal(lse, lc), "paged must equal contiguous"


def pin_page_permutation(lib=None):
    wl, kp, vp = _case(13, Hq=2, Hkv=1, d=16, ps=4, pre=(10, 21), suf=(5, 3), num_pages=40)
    o, lse, kp2, vp2 = _run_oracle(wl, kp, vp, lib)
    perm = np.random.default_rng(5).permutation(wl.num_pages)
    kpp = np.empty_like(kp)
    vpp = np.empty_like(vp)
    kpp[perm] = kp
    vpp[perm] = vp
    bt = wl.block_tables.copy()
    bt[bt >= 0] = perm[bt[bt >= 0]]
    wl.block_tables = bt
    o2, lse2, _, _ = _run_oracle(wl, kpp, vpp, lib)
    assert np.array_equal(o, o2) and np.array_equal(lse, lse2), "page permutation changed output"


def pin_chunked_equals_oneshot(lib=None):
    wl, kp, vp = _case(14, Hq=2, Hkv=1, d=16, ps=4, pre=(9,), suf=(12,), chunks=4)
    o, lse, _, _ = _run_oracle(wl, kp, vp, lib)
    wl1, kp1, vp1 = _case(14, Hq=2, Hkv=1, d=16, ps=4, pre=(9,), suf=(12,), chunks=1)
    o1, lse1, _, _ = _run_oracle(wl1, kp1, vp1, lib)
    assert np.array_equal(o, o1) and np.array_equal(lse, lse1), "chunked must equal one-shot"


def pin_gqa_identical_queries(lib=None):
    wl, kp, vp = _case(15, Hq=4, Hkv=2, d=16, ps=4, pre=(8,), suf=(5,))
    wl.q[:, 1] = wl.q[:, 0]
    wl.q[:, 3] = wl.q[:, 2]
    o, lse, _, _ = _run_oracle(wl, kp, vp, lib)
    assert np.array_equal(o[:, 0], o[:, 1]) and np.array_equal(o[:, 2], o[:, 3])
    assert not np.array_equal(o[:, 0], o[:, 2]), "different KV heads must differ"


def pin_stale_slots_ignored(lib=None):
    wl, kp, vp = _case(16, Hq=2, Hkv=1, d=16, ps=8, pre=(5, 11), suf=(2, 6))
    o, lse, _, _ = _run_oracle(wl, kp, vp, lib)
    assert np.isfinite(o).all() and np.isfinite(lse).all(), "NaN sentinels leaked"
    kz, vz = wl.pool_bits(fill=0)
    oz, lz, _, _ = _run_oracle(wl, kz, vz, lib)
    assert np.array_equal(o, oz) and np.array_equal(lse, lz), "stale slot contents matter"


def pin_append_scatter(lib=None):
    wl, kp, vp = _case(17, Hq=2, Hkv=2, d=8, ps=4, pre=(6, 0, 3), suf=(5, 9, 4), num_pages=30)
    kp2, vp2 = oracle.append_kv(wl.prefix_lens, wl.suffix_lens, wl.block_tables, wl.page_size,
                                wl.k_new, wl.v_new, kp, vp, lib_path=lib)
    ek = kp.copy()   # [page, Hkv, slot, d]
    ev = vp.copy()   # [page, Hkv, d, slot]
    toff = 0
    for b in range(wl.num_seqs):
        P, S = int(wl.prefix_lens[b]), int(wl.suffix_lens[b])
        t = np.arange(P, P + S)
        pages = wl.block_tables[b, t // 4]
        ek[pages, :, t % 4, :] = wl.k_new[toff:toff + S]
        ev[pages, :, :, t % 4] = wl.v_new[toff:toff + S]
        toff += S
    assert np.array_equal(kp2, ek) and np.array_equal(vp2, ev)


def pin_gather(lib=None):
    wl, kp, vp = _case(18, Hq=2, Hkv=2, d=8, ps=4, pre=(6, 0, 13), suf=(5, 9, 4), num_pages=30)
    _, _, kp2, vp2 = _run_oracle(wl, kp, vp, lib)
    ko, vo = oracle.gather_kv(wl.prefix_lens, wl.suffix_lens, wl.block_tables, wl.page_size,
                              kp2, vp2, lib_path=lib)
    ek, ev = [], []
    for b in range(wl.num_seqs):
        poff = int(wl.prefix_lens[:b].sum())
        toff = int(wl.suffix_lens[:b].sum())
        P, S = int(wl.prefix_lens[b]), int(wl.suffix_lens[b])
        ek += [wl.prefix_k[poff:poff + P], wl.k_new[toff:toff + S]]
        ev += [wl.prefix_v[poff:poff + P], wl.v_new[toff:toff + S]]
    assert np.array_equal(ko, np.concatenate(ek)) and np.array_equal(vo, np.concatenate(ev))


def pin_bad_page_id_rejected(lib=None):
    wl, kp, vp = _case(19, Hq=2, Hkv=1, d=8, ps=4, pre=(6,), suf=(3,))
    bt = wl.block_tables.copy()
    bt[0, 0] = wl.num_pages
    try:
        oracle.sp_attention(wl.prefix_lens, wl.suffix_lens, bt, wl.page_size, wl.q, kp, vp,
                            lib_path=lib)
    except ValueError:
        return
    raise AssertionError("out-of-range page id was accepted")


def pin_row_subset(lib=None):
    """The row-subset mode (output k belongs to flat row rows[k] = token * Hq +
    head) against brute force and, bit for bit, against the all-rows mode, on
    a permutation of every row, an unsorted list with duplicates that crosses
    sequences and heads, and a single row; for both the paged and the
    contiguous entry point."""
    wl, kp, vp = _case(20, Hq=4, Hkv=2, d=16, ps=4, pre=(9, 0, 14), suf=(5, 7, 3), num_pages=40)
    o_all, lse_all, kp2, vp2 = _run_oracle(wl, kp, vp, lib)
    bo, blse = brute_force(wl)
    T, Hq, d = wl.q.shape
    flat_o, flat_lse = o_all.reshape(T * Hq, d), lse_all.reshape(T * Hq)
    bo, blse = bo.reshape(T * Hq, d), blse.reshape(T * Hq)
    rng = np.random.default_rng(21)
    lists = [rng.permutation(T * Hq),
             np.array([T * Hq - 1, 0, 17, 17, 5, 44, 3, 17, 58, 1, 0, 29], dtype=np.int64),
             np.array([33], dtype=np.int64)]
    kc, vc = oracle.gather_kv(wl.prefix_lens, wl.suffix_lens, wl.block_tables, wl.page_size,
                              kp2, vp2, lib_path=lib)
    for i, rows in enumerate(lists):
        o, lse = oracle.sp_attention(wl.prefix_lens, wl.suffix_lens, wl.block_tables,
                                     wl.page_size, wl.q, kp2, vp2, rows=rows, lib_path=lib)
        assert np.max(np.abs(o - bo[rows])) <= TOL, f"list {i}: rows differ from brute force"
        assert np.max(np.abs(lse - blse[rows])) <= TOL, f"list {i}: lse differs from brute force"
        assert np.array_equal(o, flat_o[rows]) and np.array_equal(lse, flat_lse[rows]), \
            f"list {i}: rows mode differs from all-rows mode"
        oc, lc = oracle.attention_contiguous(wl.prefix_lens, wl.suffix_lens, wl.q, kc, vc,
                                             rows=rows, lib_path=lib)
        assert np.array_equal(oc, o) and np.array_equal(lc, lse), \
            f"list {i}: contiguous rows mode differs from paged rows mode"


ALL_PINS = [pin_bruteforce, pin_torch_sdpa, pin_constant_v, pin_zero_q, pin_first_token,
            pin_dominant_logit, pin_paged_equals_contiguous, pin_page_permutation,
            pin_chunked_equals_oneshot, pin_gqa_identical_queries, pin_stale_slots_ignored,
            pin_append_scatter, pin_gather, pin_bad_page_id_rejected, pin_row_subset]
