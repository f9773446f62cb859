"""Parity at the library's limits (needs an MI355X): a full batch of 128
sequences, the 64-split maximum on one query tile, and 32 query heads per KV
head; all against the oracle, the pool bit-exact after append."""
import numpy as np
import pytest

import oracle
import paper_2607_17181_amd as tsa
from workload import BF16_NAN, workload_from_lengths

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _check(wl, splits, decode=False):
    import gpu_harness as h
    kp, vp = wl.pool_bits(fill=int(BF16_NAN))
    kp, vp = oracle.append_kv(wl.prefix_lens, wl.suffix_lens, wl.block_tables, wl.page_size,
                              wl.k_new, wl.v_new, kp, vp)
    o_ref, lse_ref = oracle.sp_attention(wl.prefix_lens, wl.suffix_lens, wl.block_tables,
                                         wl.page_size, wl.q, kp, vp)
    db = h.DeviceBatch(wl)
    sp = db.plans(kv_splits=splits)[0]
    tsa.append_kv(sp, db.k_new, db.v_new, db.k_pool, db.v_pool, db.bt)
    call = tsa.decode if decode else tsa.prefill
    call(sp, db.q, db.k_pool, db.v_pool, db.bt, db.out, db.lse, tsa.workspace_tensor(sp))
    torch.cuda.synchronize()
    assert np.array_equal(h.host_bits(db.k_pool), kp)
    assert np.array_equal(h.host_bits(db.v_pool), vp)
    h.assert_parity(h.error_stats(h.host_bits(db.out), o_ref), wl.name)
    assert np.abs(db.lse.cpu().numpy() - lse_ref).max() <= h.LSE_ABS
    return sp


def _wl(name, seed, hq, hkv, d, ps, pre, suf):
    need = sum((p + s + ps - 1) // ps for p, s in zip(pre, suf))
    return workload_from_lengths(name, seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                                 page_size=ps, num_pages=need + 64, prefix_lens=pre,
                                 suffix_lens=suf, extra_pages_per_seq=1)


@pytest.mark.parametrize("decode", [False, True])
def test_full_batch_of_128_sequences(decode):
    rng = np.random.default_rng(77)
    pre = rng.integers(0, 400, size=tsa.MAX_SEQS).tolist()
    suf = [1] * tsa.MAX_SEQS if decode else rng.integers(0, 40, size=tsa.MAX_SEQS).tolist()
    print(f"case 128 sequences decode={decode}", flush=True)
    _check(_wl("max_batch", 78, 8, 1, 128, 16, pre, suf), 0, decode)


def test_64_splits_on_one_query_tile():
    print("case 64 splits", flush=True)
    sp = _check(_wl("max_splits", 79, 8, 1, 128, 16, [9000], [32]), 64)
    items = tsa.plan_items(sp)
    assert items.shape[0] == 64 and int(items[:, 7].max()) == 64


@pytest.mark.parametrize("d", [64, 128])
def test_group_of_32_query_heads(d):
    print(f"case group 32 d={d}", flush=True)
    _check(_wl("group32", 80, 32, 1, d, 32, [700, 0, 1500], [40, 9, 8]), 3)
