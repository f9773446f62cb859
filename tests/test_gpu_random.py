"""Seeded random small batches on the GPU against the attention oracle.

Each case draws its GQA geometry, head_dim, page size, batch size, prefix and
suffix lengths (including empty suffixes, or one token per sequence for a
decode batch) and a forced split count, so that combinations no hand-picked
case covers are exercised.  Stale pool slots hold NaN.  Checks: the pool
after append is bit-exact over the whole pool; prefill (or decode, for a
one-token batch) matches the oracle to the parity bar.
"""
import numpy as np
import pytest

import oracle
import paper_2607_17181_amd as tsa
from workload import BF16_NAN, workload_from_lengths

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

GEOMS = [(2, 1, 64), (8, 1, 128), (8, 2, 128), (16, 1, 64), (12, 4, 128), (32, 1, 128),
         (10, 2, 64), (4, 4, 128)]
PAGE_SIZES = [8, 16, 32, 64, 128, 256]
SPLITS = [0, 0, 1, 2, 5, 9]


def random_case(seed):
    rng = np.random.default_rng(1000 + seed)
    hq, hkv, d = GEOMS[int(rng.integers(len(GEOMS)))]
    ps = PAGE_SIZES[int(rng.integers(len(PAGE_SIZES)))]
    n = int(rng.integers(1, 5))
    decode = seed % 4 == 3
    pre = rng.integers(0, 3000, size=n).tolist()
    suf = [1] * n if decode else rng.integers(0, 300, size=n).tolist()
    if sum(suf) == 0:
        suf[0] = 1
    splits = SPLITS[int(rng.integers(len(SPLITS)))]
    need = sum((p + s + ps - 1) // ps for p, s in zip(pre, suf))
    wl = workload_from_lengths(f"random{seed}", 500 + seed, num_q_heads=hq, num_kv_heads=hkv,
                               head_dim=d, page_size=ps, num_pages=need + 40, prefix_lens=pre,
                               suffix_lens=suf, extra_pages_per_seq=2)
    return wl, splits, decode


@pytest.mark.parametrize("seed", range(128))
def test_random_batch_matches_oracle(seed):
    import gpu_harness as h
    wl, splits, decode = random_case(seed)
    print(f"case seed={seed} hq={wl.num_q_heads} hkv={wl.num_kv_heads} d={wl.head_dim} "
          f"ps={wl.page_size} P={list(wl.prefix_lens)} S={list(wl.suffix_lens)} "
          f"splits={splits} decode={decode}", flush=True)
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
    h.assert_parity(h.error_stats(h.host_bits(db.out), o_ref), f"seed={seed}")
    assert np.abs(db.lse.cpu().numpy() - lse_ref).max() <= h.LSE_ABS
