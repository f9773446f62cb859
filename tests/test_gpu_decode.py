"""Decode-phase attention (one new token per sequence) on the GPU vs the
attention oracle: ragged contexts from empty to 25K tokens, NaN in stale
slots, group sizes 1..32, head_dim 64/128, page sizes 8..256, forced splits."""
import numpy as np
import pytest

import oracle
import paper_2607_17181_amd as tsa
from workload import BF16_NAN, workload_from_lengths

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

CASES = {
    "g8_d128_ps16_mix": (8, 1, 128, 16, [0, 1, 7, 8, 15, 16, 100, 1000, 4097, 25000]),
    "g32_d64_ps8": (32, 1, 64, 8, [333, 2048, 77]),
    "g1_hkv4_d128_ps64": (4, 4, 128, 64, [500, 3000]),
    "g4_hkv2_d128_ps256": (8, 2, 128, 256, [1023, 9000]),
    "g16_d64_ps32": (16, 1, 64, 32, [31, 32, 33, 5000]),
}


def _wl(name, seed=21):
    hq, hkv, d, ps, pre = CASES[name]
    need = sum((p + 1 + ps - 1) // ps for p in pre)
    return workload_from_lengths(name, seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                                 page_size=ps, num_pages=need + 40, prefix_lens=pre,
                                 suffix_lens=[1] * len(pre), extra_pages_per_seq=2)


def _oracle(wl):
    kp, vp = wl.pool_bits(fill=int(BF16_NAN))
    kp, vp = oracle.append_kv(wl.prefix_lens, wl.suffix_lens, wl.block_tables, wl.page_size,
                              wl.k_new, wl.v_new, kp, vp)
    return oracle.sp_attention(wl.prefix_lens, wl.suffix_lens, wl.block_tables, wl.page_size,
                               wl.q, kp, vp)


def _decode(wl, splits):
    import gpu_harness as h
    db = h.DeviceBatch(wl)  # stale slots hold NaN
    sp = db.plans(kv_splits=splits)[0]
    tsa.append_kv(sp, db.k_new, db.v_new, db.k_pool, db.v_pool, db.bt)
    tsa.decode(sp, db.q, db.k_pool, db.v_pool, db.bt, db.out, db.lse, tsa.workspace_tensor(sp))
    return h, h.host_bits(db.out), db.lse.cpu().numpy()


@pytest.mark.parametrize("splits", [0, 1, 3, 20])
@pytest.mark.parametrize("name", list(CASES))
def test_decode_matches_oracle(name, splits):
    wl = _wl(name)
    o_ref, lse_ref = _oracle(wl)
    h, out, lse = _decode(wl, splits)
    h.assert_parity(h.error_stats(out, o_ref), f"{name} splits={splits}")
    assert np.abs(lse - lse_ref).max() <= h.LSE_ABS


def test_decode_equals_prefill_path_within_tolerance_and_is_deterministic():
    import gpu_harness as h
    wl = _wl("g8_d128_ps16_mix")
    _, a, _ = _decode(wl, 0)
    _, b, _ = _decode(wl, 0)
    assert np.array_equal(a, b)
    pre = h.host_bits(h.DeviceBatch(wl).run()[0])
    assert np.abs(h.bits_to_f64(a) - h.bits_to_f64(pre)).max() <= 2e-2
