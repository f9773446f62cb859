"""HKVR page transfer on the GPU vs the CPU oracle (bit-exact), and a restore
followed by the SP path (append + prefill) against the attention oracle."""
import numpy as np
import pytest

import oracle
from oracle import hkvr as hkvr_oracle
import paper_2607_17181_amd as tsa
from workload import BF16_NAN, workload_from_lengths

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

GEOMS = {
    "L3_hkv2_d64_ps32": (3, 2, 64, 32, 40),
    "L4_hkv1_d128_ps16": (4, 1, 128, 16, 64),
    "L1_hkv1_d128_ps256": (1, 1, 128, 256, 6),
}


def _dev16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def _pinned16(a):
    t = torch.empty(a.shape, dtype=torch.int16, pin_memory=True)
    t.copy_(torch.from_numpy(np.ascontiguousarray(a).view(np.int16)))
    return t


def _host16(t):
    return t.cpu().numpy().view(np.uint16)


def _setup(name, seed):
    L, H, d, ps, P = GEOMS[name]
    rng = np.random.default_rng(seed)
    k = rng.integers(0, 1 << 16, size=(L, P, H, ps, d), dtype=np.uint16)
    v = rng.integers(0, 1 << 16, size=(L, P, H, d, ps), dtype=np.uint16)
    n = min(P - 1, 23)
    ids = rng.permutation(P)[:n].astype(np.int32)
    ids[n // 2] = P + 5          # out of range: moves nothing
    ids[-1] = -3
    slab = rng.integers(0, 1 << 16, size=(n, L, 2, H * ps * d), dtype=np.uint16)
    return tsa.kv_cache(L, H, d, ps, P), k, v, ids, slab


@pytest.mark.parametrize("name", list(GEOMS))
def test_restore_bit_exact(name):
    c, k, v, ids, slab = _setup(name, 1)
    kd, vd = _dev16(k), _dev16(v)
    tsa.hkvr_restore(c, _pinned16(slab), torch.from_numpy(ids).cuda(), kd, vd)
    torch.cuda.synchronize()
    kr, vr = hkvr_oracle.restore(slab, ids, k, v)
    assert np.array_equal(_host16(kd), kr) and np.array_equal(_host16(vd), vr)


@pytest.mark.parametrize("name", list(GEOMS))
def test_checkpoint_bit_exact(name):
    c, k, v, ids, slab = _setup(name, 2)
    hs = _pinned16(slab)
    tsa.hkvr_checkpoint(c, _dev16(k), _dev16(v), torch.from_numpy(ids).cuda(), hs)
    torch.cuda.synchronize()
    assert np.array_equal(_host16(hs), hkvr_oracle.checkpoint(k, v, ids, slab))


def test_restore_then_sp_prefill_matches_oracle():
    """A prefix checkpointed from one layer-first cache and restored into
    freshly allocated pages of another serves the SP path exactly as a
    device-resident prefix does."""
    import gpu_harness as h
    L, layer = 3, 1
    wl = workload_from_lengths("hkvr_sp", 11, num_q_heads=8, num_kv_heads=1, head_dim=128,
                               page_size=16, num_pages=200, prefix_lens=[1024], suffix_lens=[200])
    kp, vp = wl.pool_bits(fill=int(BF16_NAN))
    npre = 1024 // 16
    ids = wl.block_tables[0, :npre].astype(np.int32)
    c = tsa.kv_cache(L, 1, 128, 16, wl.num_pages)
    # source cache: the workload's prefix pages in `layer`, other layers noise
    rng = np.random.default_rng(5)
    src_k = rng.integers(0, 1 << 16, size=(L,) + kp.shape, dtype=np.uint16)
    src_v = rng.integers(0, 1 << 16, size=(L,) + vp.shape, dtype=np.uint16)
    src_k[layer], src_v[layer] = kp, vp
    slab = _pinned16(np.zeros(tsa.slab_shape(c, npre), np.uint16))
    tsa.hkvr_checkpoint(c, _dev16(src_k), _dev16(src_v), torch.from_numpy(ids).cuda(), slab)
    # destination cache: NaN everywhere, then restore, then the SP path on `layer`
    dst_k = _dev16(np.full((L,) + kp.shape, BF16_NAN, np.uint16))
    dst_v = _dev16(np.full((L,) + vp.shape, BF16_NAN, np.uint16))
    tsa.hkvr_restore(c, slab, torch.from_numpy(ids).cuda(), dst_k, dst_v)
    db = h.DeviceBatch(wl)
    db.k_pool, db.v_pool = dst_k[layer], dst_v[layer]
    out, _ = db.run()
    kref, vref = oracle.append_kv(wl.prefix_lens, wl.suffix_lens, wl.block_tables, 16,
                                  wl.k_new, wl.v_new, kp, vp)
    o_ref, _ = oracle.sp_attention(wl.prefix_lens, wl.suffix_lens, wl.block_tables, 16, wl.q,
                                   kref, vref)
    h.assert_parity(h.error_stats(h.host_bits(out), o_ref), "restore + SP")
    # the restored layer's pool now equals the oracle's appended pool
    assert np.array_equal(h.host_bits(dst_k[layer]), kref)
    assert np.array_equal(h.host_bits(dst_v[layer]), vref)
