"""The allocation-free prefill entry point against talaria_sp_attn_prefill.

talaria_sp_attn_prefill_noalloc runs the same kernels with the library's own
per-GPU scratch in place of the caller's workspace, so on the same plan and
inputs its output and LSE must equal the workspace call's bit for bit.  Two
calls in a row, the second with a smaller batch (the scratch keeps the first
call's contents), both split so the scratch is really used; each output is
also held to the oracle's parity bar.  Called through the C ABI.
"""
import numpy as np
import pytest

import oracle
import paper_2607_17181_amd as tsa
from workload import BF16_NAN, workload_from_lengths

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _wl(seed, pre, suf):
    ps = 16
    need = sum((p + s + ps - 1) // ps for p, s in zip(pre, suf))
    return workload_from_lengths("noalloc", seed, num_q_heads=8, num_kv_heads=1, head_dim=128,
                                 page_size=ps, num_pages=need + 40, prefix_lens=pre,
                                 suffix_lens=suf)


def _run(wl, kv_splits):
    import gpu_harness as gh
    kp, vp = wl.pool_bits(fill=int(BF16_NAN))
    k_pool, v_pool = gh.dev_bits(kp), gh.dev_bits(vp)
    q, k_new, v_new = gh.dev_bits(wl.q), gh.dev_bits(wl.k_new), gh.dev_bits(wl.v_new)
    bt = torch.from_numpy(wl.block_tables).cuda()
    geom = tsa.make_geom(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.page_size,
                         wl.num_pages)
    sp = tsa.plan(geom, wl.prefix_lens, wl.suffix_lens, wl.max_pages_per_seq, kv_splits)
    assert 0 < sp.workspace_bytes <= tsa.noalloc_scratch_bytes()
    tsa.append_kv(sp, k_new, v_new, k_pool, v_pool, bt)
    out_ws, out_na = torch.zeros_like(q), torch.full_like(q, 0x7FC0)
    lse_ws = torch.zeros(q.shape[:2], dtype=torch.float32, device="cuda")
    lse_na = torch.full_like(lse_ws, float("nan"))
    tsa.prefill(sp, q, k_pool, v_pool, bt, out_ws, lse_ws, tsa.workspace_tensor(sp))
    tsa.prefill_noalloc(sp, q, k_pool, v_pool, bt, out_na, lse_na)
    torch.cuda.synchronize()
    return (gh.host_bits(out_ws), lse_ws.cpu().numpy(), gh.host_bits(out_na),
            lse_na.cpu().numpy(), kp)


def test_noalloc_matches_workspace_call_twice():
    import gpu_harness as gh
    cases = [(_wl(31, [3000, 410], [700, 333]), 5),   # larger first call
             (_wl(32, [500], [100]), 3)]              # then a smaller one
    for i, (wl, splits) in enumerate(cases):
        print(f"noalloc call {i}: P={list(wl.prefix_lens)} S={list(wl.suffix_lens)} "
              f"splits={splits}", flush=True)
        o_ws, l_ws, o_na, l_na, kp = _run(wl, splits)
        assert np.array_equal(o_na, o_ws), f"call {i}: output differs from the workspace call"
        assert np.array_equal(l_na.view(np.uint32), l_ws.view(np.uint32)), \
            f"call {i}: LSE differs from the workspace call"
        kp2, vp2 = oracle.append_kv(wl.prefix_lens, wl.suffix_lens, wl.block_tables,
                                    wl.page_size, wl.k_new, wl.v_new, *wl.pool_bits(
                                        fill=int(BF16_NAN)))
        o_ref, lse_ref = oracle.sp_attention(wl.prefix_lens, wl.suffix_lens, wl.block_tables,
                                             wl.page_size, wl.q, kp2, vp2)
        gh.assert_parity(gh.error_stats(o_na, o_ref), f"noalloc call {i}")
        assert np.abs(l_na - lse_ref).max() <= gh.LSE_ABS, f"call {i}: LSE vs oracle"
