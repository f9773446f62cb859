"""XCD placement on the GPU: calibration measures a valid order, and plans
placed by any order give bit-identical outputs and LSE to unplaced plans."""
import numpy as np
import pytest

import paper_2607_17181_amd as tsa
from workload import make_workload, workload_from_lengths

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture
def clear_xcd_order():
    tsa.set_xcd_order(None)
    yield
    tsa.set_xcd_order(None)


def _outputs(db):
    db.out.zero_()
    db.lse.zero_()
    out, lse = db.run()
    torch.cuda.synchronize()
    return out.clone(), lse.clone()


def test_calibration_sets_an_order_and_placement_is_bit_identical(clear_xcd_order):
    import gpu_harness as h
    wl = make_workload("single")  # 256 work items: one round, one per CU
    db = h.DeviceBatch(wl, fill=0)
    ref_out, ref_lse = _outputs(db)
    (sp,) = db.plans()
    ws = tsa.workspace_tensor(sp)
    tsa.append_kv(sp, db.k_new, db.v_new, db.k_pool, db.v_pool, db.bt)
    cal_out = torch.zeros_like(db.out)
    order = tsa.calibrate_xcd(sp, db.q, db.k_pool, db.v_pool, db.bt, cal_out, ws)
    print(f"single: calibrated XCD order {order}")
    assert sorted(order) == list(range(8)) and tsa.get_xcd_order() == order
    assert torch.equal(cal_out, ref_out)  # the calibration launch is an ordinary prefill
    out, lse = _outputs(db)  # plans made now are placed
    assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse)


@pytest.mark.parametrize("order", [[7, 6, 5, 4, 3, 2, 1, 0], [3, 0, 6, 1, 4, 7, 2, 5]])
@pytest.mark.parametrize("case", ["ragged", "gqa_hkv2"])
def test_forced_orders_are_bit_identical(order, case, clear_xcd_order):
    import gpu_harness as h
    if case == "ragged":
        wl = workload_from_lengths("xr", 31, num_q_heads=8, num_kv_heads=1, head_dim=128,
                                   page_size=16, num_pages=9000,
                                   prefix_lens=[0, 37, 20049, 600, 5, 9000],
                                   suffix_lens=[65, 0, 700, 1, 257, 2000],
                                   extra_pages_per_seq=2)
    else:
        wl = workload_from_lengths("xg", 32, num_q_heads=8, num_kv_heads=2, head_dim=64,
                                   page_size=32, num_pages=4000, prefix_lens=[30000, 7000],
                                   suffix_lens=[600, 300], extra_pages_per_seq=2)
    db = h.DeviceBatch(wl, fill=0)
    (sp,) = db.plans()
    n = tsa.plan_items(sp).shape[0]
    print(f"{case}: {n} work items, order {order}")
    assert 8 <= n <= 256  # a single-round plan, so placement applies
    ref_out, ref_lse = _outputs(db)
    tsa.set_xcd_order(order)
    out, lse = _outputs(db)
    assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse)
