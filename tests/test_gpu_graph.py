"""The SP step captured in a HIP graph (through torch's graph capture on the
current stream) and replayed: append + prefill + split combine, and a decode
step.  The library allocates nothing and never synchronises inside a call,
so the whole step records as plain kernel nodes.  Every replay, with eager
work and synchronisation between replays, must match the eager run bit for
bit (outputs, LSE and the appended pool)."""
import numpy as np
import pytest

import paper_2607_17181_amd as tsa
from workload import workload_from_lengths

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _workload(decode):
    pre, suf = ([2500, 700, 40], [1, 1, 1]) if decode else ([3000, 700], [300, 129])
    need = sum((p + s + 15) // 16 for p, s in zip(pre, suf))
    return workload_from_lengths("graph", 31, num_q_heads=8, num_kv_heads=1, head_dim=128,
                                 page_size=16, num_pages=need + 40, prefix_lens=pre,
                                 suffix_lens=suf, extra_pages_per_seq=2)


def _step(db, sp, ws, decode):
    tsa.append_kv(sp, db.k_new, db.v_new, db.k_pool, db.v_pool, db.bt)
    call = tsa.decode if decode else tsa.prefill
    call(sp, db.q, db.k_pool, db.v_pool, db.bt, db.out, db.lse, ws)


@pytest.mark.parametrize("decode", [False, True])
def test_step_graph_replays_match_eager(decode):
    import gpu_harness as h
    wl = _workload(decode)
    print(f"case graph decode={decode}", flush=True)
    eager = h.DeviceBatch(wl)
    sp = eager.plans(kv_splits=3)[0]
    ws = tsa.workspace_tensor(sp)
    _step(eager, sp, ws, decode)
    torch.cuda.synchronize()
    ref = (h.host_bits(eager.out), eager.lse.cpu().numpy(), h.host_bits(eager.k_pool),
           h.host_bits(eager.v_pool))

    db = h.DeviceBatch(wl)
    ws2 = tsa.workspace_tensor(sp)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _step(db, sp, ws2, decode)
    for r in range(3):
        # eager work between replays: clobber the outputs and the workspace
        db.out.fill_(r + 1)
        db.lse.fill_(float(r))
        ws2.fill_(0x7F)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = (h.host_bits(db.out), db.lse.cpu().numpy(), h.host_bits(db.k_pool),
               h.host_bits(db.v_pool))
        for name, a, b in zip(("out", "lse", "k_pool", "v_pool"), got, ref):
            assert np.array_equal(a, b), f"replay {r}: {name} differs from the eager run"
