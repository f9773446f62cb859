"""SP batch selection: the oracle pinned on cases whose answer follows from
their construction and on the first-fit property, and the C ABI selector
compared with the oracle (host only, no GPU)."""
import numpy as np
import pytest

from oracle import select as osel
import paper_2607_17181_amd as tsa

# One TP rank of a 94-layer GQA model; round numbers make costs easy to read.
M = osel.Model(num_layers=94, num_q_heads=8, num_kv_heads=1, head_dim=128, page_size=16,
               attn_flops_per_s=1e15, per_token_s=1e-5, restore_bytes_per_s=50e9,
               batch_overhead_s=1e-3)


def _c_model(m):
    return tsa.CostModel(m.num_layers, m.num_q_heads, m.num_kv_heads, m.head_dim, m.page_size,
                         m.attn_flops_per_s, m.per_token_s, m.restore_bytes_per_s,
                         m.batch_overhead_s)


def test_candidate_cost_closed_form():
    # P=25,000, S=2,048: 4*128*8*94*(2048*25000 + 2048*2049/2) FLOPs at 1 PFLOP/s
    sec, pages, P, S = osel.candidate(25_000, 2_048, False, M)
    flops = 4 * 128 * 8 * 94 * (2048 * 25000 + 2048 * 2049 / 2)
    assert sec == pytest.approx(flops / 1e15 + 2048 * 1e-5, rel=1e-15)
    assert (pages, P, S) == (1691 - 1563, 25_000, 2_048)   # 8 tokens fill the last prefix page
    # host-resident: 25,000 -> 24,992 restored (1,562 pages of 2*16*128*2*94 bytes), 8 recomputed
    sec_h, pages_h, Ph, Sh = osel.candidate(25_000, 2_048, True, M)
    flops_h = 4 * 128 * 8 * 94 * (2056 * 24992 + 2056 * 2057 / 2)
    restore = 1562 * (2 * 16 * 128 * 2 * 94) / 50e9
    assert sec_h == pytest.approx(flops_h / 1e15 + 2056 * 1e-5 + restore, rel=1e-15)
    assert (pages_h, Ph, Sh) == (1691, 24_992, 2_056)


def test_first_fit_skips_what_does_not_fit():
    small = (1000, 100, 0)
    huge = (100_000, 50_000, 0)
    t_small = osel.candidate(*small[:2], False, M)[0]
    budget = M.batch_overhead_s + 3 * t_small + 1e-9
    idx, *_ = osel.select([small, huge, small, small, small], M, budget, 10**9, 128)
    assert idx == [0, 2, 3]          # the huge call stays queued; later small ones still fit


def test_pages_and_batch_bounds():
    c = (0, 160, 0)                  # 10 new pages each, cheap in time
    idx, *_, pages = osel.select([c] * 10, M, 10.0, 35, 128)
    assert idx == [0, 1, 2] and pages == 30
    idx, *_ = osel.select([c] * 10, M, 10.0, 10**9, 4)
    assert idx == [0, 1, 2, 3]
    idx, *_ = osel.select([(5, 0, 0), (-1, 5, 0), c], M, 10.0, 10**9, 128)
    assert idx == [2]                # empty suffixes and bad prefixes are never admitted


def test_first_fit_property_random():
    rng = np.random.default_rng(0)
    for trial in range(200):
        n = int(rng.integers(1, 40))
        cands = [(int(rng.integers(0, 120_000)), int(rng.integers(1, 5000)), int(rng.random() < 0.3))
                 for _ in range(n)]
        budget, free, mb = float(rng.uniform(0, 0.5)), int(rng.integers(0, 3000)), int(rng.integers(1, 20))
        idx, pre, suf, t, pages = osel.select(cands, M, budget, free, mb)
        assert t <= budget and pages <= free and len(idx) <= mb
        # every skipped candidate before the batch filled would have broken a bound
        tt, pp, taken = 0.0, 0, 0
        for i, (P, S, h) in enumerate(cands):
            if taken >= mb:
                break
            sec, pg, _, _ = osel.candidate(P, S, bool(h), M)
            fits = tt + sec + (M.batch_overhead_s if taken == 0 else 0.0) <= budget and pp + pg <= free
            assert (i in idx) == fits
            if fits:
                tt += sec + (M.batch_overhead_s if taken == 0 else 0.0)
                pp += pg
                taken += 1


def test_c_selector_matches_oracle():
    rng = np.random.default_rng(1)
    model = _c_model(M)
    for trial in range(300):
        n = int(rng.integers(0, 200))
        cands = np.stack([rng.integers(0, 131_072, n), rng.integers(-2, 8192, n),
                          (rng.random(n) < 0.3).astype(np.int64)], axis=1).astype(np.int32)
        budget = tsa.Budget(float(rng.uniform(0, 1.0)), int(rng.integers(0, 20000)),
                            int(rng.integers(0, 129)))
        sel, pre, suf, secs, pages = tsa.sp_select(cands, model, budget)
        idx, opre, osuf, ot, opages = osel.select([tuple(int(x) for x in r) for r in cands], M,
                                                  budget.time_budget_s, budget.free_pages,
                                                  budget.max_batch)
        assert list(sel) == idx and list(pre) == opre and list(suf) == osuf
        assert pages == opages and secs == pytest.approx(ot, rel=1e-12, abs=0)


def test_c_selector_rejects_bad_model():
    m = _c_model(M)
    m.attn_flops_per_s = 0.0
    with pytest.raises(tsa.TalariaError):
        tsa.sp_select(np.zeros((1, 3), np.int32), m, tsa.Budget(1.0, 10, 4))
    with pytest.raises(tsa.TalariaError):
        tsa.sp_select(np.zeros((1, 3), np.int32), _c_model(M), tsa.Budget(1.0, 10, 129))
