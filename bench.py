#!/usr/bin/env python3
"""Benchmark: session-prefill attention for one 25K-prefix continuation.

One step = the whole hot path for one SP batch of one attention layer:
plan (host) -> append_kv (new K/V into pool pages) -> prefill (paged causal
attention; split key ranges merged by the LSE combine).  Inputs are seeded
synthetic tensors already resident in HBM when timing starts.

Workload: one continuation with a 25,000-token cached prefix and 2,048 new
tokens, Hq=8 / Hkv=1 / head_dim=128 (one TP=8 rank's head share of a
235B-class GQA model), page size 16, pages shuffled in a 100K-page pool.

Prints ONE JSON line: the single continuation's throughput, with HIP-event
step and prefill-call distributions (mean, nearest-rank p50 / p5 / p95), the
prefill call's roofline, the CPU oracle timed beside it over all 16,384 query
rows, and the parity of the timed GPU output against those rows; under
"configs", the tiny, ragged, long and cold workloads timed the same way, each
with the oracle's speed and parity on a seeded row sample.  Extra figures
(per-kernel times, standalone append/gather bandwidth) go to --extra-json.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)
sys.path.insert(0, os.path.join(HERE, "tests"))

METRIC = "SP prefill attention TFLOP/s (% bf16 MFMA peak); ms per 25K-prefix continuation"
WORKLOADS = {
    "tiny": "tiny: 1 sequence, P=256 + S=64, Hq=2 Hkv=1 d=64, page 16, 64-page pool",
    "single": "single continuation: P=25,000 cached + S=2,048 new tokens, Hq=8 Hkv=1 d=128, "
              "page 16, shuffled 100K-page pool",
    "ragged": "ragged SP batch: 16 continuations, P lognormal (median 25K, p95 105K, cap 128K), "
              "S uniform 512-4096, Hq=8 Hkv=1 d=128, page 16, 300K-page pool",
    "long": "long context: P=105,000 + S=8,192 as 4 chunked-prefill chunks of 2,048, "
            "Hq=8 Hkv=1 d=128, page 16, 100K-page pool",
    "cold": "cold recompute: 4 sequences, P=0 + S=25,000, Hq=8 Hkv=1 d=128, page 16, "
            "100K-page pool",
}
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # The GPU settles to its steady (power-limited) clock only after about
    # 50-100 ms of continuous MFMA work; a 5-step warm-up timed the single
    # continuation's prefill call at 0.201 ms p50 where the settled figure is
    # 0.189 ms.  400 warm-up steps are about 0.1 s of work.
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=400)
    ap.add_argument("--config", default="single",
                    choices=["tiny", "single", "ragged", "long", "cold"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-xcd-calibration", action="store_true",
                    help="leave XCD placement off (plans run item i on workgroup i)")
    ap.add_argument("--cpu-rows", type=int, default=16384,
                    help="query rows of the workload the oracle baseline computes")
    ap.add_argument("--extra-json", default=None,
                    help="write per-kernel / per-config figures to this file")
    ap.add_argument("--no-extra-configs", action="store_true",
                    help="time only --config (by default tiny, ragged, long and cold are also "
                         "timed and reported under \"configs\")")
    ap.add_argument("--extra-steps", type=int, default=20,
                    help="timed steps for each of the other configs")
    ap.add_argument("--extra-warmup-ms", type=float, default=150.0,
                    help="untimed warm-up of each of the other configs, in ms of steps "
                         "(at least 3 steps)")
    ap.add_argument("--extra-rows", type=int, default=4096,
                    help="seeded query rows the oracle computes for each of the other configs")
    ap.add_argument("--hbm-sweep", action="store_true",
                    help="only time append_kv / gather_kv on 0.1-2 GB batches (cache flushed) "
                         "and print one JSON line")
    ap.add_argument("--hkvr", action="store_true",
                    help="only time HKVR restore/checkpoint of a 25K-token prefix over 94 "
                         "layers and print one JSON line")
    ap.add_argument("--stage", action="store_true",
                    help="only time the D2D-staged weight gather (4 GiB) and print one JSON line")
    ap.add_argument("--select", action="store_true",
                    help="only time SP batch selection over 1000 candidates (host)")
    ap.add_argument("--decode", action="store_true",
                    help="only time a 64-sequence decode step and print one JSON line")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB three times "
                         "(reference for the HBM traffic counters) and exit")
    return ap.parse_args()


def nearest_rank(values, q):
    """p_q of `values` by the nearest-rank definition the paper's evaluation
    uses (Section 5.1): the observation at rank ceil(q N / 100), 1-based."""
    v = sorted(values)
    return float(v[max(1, math.ceil(q * len(v) / 100)) - 1])


def dist(values):
    """Mean, nearest-rank median / p5 / p95 of a list of milliseconds."""
    return {"mean": round(float(np.mean(values)), 4), "p50": round(nearest_rank(values, 50), 4),
            "p5": round(nearest_rank(values, 5), 4), "p95": round(nearest_rank(values, 95), 4)}


def time_config(name, steps, warmup, torch, tsa, harness, workload, calibrate=True):
    """Time `steps` whole-path steps after `warmup` untimed ones (a negative
    `warmup` is a warm-up length in ms); return a dict of figures."""
    wl = workload.make_workload(name)
    db = harness.DeviceBatch(wl, fill=0)
    flops = wl.flops()
    n_chunks = len(wl.chunks)
    stream = torch.cuda.current_stream()

    # Plans are made inside the timed step (host work is part of the path);
    # workspaces are allocated once up front, sized by a first plan.
    plans0 = db.plans()
    workspaces = [tsa.workspace_tensor(sp) for sp in plans0]
    chunk_t = [db.chunk_tensors(c) for c in range(n_chunks)]

    # Set-up: measure the XCD order on the first chunk (one ordinary prefill
    # with per-workgroup timing); the plans made in the timed steps are
    # placed by it.
    xcd_order = None
    tsa.set_xcd_order(None)
    if calibrate and tsa.plan_items(plans0[0]).shape[0] >= 8:
        q, kn, vn, out, _, _ = chunk_t[0]
        tsa.append_kv(plans0[0], kn, vn, db.k_pool, db.v_pool, db.bt)
        xcd_order = tsa.calibrate_xcd(plans0[0], q, db.k_pool, db.v_pool, db.bt, out,
                                      workspaces[0])

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * n_chunks + 1)]
          for _ in range(steps)]
    plan_s = 0.0

    def step(events):
        nonlocal plan_s
        t0 = time.perf_counter()
        plans = db.plans()
        plan_s += time.perf_counter() - t0
        if events is not None:
            events[0].record(stream)
        for c, sp in enumerate(plans):
            q, kn, vn, out, lse, idx = chunk_t[c]
            tsa.append_kv(sp, kn, vn, db.k_pool, db.v_pool, db.bt)
            if events is not None:
                events[2 * c + 1].record(stream)
            tsa.prefill(sp, q, db.k_pool, db.v_pool, db.bt, out, lse, workspaces[c])
            if events is not None:
                events[2 * c + 2].record(stream)

    if warmup < 0:
        # Warm-up given in ms: at least 3 steps, then as many as fill it.
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(3):
            step(None)
        torch.cuda.synchronize()
        per_step = (time.perf_counter() - t0) / 3
        warmup = max(0, math.ceil(-warmup / 1e3 / per_step) - 3)
    for _ in range(warmup):
        step(None)
    torch.cuda.synchronize()
    plan_s = 0.0
    t0 = time.perf_counter()
    for i in range(steps):
        step(ev[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    append_ms, prefill_ms, span_ms = [], [], []
    for e in ev:
        a = p = 0.0
        for c in range(n_chunks):
            a += e[2 * c].elapsed_time(e[2 * c + 1])
            p += e[2 * c + 1].elapsed_time(e[2 * c + 2])
        append_ms.append(a)
        prefill_ms.append(p)
        span_ms.append(e[0].elapsed_time(e[2 * n_chunks]))
    # Outputs of the last step, in token order (chunks scattered back).
    for c in range(n_chunks):
        _, _, _, out, lse, idx = chunk_t[c]
        if idx is not None:
            db.out[idx] = out
            db.lse[idx] = lse
    torch.cuda.synchronize()
    ms_step = wall * 1e3 / steps
    prefill_avg = float(np.mean(prefill_ms))
    append_avg = float(np.mean(append_ms))
    T = wl.total_tokens
    append_bytes = 2 * 2 * T * wl.num_kv_heads * wl.head_dim * 2   # K+V, read + write
    return {
        "workload": name,
        "flops": flops,
        "ms_per_step": ms_step,
        "tflops_step": flops / (ms_step * 1e-3) / 1e12,
        "step_gpu_ms": dist(span_ms),
        "prefill_call_ms": prefill_avg,
        "prefill_call_dist_ms": dist(prefill_ms),
        "prefill_tflops": flops / (prefill_avg * 1e-3) / 1e12,
        "append_ms": append_avg,
        "append_gbs": append_bytes / (append_avg * 1e-3) / 1e9,
        "plan_us": plan_s / steps * 1e6,
        "num_items": [int(tsa.plan_items(sp).shape[0]) for sp in plans0],
        "xcd_order": xcd_order,
        "warmup_steps": warmup,
        "workspace_bytes": [sp.workspace_bytes for sp in plans0],
        "wl": wl,
        "db": db,
    }


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_rows(wl, rows, oracle):
    """The oracle (fp64) on the flat rows `rows` of a workload: pools with the
    prefix in place, the suffix appended by the oracle's own scatter; returns
    (o [R, d], lse [R], seconds)."""
    from workload import BF16_NAN
    kp, vp = wl.pool_bits(fill=int(BF16_NAN))
    o_all, l_all = [], []
    t = 0.0
    for pre, suf, tok in wl.chunks:
        kp, vp = oracle.append_kv(pre, suf, wl.block_tables, wl.page_size, wl.k_new[tok],
                                  wl.v_new[tok], kp, vp)
    # After every chunk is appended the pool holds all positions; rows of a
    # chunk see only keys up to their own position, so attending each chunk's
    # rows over the final pool equals the chunked computation.
    Hq = wl.num_q_heads
    for pre, suf, tok in wl.chunks:
        lo, hi = int(tok[0]) * Hq, (int(tok[-1]) + 1) * Hq
        sel = rows[(rows >= lo) & (rows < hi)]
        if sel.size == 0:
            continue
        t0 = time.perf_counter()
        o, l = oracle.sp_attention(pre, suf, wl.block_tables, wl.page_size, wl.q[tok], kp, vp,
                                   rows=sel - lo)
        t += time.perf_counter() - t0
        o_all.append(o)
        l_all.append(l)
    return np.concatenate(o_all), np.concatenate(l_all), t


def row_flops(wl, rows):
    """4 d per visible (row, key) pair over the flat rows `rows`."""
    tok = rows // wl.num_q_heads
    offs = np.concatenate([[0], np.cumsum(wl.suffix_lens)])
    seq = np.searchsorted(offs, tok, side="right") - 1
    visible = wl.prefix_lens[seq].astype(np.int64) + (tok - offs[seq]) + 1
    return float(4 * wl.head_dim * visible.sum())


def parity(wl, db, rows, o_ref, lse_ref, harness):
    """The GPU output of the timed run against oracle rows."""
    import torch  # noqa: F401
    out = harness.host_bits(db.out).reshape(-1, wl.head_dim)[rows]
    st = harness.error_stats(out, o_ref)
    lse = db.lse.cpu().numpy().reshape(-1)[rows]
    return {"rows": int(len(rows)), "max_abs": float(f"{st['max_abs']:.3e}"),
            "mean_abs": float(f"{st['mean_abs']:.3e}"), "rel_l2": float(f"{st['rel_l2']:.3e}"),
            "lse_max_abs": float(f"{float(np.abs(lse - lse_ref).max()):.3e}"),
            "pass": bool(st["finite"] and st["max_abs"] <= harness.MAX_ABS and
                         st["mean_abs"] <= harness.MEAN_ABS and st["rel_l2"] <= harness.REL_L2 and
                         np.abs(lse - lse_ref).max() <= harness.LSE_ABS)}


def cpu_baseline(wl, rows, oracle, min_seconds=10.0):
    """The oracle timed on the host cores over the flat rows `rows` of the
    workload, repeated until about `min_seconds` have been timed; returns the
    baseline record and the first pass's (o, lse) for the parity check."""
    flops = row_flops(wl, rows)
    passes, dt, first = 0, 0.0, None
    while True:
        o, lse, t = oracle_rows(wl, rows, oracle)
        first = first or (o, lse)
        passes += 1
        dt += t
        if dt >= min_seconds or passes >= 50:
            break
    n_all = wl.total_tokens * wl.num_q_heads
    return ({"value": passes * flops / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
             "cpu": cpu_model(), "kind": "oracle",
             "sample": f"{len(rows)} of {n_all} query rows (seeded) of the same workload, fp64, "
                       f"{passes} pass(es) in {dt:.1f} s of oracle time"}, first)


def sample_rows(wl, n, seed=123):
    """Seeded sorted sample of n flat query rows (all of them if fewer)."""
    n_all = wl.total_tokens * wl.num_q_heads
    if n >= n_all:
        return np.arange(n_all)
    return np.sort(np.random.default_rng(seed).choice(n_all, size=n, replace=False))


def measured_traffic(config):
    """HBM bytes per prefill call from the committed counter summary, or None.

    The summary records a hash of the kernel and planner sources it was taken
    with; once those change the counters no longer describe the kernel and
    the figure is withheld (None)."""
    import hashlib
    path = os.path.join(HERE, "profiles", f"prefill_{config}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    src = b"".join(open(os.path.join(HERE, s), "rb").read() for s in rec["sources"])
    if hashlib.sha256(src).hexdigest() != rec["sources_sha256"]:
        return None
    return int(rec["traffic_bytes_per_call"])


def hbm_sweep(torch, tsa, reps=10):
    """append_kv / gather_kv GB/s on synthetic batches of 102 MB to 2 GB, with
    the 256 MB Infinity Cache flushed before every repetition by reading a
    1 GiB buffer.  (Writing the buffer instead would leave the cache full of
    dirty lines that the timed kernel then has to write back to HBM.)"""
    scratch = torch.ones(1 << 27, dtype=torch.int64, device="cuda")
    sink = torch.zeros(1, dtype=torch.int64, device="cuda")

    def timeit(fn, warm_ms=150.0):
        # Untimed calls for at least warm_ms first, so that the part has
        # settled to its steady clock.
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        while (time.perf_counter() - t0) * 1e3 < warm_ms:
            for _ in range(5):
                fn()
            torch.cuda.synchronize()
        ts = []
        for r in range(reps):
            sink.add_(scratch.sum())
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    res = []
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    for nseq, S, P in [(4, 25_000, 0), (16, 4_096, 25_000), (8, 250_000, 0)]:
        hkv, d, ps = 1, 128, 16
        pages = (P + S + ps - 1) // ps
        num_pages = nseq * pages + 64
        T = nseq * S
        sp = tsa.plan(tsa.make_geom(8, hkv, d, ps, num_pages), [P] * nseq, [S] * nseq, pages)
        perm = torch.randperm(num_pages, device="cuda", generator=gen, dtype=torch.int32)
        bt = perm[: nseq * pages].view(nseq, pages).contiguous()
        kp = torch.zeros((num_pages, hkv, ps, d), dtype=torch.int16, device="cuda")
        vp = torch.zeros((num_pages, hkv, d, ps), dtype=torch.int16, device="cuda")
        kn = torch.randint(-30000, 30000, (T, hkv, d), dtype=torch.int16, device="cuda",
                           generator=gen)
        vn = torch.randint(-30000, 30000, (T, hkv, d), dtype=torch.int16, device="cuda",
                           generator=gen)
        ms = timeit(lambda: tsa.append_kv(sp, kn, vn, kp, vp, bt))
        nbytes = 2 * 2 * T * hkv * d * 2
        res.append({"kernel": "append_kv", "batch": f"{nseq}x(P={P},S={S})", "bytes": nbytes,
                    "us": round(ms * 1e3, 1), "gbs": round(nbytes / ms / 1e6)})
        nk = nseq * (P + S)
        ko = torch.empty((nk, hkv, d), dtype=torch.int16, device="cuda")
        vo = torch.empty_like(ko)
        ms = timeit(lambda: tsa.gather_kv(sp, kp, vp, bt, ko, vo))
        nbytes = 2 * 2 * nk * hkv * d * 2
        res.append({"kernel": "gather_kv", "batch": f"{nseq}x(P={P},S={S})", "bytes": nbytes,
                    "us": round(ms * 1e3, 1), "gbs": round(nbytes / ms / 1e6)})
        del kp, vp, kn, vn, ko, vo
        torch.cuda.empty_cache()
    return res


def hkvr_bench(torch, tsa, layers=94, prefix=25_000, reps=5):
    """HKVR restore (host slab -> device pages) and checkpoint (device -> host)
    of one continuation's page-aligned prefix across all layers of one TP
    rank's share of a 94-layer GQA model (Hkv=1, d=128, page 16), against a
    plain pinned-host <-> device copy of the same bytes."""
    ps, d, hkv = 16, 128, 1
    n = prefix // ps
    num_pages = n + 1024
    cache = tsa.kv_cache(layers, hkv, d, ps, num_pages)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7)
    ids = torch.randperm(num_pages, device="cuda", generator=gen, dtype=torch.int32)[:n]
    kc = torch.zeros((layers, num_pages, hkv, ps, d), dtype=torch.int16, device="cuda")
    vc = torch.zeros((layers, num_pages, hkv, d, ps), dtype=torch.int16, device="cuda")
    slab = torch.empty(tsa.slab_shape(cache, n), dtype=torch.int16, pin_memory=True)
    slab.random_(-30000, 30000)
    flat = torch.empty(slab.numel(), dtype=torch.int16, device="cuda")

    def timeit(fn):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    nbytes = slab.numel() * 2
    out = {"workload": f"{layers} layers x {n} pages (P={n * ps}), Hkv={hkv} d={d} page {ps}",
           "bytes": nbytes}
    for name, fn in [("restore", lambda: tsa.hkvr_restore(cache, slab, ids, kc, vc)),
                     ("checkpoint", lambda: tsa.hkvr_checkpoint(cache, kc, vc, ids, slab)),
                     ("memcpy_h2d", lambda: flat.copy_(slab.view(-1), non_blocking=True)),
                     ("memcpy_d2h", lambda: slab.view(-1).copy_(flat, non_blocking=True))]:
        ms = timeit(fn)
        out[name] = {"ms": round(ms, 3), "gbs": round(nbytes / ms / 1e6, 1)}
    return out


def stage_bench(torch, tsa, weight_gib=4, chunk_mib=2, reps=5):
    """D2D-staged switch: assemble a weight region of weight_gib GiB from
    chunk_mib MiB chunks, (a) all staged and clean (pure D2D), (b) with the
    chunks under 10% of the KV pages dirty (D2D + H2D top-up), (c) all from
    host (pure H2D); plus the dirty-marking kernel."""
    chunk = chunk_mib << 20
    n = (weight_gib << 30) // chunk
    page = 64 << 10
    stage_bytes = n * chunk + (64 << 20)
    chunks = torch.tensor([[(64 << 20) + i * chunk, i * chunk, chunk] for i in range(n)],
                          dtype=torch.int64, device="cuda")
    staging = torch.zeros(stage_bytes, dtype=torch.uint8, device="cuda")
    weights = torch.empty(n * chunk, dtype=torch.uint8, device="cuda")
    host = torch.empty(n * chunk, dtype=torch.uint8, pin_memory=True)
    num_pages = stage_bytes // page
    words = (num_pages + 31) // 32
    gen = torch.Generator(device="cuda")
    gen.manual_seed(3)
    used_bits = torch.rand(num_pages, device="cuda", generator=gen) < 0.001  # scattered KV pages
    w = torch.zeros(words * 32, dtype=torch.int64, device="cuda")
    w[:num_pages] = used_bits.to(torch.int64)
    used = (w.view(words, 32) << torch.arange(32, device="cuda")).sum(1).to(torch.int32)
    cw = (n + 31) // 32
    all_set = torch.full((cw,), -1, dtype=torch.int32, device="cuda")
    none_set = torch.zeros(cw, dtype=torch.int32, device="cuda")
    dirty = torch.zeros(cw, dtype=torch.int32, device="cuda")

    def timeit(fn):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    ms_mark = timeit(lambda: tsa.stage_mark_dirty(chunks, used, num_pages, page, dirty))
    n_dirty = int(sum(bin(int(x) & 0xFFFFFFFF).count("1") for x in dirty.cpu().tolist()))
    nbytes = n * chunk
    res = {"workload": f"{n} chunks x {chunk_mib} MiB = {nbytes / 2**30:.0f} GiB of weights",
           "mark_dirty_us": round(ms_mark * 1e3, 1), "dirty_chunks": n_dirty}
    for name, stg, drt in [("all_d2d", all_set, none_set), ("d2d_plus_h2d", all_set, dirty),
                           ("all_h2d", none_set, none_set)]:
        ms = timeit(lambda: tsa.stage_gather(chunks, stg, drt, staging, host, weights))
        # weight bytes placed per second; a D2D chunk also reads as many HBM bytes
        res[name] = {"ms": round(ms, 3), "weight_gbs": round(nbytes / ms / 1e6, 1)}
    res["all_d2d"]["hbm_read_write_gbs"] = round(2 * nbytes / res["all_d2d"]["ms"] / 1e6, 1)
    return res


def select_bench(tsa, n=1000, reps=200):
    """Host latency of SP batch selection over n queued continuations."""
    rng = np.random.default_rng(11)
    cands = np.stack([np.minimum(np.round(np.exp(rng.normal(np.log(25_000), 0.87247, n))), 131_072),
                      rng.integers(512, 4097, n), (rng.random(n) < 0.3)],
                     axis=1).astype(np.int32)
    model = tsa.CostModel(94, 8, 1, 128, 16, 1.0e15, 1e-5, 50e9, 1e-3)
    budget = tsa.Budget(2.0, 200_000, 128)
    tsa.sp_select(cands, model, budget)
    t0 = time.perf_counter()
    for _ in range(reps):
        sel, *_ = tsa.sp_select(cands, model, budget)
    us = (time.perf_counter() - t0) / reps * 1e6
    return {"candidates": n, "admitted": int(len(sel)), "us_per_call": round(us, 2),
            "note": "includes the Python binding's marshalling"}


def decode_bench(torch, tsa, harness, workload, n_seqs=64, reps=100):
    """Decode step of a batch of continuations: lognormal contexts (median
    25K, p95 105K tokens), one new token each, Hq=8 Hkv=1 d=128 page 16.
    GB/s = K/V bytes of every context position read once / decode call time;
    the same plan run through the prefill kernel for comparison."""
    rng = np.random.default_rng(17)
    pre = workload.lognormal_prefix_lengths(rng, n_seqs).tolist()
    need = sum((p_ + 1 + 15) // 16 for p_ in pre)
    wl = workload.workload_from_lengths("decode", 17, num_q_heads=8, num_kv_heads=1,
                                        head_dim=128, page_size=16, num_pages=need + 1024,
                                        prefix_lens=pre, suffix_lens=[1] * n_seqs)
    db = harness.DeviceBatch(wl, fill=0)
    sp = db.plans()[0]
    ws = tsa.workspace_tensor(sp)
    tsa.append_kv(sp, db.k_new, db.v_new, db.k_pool, db.v_pool, db.bt)

    def timeit(fn, warm_ms=150.0):
        # Untimed calls first, for at least warm_ms, so that the part has
        # settled to its steady clock (as the prefill configs are timed).
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        while (time.perf_counter() - t0) * 1e3 < warm_ms:
            for _ in range(10):
                fn()
            torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    kv_bytes = int(sum(p_ + 1 for p_ in pre)) * wl.num_kv_heads * wl.head_dim * 2 * 2
    ms_dec = timeit(lambda: tsa.decode(sp, db.q, db.k_pool, db.v_pool, db.bt, db.out, db.lse, ws))
    ms_pre = timeit(lambda: tsa.prefill(sp, db.q, db.k_pool, db.v_pool, db.bt, db.out, db.lse, ws))
    ms_app = timeit(lambda: tsa.append_kv(sp, db.k_new, db.v_new, db.k_pool, db.v_pool, db.bt))
    return {"workload": f"decode step of {n_seqs} continuations, contexts lognormal median 25K "
                        f"(total {sum(pre) + n_seqs} positions), Hq=8 Hkv=1 d=128 page 16",
            "items": int(tsa.plan_items(sp).shape[0]), "kv_bytes": kv_bytes,
            "decode_call_us": round(ms_dec * 1e3, 1),
            "decode_gbs": round(kv_bytes / ms_dec / 1e6, 1),
            "prefill_path_us": round(ms_pre * 1e3, 1),
            "prefill_path_gbs": round(kv_bytes / ms_pre / 1e6, 1),
            "append_us": round(ms_app * 1e3, 1)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the path is "
              "sharded by KV head or by sequence with no exchange, see the design notes.",
              file=sys.stderr)
        sys.exit(2)
    if args.select:
        import paper_2607_17181_amd as tsa
        print(json.dumps({"select": select_bench(tsa)}), flush=True)
        return
    import torch
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n, "copy_calibration_bytes_written": n,
                          "copies": 3}), flush=True)
        return
    import paper_2607_17181_amd as tsa
    import gpu_harness as harness
    import workload

    tsa.library()  # fail loudly if the HIP library is missing
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.decode:
        import gpu_harness as harness
        import workload
        print(json.dumps({"decode": decode_bench(torch, tsa, harness, workload)}), flush=True)
        return
    if args.stage:
        print(json.dumps({"stage": stage_bench(torch, tsa)}), flush=True)
        return
    if args.hkvr:
        print(json.dumps({"hkvr": hkvr_bench(torch, tsa)}), flush=True)
        return
    if args.hbm_sweep:
        print(json.dumps({"hbm_sweep": hbm_sweep(torch, tsa), "peak_gbs": PEAK_HBM_GBS}),
              flush=True)
        return

    r = time_config(args.config, args.steps, args.warmup, torch, tsa, harness, workload,
                    calibrate=not args.no_xcd_calibration)
    wl = r.pop("wl")
    db = r.pop("db")
    achieved = r["prefill_tflops"]
    line = {
        "metric": METRIC,
        "value": round(r["tflops_step"], 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": WORKLOADS.get(args.config, args.config),
            "num_seqs": wl.num_seqs,
            "prefix_lens": wl.prefix_lens.tolist() if wl.num_seqs <= 4 else "ragged",
            "suffix_lens": wl.suffix_lens.tolist() if wl.num_seqs <= 4 else "ragged",
            "num_q_heads": wl.num_q_heads, "num_kv_heads": wl.num_kv_heads,
            "head_dim": wl.head_dim, "page_size": wl.page_size, "pool_pages": wl.num_pages,
            "algorithmic_flops": r["flops"],
        },
        "pct_bf16_peak": round(100 * r["tflops_step"] / PEAK_BF16_TFLOPS, 2),
        "ms_per_continuation": round(r["ms_per_step"] / wl.num_seqs, 4),
        "step_gpu_ms": r["step_gpu_ms"],
        "prefill_call_ms": r["prefill_call_dist_ms"],
        "xcd_order": r["xcd_order"],
        "breakdown_ms": {"plan_host": round(r["plan_us"] / 1e3, 4),
                         "append_kv": round(r["append_ms"], 4),
                         "prefill_call": round(r["prefill_call_ms"], 4)},
        "roofline": {"bound": "mfma", "kernel": "prefill_kernel + combine_kernel (one prefill call)",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic(args.config)},
    }
    import oracle
    if not args.no_cpu_baseline:
        # The oracle beside the GPU: every query row of the workload (the
        # single continuation's 16,384 rows take about 2 s a pass on 16
        # cores), and the same rows check the timed GPU output.
        rows = sample_rows(wl, args.cpu_rows)
        line["cpu_baseline"], (o_ref, lse_ref) = cpu_baseline(wl, rows, oracle)
        line["parity"] = parity(wl, db, rows, o_ref, lse_ref, harness)
    del db
    torch.cuda.empty_cache()
    extra = {"main": r}
    if not args.no_extra_configs:
        # The other configurations: the same path timed, plus the oracle on a
        # seeded row sample (its speed, and parity of the timed output there).
        line["configs"] = {}
        for name in ("tiny", "ragged", "long", "cold"):
            if name == args.config:
                continue
            rr = time_config(name, args.extra_steps, -args.extra_warmup_ms, torch, tsa, harness,
                             workload,
                             calibrate=not args.no_xcd_calibration)
            wlx, dbx = rr.pop("wl"), rr.pop("db")
            rec = {"workload": WORKLOADS[name],
                   "ms_per_continuation": round(rr["ms_per_step"] / wlx.num_seqs, 4),
                   "ms_per_step": round(rr["ms_per_step"], 4),
                   "tflops_step": round(rr["tflops_step"], 2),
                   "step_gpu_ms": rr["step_gpu_ms"],
                   "prefill_call_ms": rr["prefill_call_dist_ms"],
                   "prefill_tflops": round(rr["prefill_tflops"], 2),
                   "frac": round(rr["prefill_tflops"] / PEAK_BF16_TFLOPS, 4),
                   "append_gbs": round(rr["append_gbs"], 1),
                   "work_items": rr["num_items"], "steps": args.extra_steps,
                   "warmup": rr["warmup_steps"]}
            if not args.no_cpu_baseline:
                rows = sample_rows(wlx, args.extra_rows, seed=321)
                o_ref, lse_ref, t = oracle_rows(wlx, rows, oracle)
                rec["oracle"] = {"value": round(row_flops(wlx, rows) / t / 1e12, 5),
                                 "unit": "TFLOP/s", "rows": int(len(rows)),
                                 "seconds": round(t, 2), "cores": oracle.num_threads()}
                rec["parity"] = parity(wlx, dbx, rows, o_ref, lse_ref, harness)
            line["configs"][name] = rec
            extra[name] = rr
            del dbx, wlx
            torch.cuda.empty_cache()
    if args.extra_json:
        extra["hbm_sweep"] = hbm_sweep(torch, tsa)
        with open(args.extra_json, "w") as f:
            json.dump(extra, f, indent=1, default=float)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
