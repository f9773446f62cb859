"""Seeded synthetic workloads for session-prefill (SP) attention.

Every array here is a pure function of (config, seed).  Draw order inside one
workload is fixed and documented so that any consumer can regenerate it:

1. sequence lengths (only the ragged config draws them: prefix lengths first,
   then suffix lengths);
2. one permutation of all physical page ids of the pool;
3. Q ``[T, Hq, d]``, then K_new ``[T, Hkv, d]``, then V_new ``[T, Hkv, d]``
   (T = total suffix tokens), then the prefix K and the prefix V
   ``[sum P_b, Hkv, d]``, each as float32 N(0, 1) rounded to bf16
   (round to nearest, ties to even) and stored as uint16 bit patterns.

Page assignment: pages are taken in permutation order, first the pages that
hold every sequence's prefix (sequence by sequence), then the extra pages that
the suffixes need, so a sequence's pages are scattered over the whole pool
and its suffix pages are not adjacent to its prefix pages.  Unused
block-table entries hold -1.

Nothing in this module computes attention or appends to a pool.  The prefix
is the cache state a continuation finds on the device, so it is input: it
comes as rows plus their flat slot indices, and ``Workload.pool_bits`` lays
those rows into fresh host pools (every other slot a sentinel) for the
harnesses that want the resident state ready-made.  Appending the suffix, the
method's own step, is left to each consumer.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

BF16_NAN = np.uint16(0x7FC0)

# Prompt-length statistics of the paper's agent trace (Section 2.1, "Continuation
# inputs"): median 25K tokens, p95 105K.  The ragged config draws prefix
# lengths from a lognormal with that median and p95, capped at 128K tokens.
TRACE_MEDIAN_TOKENS = 25_000
TRACE_P95_TOKENS = 105_000
RAGGED_PREFIX_CAP = 131_072
# Phi^{-1}(0.95), the standard normal 95th percentile.
_Z95 = 1.6448536269514722


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return uint16 bits.

    NaN inputs map to the canonical quiet NaN 0x7FC0.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    rounded = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    out = rounded.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = BF16_NAN
    return out


def f32_from_bf16_bits(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 exactly."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def lognormal_prefix_lengths(rng: np.random.Generator, n: int,
                             median: int = TRACE_MEDIAN_TOKENS,
                             p95: int = TRACE_P95_TOKENS,
                             cap: int = RAGGED_PREFIX_CAP) -> np.ndarray:
    """Integer prefix lengths from a lognormal with the given median and p95."""
    mu = math.log(median)
    sigma = math.log(p95 / median) / _Z95
    draw = np.exp(rng.normal(mu, sigma, size=n))
    return np.minimum(np.rint(draw), cap).astype(np.int32)


@dataclasses.dataclass
class Workload:
    """One synthetic SP batch for one attention layer.

    Bit arrays are uint16 bf16 patterns.  ``prefix_slots`` are flat slot
    indices ``page * page_size + (t mod page_size)`` for every prefix token
    (sequence-major), aligned with the rows of ``prefix_k``/``prefix_v``.
    ``chunks`` lists, per chunked-prefill step, the (prefix_lens, suffix_lens)
    pair and the token range of that step inside ``q``/``k_new``/``v_new``.
    """

    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    num_pages: int
    prefix_lens: np.ndarray
    suffix_lens: np.ndarray
    block_tables: np.ndarray
    q: np.ndarray
    k_new: np.ndarray
    v_new: np.ndarray
    prefix_k: np.ndarray
    prefix_v: np.ndarray
    prefix_slots: np.ndarray
    chunks: List[Tuple[np.ndarray, np.ndarray, np.ndarray]]

    @property
    def num_seqs(self) -> int:
        return int(self.prefix_lens.shape[0])

    @property
    def total_tokens(self) -> int:
        return int(self.suffix_lens.sum())

    @property
    def max_pages_per_seq(self) -> int:
        return int(self.block_tables.shape[1])

    def visible_pairs(self) -> int:
        """Number of causally visible (query row, key) pairs per query head."""
        total = 0
        for pre_lens, suf_lens, _ in self.chunks:
            for p, s in zip(pre_lens.tolist(), suf_lens.tolist()):
                total += s * p + s * (s + 1) // 2
        return total

    def flops(self) -> int:
        """Algorithmic FLOPs: 4 * d * Hq * visible pairs (QK^T plus PV)."""
        return 4 * self.head_dim * self.num_q_heads * self.visible_pairs()

    def pool_bits(self, fill: int = int(BF16_NAN)) -> Tuple[np.ndarray, np.ndarray]:
        """Host K and V pools with the prefix placed; every other slot holds ``fill``.

        K pool ``[num_pages, Hkv, page_size, d]``; V pool
        ``[num_pages, Hkv, d, page_size]`` (token index innermost).
        """
        P, H, ps, d = self.num_pages, self.num_kv_heads, self.page_size, self.head_dim
        kp = np.full((P, H, ps, d), fill, dtype=np.uint16)
        vp = np.full((P, H, d, ps), fill, dtype=np.uint16)
        page = self.prefix_slots // ps
        slot = self.prefix_slots % ps
        kp[page, :, slot, :] = self.prefix_k
        vp[page, :, :, slot] = self.prefix_v
        return kp, vp


def _draw_bits(rng: np.random.Generator, shape: Sequence[int], std: float) -> np.ndarray:
    x = rng.standard_normal(size=tuple(shape), dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return bf16_bits_from_f32(x)


def workload_from_lengths(name: str, seed: int, *, num_q_heads: int, num_kv_heads: int,
                          head_dim: int, page_size: int, num_pages: int,
                          prefix_lens: Sequence[int], suffix_lens: Sequence[int],
                          num_chunks: int = 1, q_std: float = 1.0, kv_std: float = 1.0,
                          rng: Optional[np.random.Generator] = None,
                          extra_pages_per_seq: int = 0) -> Workload:
    """Build a workload from explicit lengths.

    ``num_chunks > 1`` splits every suffix into that many equal chunked-prefill
    steps (the suffix length must divide evenly); step c then has prefix
    ``P_b + c * S_b / num_chunks``.  ``extra_pages_per_seq`` widens the
    block-table stride beyond what the lengths need (unused entries are -1).
    """
    if rng is None:
        rng = np.random.default_rng(seed)
    pre = np.asarray(prefix_lens, dtype=np.int32)
    suf = np.asarray(suffix_lens, dtype=np.int32)
    if pre.shape != suf.shape or pre.ndim != 1:
        raise ValueError("prefix_lens and suffix_lens must be 1-D and equal length")
    if (pre < 0).any() or (suf < 0).any():
        raise ValueError("lengths must be non-negative")
    ps = int(page_size)
    n_pre_pages = (pre.astype(np.int64) + ps - 1) // ps
    n_all_pages = (pre.astype(np.int64) + suf + ps - 1) // ps
    need = int(n_all_pages.sum())
    if need > num_pages:
        raise ValueError(f"pool of {num_pages} pages cannot hold {need} pages")
    perm = rng.permutation(num_pages).astype(np.int32)
    max_pages = int(max(1, n_all_pages.max(initial=0))) + int(extra_pages_per_seq)
    bt = np.full((pre.shape[0], max_pages), -1, dtype=np.int32)
    cursor = 0
    for b in range(pre.shape[0]):
        n = int(n_pre_pages[b])
        bt[b, :n] = perm[cursor:cursor + n]
        cursor += n
    for b in range(pre.shape[0]):
        lo, hi = int(n_pre_pages[b]), int(n_all_pages[b])
        bt[b, lo:hi] = perm[cursor:cursor + hi - lo]
        cursor += hi - lo

    T = int(suf.sum())
    total_pre = int(pre.sum())
    q = _draw_bits(rng, (T, num_q_heads, head_dim), q_std)
    k_new = _draw_bits(rng, (T, num_kv_heads, head_dim), kv_std)
    v_new = _draw_bits(rng, (T, num_kv_heads, head_dim), kv_std)
    prefix_k = _draw_bits(rng, (total_pre, num_kv_heads, head_dim), kv_std)
    prefix_v = _draw_bits(rng, (total_pre, num_kv_heads, head_dim), kv_std)

    slots = np.empty(total_pre, dtype=np.int64)
    off = 0
    for b in range(pre.shape[0]):
        t = np.arange(int(pre[b]), dtype=np.int64)
        pages = bt[b, t // ps].astype(np.int64)
        slots[off:off + t.shape[0]] = pages * ps + (t % ps)
        off += t.shape[0]

    chunks = []
    if num_chunks <= 1:
        chunks.append((pre.copy(), suf.copy(), np.arange(T, dtype=np.int64)))
    else:
        if (suf % num_chunks).any():
            raise ValueError("suffix lengths must divide evenly into chunks")
        step = suf // num_chunks
        offs = np.concatenate([[0], np.cumsum(suf.astype(np.int64))])
        for c in range(num_chunks):
            rows = np.concatenate([np.arange(offs[b] + c * step[b], offs[b] + (c + 1) * step[b])
                                   for b in range(pre.shape[0])]).astype(np.int64)
            chunks.append((pre + c * step, step.copy(), rows))

    return Workload(name=name, seed=seed, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                    head_dim=head_dim, page_size=ps, num_pages=num_pages,
                    prefix_lens=pre, suffix_lens=suf, block_tables=bt, q=q, k_new=k_new,
                    v_new=v_new, prefix_k=prefix_k, prefix_v=prefix_v, prefix_slots=slots,
                    chunks=chunks)


# The five synthetic configurations.  Geometry Hq=8, Hkv=1, d=128 is one
# tensor-parallel rank's head share of a 235B-class GQA model at TP=8 (the
# paper's main testbed is a TP=8 server, Section 5); page size 16 tokens.
CONFIGS: Dict[str, Dict] = {
    # 1 sequence, P=256, S=64, 64-page pool.
    "tiny": dict(seed=0, num_q_heads=2, num_kv_heads=1, head_dim=64, page_size=16,
                 num_pages=64, prefix_lens=[256], suffix_lens=[64]),
    # One continuation with a median-length (25K) prefix and a 2K suffix.
    "single": dict(seed=1, num_q_heads=8, num_kv_heads=1, head_dim=128, page_size=16,
                   num_pages=100_000, prefix_lens=[25_000], suffix_lens=[2_048]),
    # 16 continuations, lognormal prefixes (median 25K, p95 105K, cap 128K),
    # suffixes uniform in [512, 4096].
    "ragged": dict(seed=2, num_q_heads=8, num_kv_heads=1, head_dim=128, page_size=16,
                   num_pages=300_000, ragged=16),
    # A p95-length (105K) prefix, 8192 new tokens as 4 chunks of 2048.
    "long": dict(seed=3, num_q_heads=8, num_kv_heads=1, head_dim=128, page_size=16,
                 num_pages=100_000, prefix_lens=[105_000], suffix_lens=[8_192], num_chunks=4),
    # Cold recompute: 4 sequences with no cached prefix, 25,000 new tokens each.
    "cold": dict(seed=4, num_q_heads=8, num_kv_heads=1, head_dim=128, page_size=16,
                 num_pages=100_000, prefix_lens=[0, 0, 0, 0],
                 suffix_lens=[25_000, 25_000, 25_000, 25_000]),
}


def make_workload(name: str, seed: Optional[int] = None, **overrides) -> Workload:
    """Generate one of the named configs (optionally with another seed)."""
    cfg = dict(CONFIGS[name])
    cfg.update(overrides)
    s = cfg.pop("seed") if seed is None else seed
    cfg.pop("seed", None)
    rng = np.random.default_rng(s)
    ragged = cfg.pop("ragged", None)
    if ragged:
        cfg["prefix_lens"] = lognormal_prefix_lengths(rng, ragged)
        cfg["suffix_lens"] = rng.integers(512, 4096, size=ragged, endpoint=True).astype(np.int32)
    return workload_from_lengths(name, s, rng=rng, **cfg)
