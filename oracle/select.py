"""CPU oracle for SP batch selection -- TEST INFRASTRUCTURE ONLY.

Only the tests may import this module; the product path never does.
Written from Section 3.4's admission rule: each SP opportunity takes a
bounded set of waiting continuations, sized so that their predicted cost
(attention, page restore, device pages) stays within what the slot has left
once decode is served; anything else waits for a later opportunity.  Reading
taken: candidates in queue order, each admitted when the batch with it still
fits (first fit).
Host-resident prefixes are restored page aligned (Appendix B), the partial
last page joining the recomputed tail.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Tuple


@dataclass
class Model:
    num_layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    attn_flops_per_s: float
    per_token_s: float
    restore_bytes_per_s: float
    batch_overhead_s: float


def candidate(P: int, S: int, host: bool, m: Model) -> Tuple[float, int, int, int]:
    """(seconds, pages, plan prefix, plan suffix) of one continuation."""
    ps = m.page_size
    if host:
        P2 = (P // ps) * ps
        S, P = S + (P - P2), P2
    attn_flops = 4.0 * m.head_dim * m.num_q_heads * m.num_layers * (S * P + S * (S + 1) / 2.0)
    seconds = attn_flops / m.attn_flops_per_s + S * m.per_token_s
    pages_all = -(-(P + S) // ps)
    if host:
        kv_page_bytes = 2.0 * m.num_kv_heads * ps * m.head_dim * 2.0 * m.num_layers
        seconds += (P // ps) * kv_page_bytes / m.restore_bytes_per_s
        pages = pages_all
    else:
        pages = pages_all - (-(-P // ps))
    return seconds, pages, P, S


def select(cands: List[Tuple[int, int, int]], m: Model, time_budget: float, free_pages: int,
           max_batch: int):
    """(indices, plan prefixes, plan suffixes, seconds, pages) of the batch."""
    idx, pre, suf = [], [], []
    t, pages = 0.0, 0
    for i, (P, S, host) in enumerate(cands):
        if len(idx) >= max_batch:
            break
        if P < 0 or S <= 0:
            continue
        sec, pg, P2, S2 = candidate(P, S, bool(host), m)
        t_new = t + sec + (m.batch_overhead_s if not idx else 0.0)
        if t_new <= time_budget and pages + pg <= free_pages:
            t, pages = t_new, pages + pg
            idx.append(i)
            pre.append(P2)
            suf.append(S2)
    return idx, pre, suf, t, pages
