"""CPU oracle for D2D-staged weight switching -- TEST INFRASTRUCTURE ONLY.

Only the tests may import this module; the product path never does.  Plain
numpy, written from the paper's description (Section 4.4): weights are
pre-staged in fixed-size chunks inside the KV region; a chunk becomes dirty
when the KV allocator hands out pages overlapping its staging range; at the
switch, clean staged chunks are copied from the staging copy and dirty or
missing chunks are reloaded from the host copy.

chunks: int64 [n, 3] rows (stage_offset, weight_offset, bytes).
used_pages: bool [num_pages]; page p covers bytes [p*page_bytes, (p+1)*page_bytes).
"""
from __future__ import annotations

import numpy as np


def mark_dirty(chunks: np.ndarray, used_pages: np.ndarray, page_bytes: int) -> np.ndarray:
    """bool [n]: chunk i overlaps a used page."""
    out = np.zeros(len(chunks), dtype=bool)
    for i, (so, _, nb) in enumerate(np.asarray(chunks, dtype=np.int64)):
        if nb <= 0 or so < 0:
            continue
        first, last = so // page_bytes, (so + nb - 1) // page_bytes
        last = min(last, len(used_pages) - 1)
        out[i] = bool(used_pages[first:last + 1].any()) if first <= last else False
    return out


def gather(chunks: np.ndarray, staged: np.ndarray, dirty: np.ndarray, staging: np.ndarray,
           host_weights: np.ndarray, weights: np.ndarray) -> np.ndarray:
    """The weight region after the switch (returns a new array)."""
    out = weights.copy()
    for i, (so, wo, nb) in enumerate(np.asarray(chunks, dtype=np.int64)):
        if nb <= 0 or (nb | wo) % 16 or wo < 0 or wo + nb > len(weights):
            continue
        stage_ok = so % 16 == 0 and so >= 0 and so + nb <= len(staging)
        if staged[i] and not dirty[i] and stage_ok:
            out[wo:wo + nb] = staging[so:so + nb]
        else:
            out[wo:wo + nb] = host_weights[wo:wo + nb]
    return out


def bits_to_words(bits: np.ndarray) -> np.ndarray:
    """bool [n] -> uint32 words, bit i in word i // 32 at position i % 32."""
    n = len(bits)
    words = np.zeros((n + 31) // 32, dtype=np.uint32)
    for i in np.nonzero(bits)[0]:
        words[i // 32] |= np.uint32(1) << np.uint32(i % 32)
    return words
