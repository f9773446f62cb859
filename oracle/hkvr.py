"""CPU oracle for HKVR page transfer -- TEST INFRASTRUCTURE ONLY.

Only the tests and the bench's CPU-baseline leg may import this module; the
product path never does.  Plain numpy, written from the paper's description
and independent of the HIP library.

What it computes (Section 4.3: the registry restores the agreed prefix into
newly allocated device pages through layer-first/page-first transfer
kernels; Appendix C: the layer-first view groups pages by layer, the
page-first view groups the per-layer fragments of one logical page under
that page):

  device cache, layer-first:  K[l][page] is a [Hkv][page_size][d] block,
                              V[l][page] is a [Hkv][d][page_size] block
  host slab, page-first:      slab[p][l][0] = K[l][page_ids[p]] (flattened)
                              slab[p][l][1] = V[l][page_ids[p]] (flattened)

restore() writes the slab's blocks into the device pages named by page_ids;
checkpoint() reads them back out.  A page id outside [0, num_pages) moves
nothing (the slab block, or the device page, keeps what it held).
"""
from __future__ import annotations

from typing import Tuple

import numpy as np


def restore(slab: np.ndarray, page_ids, k_cache: np.ndarray,
            v_cache: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Page-first host slab -> layer-first device cache (returns new arrays)."""
    k = k_cache.copy()
    v = v_cache.copy()
    num_layers, num_pages = k.shape[0], k.shape[1]
    for p, page in enumerate(np.asarray(page_ids)):
        if not 0 <= page < num_pages:
            continue
        for layer in range(num_layers):
            k[layer, page] = slab[p, layer, 0].reshape(k.shape[2:])
            v[layer, page] = slab[p, layer, 1].reshape(v.shape[2:])
    return k, v


def checkpoint(k_cache: np.ndarray, v_cache: np.ndarray, page_ids,
               slab: np.ndarray) -> np.ndarray:
    """Layer-first device cache -> page-first host slab (returns a new slab)."""
    out = slab.copy()
    num_layers, num_pages = k_cache.shape[0], k_cache.shape[1]
    for p, page in enumerate(np.asarray(page_ids)):
        if not 0 <= page < num_pages:
            continue
        for layer in range(num_layers):
            out[p, layer, 0] = k_cache[layer, page].reshape(-1)
            out[p, layer, 1] = v_cache[layer, page].reshape(-1)
    return out
