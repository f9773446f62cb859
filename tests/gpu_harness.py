"""GPU-side test and bench harness: places the generator's inputs in device
memory and drives the library chunk by chunk.  Holds no attention
arithmetic (that lives in the HIP library and, separately, in the oracle)."""
from __future__ import annotations

from typing import Dict, Optional, Tuple

import numpy as np
import torch

import paper_2607_17181_amd as tsa
from workload import BF16_NAN, Workload


def dev_bits(a: np.ndarray) -> torch.Tensor:
    """uint16 bit array -> int16 device tensor with the same bits."""
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def bits_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


class DeviceBatch:
    """One workload resident on the GPU (pools with the prefix already placed)."""

    def __init__(self, wl: Workload, fill: int = int(BF16_NAN), host_pools=None):
        self.wl = wl
        kp, vp = host_pools if host_pools is not None else wl.pool_bits(fill=fill)
        self.k_pool = dev_bits(kp)
        self.v_pool = dev_bits(vp)
        self.q = dev_bits(wl.q)
        self.k_new = dev_bits(wl.k_new)
        self.v_new = dev_bits(wl.v_new)
        self.bt = torch.from_numpy(wl.block_tables).cuda()
        self.geom = tsa.make_geom(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.page_size,
                                  wl.num_pages)
        self.out = torch.zeros_like(self.q)
        self.lse = torch.zeros(wl.q.shape[:2], dtype=torch.float32, device="cuda")
        self._chunk_cache: Dict[int, Tuple] = {}

    def chunk_tensors(self, c: int):
        """Contiguous per-chunk q/k_new/v_new/out/lse views (copies for multi-seq chunks)."""
        if c not in self._chunk_cache:
            _, _, tok = self.wl.chunks[c]
            idx = torch.from_numpy(tok).cuda()
            if len(self.wl.chunks) == 1:
                self._chunk_cache[c] = (self.q, self.k_new, self.v_new, self.out, self.lse, None)
            else:
                self._chunk_cache[c] = (self.q[idx].contiguous(), self.k_new[idx].contiguous(),
                                        self.v_new[idx].contiguous(),
                                        torch.zeros_like(self.q[idx]),
                                        torch.zeros(len(tok), self.q.shape[1], dtype=torch.float32,
                                                    device="cuda"), idx)
        return self._chunk_cache[c]

    def plans(self, kv_splits: int = 0):
        out = []
        for pre, suf, _ in self.wl.chunks:
            out.append(tsa.plan(self.geom, pre, suf, self.wl.max_pages_per_seq, kv_splits))
        return out

    def run(self, kv_splits: int = 0, plans=None, workspaces=None, with_lse: bool = True,
            sm_scale: float = 0.0):
        """append + prefill for every chunk in order; outputs land in self.out / self.lse."""
        plans = plans or self.plans(kv_splits)
        for c, sp in enumerate(plans):
            q, kn, vn, out, lse, idx = self.chunk_tensors(c)
            ws = workspaces[c] if workspaces is not None else tsa.workspace_tensor(sp)
            tsa.append_kv(sp, kn, vn, self.k_pool, self.v_pool, self.bt)
            tsa.prefill(sp, q, self.k_pool, self.v_pool, self.bt, out,
                        lse if with_lse else None, ws, sm_scale=sm_scale)
            if idx is not None:
                self.out[idx] = out
                if with_lse:
                    self.lse[idx] = lse
        return self.out, self.lse


def error_stats(gpu_bits: np.ndarray, ref: np.ndarray) -> Dict[str, float]:
    """max-abs, mean-abs and relative L2 of bf16 GPU output vs fp64 reference."""
    g = bits_to_f64(gpu_bits).reshape(ref.shape)
    diff = np.abs(g - ref)
    return {
        "max_abs": float(diff.max()) if diff.size else 0.0,
        "mean_abs": float(diff.mean()) if diff.size else 0.0,
        "rel_l2": float(np.linalg.norm(g - ref) / max(np.linalg.norm(ref), 1e-300)),
        "finite": bool(np.isfinite(g).all()),
    }


# Parity bar: the absolute bounds are the build target's; the relative-L2
# bound adds a check that an all-zero output cannot pass (|o| shrinks like
# 1/sqrt(keys)).  bf16 output rounding alone gives ~1e-3 relative RMS, P in
# bf16 a few 1e-4 more; 1e-2 leaves a 5x margin.
MAX_ABS = 2e-2
MEAN_ABS = 2e-3
REL_L2 = 1e-2
LSE_ABS = 2e-3


def assert_parity(stats: Dict[str, float], what: str = "") -> None:
    assert stats["finite"], f"{what}: non-finite output"
    assert stats["max_abs"] <= MAX_ABS, f"{what}: max-abs {stats['max_abs']:.3e}"
    assert stats["mean_abs"] <= MEAN_ABS, f"{what}: mean-abs {stats['mean_abs']:.3e}"
    assert stats["rel_l2"] <= REL_L2, f"{what}: rel-L2 {stats['rel_l2']:.3e}"
