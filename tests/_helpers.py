"""Small seeded host layouts for oracle and parity tests (inputs only)."""
from __future__ import annotations

import numpy as np

from oracle.layercheck_oracle import DT_BF16, DT_F32, OSegment


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16, returned as raw uint16 bits (finite inputs)."""
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    r = (b + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


class HostLayout:
    """A tiny layout: per layer a list of tensor sizes, host arrays per tensor."""

    def __init__(self, sizes, dtype=DT_BF16, has_master=True, seed=0, scale=0.02):
        self.sizes = [list(s) for s in sizes]
        self.dtype = dtype
        self.has_master = has_master
        self.rng = np.random.default_rng(seed)
        self.segs = []
        for l, layer in enumerate(self.sizes):
            for n in layer:
                base = (self.rng.standard_normal(n) * scale).astype(np.float32)
                if dtype == DT_BF16:
                    w = f32_to_bf16_bits(base)
                    sh = np.zeros(n, dtype=np.uint16)
                else:
                    w = base.copy()
                    sh = np.zeros(n, dtype=np.float32)
                master = base.copy() if has_master else None
                m = (self.rng.standard_normal(n) * 1e-3).astype(np.float32)
                v = np.abs(self.rng.standard_normal(n) * 1e-6).astype(np.float32)
                self.segs.append(OSegment(l, w, sh, master, m, v))

    @property
    def n_layers(self):
        return len(self.sizes)

    def step(self, scales, zero_layers=()):
        """Synthetic optimizer step: per-layer scaled Gaussian update."""
        for s in self.segs:
            if s.layer in zero_layers:
                continue
            d = (self.rng.standard_normal(s.numel) * scales[s.layer] * 1e-3).astype(np.float32)
            if self.has_master:
                s.master += d
                w = s.master
            else:
                w = (bf16_bits_to_f32(s.weight) if self.dtype == DT_BF16 else s.weight) + d
            if self.dtype == DT_BF16:
                s.weight[...] = f32_to_bf16_bits(w)
            else:
                s.weight[...] = w
            s.exp_avg[...] = (self.rng.standard_normal(s.numel) * 1e-3).astype(np.float32)
            s.exp_avg_sq[...] = np.abs(self.rng.standard_normal(s.numel) * 1e-6).astype(np.float32)

    def snapshot(self):
        return [(s.weight.copy(), s.shadow.copy(),
                 None if s.master is None else s.master.copy(),
                 s.exp_avg.copy(), s.exp_avg_sq.copy()) for s in self.segs]
