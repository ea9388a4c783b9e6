"""Seeded synthetic model states for the layer-wise checkpoint decision path.

This module only *produces inputs*: layer-grouped parameter shapes, initial
weights, fp32 master copies, Adam moments, and a stand-in for one optimizer
step.  It computes none of the checkpointing method itself (no update score,
no threshold, no packing, no recovery), so both the HIP path and the CPU
oracle may draw their inputs from it without sharing any of the method's
arithmetic.

Layer grouping follows the paper's Section 2.2: the trainable parameters of a
decoder are split at module granularity into ``embed_tokens``, one group per
transformer block, the final normalisation and ``lm_head`` (N = B + 3, or
B + 2 when ``lm_head`` is tied to the embedding).

Value recipe (the paper trains real models; these synthetic states stand in
for them, with the same shapes):

* matrices, biases and embeddings start from N(0, 0.02) in fp32; RMSNorm
  weights start at 1.0 (the toy model draws every tensor from N(0, 0.02));
* bf16 weights are the round-to-nearest-even image of the fp32 master copy;
* one synthetic optimizer step adds ``s_l * 1e-3 * N(0, 1)`` to every element
  of layer ``l`` (to the master copy when there is one, otherwise directly to
  the weights), with a per-layer scale ``s_l`` drawn per workload;
* Adam moments are redrawn every step: m ~ N(0, 1e-3), v = |N(0, 1e-6)|
  (second argument read as the standard deviation).

Random numbers come from ``torch.Generator`` seeded with a 64-bit mix of
(workload seed, layer, tensor, array, step); values are reproducible on one
device type (CPU and GPU generators produce different streams, which is fine:
every consumer copies the arrays it needs).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

# ----------------------------------------------------------------------------
# Shapes
# ----------------------------------------------------------------------------


@dataclass(frozen=True)
class TensorSpec:
    name: str
    numel: int
    kind: str  # "matrix" | "embed" | "norm" | "bias" | "shard"


@dataclass(frozen=True)
class LayerSpec:
    name: str
    tensors: Tuple[TensorSpec, ...]

    @property
    def numel(self) -> int:
        return sum(t.numel for t in self.tensors)


@dataclass(frozen=True)
class ModelSpec:
    name: str
    layers: Tuple[LayerSpec, ...]
    weight_dtype: str            # "bf16" or "f32"
    has_master: bool             # fp32 master copy present
    scale_rule: str              # name of the per-layer update-scale distribution
    target_fraction: float       # fraction of layers the threshold should select
    s_max: int                   # staleness bound S_max
    seed: int = 0
    norm_init_one: bool = True   # RMSNorm weights start at 1.0
    description: str = ""

    @property
    def n_layers(self) -> int:
        return len(self.layers)

    @property
    def numel(self) -> int:
        return sum(l.numel for l in self.layers)

    @property
    def weight_bytes(self) -> int:
        return 2 if self.weight_dtype == "bf16" else 4

    def embed_layers(self) -> List[int]:
        return [i for i, l in enumerate(self.layers) if l.name == "embed_tokens"]


def layer_group_count(n_blocks: int, tied_lm_head: bool) -> int:
    """Number of layer groups of a decoder with ``n_blocks`` transformer blocks
    (Section 2.2): embed_tokens, the blocks, the final norm and lm_head; a tied
    lm_head is the embedding itself and adds no group."""
    return n_blocks + (2 if tied_lm_head else 3)


def _decoder_layers(hidden: int, ffn: int, n_blocks: int, vocab: int,
                    n_q_heads: int, n_kv_heads: int, qkv_bias: bool = False,
                    tied: bool = False, gated_mlp: bool = True) -> Tuple[LayerSpec, ...]:
    head_dim = hidden // n_q_heads
    kv = n_kv_heads * head_dim
    blk = [TensorSpec("q_proj", hidden * hidden, "matrix")]
    if qkv_bias:
        blk.append(TensorSpec("q_bias", hidden, "bias"))
    blk.append(TensorSpec("k_proj", hidden * kv, "matrix"))
    if qkv_bias:
        blk.append(TensorSpec("k_bias", kv, "bias"))
    blk.append(TensorSpec("v_proj", hidden * kv, "matrix"))
    if qkv_bias:
        blk.append(TensorSpec("v_bias", kv, "bias"))
    blk.append(TensorSpec("o_proj", hidden * hidden, "matrix"))
    if gated_mlp:
        blk.append(TensorSpec("gate_proj", hidden * ffn, "matrix"))
    blk.append(TensorSpec("up_proj", hidden * ffn, "matrix"))
    blk.append(TensorSpec("down_proj", ffn * hidden, "matrix"))
    blk.append(TensorSpec("input_layernorm", hidden, "norm"))
    blk.append(TensorSpec("post_attention_layernorm", hidden, "norm"))
    layers = [LayerSpec("embed_tokens", (TensorSpec("embed_tokens", vocab * hidden, "embed"),))]
    for i in range(n_blocks):
        layers.append(LayerSpec(f"block_{i}", tuple(blk)))
    layers.append(LayerSpec("norm", (TensorSpec("norm", hidden, "norm"),)))
    if not tied:
        layers.append(LayerSpec("lm_head", (TensorSpec("lm_head", vocab * hidden, "embed"),)))
    return tuple(layers)


def _zero3_shard(layers: Sequence[LayerSpec], world: int, rank: int) -> Tuple[LayerSpec, ...]:
    """Each layer's tensors flattened in order and cut into ``world`` equal
    contiguous pieces; only piece ``rank`` is held (one segment per layer)."""
    out = []
    for l in layers:
        total = l.numel
        if total % world:
            raise ValueError(f"layer {l.name}: {total} not divisible by {world}")
        out.append(LayerSpec(l.name, (TensorSpec(f"{l.name}.shard{rank}", total // world, "shard"),)))
    return tuple(out)


def _shard_kinds(full: LayerSpec, world: int, rank: int) -> List[Tuple[int, int, str]]:
    """(start, length, kind) runs of the flattened layer inside shard ``rank``."""
    per = full.numel // world
    lo, hi = rank * per, (rank + 1) * per
    runs, pos = [], 0
    for t in full.tensors:
        a, b = max(lo, pos), min(hi, pos + t.numel)
        if a < b:
            runs.append((a - lo, b - a, t.kind))
        pos += t.numel
    return runs


def toy_spec() -> ModelSpec:
    """4 blocks, hidden 256, two-matrix MLP with FFN 1024, vocab 1024, untied
    head, fp32 weights and Adam m/v (no separate master): 3,672,320 params."""
    hidden, ffn, vocab = 256, 1024, 1024
    return ModelSpec(
        name="toy-decoder-4L-h256", weight_dtype="f32", has_master=False,
        layers=_decoder_layers(hidden, ffn, 4, vocab, 4, 4, gated_mlp=False),
        scale_rule="loguniform_0.01_1", target_fraction=0.25, s_max=4,
        norm_init_one=False,
        description="toy decoder, fp32 weights + Adam m/v, 10 steps, S_max=4")


def llama3_8b_spec() -> ModelSpec:
    return ModelSpec(
        name="llama-3-8b", weight_dtype="bf16", has_master=True,
        layers=_decoder_layers(4096, 14336, 32, 128256, 32, 8),
        scale_rule="loguniform_2dec_embed0.1", target_fraction=0.20, s_max=8,
        description="Llama-3-8B-shaped state, bf16 W + fp32 master/m/v + bf16 shadow, S_max=8")


def llama2_13b_spec() -> ModelSpec:
    return ModelSpec(
        name="llama-2-13b", weight_dtype="bf16", has_master=True,
        layers=_decoder_layers(5120, 13824, 40, 32000, 40, 40),
        scale_rule="ramp_0.1_1", target_fraction=0.15, s_max=8,
        description="Llama-2-13B-shaped state, late blocks 10x early, S_max=8")


def qwen25_14b_spec() -> ModelSpec:
    return ModelSpec(
        name="qwen2.5-14b", weight_dtype="bf16", has_master=False,
        layers=_decoder_layers(5120, 13824, 48, 152064, 40, 8, qkv_bias=True),
        scale_rule="bimodal_0.3", target_fraction=0.30, s_max=6,
        description="Qwen2.5-14B-shaped state, bf16 W + fp32 m/v (no master), S_max=6")


def llama3_70b_shard_spec(world: int = 8, rank: int = 0) -> ModelSpec:
    full = _decoder_layers(8192, 28672, 80, 128256, 64, 8)
    return ModelSpec(
        name=f"llama-3-70b-zero3-shard{rank}of{world}", weight_dtype="bf16", has_master=True,
        layers=_zero3_shard(full, world, rank),
        scale_rule="pareto_1.5", target_fraction=0.10, s_max=10,
        description="one 1/8 ZeRO-3 shard of a Llama-3-70B-shaped state, S_max=10")


def llama32_1b_spec() -> ModelSpec:
    """Llama-3.2-1B shape (tied lm_head: N = 18, as in the paper's Table 1),
    used for the persistence-store measurement, whose whole record set
    (17.3 GB) fits a local disk."""
    return ModelSpec(
        name="llama-3.2-1b", weight_dtype="bf16", has_master=True,
        layers=_decoder_layers(2048, 8192, 16, 128256, 32, 8, tied=True),
        scale_rule="loguniform_2dec_embed0.1", target_fraction=0.20, s_max=8,
        description="Llama-3.2-1B-shaped state (tied embeddings), bf16 W + fp32 master/m/v")


def _full_70b_layers():
    return _decoder_layers(8192, 28672, 80, 128256, 64, 8)


def scaled_spec(base: ModelSpec, hidden: int, ffn: int, n_blocks: int, vocab: int,
                n_q: int, n_kv: int, qkv_bias: bool = False) -> ModelSpec:
    """Same dtypes and update-scale rule as ``base`` at a reduced width, for
    parity runs that span many chunks but finish quickly on the CPU."""
    return ModelSpec(
        name=f"{base.name}-reduced-h{hidden}", weight_dtype=base.weight_dtype,
        has_master=base.has_master,
        layers=_decoder_layers(hidden, ffn, n_blocks, vocab, n_q, n_kv, qkv_bias=qkv_bias),
        scale_rule=base.scale_rule, target_fraction=base.target_fraction,
        s_max=base.s_max, seed=base.seed, description=f"reduced {base.description}")


WORKLOADS = {
    "toy": toy_spec,
    "llama3-8b": llama3_8b_spec,
    "llama2-13b": llama2_13b_spec,
    "qwen2.5-14b": qwen25_14b_spec,
    "llama3-70b-shard0": llama3_70b_shard_spec,
    "llama3.2-1b": llama32_1b_spec,
}

# ----------------------------------------------------------------------------
# Seeds and per-layer update scales
# ----------------------------------------------------------------------------

ARRAY_IDS = {"init": 1, "update": 2, "exp_avg": 3, "exp_avg_sq": 4, "scale": 5, "misc": 6, "grad": 7,
             "direction": 8}
_M64 = (1 << 64) - 1


def _splitmix64(x: int) -> int:
    x = (x + 0x9E3779B97F4A7C15) & _M64
    x = ((x ^ (x >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    x = ((x ^ (x >> 27)) * 0x94D049BB133111EB) & _M64
    return x ^ (x >> 31)


def seed_of(workload_seed: int, layer: int, tensor: int, array: str, step: int) -> int:
    h = _splitmix64(workload_seed)
    for v in (layer, tensor, ARRAY_IDS[array], step):
        h = _splitmix64(h ^ (v & _M64))
    return h & ((1 << 63) - 1)


def update_scales(spec: ModelSpec) -> np.ndarray:
    """Per-layer synthetic update scale s_l (float64[N])."""
    rng = np.random.Generator(np.random.Philox(seed_of(spec.seed, 0, 0, "scale", 0)))
    n = spec.n_layers
    names = [l.name for l in spec.layers]
    rule = spec.scale_rule
    if rule == "loguniform_0.01_1":
        s = np.exp(rng.uniform(math.log(0.01), math.log(1.0), n))
    elif rule == "loguniform_2dec_embed0.1":
        s = 10.0 ** rng.uniform(-2.0, 0.0, n)
        for i, nm in enumerate(names):
            if nm in ("embed_tokens", "lm_head"):
                s[i] *= 0.1
    elif rule == "ramp_0.1_1":
        blocks = [i for i, nm in enumerate(names) if nm.startswith("block_")]
        s = np.zeros(n)
        nb = len(blocks)
        for j, i in enumerate(blocks):
            s[i] = 0.1 * (10.0 ** (j / max(nb - 1, 1)))
        first, last = s[blocks[0]], s[blocks[-1]]
        for i, nm in enumerate(names):
            if nm == "embed_tokens":
                s[i] = first
            elif nm in ("norm", "lm_head"):
                s[i] = last
    elif rule == "bimodal_0.3":
        k = int(round(0.3 * n))
        fast = rng.permutation(n)[:k]
        s = np.full(n, 0.02)
        s[fast] = 1.0
    elif rule == "pareto_1.5":
        u = rng.uniform(0.0, 1.0, n)
        s = 0.01 * (1.0 - u) ** (-1.0 / 1.5)
    elif rule == "constant_1":
        s = np.ones(n)
    else:
        raise ValueError(f"unknown scale rule {rule}")
    return s.astype(np.float64)


# ----------------------------------------------------------------------------
# The state itself (torch tensors, flat per array, layer-grouped)
# ----------------------------------------------------------------------------


@dataclass
class SegmentView:
    layer: int
    tensor: int
    offset: int  # element offset inside the flat arrays
    numel: int
    kind: str


def segment_table(spec: ModelSpec) -> List[SegmentView]:
    segs, off = [], 0
    for li, l in enumerate(spec.layers):
        for ti, t in enumerate(l.tensors):
            segs.append(SegmentView(li, ti, off, t.numel, t.kind))
            off += t.numel
    return segs


class SyntheticState:
    """Flat, layer-grouped arrays of one workload on one device.

    Arrays: ``weight`` (bf16 or fp32), ``shadow`` (same dtype, left
    uninitialised: the checkpoint library fills it), ``master`` (fp32, or
    None), ``exp_avg`` and ``exp_avg_sq`` (fp32).  ``segments`` lists one
    entry per parameter tensor in layer order.
    """

    def __init__(self, spec: ModelSpec, device="cpu", init: bool = True, shadow: bool = True):
        import torch
        self.torch = torch
        self.spec = spec
        self.device = torch.device(device)
        self.segments = segment_table(spec)
        self.scales = update_scales(spec)
        P = spec.numel
        wdt = torch.bfloat16 if spec.weight_dtype == "bf16" else torch.float32
        self.weight = torch.empty(P, dtype=wdt, device=self.device)
        self.shadow = torch.empty(P, dtype=wdt, device=self.device) if shadow else None
        self.master = torch.empty(P, dtype=torch.float32, device=self.device) if spec.has_master else None
        self.exp_avg = torch.empty(P, dtype=torch.float32, device=self.device)
        self.exp_avg_sq = torch.empty(P, dtype=torch.float32, device=self.device)
        self.step_index = 0
        self._full_70b = None
        if spec.name.startswith("llama-3-70b-zero3"):
            self._full_70b = _full_70b_layers()
        if init:
            self.initialise()

    # -- helpers ---------------------------------------------------------
    def _gen(self, seed: int):
        g = self.torch.Generator(device=self.device)
        g.manual_seed(seed)
        return g

    def _randn(self, n: int, seed: int):
        return self.torch.randn(n, generator=self._gen(seed), device=self.device, dtype=self.torch.float32)

    def layer_range(self, li: int) -> Tuple[int, int]:
        segs = [s for s in self.segments if s.layer == li]
        return segs[0].offset, segs[-1].offset + segs[-1].numel

    def _kind_runs(self, seg: SegmentView) -> List[Tuple[int, int, str]]:
        if seg.kind == "shard" and self._full_70b is not None:
            name = self.spec.layers[seg.layer].name
            full = [l for l in self._full_70b if l.name == name][0]
            return _shard_kinds(full, 8, 0)
        return [(0, seg.numel, seg.kind)]

    # -- initial state -----------------------------------------------------
    def initialise(self):
        torch = self.torch
        for seg in self.segments:
            base = self._randn(seg.numel, seed_of(self.spec.seed, seg.layer, seg.tensor, "init", 0)) * 0.02
            if self.spec.norm_init_one:
                for a, n, kind in self._kind_runs(seg):
                    if kind == "norm":
                        base[a:a + n] = 1.0
            sl = slice(seg.offset, seg.offset + seg.numel)
            if self.master is not None:
                self.master[sl] = base
            self.weight[sl] = base.to(self.weight.dtype)
            del base
        self._redraw_moments(0)
        self.step_index = 0

    def _redraw_moments(self, step: int):
        for li in range(self.spec.n_layers):
            a, b = self.layer_range(li)
            n = b - a
            self.exp_avg[a:b] = self._randn(n, seed_of(self.spec.seed, li, 0, "exp_avg", step)) * 1e-3
            self.exp_avg_sq[a:b] = self._randn(n, seed_of(self.spec.seed, li, 0, "exp_avg_sq", step)).abs_() * 1e-6

    # -- one synthetic optimizer step ------------------------------------
    def step(self, t: Optional[int] = None):
        """Advance every layer by one synthetic update (the stand-in for an
        AdamW step) and redraw the Adam moments."""
        t = self.step_index + 1 if t is None else t
        for li in range(self.spec.n_layers):
            a, b = self.layer_range(li)
            n = b - a
            delta = self._randn(n, seed_of(self.spec.seed, li, 0, "update", t))
            delta.mul_(float(self.scales[li]) * 1e-3)
            if self.master is not None:
                self.master[a:b].add_(delta)
                self.weight[a:b] = self.master[a:b].to(self.weight.dtype)
            elif self.weight.dtype == self.torch.float32:
                self.weight[a:b].add_(delta)
            else:
                self.weight[a:b] = (self.weight[a:b].float() + delta).to(self.weight.dtype)
            del delta
        self._redraw_moments(t)
        self.step_index = t

    # -- synthetic gradients for an optimizer-driven run ------------------
    def gradients(self, t: int, dtype=None):
        """Flat gradient tensor for step ``t``: per element N(0, 1) noise plus
        4 * s_l times a fixed per-element direction of layer l, so layers with
        a larger update scale see more consistent gradients and an Adam-type
        optimizer moves them further.  Returned in ``dtype`` (bf16 default)."""
        torch = self.torch
        dtype = torch.bfloat16 if dtype is None else dtype
        g = torch.empty(self.spec.numel, dtype=dtype, device=self.device)
        for li in range(self.spec.n_layers):
            a, b = self.layer_range(li)
            x = self._randn(b - a, seed_of(self.spec.seed, li, 0, "grad", t))
            d = self._randn(b - a, seed_of(self.spec.seed, li, 0, "direction", 0))
            x.add_(d, alpha=4.0 * float(self.scales[li]))
            g[a:b] = x.to(dtype)
            del x, d
        return g

    def decay_mask(self):
        """Weight decay applies to matrices and embeddings, not to norms and
        biases (the paper's with/without weight-decay parameter groups)."""
        return [0 if s.kind in ("norm", "bias") else 1 for s in self.segments]

    # -- views -------------------------------------------------------------
    def seg_views(self, seg: SegmentView):
        sl = slice(seg.offset, seg.offset + seg.numel)
        return (self.weight[sl], None if self.shadow is None else self.shadow[sl],
                None if self.master is None else self.master[sl],
                self.exp_avg[sl], self.exp_avg_sq[sl])

    def nbytes(self) -> int:
        tot = 0
        for t in (self.weight, self.shadow, self.master, self.exp_avg, self.exp_avg_sq):
            if t is not None:
                tot += t.numel() * t.element_size()
        return tot


def to_numpy_weight(t) -> np.ndarray:
    """Host copy of a weight-like tensor: bf16 as raw uint16 bits, fp32 as float32."""
    import torch
    t = t.detach()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16).copy()
    return t.cpu().numpy().copy()
