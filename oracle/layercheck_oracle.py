"""CPU oracle for the LayerCheck decision step -- TEST INFRASTRUCTURE ONLY.

Only the tests, the package's smoke check and the benchmark's CPU-baseline leg
may import this module.  It is a plain, slow, obviously-correct restatement
of the paper's method (Section 3.2, per-layer drift monitoring and selective
persistence; Section 3.3, the bound on mixed-timestamp staleness; Section 3.5,
recovery from the persisted records; Equations 1-5 and 8) on host numpy arrays, in fp64.
It shares no code with the HIP library and imports nothing from it.

What it computes, in the paper's notation:

* Eq. 1: for layer l, u_l(t) = mean|W_l(t) - W_l(t-1)| / (mean|W_l(t-1)| + eps_w),
  the means taken jointly over every element of every tensor of the layer.
  W_l(t-1) is the caller-held shadow copy S of the weights.
* Eq. 2: Delta_l <- Delta_l + u_l(t)   (ACCUM mode, the paper's rule).
  SNAPSHOT mode instead keeps S equal to the last *persisted* weights and sets
  Delta_l <- u_l(t) (distance to the last persisted version).
* Eq. 3 and the LR adaptation: persist l if Delta_l >= K(t), K(t) = K0_l * s(lr(t));
  the caller passes s(lr(t)) as ``lr_scale``.
* Section 3.3 staleness guard: persist l also when t - t_l >= S_max.
* Eq. 4: a persisted layer gets Delta_l <- 0 and t_l <- t.
* Section 3.3 reporting metric: size-weighted staleness sum_l n_l (t - t_l) / sum_l n_l.
* Section 3.4 warm-up: no selective persistence during the warm-up window,
  then a full base checkpoint, after which every layer counts as persisted
  at the base step (``rebase``).
* Section 3.4 / 4.1 / 4.7: the drift taken from the optimizer's own update,
  for AdamW (``adamw_step_score``) and for plain SGD (``sgd_step_score``),
  in fp32 with one rounding per operation (the optimizer's precision).
* Section 3.1 / Eq. 8 recovery: each layer takes its newest persisted record
  with step <= t_fail; the base full checkpoint is simply a version holding
  every layer.

Readings where the paper is silent: eps_w is added to the *mean* exactly as
Eq. 1 is typeset; the
comparison operators are ">=" for both rules; the payload format (records of
selected layers in ascending layer id, each record [W | master | m | v],
every (array, tensor) block zero-padded to a multiple of 256 bytes) is this
implementation's own, since the paper only says a DeepSpeed-compatible
checkpoint is assembled; after recovery Delta_l = 0, t_l = the restored step
and S = W; with eps_w = 0 an all-zero, unchanged layer scores 0/0 = NaN,
which never meets the threshold, so only the staleness guard persists it.

A selection made by ``select`` or ``rebase`` has reset Delta_l and t_l of its
layers (Eq. 4), so it must be packed in full before the next score or
optimizer step (otherwise recovery would silently take older records and the
Section 3.3 bound would fail); the base selected at construction resets
nothing and may stay unpacked in ACCUM mode (a warm-up), while SNAPSHOT mode
needs it packed.

Parity status: every function here is pinned by the ``-m "not gpu"`` tests
(closed forms, exact-rational brute force, invariants, the paper's Table 1
record-size and layer-count figures; ``bf16_round`` against hand-worked bit
patterns and torch's independent conversion; ``resync`` against taking the
same decision directly; the call and layout rules against the interface's
refusals), and the pins are themselves checked to fail on planted mistakes;
no function is "parity unpinned".
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

# Status codes (same numbering as the C interface, so tests can compare).
LC_OK = 0
LC_ERR_INVALID_ARG = 1
LC_ERR_BAD_STATE = 2
LC_ERR_CAPACITY = 3
LC_ERR_NO_VERSION = 4

DT_BF16 = 1
DT_F32 = 2
MODE_ACCUM = 0
MODE_SNAPSHOT = 1

PAD = 256  # block alignment inside a packed record (this implementation's format)


class OracleError(Exception):
    def __init__(self, code: int, msg: str):
        super().__init__(msg)
        self.code = code


@dataclass
class OSegment:
    """One tensor of one layer, as host arrays (bf16 weights are raw uint16)."""
    layer: int
    weight: np.ndarray
    shadow: np.ndarray
    master: Optional[np.ndarray]
    exp_avg: np.ndarray
    exp_avg_sq: np.ndarray

    @property
    def numel(self) -> int:
        return int(self.weight.size)


def widen(values: np.ndarray, dtype: int) -> np.ndarray:
    """Exact fp64 value of each stored weight (bf16 is the top half of an fp32)."""
    if dtype == DT_BF16:
        return (values.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return values.astype(np.float64)


def layer_update_score(weights: Sequence[np.ndarray], previous: Sequence[np.ndarray],
                       dtype: int, eps_w: float):
    """Eq. 1 for one layer.  Returns (sum|W-S|, sum|S|, n, u)."""
    A = 0.0
    B = 0.0
    n = 0
    for w, s in zip(weights, previous):
        x = widen(w, dtype)
        y = widen(s, dtype)
        A += float(np.sum(np.abs(x - y)))
        B += float(np.sum(np.abs(y)))
        n += int(w.size)
    with np.errstate(divide="ignore", invalid="ignore"):
        u = float(np.float64(A / n) / np.float64(B / n + eps_w))
    return A, B, n, u


def padded(nbytes: int) -> int:
    return (nbytes + PAD - 1) // PAD * PAD


def _arrays_in_record(has_master: bool, has_moments: bool = True) -> List[str]:
    """Weights and their optimizer tensors (Section 3.2); without Adam moments
    (the SGD variant of Section 4.7) a record holds the weights only."""
    return (["weight"] + (["master"] if has_master else [])
            + (["exp_avg", "exp_avg_sq"] if has_moments else []))


def record_bytes(seg_numels: Sequence[int], weight_itemsize: int, has_master: bool,
                 has_moments: bool = True) -> int:
    """Size of one layer's packed record: every (array, tensor) block padded."""
    total = 0
    for arr in _arrays_in_record(has_master, has_moments):
        item = weight_itemsize if arr == "weight" else 4
        for n in seg_numels:
            total += padded(n * item)
    return total


def decide(delta, t_last, k0, lr_scale: float, s_max: int, step: int):
    """Eq. 3 with K(t) = K0 * s(lr(t)), and the Section 3.3 staleness guard.
    Returns (selected, selected-by-the-guard-alone) as uint8 arrays."""
    n = len(delta)
    mask = np.zeros(n, dtype=np.uint8)
    forced = np.zeros(n, dtype=np.uint8)
    for l in range(n):
        K = k0[l] * lr_scale
        age = step - t_last[l]
        by_drift = delta[l] >= K
        by_age = age >= s_max
        if by_drift or by_age:
            mask[l] = 1
            forced[l] = 0 if by_drift else 1
    return mask, forced


def plan_versions(versions: Sequence[dict], n_layers: int, t_fail: int) -> List[int]:
    """Section 3.5 step 1: for each layer, the index of the version with the
    greatest step <= t_fail whose mask holds the layer (the base full
    checkpoint is one such version).  Only ``step`` and ``mask`` are read."""
    choice = []
    for l in range(n_layers):
        best, best_step, dup = None, None, False
        for i, v in enumerate(versions):
            if v["step"] <= t_fail and v["mask"][l]:
                if best is None or v["step"] > best_step:
                    best, best_step, dup = i, v["step"], False
                elif v["step"] == best_step:
                    dup = True
        if best is None:
            raise OracleError(LC_ERR_NO_VERSION, f"layer {l}: no persisted version <= {t_fail}")
        if dup:
            raise OracleError(LC_ERR_INVALID_ARG, f"layer {l}: two versions at step {best_step}")
        choice.append(best)
    return choice


# ----------------------------------------------------------------------------
# AdamW with drift taken from the update itself (Section 3.4 computes the
# drift inside the optimizer step).  The paper trains with AdamW
# (Section 4.1) but does not restate it; this follows the published
# definition (Adam with bias correction, decoupled weight decay):
#   m <- b1 m + (1 - b1) g ;  v <- b2 v + (1 - b2) g^2
#   m_hat = m / (1 - b1^t) ;  v_hat = v / (1 - b2^t)
#   p <- p (1 - lr wd) - lr m_hat / (sqrt(v_hat) + eps)
# evaluated in fp32 (the optimizer state's precision) with every operation
# rounded once, in this order; the per-step scalars are formed in fp64 and
# rounded to fp32 once.  Drift is Eq. 1 on the optimizer's parameters:
# u = mean|p_new - p_old| / (mean|p_old| + eps_w).


def adamw_scalars(lr: float, beta1: float, beta2: float, eps: float, weight_decay: float, t: int) -> dict:
    f = np.float32
    return {"b1": f(beta1), "omb1": f(1.0 - beta1), "b2": f(beta2), "omb2": f(1.0 - beta2),
            "c1": f(1.0 / (1.0 - beta1 ** t)), "c2": f(1.0 / (1.0 - beta2 ** t)),
            "eps": f(eps), "lr": f(lr), "decay": f(1.0 - lr * weight_decay)}


def adamw_update(p: np.ndarray, m: np.ndarray, v: np.ndarray, g: np.ndarray, sc: dict, decayed: bool):
    """One AdamW step on fp32 arrays; returns (p_new, m_new, v_new)."""
    f = np.float32
    g = g.astype(f)
    m_new = (sc["b1"] * m).astype(f) + (sc["omb1"] * g).astype(f)
    v_new = (sc["b2"] * v).astype(f) + (sc["omb2"] * (g * g).astype(f)).astype(f)
    m_hat = (m_new * sc["c1"]).astype(f)
    v_hat = (v_new * sc["c2"]).astype(f)
    denom = (np.sqrt(v_hat).astype(f) + sc["eps"]).astype(f)
    upd = (m_hat / denom).astype(f)
    p1 = (p * sc["decay"]).astype(f) if decayed else p.astype(f)
    p_new = (p1 - (sc["lr"] * upd).astype(f)).astype(f)
    return p_new, m_new.astype(f), v_new.astype(f)


# Section 4.7 notes the method applies to plain SGD, persisting the weights
# without per-parameter optimizer state.  One SGD step with decoupled weight
# decay, fp32, one rounding per operation:
#   p_new = p * (1 - lr * wd) - lr * g      (the decay only for decayed groups)


def sgd_scalars(lr: float, weight_decay: float) -> dict:
    f = np.float32
    return {"lr": f(lr), "decay": f(1.0 - lr * weight_decay)}


def sgd_update(p: np.ndarray, g: np.ndarray, sc: dict, decayed: bool) -> np.ndarray:
    """One SGD step on fp32 arrays; returns p_new."""
    f = np.float32
    p1 = (p * sc["decay"]).astype(f) if decayed else p.astype(f)
    return (p1 - (sc["lr"] * g.astype(f)).astype(f)).astype(f)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits, round to nearest even (NaN kept as a quiet NaN)."""
    b = x.astype(np.float32).view(np.uint32).astype(np.uint64)
    r = ((b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        r[nan] = np.uint16(0x7FC0)
    return r


class LayerCheckOracle:
    """Stateful mirror of the decision step on host arrays."""

    def __init__(self, segments: Sequence[OSegment], n_layers: int, weight_dtype: int,
                 has_master: bool, mode: int, k0: Sequence[float], s_max: int,
                 eps_w: float = 1e-8, t_base: int = 0):
        if n_layers <= 0 or len(segments) == 0:
            raise OracleError(LC_ERR_INVALID_ARG, "empty layout")
        if weight_dtype not in (DT_BF16, DT_F32) or mode not in (MODE_ACCUM, MODE_SNAPSHOT):
            raise OracleError(LC_ERR_INVALID_ARG, "bad dtype or mode")
        if len(k0) != n_layers or s_max < 1 or not (eps_w >= 0.0) or eps_w == float("inf"):
            raise OracleError(LC_ERR_INVALID_ARG, "bad thresholds")
        if not all(k >= 0.0 for k in k0):  # refuses NaN too
            raise OracleError(LC_ERR_INVALID_ARG, "K0 must be >= 0")
        self.by_layer: List[List[OSegment]] = [[] for _ in range(n_layers)]
        self.has_moments = segments[0].exp_avg is not None
        last = -1
        for s in segments:
            if (s.exp_avg is None) == self.has_moments or (s.exp_avg_sq is None) == self.has_moments:
                raise OracleError(LC_ERR_INVALID_ARG, "Adam moments must be given for every segment or none")
            if not (0 <= s.layer < n_layers) or s.layer < last or s.numel == 0:
                raise OracleError(LC_ERR_INVALID_ARG, "segments must be grouped by ascending layer")
            if (s.master is None) == has_master:
                raise OracleError(LC_ERR_INVALID_ARG, "master presence mismatch")
            last = s.layer
            self.by_layer[s.layer].append(s)
        if any(len(g) == 0 for g in self.by_layer):
            raise OracleError(LC_ERR_INVALID_ARG, "layer without tensors")
        self.N = n_layers
        self.dtype = weight_dtype
        self.itemsize = 2 if weight_dtype == DT_BF16 else 4
        self.has_master = has_master
        self.mode = mode
        self.k0 = [float(k) for k in k0]
        self.s_max = int(s_max)
        self.eps_w = float(eps_w)
        self.t_base = int(t_base)
        self.n = [sum(s.numel for s in g) for g in self.by_layer]
        self.R = [record_bytes([s.numel for s in g], self.itemsize, has_master, self.has_moments)
                  for g in self.by_layer]
        # Section 3.2: accumulators start at 0; every layer counts as persisted
        # by the base full checkpoint at t_base; the shadow starts equal to W.
        self.delta = [0.0] * n_layers
        self.u = [0.0] * n_layers
        self.t_last = [self.t_base] * n_layers
        for g in self.by_layer:
            for s in g:
                s.shadow[...] = s.weight
        self.last_step = self.t_base
        self.scored_step: Optional[int] = None
        # the base version is pending: every layer selected at t_base
        self.mask = np.ones(n_layers, dtype=np.uint8)
        self.mask_step = self.t_base
        self.unpacked = set(range(n_layers))
        # The base selected at init resets nothing (Delta is 0 and t_l = t_base
        # already), so a warm-up may leave it unpacked in ACCUM mode; a
        # selection made by ``select`` or ``rebase`` has reset its layers.
        self.pending_persists = False

    def _require_packed(self) -> None:
        """Eq. 4 resets Delta_l and t_l of a selected layer as if it were
        already persisted, so the layers of a selection made by ``select`` or
        ``rebase`` must all be packed before the state moves on (otherwise a
        recovery would silently fall back to an older record and the Section
        3.3 bound would not hold).  SNAPSHOT mode also needs the base packed:
        its pack is what refreshes the shadow."""
        if self.unpacked and (self.pending_persists or self.mode == MODE_SNAPSHOT):
            raise OracleError(LC_ERR_BAD_STATE, "previous selection not fully packed")

    # -- Section 3.4: AdamW step with the drift taken from the update --------
    def _optimizer_step(self, step: int, grads, decayed, update) -> None:
        """Section 3.4: the optimizer updates every segment's parameters (the
        fp32 master when present, else the weights widened to fp32); the
        weights are written back (round to nearest even for bf16), and the
        drift of each layer is Eq. 1 on its parameters before and after the
        update, accumulated by Eq. 2.  ``update(segment, p_old, g, decayed)``
        returns p_new and updates any optimizer state of the segment."""
        if step <= self.last_step:
            raise OracleError(LC_ERR_BAD_STATE, "decision steps must strictly increase")
        if self.mode != MODE_ACCUM:
            raise OracleError(LC_ERR_BAD_STATE, "the fused optimizer step accumulates (ACCUM mode)")
        self._require_packed()
        segs = [s for g in self.by_layer for s in g]
        for i, (s, g) in enumerate(zip(segs, grads)):
            if s.master is not None:
                p_old = s.master.copy()
            else:
                p_old = widen(s.weight, self.dtype).astype(np.float32)
            dec = True if decayed is None else bool(decayed[i])
            p_new = update(s, p_old, g, dec)
            if s.master is not None:
                s.master[...] = p_new
            s.weight[...] = bf16_round(p_new) if self.dtype == DT_BF16 else p_new
            s._p_old = p_old
            s._p_new = p_new
        for l, g in enumerate(self.by_layer):
            _, _, _, u = layer_update_score([s._p_new for s in g], [s._p_old for s in g], DT_F32, self.eps_w)
            self.u[l] = u
            self.delta[l] = self.delta[l] + u
            for s in g:
                del s._p_old, s._p_new
        self.last_step = step
        self.scored_step = step
        self.unpacked = set()
        self.mask = None

    def adamw_step_score(self, step: int, grads, lr: float, beta1: float, beta2: float, eps: float,
                         weight_decay: float, adam_t: int, decayed=None) -> None:
        """``grads``: one fp32 array per segment (bf16 gradients widened
        exactly); ``decayed``: per-segment weight-decay flags (the paper's
        with/without weight-decay parameter groups, Section 3.4), all True
        when None."""
        if step > self.last_step and self.mode == MODE_ACCUM and not self.has_moments:
            raise OracleError(LC_ERR_BAD_STATE, "AdamW needs the moment arrays")
        sc = adamw_scalars(lr, beta1, beta2, eps, weight_decay, adam_t)

        def update(s, p_old, g, dec):
            p_new, m_new, v_new = adamw_update(p_old, s.exp_avg, s.exp_avg_sq, g, sc, dec)
            s.exp_avg[...] = m_new
            s.exp_avg_sq[...] = v_new
            return p_new

        self._optimizer_step(step, grads, decayed, update)

    # -- Section 4.7: SGD step with the drift taken from the update ----------
    def sgd_step_score(self, step: int, grads, lr: float, weight_decay: float, decayed=None) -> None:
        """As ``adamw_step_score`` for plain SGD; Adam moments, if the layout
        has them, are left as they are."""
        sc = sgd_scalars(lr, weight_decay)
        self._optimizer_step(step, grads, decayed, lambda s, p_old, g, dec: sgd_update(p_old, g, sc, dec))

    # -- Eq. 1-2 -------------------------------------------------------------
    def score(self, step: int) -> None:
        if step <= self.last_step:
            raise OracleError(LC_ERR_BAD_STATE, "decision steps must strictly increase")
        self._require_packed()
        for l, g in enumerate(self.by_layer):
            _, _, _, u = layer_update_score([s.weight for s in g], [s.shadow for s in g],
                                            self.dtype, self.eps_w)
            self.u[l] = u
            if self.mode == MODE_ACCUM:
                self.delta[l] = self.delta[l] + u
            else:
                self.delta[l] = u
        if self.mode == MODE_ACCUM:
            # the next step's W(t-1) is this step's W(t)
            for g in self.by_layer:
                for s in g:
                    s.shadow[...] = s.weight
        self.last_step = step
        self.scored_step = step
        self.unpacked = set()
        self.mask = None

    # -- Eq. 3-5 -------------------------------------------------------------
    def select(self, step: int, lr_scale: float):
        if self.scored_step is None or self.scored_step != step:
            raise OracleError(LC_ERR_BAD_STATE, "select must follow score at the same step")
        if not (lr_scale > 0.0) or lr_scale == float("inf"):
            raise OracleError(LC_ERR_INVALID_ARG, "lr_scale must be positive and finite")
        self._pre_delta = list(self.delta)
        self._pre_t_last = list(self.t_last)
        mask, forced = decide(self.delta, self.t_last, self.k0, lr_scale, self.s_max, step)
        n_forced = int(forced.sum())
        for l in range(self.N):
            if mask[l]:  # Eq. 4: reset on persist
                self.delta[l] = 0.0
                self.t_last[l] = step
        self.scored_step = None
        self.mask = mask
        self.mask_step = step
        self.unpacked = {l for l in range(self.N) if mask[l]}
        self.pending_persists = True
        return mask.copy(), self.stats(step, mask, n_forced)

    # -- Section 3.4 warm-up and base checkpoint ------------------------------
    def rebase(self, step: int) -> None:
        """A full base checkpoint at ``step``: the end of the warm-up window
        during which selective persistence is off, or any later full
        checkpoint.  Every layer counts as persisted at ``step`` (Delta_l = 0,
        t_l = step, S = W) and every layer is selected for packing; any
        selection still pending is replaced.  ``step`` may equal the last
        optimizer or score step (the rebase follows that step's update)."""
        if step < self.last_step:
            raise OracleError(LC_ERR_BAD_STATE, "a base checkpoint cannot precede the last step")
        for l, g in enumerate(self.by_layer):
            self.delta[l] = 0.0
            self.t_last[l] = step
            for s in g:
                if s.shadow is not None:
                    s.shadow[...] = s.weight
        self.last_step = step
        self.scored_step = None
        self.mask = np.ones(self.N, dtype=np.uint8)
        self.mask_step = step
        self.unpacked = set(range(self.N))
        self.pending_persists = True

    def stats(self, step: int, mask: np.ndarray, n_forced: int) -> dict:
        ages = [step - self.t_last[l] for l in range(self.N)]
        num = sum(self.n[l] * ages[l] for l in range(self.N))
        den = sum(self.n)
        return {
            "n_selected": int(mask.sum()),
            "n_forced": n_forced,
            "payload_bytes": sum(self.R[l] for l in range(self.N) if mask[l]),
            "max_age": max(ages),
            "weighted_age": float(num) / float(den),
        }

    def resync(self, layer: int, selected: bool) -> None:
        """Parity-protocol helper: adopt another implementation's decision for
        a layer whose accumulator lies within the tolerance band of K."""
        if self.mask is None:
            raise OracleError(LC_ERR_BAD_STATE, "no selection to resync")
        if selected and not self.mask[layer]:
            self.mask[layer] = 1
            self.delta[layer] = 0.0
            self.t_last[layer] = self.mask_step
            self.unpacked.add(layer)
        elif not selected and self.mask[layer]:
            self.mask[layer] = 0
            self.delta[layer] = self._pre_delta[layer]
            self.t_last[layer] = self._pre_t_last[layer]
            self.unpacked.discard(layer)

    # -- Section 3.2: a persisted layer's record holds all of its state ---------
    def layer_record(self, l: int) -> bytes:
        out = bytearray()
        g = self.by_layer[l]
        for arr in _arrays_in_record(self.has_master, self.has_moments):
            for s in g:
                raw = getattr(s, arr).tobytes()
                out += raw
                out += bytes(padded(len(raw)) - len(raw))
        assert len(out) == self.R[l]
        return bytes(out)

    def pack(self, first_rank: int, capacity: int):
        if self.mask is None:
            raise OracleError(LC_ERR_BAD_STATE, "nothing selected")
        sel = [l for l in range(self.N) if self.mask[l]]
        if first_rank < 0 or first_rank > len(sel):
            raise OracleError(LC_ERR_INVALID_ARG, "first_rank out of range")
        last, total = first_rank, 0
        while last < len(sel) and total + self.R[sel[last]] <= capacity:
            total += self.R[sel[last]]
            last += 1
        if last == first_rank and first_rank < len(sel):
            raise OracleError(LC_ERR_CAPACITY, "record does not fit")
        payload = b"".join(self.layer_record(l) for l in sel[first_rank:last])
        if self.mode == MODE_SNAPSHOT:
            for l in sel[first_rank:last]:
                for s in self.by_layer[l]:
                    s.shadow[...] = s.weight
        for l in sel[first_rank:last]:
            self.unpacked.discard(l)
        return np.frombuffer(payload, dtype=np.uint8).copy(), {
            "bytes_written": total, "n_packed": last - first_rank,
            "next_rank": last, "done": int(last == len(sel))}

    # -- Section 3.5 / Eq. 8 -------------------------------------------------
    def plan(self, versions: Sequence[dict], t_fail: int) -> List[int]:
        """Index of the version each layer is restored from."""
        for v in versions:
            m = np.asarray(v["mask"])
            if m.shape != (self.N,):
                raise OracleError(LC_ERR_INVALID_ARG, "mask length")
            need = sum(self.R[l] for l in range(self.N) if m[l])
            if len(v["payload"]) != need:
                raise OracleError(LC_ERR_INVALID_ARG, "payload size does not match mask")
        return plan_versions(versions, self.N, t_fail)

    def restore(self, versions: Sequence[dict], t_fail: int) -> np.ndarray:
        choice = self.plan(versions, t_fail)
        chosen = np.zeros(self.N, dtype=np.int64)
        for l in range(self.N):
            v = versions[choice[l]]
            off = sum(self.R[j] for j in range(l) if v["mask"][j])
            rec = bytes(np.asarray(v["payload"], dtype=np.uint8)[off:off + self.R[l]])
            pos = 0
            for arr in _arrays_in_record(self.has_master, self.has_moments):
                for s in self.by_layer[l]:
                    dst = getattr(s, arr)
                    nb = dst.nbytes
                    dst[...] = np.frombuffer(rec[pos:pos + nb], dtype=dst.dtype)
                    pos += padded(nb)
            for s in self.by_layer[l]:
                s.shadow[...] = s.weight
            self.delta[l] = 0.0
            self.t_last[l] = int(v["step"])
            chosen[l] = int(v["step"])
        self.last_step = t_fail
        self.scored_step = None
        self.mask = None
        self.unpacked = set()
        return chosen
