"""Side-by-side runner: the HIP library (through the C interface) and the CPU
oracle on the same seeded inputs, compared with the parity protocol.

Protocol (scores to 1e-5 relative; everything else exact):
* u_l and Delta_l within 1e-5 relative; a zero on one side is an exact zero
  on the other;
* masks bit-exact except layers with |Delta_gpu - K| <= 1e-5 K, which are
  reported and excluded; when the two sides decide differently on such a
  layer the oracle adopts the GPU's decision (resync);
* the oracle's decision rule fed the GPU's own accumulators reproduces the
  GPU mask with no exclusions;
* packed payloads, shadows, restored arrays and last-persist steps: memcmp.
"""
from __future__ import annotations

import sys

import numpy as np

from oracle import layercheck_oracle as O
from paper_2609_27193_amd import layercheck as LC
from paper_2609_27193_amd.inputs import SyntheticState, to_numpy_weight

REL = 1e-5


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel_ok(g, o):
    """Within REL relative; a zero, an infinity or a NaN (Eq. 1 with eps_w = 0
    on an all-zero layer is 0/0) must appear on both sides."""
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    if np.any(np.isnan(g) != np.isnan(o)):
        return False
    zero = (o == 0) | (g == 0)
    if np.any(zero & (g != o)):
        return False
    both_inf = np.isinf(o) & np.isinf(g) & (np.sign(o) == np.sign(g))
    nz = ~zero & ~both_inf & ~np.isnan(o)
    return bool(np.all(np.abs(g[nz] - o[nz]) <= REL * np.abs(o[nz])))


def torch_bytes(t):
    import torch
    return t.detach().contiguous().view(torch.uint8).cpu().numpy()


class Pair:
    """Owns one synthetic state, its device copy for the library, its host
    copy for the oracle, and both implementations."""

    def __init__(self, spec, mode, k0, eps_w=1e-8, t_base=0, moments=True):
        import torch
        self.torch = torch
        self.spec = spec
        self.mode = mode
        self.N = spec.n_layers
        self.k0 = list(k0)
        self.dtype = LC.LC_DT_BF16 if spec.weight_dtype == "bf16" else LC.LC_DT_F32
        self.gen = SyntheticState(spec, device="cpu")
        dev = torch.device("cuda")
        g = self.gen
        self.dW = g.weight.to(dev)
        self.dS = torch.zeros_like(self.dW)
        self.dM = None if g.master is None else g.master.to(dev)
        self.dm = g.exp_avg.to(dev)
        self.dv = g.exp_avg_sq.to(dev)
        self.hW = to_numpy_weight(g.weight)
        self.hS = np.zeros_like(self.hW)
        self.hM = None if g.master is None else g.master.numpy().copy()
        self.hm = g.exp_avg.numpy().copy()
        self.hv = g.exp_avg_sq.numpy().copy()
        osegs, lsegs = [], []
        for s in g.segments:
            a, b = s.offset, s.offset + s.numel
            osegs.append(O.OSegment(s.layer, self.hW[a:b], self.hS[a:b],
                                    None if self.hM is None else self.hM[a:b],
                                    self.hm[a:b] if moments else None, self.hv[a:b] if moments else None))
            lsegs.append(LC.Segment(s.layer, s.numel, self.dW[a:b].data_ptr(), self.dS[a:b].data_ptr(),
                                    None if self.dM is None else self.dM[a:b].data_ptr(),
                                    self.dm[a:b].data_ptr() if moments else None,
                                    self.dv[a:b].data_ptr() if moments else None))
        self.lsegs = lsegs
        self.orc = O.LayerCheckOracle(osegs, self.N, self.dtype, spec.has_master, mode, self.k0,
                                      spec.s_max, eps_w=eps_w, t_base=t_base)
        self.stream = torch.cuda.current_stream().cuda_stream
        self.layout = LC.LayoutDesc(lsegs, self.N, self.dtype, spec.has_master, mode, self.k0,
                                    spec.s_max, eps_w=eps_w, t_base=t_base, stream=self.stream)
        self.ctx = LC.lc_init_layout(self.layout)
        self.R = [LC.lc_record_bytes(self.ctx, l) for l in range(self.N)]
        assert self.R == self.orc.R
        self.near_excluded = 0
        self.resyncs = 0
        self.max_pack_calls = 0  # most lc_pack_selected calls one pack needed
        self.versions_dev = []  # (step, mask, device tensor)
        self.versions_host = []  # (step, mask, numpy payload from the oracle)

    def close(self):
        if self.ctx is not None:
            LC.lc_destroy(self.ctx)
            self.ctx = None

    # -- inputs -------------------------------------------------------------
    def advance(self, t):
        g = self.gen
        g.step(t)
        self.dW.copy_(g.weight)
        if self.dM is not None:
            self.dM.copy_(g.master)
            self.hM[...] = g.master.numpy()
        self.dm.copy_(g.exp_avg)
        self.dv.copy_(g.exp_avg_sq)
        self.hW[...] = to_numpy_weight(g.weight)
        self.hm[...] = g.exp_avg.numpy()
        self.hv[...] = g.exp_avg_sq.numpy()
        self.torch.cuda.synchronize()

    # -- one decision step on both sides -------------------------------------
    def score(self, t):
        LC.lc_score_layers(self.ctx, t)
        self.orc.score(t)
        u, d, tl = LC.lc_read_state(self.ctx, self.N)
        assert rel_ok(u, self.orc.u), (t, u, self.orc.u)
        assert rel_ok(d, self.orc.delta), (t, d, self.orc.delta)
        assert list(tl) == list(self.orc.t_last)
        return d, tl

    def select(self, t, lr_scale=1.0, gpu_delta=None, gpu_t_last=None):
        mask_g, st_g = LC.lc_select(self.ctx, t, lr_scale, self.N)
        if gpu_delta is not None:
            m_fed, f_fed = O.decide(list(gpu_delta), list(gpu_t_last), self.k0, lr_scale, self.spec.s_max, t)
            assert np.array_equal(m_fed, mask_g), (t, m_fed, mask_g)
            assert int(f_fed.sum()) == st_g["n_forced"]
        mask_o, st_o = self.orc.select(t, lr_scale)
        resynced = False
        for l in range(self.N):
            if mask_g[l] == mask_o[l]:
                continue
            K = self.k0[l] * lr_scale
            dl = gpu_delta[l] if gpu_delta is not None else self.orc._pre_delta[l]
            assert abs(dl - K) <= REL * K, f"step {t} layer {l}: mask differs outside the tolerance band"
            self.orc.resync(l, bool(mask_g[l]))
            self.resyncs += 1
            resynced = True
        if gpu_delta is not None:
            for l in range(self.N):
                if abs(gpu_delta[l] - self.k0[l] * lr_scale) <= REL * self.k0[l] * lr_scale:
                    self.near_excluded += 1
        mask_o = self.orc.mask.copy()
        assert np.array_equal(mask_g, mask_o)
        if not resynced:
            for k in ("n_selected", "n_forced", "payload_bytes", "max_age"):
                assert st_g[k] == st_o[k], (k, st_g[k], st_o[k])
            assert abs(st_g["weighted_age"] - st_o["weighted_age"]) <= 1e-12 * max(1.0, st_o["weighted_age"])
        assert st_g["payload_bytes"] == sum(self.R[l] for l in range(self.N) if mask_g[l])
        _, _, tl = LC.lc_read_state(self.ctx, self.N)
        assert list(tl) == list(self.orc.t_last)
        return mask_g, st_g

    def pack(self, t, mask, capacity=None, keep_versions=True):
        total = int(sum(self.R[l] for l in range(self.N) if mask[l]))
        staging = self.torch.empty(max(total, 1), dtype=self.torch.uint8, device="cuda")
        cap = total if capacity is None else capacity
        parts_g, parts_o = [], []
        rank, calls = 0, 0
        while True:
            res = LC.lc_pack_selected(self.ctx, staging.data_ptr(), cap, rank)
            calls += 1
            pay_o, res_o = self.orc.pack(rank, cap)
            assert res == res_o, (res, res_o)
            self.torch.cuda.synchronize()
            got = torch_bytes(staging[:res["bytes_written"]]) if res["bytes_written"] else np.zeros(0, np.uint8)
            assert np.array_equal(got, pay_o), f"step {t}: payload differs at rank {rank}"
            # SNAPSHOT refreshes the shadow of the layers each call writes, and only
            # those: compare after every call, not only after the last
            self.check_shadow()
            parts_g.append(got)
            parts_o.append(pay_o)
            if res["done"]:
                break
            rank = res["next_rank"]
        self.max_pack_calls = max(self.max_pack_calls, calls)
        payload = np.concatenate(parts_o) if parts_o else np.zeros(0, np.uint8)
        assert len(payload) == total
        if keep_versions:
            dev = self.torch.from_numpy(np.concatenate(parts_g)).to("cuda") if total else None
            self.versions_dev.append((t, mask.copy(), dev))
            self.versions_host.append((t, mask.copy(), payload))
        return payload

    def check_shadow(self):
        self.torch.cuda.synchronize()
        assert np.array_equal(torch_bytes(self.dS), self.hS.view(np.uint8)), "shadow differs"

    def check_arrays(self):
        self.torch.cuda.synchronize()
        assert np.array_equal(torch_bytes(self.dW), self.hW.view(np.uint8))
        assert np.array_equal(torch_bytes(self.dS), self.hS.view(np.uint8))
        if self.dM is not None:
            assert np.array_equal(torch_bytes(self.dM), self.hM.view(np.uint8))
        assert np.array_equal(torch_bytes(self.dm), self.hm.view(np.uint8))
        assert np.array_equal(torch_bytes(self.dv), self.hv.view(np.uint8))

    def adopt_restored(self):
        """Continue the synthetic trajectory from the restored live state."""
        import torch
        g = self.gen
        if g.weight.dtype == torch.bfloat16:
            g.weight.copy_(torch.from_numpy(self.hW.view(np.int16)).view(torch.bfloat16))
        else:
            g.weight.copy_(torch.from_numpy(self.hW))
        if g.master is not None:
            g.master.copy_(torch.from_numpy(self.hM))

    def rebase(self, t):
        """A full base checkpoint at t on both sides (every layer selected)."""
        LC.lc_rebase(self.ctx, t)
        self.orc.rebase(t)
        u, d, tl = LC.lc_read_state(self.ctx, self.N)
        assert not d.any() and tl.tolist() == [t] * self.N == list(self.orc.t_last)
        self.check_arrays()
        return np.ones(self.N, np.uint8)

    def fused_step(self, t, adam_t, lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, wd=0.01, grad_dtype="bf16",
                   lr_scale=1.0, capacity=None, decide=True):
        """One AdamW step with the drift taken from the update, on both sides,
        then (with ``decide``) select and pack."""
        torch = self.torch
        gdt = torch.bfloat16 if grad_dtype == "bf16" else torch.float32
        g = self.gen.gradients(t, gdt)
        dg = g.to("cuda")
        gf = g.float().numpy()  # exact widening of bf16 gradients
        decay = self.gen.decay_mask()
        ptrs = [dg[s.offset:s.offset + s.numel].data_ptr() for s in self.gen.segments]
        LC.lc_adamw_step_score(self.ctx, t, ptrs, LC.LC_DT_BF16 if grad_dtype == "bf16" else LC.LC_DT_F32,
                               lr, beta1, beta2, eps, wd, adam_t, decay)
        self.orc.adamw_step_score(t, [gf[s.offset:s.offset + s.numel] for s in self.gen.segments],
                                  lr, beta1, beta2, eps, wd, adam_t, decay)
        u, d, tl = LC.lc_read_state(self.ctx, self.N)
        assert rel_ok(u, self.orc.u), (t, u, self.orc.u)
        assert rel_ok(d, self.orc.delta), (t, d, self.orc.delta)
        self.check_arrays()  # optimizer state and weights bit-exact
        if not decide:
            return None, None
        mask, st = self.select(t, lr_scale, d, tl)
        self.pack(t, mask, capacity)
        return mask, st

    def fused_sgd_step(self, t, lr=1e-3, wd=0.01, grad_dtype="bf16", lr_scale=1.0, capacity=None, decide=True):
        """One SGD step with the drift taken from the update, on both sides,
        then (with ``decide``) select and pack."""
        torch = self.torch
        gdt = torch.bfloat16 if grad_dtype == "bf16" else torch.float32
        g = self.gen.gradients(t, gdt)
        dg = g.to("cuda")
        gf = g.float().numpy()
        decay = self.gen.decay_mask()
        ptrs = [dg[s.offset:s.offset + s.numel].data_ptr() for s in self.gen.segments]
        LC.lc_sgd_step_score(self.ctx, t, ptrs, LC.LC_DT_BF16 if grad_dtype == "bf16" else LC.LC_DT_F32,
                             lr, wd, decay)
        self.orc.sgd_step_score(t, [gf[s.offset:s.offset + s.numel] for s in self.gen.segments], lr, wd, decay)
        u, d, tl = LC.lc_read_state(self.ctx, self.N)
        assert rel_ok(u, self.orc.u), (t, u, self.orc.u)
        assert rel_ok(d, self.orc.delta), (t, d, self.orc.delta)
        self.check_arrays()  # master and weights bit-exact, moments untouched
        if not decide:
            return None, None
        mask, st = self.select(t, lr_scale, d, tl)
        self.pack(t, mask, capacity)
        return mask, st

    def step(self, t, lr_scale=1.0, capacity=None):
        self.advance(t)
        d, tl = self.score(t)
        mask, st = self.select(t, lr_scale, d, tl)
        self.pack(t, mask, capacity)
        return mask, st
