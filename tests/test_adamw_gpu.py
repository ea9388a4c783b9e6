"""GPU parity of the fused optimizer step (AdamW with the drift taken from
its update, Section 3.4) against the oracle: optimizer state and weights
bit-exact (both sides round every fp32 operation once, in the same order),
scores within 1e-5, then selection and records as in the plain path."""
import numpy as np
import pytest

from paper_2609_27193_amd import inputs as I
from paper_2609_27193_amd import layercheck as LC
from tests.conftest import gpu_available
from tests.gpu_harness import Pair, log
from tests.test_edges_gpu import odd_spec
from tests.test_parity_gpu import k0_for, reduced_8b, reduced_qwen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not gpu_available():
        pytest.skip("needs an MI355X")
    LC.load_library()


CASES = [("8b-bf16-master", reduced_8b, "bf16"), ("qwen-bf16-nomaster", reduced_qwen, "bf16"),
         ("toy-f32", I.toy_spec, "f32"), ("odd-misaligned", lambda: odd_spec("bf16", True), "bf16"),
         ("odd-f32-grads", lambda: odd_spec("f32", False), "f32")]


@pytest.mark.parametrize("name,maker,gdt", CASES, ids=[c[0] for c in CASES])
def test_fused_adamw_steps(name, maker, gdt):
    spec = maker()
    p = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 0.02))
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        for t in range(1, 7):
            mask, st = p.fused_step(t, adam_t=t, lr=1e-3 if t < 4 else 5e-4, grad_dtype=gdt,
                                    capacity=max(p.R) if t % 2 else None)
            log(f"  {name} t={t}: selected {st['n_selected']}/{p.N}")
    finally:
        p.close()


def test_fused_step_state_rules():
    spec = reduced_8b()
    p = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 0.02))
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        p.fused_step(1, adam_t=1)
        with pytest.raises(LC.LCError) as e:
            LC.lc_score_layers(p.ctx, 2)  # shadow stale after a fused step
        assert e.value.code == LC.LC_ERR_BAD_STATE
        with pytest.raises(LC.LCError) as e:
            LC.lc_adamw_step_score(p.ctx, 1, [1] * len(p.lsegs), LC.LC_DT_BF16, 1e-3, 0.9, 0.95, 1e-8, 0, 1)
        assert e.value.code == LC.LC_ERR_BAD_STATE  # step not increasing
        # a full base checkpoint re-synchronises the shadow: the standalone score works again
        p.rebase(1)
        p.pack(1, np.ones(p.N, np.uint8))
        p.step(2)
        for bad in (dict(beta1=1.0), dict(eps=0.0), dict(lr=-1.0), dict(weight_decay=float("nan")),
                    dict(adam_step=0)):
            args = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0, adam_step=2)
            args.update(bad)
            with pytest.raises(LC.LCError) as e:
                LC.lc_adamw_step_score(p.ctx, 3, [s.weight for s in p.lsegs], LC.LC_DT_BF16, **args)
            assert e.value.code == LC.LC_ERR_INVALID_ARG
        p.check_arrays()
    finally:
        p.close()
    q = Pair(spec, LC.LC_MODE_SNAPSHOT, k0_for(spec, 0.02))
    try:
        with pytest.raises(LC.LCError) as e:
            LC.lc_adamw_step_score(q.ctx, 1, [s.weight for s in q.lsegs], LC.LC_DT_BF16, 1e-3, 0.9, 0.95, 1e-8,
                                   0.0, 1)
        assert e.value.code == LC.LC_ERR_BAD_STATE
    finally:
        q.close()


def test_layout_without_shadow():
    """A context fed only by the fused step needs no shadow copies (16 GB less
    on an 8B-parameter state); it refuses the standalone score, packs and
    restores its records like any other layout."""
    import torch
    spec = reduced_8b()
    p = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 0.02))
    try:
        segs = [LC.Segment(s.layer, s.numel, s.weight, None, s.master, s.exp_avg, s.exp_avg_sq) for s in p.lsegs]
        lay = LC.LayoutDesc(segs, p.N, p.dtype, True, LC.LC_MODE_ACCUM, p.k0, spec.s_max, stream=p.stream)
        ctx = LC.lc_init_layout(lay)
        try:
            with pytest.raises(LC.LCError) as e:
                LC.lc_score_layers(ctx, 1)
            assert e.value.code == LC.LC_ERR_BAD_STATE
            # the base version (every layer, pending since init), then one fused step
            base = torch.empty(sum(p.R), dtype=torch.uint8, device="cuda")
            assert LC.lc_pack_selected(ctx, base.data_ptr(), base.numel(), 0)["done"] == 1
            arrays = (p.dW, p.dM, p.dm, p.dv)
            before = [a.clone() for a in arrays]
            g = torch.randn(spec.numel, device="cuda").to(torch.bfloat16)
            ptrs = [g[s.offset:s.offset + s.numel].data_ptr() for s in p.gen.segments]
            LC.lc_adamw_step_score(ctx, 1, ptrs, LC.LC_DT_BF16, 1e-3, 0.9, 0.95, 1e-8, 0.0, 1)
            u = LC.lc_read_state(ctx, p.N)[0]
            assert (u > 0).all()
            mask, st = LC.lc_select(ctx, 1, 1.0, p.N)
            assert st["n_selected"] == int(mask.sum())
            assert not torch.equal(p.dm, before[2])
            # recovery to the base: every array as it was (there is no shadow to refresh)
            chosen = LC.lc_restore_composite(ctx, [{"step": 0, "mask": np.ones(p.N, np.uint8),
                                                    "payload": base.data_ptr(), "payload_bytes": base.numel()}],
                                             0, p.N)
            torch.cuda.synchronize()
            assert chosen.tolist() == [0] * p.N
            for a, b in zip(arrays, before):
                assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))
            _, d, tl = LC.lc_read_state(ctx, p.N)
            assert not d.any() and tl.tolist() == [0] * p.N
            LC.lc_adamw_step_score(ctx, 1, ptrs, LC.LC_DT_BF16, 1e-3, 0.9, 0.95, 1e-8, 0.0, 1)  # resumes
        finally:
            LC.lc_destroy(ctx)
        with pytest.raises(LC.LCError) as e:
            LC.lc_init_layout(LC.LayoutDesc(segs, p.N, p.dtype, True, LC.LC_MODE_SNAPSHOT, p.k0, spec.s_max,
                                            stream=p.stream))
        assert e.value.code == LC.LC_ERR_INVALID_ARG
    finally:
        p.close()


SGD_CASES = [("8b-master-weights-only", reduced_8b, "bf16", False), ("qwen-nomaster", reduced_qwen, "bf16", True),
             ("toy-f32-grads", I.toy_spec, "f32", False), ("odd-misaligned", lambda: odd_spec("bf16", True), "bf16", True)]


@pytest.mark.parametrize("name,maker,gdt,moments", SGD_CASES, ids=[c[0] for c in SGD_CASES])
def test_fused_sgd_steps(name, maker, gdt, moments):
    """Plain SGD with the drift taken from its update (Section 4.7): the
    parameters and weights bit-exact against the oracle, moments (when the
    layout has them) untouched, then selection and records; the records of
    a layout without moments hold the weights (and master) only."""
    spec = maker()
    p = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 0.02), moments=moments)
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        for t in range(1, 7):
            mask, st = p.fused_sgd_step(t, lr=1e-2 if t < 4 else 5e-3, grad_dtype=gdt,
                                        capacity=max(p.R) if t % 2 else None)
            log(f"  {name} t={t}: selected {st['n_selected']}/{p.N}")
    finally:
        p.close()


def test_fused_sgd_state_rules():
    spec = reduced_8b()
    q = Pair(spec, LC.LC_MODE_SNAPSHOT, k0_for(spec, 0.02))
    try:
        with pytest.raises(LC.LCError) as e:
            LC.lc_sgd_step_score(q.ctx, 1, [s.weight for s in q.lsegs], LC.LC_DT_BF16, 1e-3, 0.0)
        assert e.value.code == LC.LC_ERR_BAD_STATE  # the drift accumulates: ACCUM only
    finally:
        q.close()
    p = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 0.02), moments=False)
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        for bad in (dict(lr=-1.0), dict(lr=float("inf")), dict(weight_decay=-0.1)):
            args = dict(lr=1e-3, weight_decay=0.0)
            args.update(bad)
            with pytest.raises(LC.LCError) as e:
                LC.lc_sgd_step_score(p.ctx, 1, [s.weight for s in p.lsegs], LC.LC_DT_BF16, **args)
            assert e.value.code == LC.LC_ERR_INVALID_ARG
        with pytest.raises(LC.LCError) as e:  # AdamW needs the moments this layout lacks
            LC.lc_adamw_step_score(p.ctx, 1, [s.weight for s in p.lsegs], LC.LC_DT_BF16, 1e-3, 0.9, 0.95, 1e-8, 0.0, 1)
        assert e.value.code == LC.LC_ERR_BAD_STATE
        p.fused_sgd_step(1)  # the failed calls left the context usable
        p.check_arrays()
    finally:
        p.close()
