"""CPU: the seeded synthetic inputs follow their stated recipe (shapes, update
scales, value distributions, determinism).  The inputs module serves both the
library's tests and the oracle; it holds no arithmetic of the method."""
import numpy as np
import pytest

from paper_2609_27193_amd import inputs as I


@pytest.mark.parametrize("name,n_layers,params", [
    ("toy", 7, 3_672_320),
    ("llama3-8b", 35, 8_030_261_248),
    ("llama2-13b", 43, 13_015_864_320),
    ("qwen2.5-14b", 51, 14_770_033_664),
    ("llama3-70b-shard0", 83, 8_819_213_312),
    ("llama3.2-1b", 18, 1_235_814_400),
])
def test_workload_shapes(name, n_layers, params):
    spec = I.WORKLOADS[name]()
    assert spec.n_layers == n_layers
    assert spec.numel == params


def test_update_scale_rules():
    s = I.update_scales(I.llama3_8b_spec())
    names = [l.name for l in I.llama3_8b_spec().layers]
    for nm, v in zip(names, s):
        lo, hi = (0.001, 0.1) if nm in ("embed_tokens", "lm_head") else (0.01, 1.0)
        assert lo <= v <= hi, (nm, v)
    spec = I.llama2_13b_spec()
    s = I.update_scales(spec)
    blocks = [v for l, v in zip(spec.layers, s) if l.name.startswith("block_")]
    assert np.all(np.diff(blocks) > 0) and blocks[0] == pytest.approx(0.1) and blocks[-1] == pytest.approx(1.0)
    spec = I.qwen25_14b_spec()
    s = I.update_scales(spec)
    assert int(np.sum(s == 1.0)) == round(0.3 * spec.n_layers) and np.all((s == 1.0) | (s == 0.02))
    assert np.all(I.update_scales(I.llama3_70b_shard_spec()) >= 0.01)


def test_toy_state_is_seeded_and_follows_its_distributions():
    import torch
    a = I.SyntheticState(I.toy_spec(), device="cpu")
    b = I.SyntheticState(I.toy_spec(), device="cpu")
    assert torch.equal(a.weight, b.weight) and torch.equal(a.exp_avg, b.exp_avg)
    w = a.weight.double()
    assert abs(w.std().item() - 0.02) < 0.001 and abs(w.mean().item()) < 0.001
    assert abs(a.exp_avg.double().std().item() - 1e-3) < 1e-4
    assert (a.exp_avg_sq >= 0).all() and abs(a.exp_avg_sq.double().mean().item() - 1e-6 * np.sqrt(2 / np.pi)) < 1e-7
    a.step(1)
    b.step(1)
    assert torch.equal(a.weight, b.weight)
    w1 = a.weight.clone()
    a.step(2)
    assert not torch.equal(a.weight, w1)
    # the per-step change of a layer has the layer's scale: 1e-3 * s_l * N(0, 1)
    s = I.update_scales(I.toy_spec())
    for li in range(len(s)):
        lo, hi = a.layer_range(li)
        d = (a.weight[lo:hi].double() - w1[lo:hi].double()).std().item()
        assert d == pytest.approx(1e-3 * s[li], rel=0.05), li
