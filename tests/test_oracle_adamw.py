"""Pins of the oracle's AdamW-with-drift step (CPU only).

The paper trains with AdamW and piggybacks the drift statistic on its
update (Sections 3.4 and 4.1) without restating the optimizer, so the
oracle follows the published AdamW definition.  Pins: the closed form of the
first step (bias correction makes the update lr * sign(g)), decoupled weight
decay on a zero gradient (p * (1 - lr wd), and nothing on a non-decayed
group), eps added beside the root of v_hat (a gradient as small as eps),
agreement with torch.optim.AdamW (an independent implementation,
different rounding order) over several steps, and Eq. 1 on the optimizer's
parameters for the drift.
"""
import numpy as np
import pytest

from oracle import layercheck_oracle as O_real


def test_first_step_is_lr_times_sign(O=O_real):
    sc = O.adamw_scalars(1e-3, 0.9, 0.999, 1e-8, 0.0, 1)
    p = np.full(6, 0.5, np.float32)
    g = np.array([2.0, -3.0, 0.25, -0.5, 7.0, -1e-3], np.float32)
    p_new, m, v = O.adamw_update(p, np.zeros(6, np.float32), np.zeros(6, np.float32), g, sc, True)
    ulp = np.spacing(np.float32(0.5))
    assert np.all(np.abs(p_new - (0.5 - 1e-3 * np.sign(g))) <= 2 * ulp), p_new
    assert np.allclose(m, 0.1 * g, rtol=2e-7) and np.allclose(v, 0.001 * g * g, rtol=4e-7)


def test_eps_beside_the_root(O=O_real):
    # A gradient as small as eps: on the first step m_hat = g and
    # sqrt(v_hat) = |g|, so the step is lr * g / (|g| + eps) = lr / 2 * sign(g)
    # when |g| = eps (eps inside the root, or squared, gives about lr instead)
    sc = O.adamw_scalars(1.0, 0.9, 0.999, 1e-8, 0.0, 1)
    g = np.array([1e-8, -1e-8], np.float32)
    p = np.zeros(2, np.float32)
    p_new, _, _ = O.adamw_update(p, np.zeros(2, np.float32), np.zeros(2, np.float32), g, sc, True)
    assert np.allclose(p_new, [-0.5, 0.5], rtol=1e-5), p_new


def test_decoupled_weight_decay_on_zero_gradient(O=O_real):
    sc = O.adamw_scalars(1e-2, 0.9, 0.999, 1e-8, 0.1, 3)
    p = np.array([1.0, -2.0, 0.375], np.float32)
    z = np.zeros(3, np.float32)
    p_dec, m, v = O.adamw_update(p, z, z, z, sc, True)
    assert np.array_equal(p_dec, p * np.float32(1.0 - 1e-2 * 0.1))  # shrink only; no Adam step
    assert not m.any() and not v.any()
    p_nodec, _, _ = O.adamw_update(p, z, z, z, sc, False)
    assert np.array_equal(p_nodec, p)


def test_matches_torch_adamw_over_steps(O=O_real):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    n = 4096
    p0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    lr, b1, b2, eps, wd = 1e-3, 0.9, 0.95, 1e-8, 0.05
    tp = torch.nn.Parameter(torch.from_numpy(p0.copy()))
    opt = torch.optim.AdamW([tp], lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd, foreach=False)
    p, m, v = p0.copy(), np.zeros(n, np.float32), np.zeros(n, np.float32)
    for t in range(1, 9):
        g = (rng.standard_normal(n) * (1 + t)).astype(np.float32)
        tp.grad = torch.from_numpy(g.copy())
        opt.step()
        p, m, v = O.adamw_update(p, m, v, g, O.adamw_scalars(lr, b1, b2, eps, wd, t), True)
        st = opt.state[tp]
        gs = float(np.abs(g).max())  # rounding-order differences scale with the gradient
        assert np.allclose(m, st["exp_avg"].numpy(), rtol=1e-5, atol=1e-6 * gs)
        assert np.allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-5, atol=1e-6 * gs * gs)
        assert np.allclose(p, tp.detach().numpy(), rtol=1e-5, atol=1e-8)


def test_fused_step_drift_is_eq1_on_the_parameters(O=O_real):
    from tests._helpers import HostLayout
    lay = HostLayout([[33, 7], [64]], dtype=O.DT_BF16, has_master=True, seed=3)
    for s in lay.segs:  # fresh optimizer state
        s.exp_avg[...] = 0
        s.exp_avg_sq[...] = 0
    orc = O.LayerCheckOracle(lay.segs, 2, O.DT_BF16, True, O.MODE_ACCUM, [1e9, 1e9], 10)
    rng = np.random.default_rng(1)
    grads = [rng.standard_normal(s.numel).astype(np.float32) for s in lay.segs]
    before = [s.master.copy() for s in lay.segs]
    orc.adamw_step_score(1, grads, 1e-3, 0.9, 0.999, 1e-8, 0.0, 1)
    # first step moves every parameter by lr (up to rounding): u = lr / mean|p_old|
    for l in range(2):
        idx = [i for i, s in enumerate(lay.segs) if s.layer == l]
        old = np.concatenate([before[i] for i in idx]).astype(np.float64)
        new = np.concatenate([lay.segs[i].master for i in idx]).astype(np.float64)
        u = np.mean(np.abs(new - old)) / (np.mean(np.abs(old)) + 1e-8)
        assert abs(orc.u[l] - u) <= 1e-12 * u
        assert abs(orc.u[l] - 1e-3 / np.mean(np.abs(old))) <= 2e-3 * orc.u[l]
        assert orc.delta[l] == orc.u[l]
    # bf16 weights are the round-to-nearest-even image of the new master
    for s in lay.segs:
        assert np.array_equal(s.weight, O.bf16_round(s.master))
    # Eq. 2: a second step adds its drift to the accumulator
    u1 = list(orc.u)
    orc.adamw_step_score(2, grads, 1e-3, 0.9, 0.999, 1e-8, 0.0, 2)
    assert orc.delta == [a + b for a, b in zip(u1, orc.u)]
    try:
        orc.adamw_step_score(2, grads, 1e-3, 0.9, 0.999, 1e-8, 0.0, 3)  # step must increase
        raise AssertionError("expected an error")
    except AssertionError:
        raise
    except Exception as e:  # noqa: BLE001 - any oracle copy's error class
        assert getattr(e, "code", None) == O.LC_ERR_BAD_STATE
