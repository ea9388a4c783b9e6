"""Pins of the oracle's SGD-with-drift step (CPU only).

Section 4.7 says the method carries over to plain SGD, persisting the
weights without optimizer state.  Pins: the closed form p - lr*g on values
where every operation is exact; decoupled weight decay (p * (1 - lr wd) on a
zero gradient, nothing for a non-decayed group); with no decay, agreement
with torch.optim.SGD (an independent implementation) over several steps;
and Eq. 1 on the parameters before and after the update for the drift,
accumulated by Eq. 2.
"""
import numpy as np
import pytest

from oracle import layercheck_oracle as O_real


def test_closed_form_exact(O=O_real):
    sc = O.sgd_scalars(2.0 ** -4, 0.0)
    p = np.array([0.5, -0.25, 1.0, 0.0], np.float32)
    g = np.array([2.0, -4.0, 0.5, 8.0], np.float32)
    assert np.array_equal(O.sgd_update(p, g, sc, True), p - np.float32(2.0 ** -4) * g)
    assert O.sgd_update(p, g, sc, True)[3] == -0.5


def test_decay_and_gradient_together(O=O_real):
    # lr = 2^-4, wd = 2^-2: decay = 1 - 2^-6 exactly; p (1 - lr wd) - lr g with
    # every operation exact, so the decay multiplies p alone, not the step
    sc = O.sgd_scalars(2.0 ** -4, 2.0 ** -2)
    assert sc["decay"] == np.float32(1.0 - 2.0 ** -6)
    p = np.array([1.0, 0.5, -2.0], np.float32)
    g = np.array([1.0, -2.0, 4.0], np.float32)
    exp = np.array([1.0 - 2.0 ** -6 - 2.0 ** -4, 0.5 - 2.0 ** -7 + 2.0 ** -3, -2.0 + 2.0 ** -5 - 2.0 ** -2], np.float32)
    assert np.array_equal(O.sgd_update(p, g, sc, True), exp)
    assert np.array_equal(O.sgd_update(p, g, sc, False), p - np.float32(2.0 ** -4) * g)


def test_decoupled_weight_decay(O=O_real):
    sc = O.sgd_scalars(1e-2, 0.1)
    p = np.array([1.0, -2.0, 0.375], np.float32)
    z = np.zeros(3, np.float32)
    assert np.array_equal(O.sgd_update(p, z, sc, True), p * np.float32(1.0 - 1e-2 * 0.1))
    assert np.array_equal(O.sgd_update(p, z, sc, False), p)


def test_matches_torch_sgd(O=O_real):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(2)
    n = 4096
    p0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    tp = torch.nn.Parameter(torch.from_numpy(p0.copy()))
    opt = torch.optim.SGD([tp], lr=1e-2, foreach=False)
    p = p0.copy()
    p_prev = p0.copy()
    for t in range(6):
        g = rng.standard_normal(n).astype(np.float32)
        tp.grad = torch.from_numpy(g.copy())
        opt.step()
        p = O.sgd_update(p, g, O.sgd_scalars(1e-2, 0.0), True)
        # torch may fuse the multiply-add (one rounding instead of two): the two
        # results differ by at most one ulp of the largest operand or result
        tq = tp.detach().numpy()
        prev = p_prev if t else p0
        big = np.maximum.reduce([np.abs(prev), np.abs(np.float32(1e-2) * g), np.abs(tq)])
        assert np.all(np.abs(p - tq) <= np.spacing(big)), t
        p = tq.copy()  # continue from torch's values so the bound applies per step
        p_prev = p.copy()


def test_drift_is_eq1_on_the_parameters(O=O_real):
    from tests._helpers import HostLayout
    lay = HostLayout([[33, 7], [64]], dtype=O.DT_BF16, has_master=True, seed=5)
    orc = O.LayerCheckOracle(lay.segs, 2, O.DT_BF16, True, O.MODE_ACCUM, [1e9, 1e9], 10)
    rng = np.random.default_rng(4)
    deltas = [0.0, 0.0]
    for t in (1, 2):
        grads = [rng.standard_normal(s.numel).astype(np.float32) for s in lay.segs]
        before = [s.master.copy() for s in lay.segs]
        m_before = [s.exp_avg.copy() for s in lay.segs]
        orc.sgd_step_score(t, grads, 1e-3, 0.0)
        for l in range(2):
            idx = [i for i, s in enumerate(lay.segs) if s.layer == l]
            old = np.concatenate([before[i] for i in idx]).astype(np.float64)
            exp = np.concatenate([before[i] - np.float32(1e-3) * grads[i] for i in idx]).astype(np.float64)
            new = np.concatenate([lay.segs[i].master for i in idx]).astype(np.float64)
            assert np.array_equal(new, exp)
            u = np.mean(np.abs(new - old)) / (np.mean(np.abs(old)) + 1e-8)
            assert abs(orc.u[l] - u) <= 1e-12 * u
            deltas[l] += orc.u[l]
            assert orc.delta[l] == deltas[l]  # Eq. 2 across the two steps
        for s, mb in zip(lay.segs, m_before):
            assert np.array_equal(s.exp_avg, mb)  # SGD leaves Adam moments alone
            assert np.array_equal(s.weight, O.bf16_round(s.master))
