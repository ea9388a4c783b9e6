"""Exact-rational brute force of the decision rule on tiny layouts (CPU).

An independent restatement of Eq. 1-5 in ``fractions.Fraction`` arithmetic
that shares no code with the oracle: it keeps the whole weight history and
recomputes every accumulator from scratch as the sum of exact per-step scores
since the layer's last persist (ACCUM), or as the exact distance to the last
persisted weights (SNAPSHOT).  The oracle's fp64 accumulators must agree to
1e-12 relative and its selected sets must equal exhaustive thresholding;
layers whose exact accumulator lies within 1e-9 of K are reported and take the
oracle's decision (the same protocol the GPU parity tests use with 1e-5).
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import layercheck_oracle as O
from tests._helpers import HostLayout


def exact_layer_values(lay, layer, dtype):
    vals = []
    for s in lay.segs:
        if s.layer != layer:
            continue
        if dtype == O.DT_BF16:
            f = (s.weight.astype(np.uint32) << np.uint32(16)).view(np.float32)
        else:
            f = s.weight
        vals.extend(Fraction(float(x)) for x in f.tolist())
    return vals


def exact_score(cur, prev, eps):
    n = len(cur)
    A = sum((abs(a - b) for a, b in zip(cur, prev)), Fraction(0))
    B = sum((abs(b) for b in prev), Fraction(0))
    return (A / n) / (B / n + Fraction(eps))


@pytest.mark.parametrize("mode", [O.MODE_ACCUM, O.MODE_SNAPSHOT])
@pytest.mark.parametrize("dtype", [O.DT_BF16, O.DT_F32])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_selected_sets_equal_exhaustive_thresholding(mode, dtype, seed):
    run_bruteforce(O, mode, dtype, seed)


def run_bruteforce(O, mode, dtype, seed, steps=20):
    rng = np.random.default_rng(100 + seed)
    N = int(rng.integers(2, 9))
    sizes = [[int(x) for x in rng.integers(1, 24, rng.integers(1, 4))] for _ in range(N)]
    lay = HostLayout(sizes, dtype=dtype, has_master=(dtype == O.DT_BF16), seed=seed)
    scales = list(10.0 ** rng.uniform(-1.0, 1.5, N))
    k0 = list(10.0 ** rng.uniform(-2.5, -1.0, N))
    s_max = int(rng.integers(2, 7))
    eps = 1e-8
    orc = O.LayerCheckOracle(lay.segs, N, dtype, dtype == O.DT_BF16, mode, k0, s_max, eps_w=eps)
    orc.pack(0, 1 << 40)
    history = {0: [exact_layer_values(lay, l, dtype) for l in range(N)]}
    t_last = [0] * N
    near_count = 0
    for t in range(1, steps + 1):
        lay.step(scales)
        history[t] = [exact_layer_values(lay, l, dtype) for l in range(N)]
        lr = float(rng.choice([1.0, 0.5, 2.0]))
        orc.score(t)
        exact_delta = []
        for l in range(N):
            if mode == O.MODE_ACCUM:
                d = sum((exact_score(history[s][l], history[s - 1][l], eps)
                         for s in range(t_last[l] + 1, t + 1)), Fraction(0))
            else:
                d = exact_score(history[t][l], history[t_last[l]][l], eps)
            exact_delta.append(d)
            got = Fraction(orc.delta[l])
            assert abs(got - d) <= Fraction(1, 10 ** 12) * d, (t, l)
        mask, st = orc.select(t, lr)
        for l in range(N):
            K = Fraction(k0[l] * lr)
            expect = exact_delta[l] >= K or (t - t_last[l]) >= s_max
            if abs(exact_delta[l] - K) <= Fraction(1, 10 ** 9) * K:
                near_count += 1
                expect = bool(mask[l])  # reported, decision adopted
            assert bool(mask[l]) == expect, (t, l, float(exact_delta[l]), float(K))
            if expect:
                t_last[l] = t
        assert st["max_age"] == max(t - x for x in t_last) <= s_max - 1
        orc.pack(0, 1 << 40)
    assert near_count <= 2
