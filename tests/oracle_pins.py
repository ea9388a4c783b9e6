"""Pins for the CPU oracle, written as reusable checks.

Each ``check_*`` takes the oracle class under test (and, for the score pins,
its Eq. 1 function) so that the same checks run against the real oracle and
against deliberately broken copies (see test_oracle_mutations.py): a check
that never fails on a planted mistake is not pinning anything.

What pins what (the paper prints no worked example of u, Delta or a
selection trace, so the pins are closed forms, exact-rational brute force,
invariants and the paper's Table 1 figures):

* Eq. 1 closed forms: constant shadow a and constant change c give
  |c| / (|a| + eps_w); the denominator is the *previous* weights; the mean is
  joint over all tensors of a layer; zero change gives exactly 0.
* Eq. 3 uses ">=": an accumulator exactly equal to K persists.
* Section 3.3 guard: with zero drift a layer persists exactly every S_max steps.
* Eq. 4: reset to 0 after persisting (brute force checks Delta as the sum of
  exact per-step scores since the layer's last persist).
* Stats: size-weighted staleness <= max staleness <= S_max - 1 after a decision.
* Records: 14 bytes per parameter for bf16 + fp32 master + m + v (Section 4.1
  with Table 1); padded blocks hold the raw bytes in order.
* Recovery: newest version <= t_fail per layer; round trip is bit-exact.
* Section 3.4 base checkpoint: a rebase resets Delta, t_l and the shadow and
  selects every layer.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

from oracle import layercheck_oracle as O
from tests._helpers import HostLayout, f32_to_bf16_bits


def expect_error(fn, code):
    """Run fn; it must raise an error carrying status ``code`` (any oracle copy)."""
    try:
        fn()
    except AssertionError:
        raise
    except Exception as e:  # noqa: BLE001 - mutant copies define their own error class
        assert getattr(e, "code", None) == code, (getattr(e, "code", None), code, e)
        return
    raise AssertionError(f"expected error code {code}")


def _seg(layer, w, s, dtype, master=True):
    n = w.size
    return O.OSegment(layer, w, s, np.zeros(n, np.float32) if master else None,
                      np.zeros(n, np.float32), np.zeros(n, np.float32))


# ---------------------------------------------------------------- Eq. 1 -----

def check_closed_form(score_fn):
    # S = 0.5 everywhere, W = 0.5 + 2^-8 everywhere (both exact in bf16).
    for dtype in (O.DT_BF16, O.DT_F32):
        n = 37
        if dtype == O.DT_BF16:
            s = f32_to_bf16_bits(np.full(n, 0.5, np.float32))
            w = f32_to_bf16_bits(np.full(n, 0.5 + 2.0 ** -8, np.float32))
        else:
            s = np.full(n, 0.5, np.float32)
            w = np.full(n, 0.5 + 2.0 ** -8, np.float32)
        A, B, cnt, u = score_fn([w], [s], dtype, 0.0)
        assert cnt == n
        assert A == n * 2.0 ** -8 and B == n * 0.5
        assert u == 2.0 ** -7, u
        # negative change of the same size gives the same score (absolute values)
        if dtype == O.DT_F32:
            w2 = np.full(n, 0.5 - 2.0 ** -8, np.float32)
            assert score_fn([w2], [s], dtype, 0.0)[3] == 2.0 ** -7


def check_denominator_is_previous(score_fn):
    # S = 0.5, W = 1.0: mean|W-S| / mean|S| = 1 (dividing by mean|W| would give 0.5)
    s = np.full(8, 0.5, np.float32)
    w = np.full(8, 1.0, np.float32)
    assert score_fn([w], [s], O.DT_F32, 0.0)[3] == 1.0


def check_joint_mean(score_fn):
    # Layer of two tensors (3 and 1 elements); only the first changes by 2^-8.
    s1, s2 = np.full(3, 0.5, np.float32), np.full(1, 0.5, np.float32)
    w1, w2 = np.full(3, 0.5 + 2.0 ** -8, np.float32), s2.copy()
    u = score_fn([w1, w2], [s1, s2], O.DT_F32, 0.0)[3]
    assert u == 3.0 * 2.0 ** -9, u  # joint mean; a mean of per-tensor means gives 2^-8


def check_zero_change(score_fn):
    rng = np.random.default_rng(1)
    for dtype in (O.DT_BF16, O.DT_F32):
        x = (rng.standard_normal(1000) * 0.02).astype(np.float32)
        w = f32_to_bf16_bits(x) if dtype == O.DT_BF16 else x
        u = score_fn([w], [w.copy()], dtype, 1e-8)[3]
        assert u == 0.0 and not np.signbit(u)


def check_eps_in_denominator(score_fn):
    # all-zero previous weights: u = mean|W| / eps_w exactly when eps_w = 2^-10
    s = np.zeros(4, np.float32)
    w = np.full(4, 2.0 ** -12, np.float32)
    assert score_fn([w], [s], O.DT_F32, 2.0 ** -10)[3] == 0.25


def check_scale_invariance(score_fn):
    rng = np.random.default_rng(2)
    s = (rng.standard_normal(257) * 0.02).astype(np.float32)
    w = (s + rng.standard_normal(257).astype(np.float32) * 1e-4).astype(np.float32)
    u0 = score_fn([w], [s], O.DT_F32, 0.0)[3]
    for k in (-3, 5):
        u1 = score_fn([w * np.float32(2.0 ** k)], [s * np.float32(2.0 ** k)], O.DT_F32, 0.0)[3]
        assert u1 == u0


def check_exact_rational(score_fn):
    """u within 1e-12 of the exact rational value on random tiny tensors."""
    rng = np.random.default_rng(3)
    for trial in range(20):
        n1, n2 = rng.integers(1, 40, 2)
        dt = O.DT_BF16 if trial % 2 else O.DT_F32
        xs = [(rng.standard_normal(n) * 0.02).astype(np.float32) for n in (n1, n2)]
        ys = [(x + rng.standard_normal(x.size).astype(np.float32) * 1e-3).astype(np.float32) for x in xs]
        if dt == O.DT_BF16:
            xs = [f32_to_bf16_bits(x) for x in xs]
            ys = [f32_to_bf16_bits(y) for y in ys]
        eps = 1e-8
        u = score_fn(ys, xs, dt, eps)[3]
        exact = exact_u(ys, xs, dt, eps)
        assert abs(Fraction(u) - exact) <= Fraction(1, 10 ** 12) * abs(exact)


def exact_value(v, dtype):
    if dtype == O.DT_BF16:
        return Fraction(float(np.array([int(v) << 16], dtype=np.uint32).view(np.float32)[0]))
    return Fraction(float(v))


def exact_u(ws, ss, dtype, eps):
    A = Fraction(0)
    B = Fraction(0)
    n = 0
    for w, s in zip(ws, ss):
        for a, b in zip(w.tolist(), s.tolist()):
            x, y = exact_value(a, dtype), exact_value(b, dtype)
            A += abs(x - y)
            B += abs(y)
            n += 1
    return (A / n) / (B / n + Fraction(eps))


# ---------------------------------------------------------------- Eq. 3-5 ---

def _const_layout(n_layers, per_layer=4):
    segs = []
    for l in range(n_layers):
        s = np.full(per_layer, 0.5, np.float32)
        segs.append(_seg(l, s.copy(), np.zeros(per_layer, np.float32), O.DT_F32))
    return segs


def check_ge_threshold(cls):
    # u = 2^-7 exactly; K0 = 2^-7: Delta == K must persist under Eq. 3's ">=".
    segs = _const_layout(2)
    orc = cls(segs, 2, O.DT_F32, True, O.MODE_ACCUM, [2.0 ** -7, 2.0 ** -6], s_max=100, eps_w=0.0)
    orc.pack(0, 1 << 30)  # base version
    for s in segs:
        s.weight[...] = 0.5 + 2.0 ** -8
    orc.score(1)
    mask, st = orc.select(1, 1.0)
    assert list(mask) == [1, 0], mask
    assert st["n_forced"] == 0
    # lr_scale = 0.5 halves K: layer 1 holds 2^-7 + u(2) ~= 0.01556, which is
    # below K0 = 2^-6 but above K0 * 0.5 (ignoring or inverting s(lr) fails here)
    orc.pack(0, 1 << 30)
    for s in segs:
        s.weight[...] = 0.5 + 2.0 ** -7
    orc.score(2)
    mask, _ = orc.select(2, 0.5)
    assert list(mask) == [1, 1], mask


def check_delta_in_fp64(cls):
    # Reading #14: Delta accumulates in fp64.  One fp32 layer of 1024 elements
    # at 1.0: step 1 doubles every element (u = 1 exactly), step 2 moves one
    # element by one ulp of 2.0 (u = 2^-22 / 1024 / 2 = 2^-33 exactly).  With
    # K0 = 1 + 2^-34 only an fp64 accumulator (1 + 2^-33) crosses; an fp32
    # one stays at 1.0.
    n = 1024
    w = np.ones(n, np.float32)
    segs = [O.OSegment(0, w, np.zeros(n, np.float32), w.copy(), np.zeros(n, np.float32), np.zeros(n, np.float32))]
    orc = cls(segs, 1, O.DT_F32, True, O.MODE_ACCUM, [1.0 + 2.0 ** -34], s_max=100, eps_w=0.0)
    orc.pack(0, 1 << 30)
    w[...] = 2.0
    orc.score(1)
    assert orc.u == [1.0]
    mask, _ = orc.select(1, 1.0)
    assert list(mask) == [0]
    w[0] = np.float32(2.0 + 2.0 ** -22)
    orc.score(2)
    assert orc.u == [2.0 ** -33] and orc.delta == [1.0 + 2.0 ** -33]
    mask, _ = orc.select(2, 1.0)
    assert list(mask) == [1]


def check_staleness_period(cls, mode=O.MODE_ACCUM):
    # zero drift: each layer persists exactly at t_base + k*S_max
    for s_max in (1, 3, 4):
        for t_base in (0, 7):
            segs = _const_layout(3)
            orc = cls(segs, 3, O.DT_F32, True, mode, [1e-3] * 3, s_max=s_max, t_base=t_base)
            orc.pack(0, 1 << 30)
            for t in range(t_base + 1, t_base + 4 * s_max + 2):
                orc.score(t)
                mask, st = orc.select(t, 1.0)
                expect = int((t - t_base) % s_max == 0)
                assert list(mask) == [expect] * 3, (s_max, t, mask)
                assert st["n_forced"] == 3 * expect
                assert st["max_age"] == (t - t_base) % s_max
                orc.pack(0, 1 << 30)


def check_irregular_steps(cls, mode=O.MODE_ACCUM):
    # Decisions need not come every iteration.  (a) zero drift, S_max = 4,
    # decisions at 1, 2, 3, 9, 10, 12, 13: nothing is due until the gap from
    # t_base reaches S_max (step 9, age 9), then every layer is forced and its
    # age is 0; the next forcing is exactly S_max after that (step 13).
    segs = _const_layout(3)
    orc = cls(segs, 3, O.DT_F32, True, mode, [1e-3] * 3, s_max=4)
    orc.pack(0, 1 << 30)
    last = 0
    for t in (1, 2, 3, 9, 10, 12, 13):
        orc.score(t)
        mask, st = orc.select(t, 1.0)
        due = int(t - last >= 4)
        assert list(mask) == [due] * 3, (t, mask)
        assert st["n_forced"] == 3 * due
        assert st["max_age"] == (0 if due else t - last), (t, st)
        last = t if due else last
        orc.pack(0, 1 << 30)
    # (b) Eq. 1 sees only the weights at decision steps.  Layer 0 holds four
    # elements at 1/2; each unscored iteration moves the first two up and the
    # last two down by d = 2^-9, which keeps mean|W| at 1/2.  Layer 1 never
    # moves.  K0 = 2^-6, S_max far away, eps_w = 0.
    d = 2.0 ** -9
    segs = _const_layout(2)
    orc = cls(segs, 2, O.DT_F32, True, mode, [2.0 ** -6] * 2, s_max=100, eps_w=0.0)
    orc.pack(0, 1 << 30)

    def move(k):
        w = segs[0].weight
        w[:2] += k * d
        w[2:] -= k * d

    def decide_at(t):
        orc.score(t)
        u = list(orc.u)
        mask, _ = orc.select(t, 1.0)
        orc.pack(0, 1 << 30)
        return u, list(mask)

    u, mask = decide_at(1)
    assert u == [0.0, 0.0] and mask == [0, 0]
    move(1)
    move(1)  # iterations 2 and 3, decision at 3: |W - W(1)| = 2d per element
    u, mask = decide_at(3)
    assert u == [2.0 ** -7, 0.0] and mask == [0, 0], (u, mask)
    move(-1)
    move(-1)  # back to 1/2 by step 6
    u, mask = decide_at(6)
    if mode == O.MODE_ACCUM:
        # reference W(3): the path length adds up, Delta = 2^-7 + 2^-7 = K0
        assert u == [2.0 ** -7, 0.0] and mask == [1, 0], (u, mask)
    else:
        # reference: the base persist; the net displacement is zero
        assert u == [0.0, 0.0] and mask == [0, 0], (u, mask)
    for k in (1, 1, -1, -1):
        move(k)  # a round trip between two decisions is invisible to Eq. 1
    u, mask = decide_at(11)
    assert u == [0.0, 0.0] and mask == [0, 0], (u, mask)


def check_k0_extremes(cls):
    lay = HostLayout([[5, 3], [4], [7]], seed=4)
    # K0 = 0: every layer persists by drift every step.  With S_max = 1 every
    # layer is also due by age, and n_forced counts only age-only selections.
    orc = cls(lay.segs, 3, O.DT_BF16, True, O.MODE_ACCUM, [0.0] * 3, s_max=1)
    orc.pack(0, 1 << 40)
    for t in range(1, 5):
        lay.step([1.0, 0.0, 0.5], zero_layers=(1,))
        orc.score(t)
        mask, st = orc.select(t, 1.0)
        assert mask.tolist() == [1, 1, 1] and st["n_forced"] == 0
        orc.pack(0, 1 << 40)
    lay = HostLayout([[5, 3], [4], [7]], seed=4)
    orc = cls(lay.segs, 3, O.DT_BF16, True, O.MODE_ACCUM, [1e300] * 3, s_max=2)
    orc.pack(0, 1 << 40)
    for t in range(1, 7):
        lay.step([1.0, 1.0, 1.0])
        orc.score(t)
        mask, st = orc.select(t, 1.0)
        assert mask.tolist() == [t % 2 == 0] * 3
        assert st["n_forced"] == (3 if t % 2 == 0 else 0)
        orc.pack(0, 1 << 40)


def check_zero_layer(cls, mode=O.MODE_ACCUM):
    # A layer that is all zeros and stays zero.  With eps_w = 0, Eq. 1 is 0/0
    # for it: u and Delta are NaN, the drift rule (Delta >= K) never holds for
    # it, and the staleness guard still persists it every S_max steps.  With
    # eps_w > 0 the same layer scores exactly 0.  The other layer moves every
    # step and persists by drift every step.
    for eps in (0.0, 1e-8):
        segs = [_seg(0, np.zeros(4, np.float32), np.zeros(4, np.float32), O.DT_F32),
                _seg(1, np.full(4, 0.5, np.float32), np.full(4, 0.5, np.float32), O.DT_F32)]
        orc = cls(segs, 2, O.DT_F32, True, mode, [1e-30, 1e-30], s_max=3, eps_w=eps)
        orc.pack(0, 1 << 30)
        for t in range(1, 8):
            segs[1].weight[...] = 0.5 + t * 2.0 ** -8
            orc.score(t)
            if eps == 0.0:
                assert np.isnan(orc.u[0]) and np.isnan(orc.delta[0]), (t, orc.u[0])
            else:
                assert orc.u[0] == 0.0 and orc.delta[0] == 0.0
            assert orc.u[1] > 0
            mask, st = orc.select(t, 1.0)
            assert list(mask) == [int(t % 3 == 0), 1], (eps, t, mask)
            assert st["n_forced"] == int(t % 3 == 0)
            orc.pack(0, 1 << 30)


def check_rebase(cls, mode=O.MODE_ACCUM):
    # Section 3.4: a full base checkpoint at the end of the warm-up window.
    # (1) It resets Delta and t_l: u(1) = 2^-7 exactly, then the rebase at
    # step 1; at step 2, u(2) = 2^-8 / (0.5 + 2^-8) < K0 = 1.5 * 2^-7, which
    # only a reset keeps below K in ACCUM mode; W then stays put.  Both layers
    # are forced S_max = 3 steps after the rebase, not after the old base.
    segs = _const_layout(2)
    orc = cls(segs, 2, O.DT_F32, True, mode, [1.5 * 2.0 ** -7, 1e300], s_max=3, eps_w=0.0)
    orc.pack(0, 1 << 30)
    for s in segs:
        s.weight[...] = 0.5 + 2.0 ** -8
    orc.score(1)  # warm-up: scored, no selection
    assert orc.delta == [2.0 ** -7] * 2
    orc.rebase(1)
    expect_error(lambda: orc.select(1, 1.0), O.LC_ERR_BAD_STATE)  # the rebase is the decision
    payload, res = orc.pack(0, 1 << 30)
    assert res["n_packed"] == 2 and res["bytes_written"] == sum(orc.R)
    assert bytes(payload) == orc.layer_record(0) + orc.layer_record(1)
    expect_error(lambda: orc.rebase(0), O.LC_ERR_BAD_STATE)  # before the last step
    for s in segs:
        s.weight[...] = 0.5 + 2 * 2.0 ** -8
    for t in (2, 3, 4):
        orc.score(t)
        mask, st = orc.select(t, 1.0)
        assert mask.tolist() == [int(t == 4)] * 2, (mode, t, mask)
        assert st["max_age"] == (0 if t == 4 else t - 1) and st["n_forced"] == (2 if t == 4 else 0)
        orc.pack(0, 1 << 30)
    # (2) It re-synchronises the shadow: W moves at steps 1 and 2 with no
    # score (a warm-up that does not score), rebase at 2; the score at 3 must
    # measure one step, 2^-8 / (0.5 + 2^-7) < K0, not three.
    segs = _const_layout(1)
    orc = cls(segs, 1, O.DT_F32, True, mode, [1.5 * 2.0 ** -7], s_max=100, eps_w=0.0)
    orc.pack(0, 1 << 30)
    for t in (1, 2):
        segs[0].weight[...] = 0.5 + t * 2.0 ** -8
    orc.rebase(2)
    orc.pack(0, 1 << 30)
    segs[0].weight[...] = 0.5 + 3 * 2.0 ** -8
    orc.score(3)
    assert orc.u[0] == (2.0 ** -8) / (0.5 + 2.0 ** -7)
    mask, _ = orc.select(3, 1.0)
    assert mask.tolist() == [0]


def check_stats_invariants(cls, mode=O.MODE_ACCUM):
    rng = np.random.default_rng(5)
    for trial in range(6):
        sizes = [[int(x) for x in rng.integers(1, 30, rng.integers(1, 4))] for _ in range(rng.integers(2, 7))]
        lay = HostLayout(sizes, seed=trial)
        N = len(sizes)
        s_max = int(rng.integers(1, 6))
        k0 = list(10.0 ** rng.uniform(-3, -1, N))
        orc = cls(lay.segs, N, O.DT_BF16, True, mode, k0, s_max=s_max)
        orc.pack(0, 1 << 40)
        scales = list(10.0 ** rng.uniform(-1.5, 1.0, N))
        for t in range(1, 15):
            lay.step(scales)
            orc.score(t)
            mask, st = orc.select(t, 1.0)
            assert st["weighted_age"] <= st["max_age"] <= s_max - 1
            n = [sum(s.numel for s in lay.segs if s.layer == l) for l in range(N)]
            ages = [t - orc.t_last[l] for l in range(N)]
            assert st["max_age"] == max(ages)
            # weighted staleness: an explicit sum over layers
            assert abs(st["weighted_age"] - sum(a * b for a, b in zip(n, ages)) / sum(n)) <= 1e-12 * max(1, st["max_age"])
            assert st["n_selected"] == int(mask.sum())
            # payload: the selected layers' records, each block (bf16 W, fp32
            # master, m, v of every tensor) padded to 256 B, written out here
            rec = [sum(-(-x * 2 // 256) * 256 + 3 * (-(-x * 4 // 256) * 256) for x in sizes[l]) for l in range(N)]
            assert st["payload_bytes"] == sum(rec[l] for l in range(N) if mask[l]), (st, rec, list(mask))
            payload, res = orc.pack(0, 1 << 40)
            assert res["bytes_written"] == len(payload) == st["payload_bytes"]


# ---------------------------------------------------------------- records ---

def check_record_format(cls):
    lay = HostLayout([[3, 200], [128]], dtype=O.DT_BF16, has_master=True, seed=6)
    orc = cls(lay.segs, 2, O.DT_BF16, True, O.MODE_ACCUM, [1e-3, 1e-3], s_max=4)
    payload, res = orc.pack(0, 1 << 30)
    # layer 0 record: W blocks (6 B -> 256, 400 B -> 512), master (12 -> 256, 800 -> 1024),
    # m and v like master: 768 + 1280 * 3 = 4608; layer 1: 256 + 512 * 3 = 1792
    assert res["bytes_written"] == len(payload) == 4608 + 1792
    s0, s1, s2 = lay.segs
    assert bytes(payload[0:6]) == s0.weight.tobytes()
    assert not payload[6:256].any()
    assert bytes(payload[256:656]) == s1.weight.tobytes()
    assert not payload[656:768].any()
    assert bytes(payload[768:780]) == s0.master.tobytes()
    off = 768 + 256 + 1024
    assert bytes(payload[off:off + 12]) == s0.exp_avg.tobytes()
    off = 768 + 2 * 1280
    assert bytes(payload[off + 256:off + 256 + 800]) == s1.exp_avg_sq.tobytes()
    off = 4608
    assert bytes(payload[off:off + 256]) == s2.weight.tobytes()
    assert bytes(payload[off + 256:off + 768]) == s2.master.tobytes()
    assert bytes(payload[off + 1280:off + 1792]) == s2.exp_avg_sq.tobytes()


def check_record_format_weights_only(cls):
    # Section 4.7 (SGD): a layout without Adam moments persists the weights
    # (and the fp32 master) only: bf16 W blocks, then master blocks, each
    # padded to 256 B -- 6 B per parameter when nothing is padded.
    rng = np.random.default_rng(13)
    segs = []
    for l, n in ((0, 128), (0, 3), (1, 256)):
        base = (rng.standard_normal(n) * 0.02).astype(np.float32)
        segs.append(O.OSegment(l, f32_to_bf16_bits(base), np.zeros(n, np.uint16), base.copy(), None, None))
    orc = cls(segs, 2, O.DT_BF16, True, O.MODE_ACCUM, [1e-3, 1e-3], s_max=4)
    assert orc.R == [256 + 256 + 512 + 256, 512 + 1024], orc.R
    payload, res = orc.pack(0, 1 << 30)
    assert res["bytes_written"] == len(payload) == 1280 + 1536
    s0, s1, s2 = segs
    assert bytes(payload[0:256]) == s0.weight.tobytes()
    assert bytes(payload[256:262]) == s1.weight.tobytes() and not payload[262:512].any()
    assert bytes(payload[512:1024]) == s0.master.tobytes()
    assert bytes(payload[1024:1036]) == s1.master.tobytes() and not payload[1036:1280].any()
    assert bytes(payload[1280:1792]) == s2.weight.tobytes()
    assert bytes(payload[1792:2816]) == s2.master.tobytes()


def check_fused_step_rules(cls):
    # The fused optimizer step replaces the score of its step: select follows
    # it at the same step; it accumulates (Eq. 2), so SNAPSHOT mode refuses
    # it; AdamW needs the moment arrays.
    lay = HostLayout([[40], [24, 8]], seed=14)
    grads = [np.full(s.numel, 0.5, np.float32) for s in lay.segs]
    orc = cls(lay.segs, 2, O.DT_BF16, True, O.MODE_ACCUM, [1e9, 1e9], s_max=2)
    orc.pack(0, 1 << 30)
    orc.adamw_step_score(1, grads, 1e-3, 0.9, 0.95, 1e-8, 0.0, 1)
    u1 = list(orc.u)
    mask, st = orc.select(1, 1.0)
    assert list(mask) == [0, 0] and st["max_age"] == 1
    orc.pack(0, 1 << 30)
    orc.sgd_step_score(2, grads, 1e-3, 0.0)
    mask, st = orc.select(2, 1.0)  # age 2 = S_max: both forced, Delta reset
    assert list(mask) == [1, 1] and st["n_forced"] == 2 and orc.delta == [0.0, 0.0]
    assert all(x > 0 for x in u1)
    lay2 = HostLayout([[40]], seed=15)
    snap = cls(lay2.segs, 1, O.DT_BF16, True, O.MODE_SNAPSHOT, [1e9], s_max=2)
    snap.pack(0, 1 << 30)
    g2 = [np.full(s.numel, 0.5, np.float32) for s in lay2.segs]
    expect_error(lambda: snap.adamw_step_score(1, g2, 1e-3, 0.9, 0.95, 1e-8, 0.0, 1), O.LC_ERR_BAD_STATE)
    expect_error(lambda: snap.sgd_step_score(1, g2, 1e-3, 0.0), O.LC_ERR_BAD_STATE)
    n = 16
    base = np.full(n, 0.25, np.float32)
    bare = cls([O.OSegment(0, f32_to_bf16_bits(base), np.zeros(n, np.uint16), base.copy(), None, None)], 1,
               O.DT_BF16, True, O.MODE_ACCUM, [1e9], s_max=2)
    expect_error(lambda: bare.adamw_step_score(1, [np.ones(n, np.float32)], 1e-3, 0.9, 0.95, 1e-8, 0.0, 1),
                 O.LC_ERR_BAD_STATE)
    bare.sgd_step_score(1, [np.ones(n, np.float32)], 2.0 ** -4, 0.0)  # SGD needs none
    assert bare.by_layer[0][0].master[0] == np.float32(0.25 - 2.0 ** -4)


def check_fourteen_bytes_per_param():
    # pad-free blocks (every tensor a multiple of 128 elements): 2 + 4 + 4 + 4 bytes
    assert O.record_bytes([128 * 7, 4096], 2, True) == 14 * (128 * 7 + 4096)
    assert O.record_bytes([128 * 7, 4096], 2, False) == 10 * (128 * 7 + 4096)
    assert O.record_bytes([64 * 3], 4, False) == 12 * 64 * 3
    assert O.record_bytes([1], 2, True) == 4 * 256
    # without Adam moments (Section 4.7): weights and master only
    assert O.record_bytes([128 * 5], 2, True, False) == 6 * 128 * 5
    assert O.record_bytes([128 * 5], 2, False, False) == 2 * 128 * 5


def check_capacity(cls):
    lay = HostLayout([[100], [300], [50]], seed=7)
    orc = cls(lay.segs, 3, O.DT_BF16, True, O.MODE_ACCUM, [1e-3] * 3, s_max=4)
    R = orc.R
    p0, r0 = orc.pack(0, R[0] + R[1] - 1)
    assert r0 == {"bytes_written": R[0], "n_packed": 1, "next_rank": 1, "done": 0}
    expect_error(lambda: orc.pack(1, R[1] - 1), O.LC_ERR_CAPACITY)
    p1, r1 = orc.pack(1, R[1] + R[2])
    assert r1["done"] == 1 and r1["n_packed"] == 2
    full = O.LayerCheckOracle(HostLayout([[100], [300], [50]], seed=7).segs, 3, O.DT_BF16, True,
                              O.MODE_ACCUM, [1e-3] * 3, s_max=4).pack(0, 1 << 30)[0]
    assert bytes(np.concatenate([p0, p1])) == bytes(full)


def check_snapshot_partial_pack_refresh(cls):
    # SNAPSHOT mode refreshes the shadow of the layers a pack call writes, and
    # only those: after a capacity-limited first call the other selected
    # layers still hold their last persisted weights in the shadow.
    lay = HostLayout([[100], [300], [50]], seed=16)
    orc = cls(lay.segs, 3, O.DT_BF16, True, O.MODE_SNAPSHOT, [0.0] * 3, s_max=4)
    orc.pack(0, 1 << 30)
    old = [s.weight.copy() for s in lay.segs]
    lay.step([1.0, 1.0, 1.0])
    orc.score(1)
    mask, _ = orc.select(1, 1.0)
    assert list(mask) == [1, 1, 1]
    _, r = orc.pack(0, orc.R[0])
    assert r["n_packed"] == 1
    segs = lay.segs
    assert np.array_equal(segs[0].shadow, segs[0].weight)
    for i in (1, 2):
        assert np.array_equal(segs[i].shadow, old[i]) and not np.array_equal(segs[i].shadow, segs[i].weight)
    orc.pack(1, 1 << 30)
    assert all(np.array_equal(s_.shadow, s_.weight) for s_ in segs)


def check_layout_validation(cls):
    # Layouts the interface refuses (LC_ERR_INVALID_ARG), mirrored by the oracle.
    def segs(layers, master=(True,), moments=(True,)):
        out = []
        for i, l in enumerate(layers):
            n = 4
            base = np.full(n, 0.5, np.float32)
            ma = master[i % len(master)]
            mo = moments[i % len(moments)]
            out.append(O.OSegment(l, f32_to_bf16_bits(base), np.zeros(n, np.uint16), base.copy() if ma else None,
                                  np.zeros(n, np.float32) if mo else None, np.zeros(n, np.float32) if mo else None))
        return out

    def refused(fn):
        expect_error(fn, O.LC_ERR_INVALID_ARG)

    ok = dict(weight_dtype=O.DT_BF16, has_master=True, mode=O.MODE_ACCUM, k0=[1e-3, 1e-3], s_max=4)
    cls(segs([0, 1]), 2, **ok)  # the accepted form
    refused(lambda: cls(segs([1, 0]), 2, **ok))                       # layers not grouped in order
    refused(lambda: cls(segs([0, 0]), 2, **ok))                       # layer 1 has no tensor
    refused(lambda: cls(segs([0, 2]), 2, **ok))                       # layer out of range
    refused(lambda: cls([], 2, **ok))                                 # empty layout
    refused(lambda: cls(segs([0, 1], master=(True, False)), 2, **ok))  # master on some tensors only
    refused(lambda: cls(segs([0, 1], moments=(True, False)), 2, **ok))  # moments on some tensors only
    refused(lambda: cls(segs([0, 1]), 2, **dict(ok, s_max=0)))        # S_max < 1
    refused(lambda: cls(segs([0, 1]), 2, **dict(ok, k0=[1e-3])))      # one K0 per layer
    refused(lambda: cls(segs([0, 1]), 2, **dict(ok, mode=7)))         # unknown mode
    refused(lambda: cls(segs([0, 1]), 2, **dict(ok, weight_dtype=9)))  # unknown weight type
    for eps in (-1e-8, float("nan"), float("inf")):
        refused(lambda: cls(segs([0, 1]), 2, eps_w=eps, **ok))         # eps_w finite, >= 0
    for k in (-1e-3, float("nan")):
        refused(lambda: cls(segs([0, 1]), 2, **dict(ok, k0=[1e-3, k])))  # K0 >= 0


# ---------------------------------------------------------------- recovery --

def check_restore_roundtrip(cls, mode=O.MODE_ACCUM):
    sizes = [[17, 5], [64], [9, 9, 9], [1]]
    lay = HostLayout(sizes, seed=8)
    N = len(sizes)
    orc = cls(lay.segs, N, O.DT_BF16, True, mode, [2e-2] * N, s_max=3)
    versions = []
    payload, _ = orc.pack(0, 1 << 40)
    versions.append({"step": 0, "mask": np.ones(N, np.uint8), "payload": payload})
    truth = {}  # (layer, step) -> arrays as persisted
    for s in lay.segs:
        truth.setdefault((s.layer, 0), []).append((s.weight.copy(), s.master.copy(), s.exp_avg.copy(), s.exp_avg_sq.copy()))
    for t in range(1, 8):
        lay.step([3.0, 0.2, 1.0, 0.05])
        orc.score(t)
        mask, _ = orc.select(t, 1.0)
        payload, _ = orc.pack(0, 1 << 40)
        versions.append({"step": t, "mask": mask, "payload": payload})
        for s in lay.segs:
            if mask[s.layer]:
                truth.setdefault((s.layer, t), []).append((s.weight.copy(), s.master.copy(), s.exp_avg.copy(), s.exp_avg_sq.copy()))
    t_fail = 5
    # brute-force plan: newest persisted step <= t_fail per layer
    expect = [max(v["step"] for v in versions if v["step"] <= t_fail and v["mask"][l]) for l in range(N)]
    for s in lay.segs:  # lose the live state
        for a in (s.weight, s.shadow, s.master, s.exp_avg, s.exp_avg_sq):
            a[...] = 0
    chosen = orc.restore(versions, t_fail)
    assert chosen.tolist() == expect
    per_layer = {}
    for s in lay.segs:
        k = per_layer.get(s.layer, 0)
        w, m0, m, v = truth[(s.layer, expect[s.layer])][k]
        per_layer[s.layer] = k + 1
        assert np.array_equal(s.weight, w) and np.array_equal(s.master, m0)
        assert np.array_equal(s.exp_avg, m) and np.array_equal(s.exp_avg_sq, v)
        assert np.array_equal(s.shadow, s.weight)
    assert orc.t_last == expect and orc.delta == [0.0] * N
    # restore -> re-pack of every layer reproduces each layer's chosen record
    orc2 = cls(lay.segs, N, O.DT_BF16, True, mode, [2e-2] * N, s_max=3)
    allrec, _ = orc2.pack(0, 1 << 40)
    pos = 0
    for l in range(N):
        v = versions[[i for i, vv in enumerate(versions) if vv["step"] == expect[l]][0]]
        off = sum(orc.R[j] for j in range(l) if v["mask"][j])
        assert bytes(allrec[pos:pos + orc.R[l]]) == bytes(v["payload"][off:off + orc.R[l]])
        pos += orc.R[l]
    # dropping the newest version of a layer moves it to the next-newest
    newest = max(range(len(versions)), key=lambda i: versions[i]["step"] if versions[i]["step"] <= t_fail else -1)
    rest = [v for i, v in enumerate(versions) if i != newest]
    plan = orc.plan(rest, t_fail)
    for l in range(N):
        exp2 = max(v["step"] for v in rest if v["step"] <= t_fail and v["mask"][l])
        assert rest[plan[l]]["step"] == exp2


def check_restore_errors(cls):
    lay = HostLayout([[4], [4]], seed=9)
    orc = cls(lay.segs, 2, O.DT_BF16, True, O.MODE_ACCUM, [1e-3] * 2, s_max=3)
    payload, _ = orc.pack(0, 1 << 30)
    base = {"step": 0, "mask": np.ones(2, np.uint8), "payload": payload}
    part = {"step": 3, "mask": np.array([1, 0], np.uint8), "payload": payload[:orc.R[0]]}
    for versions, t_fail, code in (
            ([part], 3, O.LC_ERR_NO_VERSION),
            ([base, part], -1, O.LC_ERR_NO_VERSION),
            ([base, dict(base)], 2, O.LC_ERR_INVALID_ARG),
            ([base, {"step": 3, "mask": np.array([1, 0], np.uint8), "payload": payload}], 5, O.LC_ERR_INVALID_ARG),
            ([base, {"step": 3, "mask": np.array([1, 0, 0], np.uint8), "payload": payload[:orc.R[0]]}], 5,
             O.LC_ERR_INVALID_ARG)):
        expect_error(lambda: orc.restore(versions, t_fail), code)
    # a version newer than t_fail is ignored
    assert orc.restore([base, part], 2).tolist() == [0, 0]
    assert orc.restore([base, part], 3).tolist() == [3, 0]


def check_call_order_errors(cls):
    # The interface's call rules, which the oracle mirrors so that refusals
    # compare between the two sides: decision steps strictly increase; select
    # takes a positive, finite s(lr); a pack starts at a rank inside the
    # selection; a restore at t_fail resumes the run at t_fail + 1, also below
    # the last step before the failure; a base may not precede the last step.
    lay = HostLayout([[5], [3, 2]], seed=12)
    orc = cls(lay.segs, 2, O.DT_BF16, True, O.MODE_ACCUM, [1e-3] * 2, s_max=4)
    payload, _ = orc.pack(0, 1 << 30)
    base = {"step": 0, "mask": np.ones(2, np.uint8), "payload": payload}
    for t in (1, 2, 3):
        lay.step([1.0, 1.0])
        orc.score(t)
        expect_error(lambda: orc.score(t), O.LC_ERR_BAD_STATE)
        expect_error(lambda: orc.pack(0, 1 << 30), O.LC_ERR_BAD_STATE)  # nothing selected yet
        for bad in (0.0, -1.0, float("nan"), float("inf")):
            expect_error(lambda: orc.select(t, bad), O.LC_ERR_INVALID_ARG)
        mask, st = orc.select(t, 1.0)
        expect_error(lambda: orc.select(t, 1.0), O.LC_ERR_BAD_STATE)  # one select per score
        expect_error(lambda: orc.pack(st["n_selected"] + 1, 1 << 30), O.LC_ERR_INVALID_ARG)
        orc.pack(0, 1 << 30)
    expect_error(lambda: orc.score(2), O.LC_ERR_BAD_STATE)
    expect_error(lambda: orc.rebase(2), O.LC_ERR_BAD_STATE)
    lay.step([1.0, 1.0])
    orc.score(4)
    orc.select(4, 1.0)  # a selection left unpacked ...
    assert orc.restore([base], 1).tolist() == [0, 0]  # ... is replaced by the restore
    expect_error(lambda: orc.score(1), O.LC_ERR_BAD_STATE)
    expect_error(lambda: orc.select(1, 1.0), O.LC_ERR_BAD_STATE)  # a restore is no score
    lay.step([1.0, 1.0])
    orc.score(2)  # below the step reached before the failure: the resumed run
    orc.select(2, 1.0)
    orc.pack(0, 1 << 30)
    orc.rebase(2)  # a base at the last step is allowed


def check_accum_equals_snapshot_first_step(cls):
    la = HostLayout([[30, 2], [50]], seed=10)
    lb = HostLayout([[30, 2], [50]], seed=10)
    oa = cls(la.segs, 2, O.DT_BF16, True, O.MODE_ACCUM, [1e9, 1e9], s_max=100)
    ob = cls(lb.segs, 2, O.DT_BF16, True, O.MODE_SNAPSHOT, [1e9, 1e9], s_max=100)
    oa.pack(0, 1 << 30)
    ob.pack(0, 1 << 30)
    acc = [0.0, 0.0]  # summed per-step drift numerators sum|W(t) - W(t-1)|
    for t in range(1, 6):
        la.step([1.0, 0.3])
        lb.step([1.0, 0.3])
        for l in range(2):
            g = [s for s in la.segs if s.layer == l]
            acc[l] += O.layer_update_score([s.weight for s in g], [s.shadow for s in g], O.DT_BF16, 0.0)[0]
        oa.score(t)
        ob.score(t)
        if t == 1:  # first step after a persist: both modes see the same drift
            assert oa.delta == ob.delta and oa.delta[0] > 0
        oa.select(t, 1.0)
        ob.select(t, 1.0)
    # triangle inequality: distance to the last persisted weights (SNAPSHOT's
    # numerator) is bounded by the summed per-step distances
    for l in range(2):
        g = [s for s in lb.segs if s.layer == l]
        a_snap = O.layer_update_score([s.weight for s in g], [s.shadow for s in g], O.DT_BF16, 0.0)[0]
        assert 0 < a_snap <= acc[l] * (1 + 1e-12)


# ------------------------------------------------------ bf16 weight copy ----
# Section 4.1: every checkpoint stores a bf16 copy of the weights, and the
# fused optimizer step (Section 3.4) writes those weights back from its fp32
# parameters.  Converting fp32 to bf16 keeps the sign, the 8 exponent bits
# and the top 7 fraction bits; the 16 dropped bits decide the rounding, to
# the nearest representable value and, on an exact tie (dropped bits
# 0x8000), to the neighbour whose last kept bit is 0.  Each case below is
# worked out by hand from that rule: (fp32 bits, bf16 bits).
BF16_CASES = [
    (0x3F800000, 0x3F80),  # 1.0 is exact
    (0x3F808000, 0x3F80),  # tie between 0x3F80 (even) and 0x3F81
    (0x3F818000, 0x3F82),  # tie between 0x3F81 and 0x3F82 (even)
    (0xBF808000, 0xBF80),  # the same ties, negated
    (0xBF818000, 0xBF82),
    (0x3F808001, 0x3F81),  # just above a tie rounds up
    (0x3F807FFF, 0x3F80),  # just below a tie rounds down
    (0x3F81FFFF, 0x3F82),  # carry into the kept bits
    (0x3FFF8000, 0x4000),  # tie to even carries into the exponent
    (0x7F7F7FFF, 0x7F7F),  # large finite, rounds down
    (0x7F7FFFFF, 0x7F80),  # FLT_MAX rounds up to +inf
    (0x7F7F8000, 0x7F80),  # tie between 0x7F7F and +inf (even)
    (0xFF7FFFFF, 0xFF80),  # -FLT_MAX rounds to -inf
    (0x00000000, 0x0000),  # +0
    (0x80000000, 0x8000),  # -0 keeps its sign
    (0x7F800000, 0x7F80),  # +inf
    (0xFF800000, 0xFF80),  # -inf
    (0x00000001, 0x0000),  # smallest subnormal rounds to +0
    (0x00008000, 0x0000),  # subnormal tie to even (0)
    (0x00018000, 0x0002),  # subnormal tie to even (2)
    (0x80018000, 0x8002),
    (0x007FFFFF, 0x0080),  # largest subnormal rounds up to the smallest normal
    (0x00400000, 0x0040),  # a subnormal that is exact in bf16
    (0x7FC00000, 0x7FC0),  # NaN: the quiet pattern
    (0x7F800001, 0x7FC0),  # a signalling NaN whose payload would round into +inf
    (0xFFC00000, 0x7FC0),  # a negative NaN
    (0xFFFFFFFF, 0x7FC0),
]


def check_bf16_round(bf16_round):
    bits = np.array([c[0] for c in BF16_CASES], dtype=np.uint32)
    got = bf16_round(bits.view(np.float32))
    assert got.dtype == np.uint16 and got.shape == bits.shape
    for (x, want), g in zip(BF16_CASES, got.tolist()):
        assert g == want, f"fp32 {x:#010x}: got {g:#06x}, want {want:#06x}"
    # Against an independent implementation: torch's fp32 -> bf16 conversion,
    # over random bit patterns (every exponent, both signs, subnormals, inf,
    # NaN), exact ties of both parities and their neighbours.  torch writes
    # NaN as 0xFFFF; the oracle writes the quiet NaN 0x7FC0 (checked above),
    # so NaN inputs need only give a NaN here.
    import torch
    rng = np.random.default_rng(2609)
    rand = rng.integers(0, 1 << 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    hi = rng.integers(0, 1 << 16, size=1 << 16, dtype=np.uint64).astype(np.uint32) << np.uint32(16)
    ties = np.concatenate([hi | np.uint32(0x8000), hi | np.uint32(0x7FFF), hi | np.uint32(0x8001), hi])
    bits = np.concatenate([rand, ties])
    x = bits.view(np.float32)
    got = bf16_round(x)
    want = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(x)
    assert nan.any() and np.array_equal(got[~nan], want[~nan])
    assert np.all(got[nan] == 0x7FC0)
    # and the value view: each result is one of the two bf16 neighbours of x,
    # the nearer one (finite, non-overflowing inputs)
    with np.errstate(invalid="ignore"):  # signalling NaNs raise the flag when widened
        fin = np.isfinite(x) & (np.abs(x.astype(np.float64)) < 3.38e38)
    xv = x[fin].astype(np.float64)
    gv = (got[fin].astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    down = ((bits[fin] >> np.uint32(16)) << np.uint32(16)).view(np.float32).astype(np.float64)
    up = (((bits[fin] >> np.uint32(16)) + np.uint32(1)) << np.uint32(16)).view(np.float32).astype(np.float64)
    assert np.all((gv == down) | (gv == up))
    assert np.all(np.abs(gv - xv) <= np.minimum(np.abs(down - xv), np.abs(up - xv)))


# ------------------------------------------------ the parity-protocol resync -
def _resync_pair(cls, mode, k0_a, k0_b):
    """Two identical three-layer states; W moves by 2^-8 from 0.5, so every
    layer scores u = 2^-7 exactly at step 1 (eps_w = 0)."""
    out = []
    for k0 in (k0_a, k0_b):
        segs = _const_layout(3)
        orc = cls(segs, 3, O.DT_F32, True, mode, k0, s_max=100, eps_w=0.0)
        orc.pack(0, 1 << 30)
        for s in segs:
            s.weight[...] = 0.5 + 2.0 ** -8
        orc.score(1)
        orc.select(1, 1.0)
        out.append((orc, segs))
    return out


def _same_state(a, b, segs_a, segs_b):
    assert a.delta == b.delta, (a.delta, b.delta)
    assert a.t_last == b.t_last, (a.t_last, b.t_last)
    assert np.array_equal(a.mask, b.mask), (a.mask, b.mask)
    assert a.unpacked == b.unpacked, (a.unpacked, b.unpacked)
    pa, ra = a.pack(0, 1 << 30)
    pb, rb = b.pack(0, 1 << 30)
    assert np.array_equal(pa, pb) and ra == rb
    for x, y in zip(segs_a, segs_b):
        assert np.array_equal(x.shadow, y.shadow)
    # one more step: the accumulators carry on from the same values
    for segs in (segs_a, segs_b):
        for s in segs:
            s.weight[...] = 0.5 + 2.0 ** -7
    a.score(2)
    b.score(2)
    assert a.delta == b.delta and a.u == b.u


def check_resync(cls):
    """The parity protocol lets the oracle adopt the other side's decision on
    a layer whose accumulator lies within the tolerance band of K.  Adopting
    a decision must leave exactly the state that taking it directly leaves:
    persisting resets Delta and t_l (Eq. 4) and the layer joins the pack;
    not persisting keeps the accumulated Delta and the older t_l."""
    never, always = 1e300, 0.0
    for mode in (O.MODE_ACCUM, O.MODE_SNAPSHOT):
        # persist layer 1 by resync == persist it by drift
        (direct, sd), (adopted, sa) = _resync_pair(cls, mode, [never, always, never], [never, never, never])
        assert list(adopted.mask) == [0, 0, 0]
        adopted.resync(1, True)
        _same_state(direct, adopted, sd, sa)
        # drop layer 1 by resync == never select it
        (direct, sd), (adopted, sa) = _resync_pair(cls, mode, [never, never, always], [never, always, always])
        assert list(adopted.mask) == [0, 1, 1]
        adopted.resync(1, False)
        assert adopted.delta[1] == 2.0 ** -7  # the accumulated drift is back
        _same_state(direct, adopted, sd, sa)
        # adopting the decision already taken changes nothing
        (direct, sd), (adopted, sa) = _resync_pair(cls, mode, [never, always, never], [never, always, never])
        adopted.resync(0, False)
        adopted.resync(1, True)
        _same_state(direct, adopted, sd, sa)
    segs = _const_layout(2)
    orc = cls(segs, 2, O.DT_F32, True, O.MODE_ACCUM, [1.0, 1.0], s_max=100)
    orc.pack(0, 1 << 30)
    orc.score(1)
    expect_error(lambda: orc.resync(0, True), O.LC_ERR_BAD_STATE)  # no selection to adjust


# -------------------------------------------- a selection must be packed ----
def check_unpacked_selection_blocks(cls):
    """Eq. 4 resets Delta and t_l of a selected layer as if it were persisted,
    so the next score or optimizer step refuses while a selection made by
    ``select`` or ``rebase`` has layers not yet packed (both modes; the state
    is left as it was), and goes ahead once the rest is packed.  The base
    pending at init resets nothing: in ACCUM mode a warm-up may leave it
    unpacked, while SNAPSHOT mode needs it packed first."""
    for mode in (O.MODE_ACCUM, O.MODE_SNAPSHOT):
        segs = _const_layout(3)
        orc = cls(segs, 3, O.DT_F32, True, mode, [0.0, 0.0, 1e300], s_max=100, eps_w=0.0)
        if mode == O.MODE_SNAPSHOT:
            expect_error(lambda: orc.score(1), O.LC_ERR_BAD_STATE)
        orc.pack(0, 1 << 30)
        for s in segs:
            s.weight[...] = 0.5 + 2.0 ** -8
        orc.score(1)
        mask, _ = orc.select(1, 1.0)
        assert list(mask) == [1, 1, 0]
        state = (list(orc.delta), list(orc.t_last))
        expect_error(lambda: orc.score(2), O.LC_ERR_BAD_STATE)
        orc.pack(0, orc.R[0])  # the first record only
        expect_error(lambda: orc.score(2), O.LC_ERR_BAD_STATE)
        if mode == O.MODE_ACCUM:
            grads = [np.zeros(3, np.float32) for _ in segs]
            expect_error(lambda: orc.sgd_step_score(2, grads, 1e-3, 0.0), O.LC_ERR_BAD_STATE)
        assert (list(orc.delta), list(orc.t_last)) == state
        orc.pack(1, 1 << 30)
        orc.score(2)
        # a base checkpoint taken again blocks the same way until packed
        orc.select(2, 1.0)
        orc.pack(0, 1 << 30)
        orc.rebase(2)
        expect_error(lambda: orc.score(3), O.LC_ERR_BAD_STATE)
        orc.pack(0, 1 << 30)
        orc.score(3)
    # ACCUM warm-up: the init base may stay unpacked; the first step drops it
    segs = _const_layout(2)
    orc = cls(segs, 2, O.DT_F32, True, O.MODE_ACCUM, [1e300, 1e300], s_max=100)
    orc.score(1)
    assert orc.unpacked == set()
    # ... and the base that ends the warm-up must be packed before the next step
    orc.rebase(1)
    expect_error(lambda: orc.score(2), O.LC_ERR_BAD_STATE)
    orc.pack(0, 1 << 30)
    orc.score(2)
    orc.select(2, 1.0)  # nothing is due: the next step goes ahead
    orc.score(3)
