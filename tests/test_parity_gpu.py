"""GPU parity: the HIP library through its C interface against the CPU oracle.

Sizes are chosen so the oracle finishes in seconds while the layouts still
span many score chunks and pack pieces (8 KiB each: 4096 bf16 / 2048 fp32
elements per chunk) with ragged tails; test_reduced_layouts_span_tiles
checks that against the tile sizes the library reports.
"""
import numpy as np
import pytest

from oracle import layercheck_oracle as O
from paper_2609_27193_amd import layercheck as LC
from paper_2609_27193_amd import inputs as I
from tests.conftest import gpu_available
from tests.gpu_harness import Pair, log, torch_bytes

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not gpu_available():
        pytest.skip("needs an MI355X")
    LC.load_library()  # a missing build fails here, loudly


def k0_for(spec, base):
    return [base * (10.0 if l.name == "embed_tokens" else 1.0) for l in spec.layers]


def reduced_8b():
    return I.scaled_spec(I.llama3_8b_spec(), hidden=256, ffn=896, n_blocks=4, vocab=1003, n_q=8, n_kv=2)


def reduced_qwen():
    return I.scaled_spec(I.qwen25_14b_spec(), hidden=320, ffn=864, n_blocks=3, vocab=777, n_q=5, n_kv=1,
                         qkv_bias=True)


def reduced_13b():
    return I.scaled_spec(I.llama2_13b_spec(), hidden=320, ffn=864, n_blocks=4, vocab=641, n_q=5, n_kv=5)


def run_steps(p, steps, lr=lambda t: 1.0, capacity=None, stats=None):
    fracs = []
    for t in steps:
        mask, st = p.step(t, lr(t), capacity(t) if capacity else None)
        fracs.append(mask.mean())
        if stats is not None:
            stats.append(st)
        log(f"  step {t}: selected {st['n_selected']}/{p.N} forced {st['n_forced']} "
            f"payload {st['payload_bytes']} max_age {st['max_age']} w_age {st['weighted_age']:.3f}")
    return fracs


def assert_both_rules_fired(stats):
    """Some layer was persisted by its accumulated drift (Eq. 3) and some only
    by the staleness guard (Section 3.3) during the run."""
    assert any(st["n_selected"] > st["n_forced"] for st in stats), stats
    assert any(st["n_forced"] > 0 for st in stats), stats


@pytest.mark.parametrize("mode", [LC.LC_MODE_ACCUM, LC.LC_MODE_SNAPSHOT], ids=["accum", "snapshot"])
def test_toy_ten_steps(mode):
    """The toy decoder (fp32 weights, 3.67M params, S_max = 4) for 10 steps;
    K0 = 0.02 persists about a quarter of the layers per step, by drift on
    some steps and by the staleness guard on others."""
    spec = I.toy_spec()
    log(f"toy mode={mode}")
    p = Pair(spec, mode, k0_for(spec, 0.02))
    try:
        p.pack(0, np.ones(p.N, np.uint8))  # base version
        stats = []
        fracs = run_steps(p, range(1, 11), stats=stats)
        log(f"  mean selected fraction {np.mean(fracs):.3f}; near-threshold excluded {p.near_excluded}, "
            f"resyncs {p.resyncs}")
        assert 0.15 <= np.mean(fracs) <= 0.35
        assert_both_rules_fired(stats)
        p.check_arrays()
    finally:
        p.close()


@pytest.mark.parametrize("maker,mode", [(reduced_8b, LC.LC_MODE_ACCUM), (reduced_8b, LC.LC_MODE_SNAPSHOT),
                                        (reduced_qwen, LC.LC_MODE_ACCUM), (reduced_13b, LC.LC_MODE_SNAPSHOT)],
                         ids=["8b-accum", "8b-snapshot", "qwen-accum", "13b-snapshot"])
def test_reduced_bf16(maker, mode):
    """bf16 weights (with and without master), learning-rate scaling and
    capacity-limited packing in several calls."""
    spec = maker()
    log(f"{spec.name} mode={mode} P={spec.numel}")
    p = Pair(spec, mode, k0_for(spec, 0.01))
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        cap = lambda t: (max(p.R) + 4096) if t % 3 == 0 else None  # several pack calls on some steps
        stats = []
        run_steps(p, range(1, 13), lr=lambda t: 1.0 if t < 6 else 0.5, capacity=cap, stats=stats)
        assert_both_rules_fired(stats)
        assert p.max_pack_calls > 1
        p.check_arrays()
    finally:
        p.close()


def _restore_and_compare(p, t_fail, where):
    import torch
    versions_c, versions_o = [], []
    keep = []
    for (step, mask, dev), (_, _, host) in zip(p.versions_dev, p.versions_host):
        if where == "device":
            ptr = dev.data_ptr() if dev is not None else 0
        elif where == "pinned":
            t = torch.from_numpy(host).pin_memory() if len(host) else None
            keep.append(t)
            ptr = t.data_ptr() if t is not None else 0
        else:
            arr = np.ascontiguousarray(host)
            keep.append(arr)
            ptr = arr.ctypes.data if len(arr) else 0
        versions_c.append({"step": step, "mask": mask, "payload": ptr, "payload_bytes": len(host)})
        versions_o.append({"step": step, "mask": mask, "payload": host})
    # fail-stop: the live state is lost on both sides
    for t in (p.dW, p.dS, p.dm, p.dv) + ((p.dM,) if p.dM is not None else ()):
        t.fill_(0)
    for a in (p.hW, p.hS, p.hm, p.hv) + ((p.hM,) if p.hM is not None else ()):
        a[...] = 0
    torch.cuda.synchronize()
    chosen = LC.lc_restore_composite(p.ctx, versions_c, t_fail, p.N)
    chosen_o = p.orc.restore(versions_o, t_fail)
    assert chosen.tolist() == chosen_o.tolist()
    p.check_arrays()
    u, d, tl = LC.lc_read_state(p.ctx, p.N)
    assert tl.tolist() == chosen.tolist() and not d.any()
    return chosen


@pytest.mark.parametrize("where", ["device", "pinned", "pageable"])
def test_restore_composite_then_continue(where):
    """Mixed-timestamp recovery (Section 3.5) from versions held in device,
    pinned-host and pageable-host memory; training then resumes after t_fail
    and both sides keep agreeing."""
    spec = reduced_8b()
    p = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 0.01))
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        run_steps(p, range(1, 9))
        t_fail = 6
        chosen = _restore_and_compare(p, t_fail, where)
        log(f"  restored from steps {sorted(set(chosen.tolist()))}")
        assert len(set(chosen.tolist())) >= 2
        with pytest.raises(LC.LCError) as e:  # the resumed run starts after t_fail
            LC.lc_score_layers(p.ctx, t_fail)
        assert e.value.code == LC.LC_ERR_BAD_STATE
        p.adopt_restored()  # resume from the composite state
        run_steps(p, range(t_fail + 1, t_fail + 4))
    finally:
        p.close()


@pytest.mark.parametrize("mode", [LC.LC_MODE_ACCUM, LC.LC_MODE_SNAPSHOT], ids=["accum", "snapshot"])
def test_long_horizon_lr_schedule(mode):
    """120 decision steps, about 15 staleness periods (S_max = 8), with a
    cosine learning-rate schedule from lr_0 to 0.1 lr_0 driving the
    threshold K(t) = K0 s(lr(t)) (Eq. 3).  At every step both sides agree
    (u and Delta within 1e-5, masks, stats, payloads and shadow exact), so the
    accumulators stay in step over many persist cycles; the staleness bound
    holds at every step (Section 3.3); both rules fire; as K falls, more
    layers are persisted by drift in the last stretch than in the first.  A
    composite restore from the whole history at a mid-schedule t_fail then
    matches the oracle (mixed timestamps, all within the staleness bound),
    and the run resumes from it."""
    import math
    spec = reduced_8b()
    T = 120
    p = Pair(spec, mode, k0_for(spec, 0.01))
    lr = lambda t: 0.1 + 0.9 * 0.5 * (1.0 + math.cos(math.pi * t / T))
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        stats = []
        run_steps(p, range(1, T + 1), lr=lr, stats=stats)
        assert all(st["max_age"] <= spec.s_max - 1 for st in stats)
        assert_both_rules_fired(stats)
        by_drift = [st["n_selected"] - st["n_forced"] for st in stats]
        assert sum(by_drift[-30:]) > sum(by_drift[:30]), by_drift
        log(f"  {T} steps: drift-selected layer-steps {sum(by_drift)}, forced "
            f"{sum(st['n_forced'] for st in stats)}; near-threshold excluded {p.near_excluded}, "
            f"resyncs {p.resyncs}")
        t_fail = T // 2 + 3  # mid-schedule; later, K is so low that nearly every layer persists each step
        chosen = _restore_and_compare(p, t_fail, "device")
        log(f"  restored at t_fail={t_fail} from steps {sorted(set(chosen.tolist()))}")
        assert len(set(chosen.tolist())) >= 2
        assert min(chosen.tolist()) >= t_fail - spec.s_max + 1  # every layer within the staleness bound
        p.adopt_restored()
        run_steps(p, range(t_fail + 1, t_fail + 4), lr=lr)
    finally:
        p.close()


@pytest.mark.parametrize("mode", [LC.LC_MODE_ACCUM, LC.LC_MODE_SNAPSHOT], ids=["accum", "snapshot"])
def test_decisions_at_irregular_steps(mode):
    """The weights move every iteration, decisions come only at steps 1, 2,
    5, 6, 7, 19, 20 and 35 (S_max = 8).  A score after skipped iterations
    measures the change since the previous scored step (ACCUM) or since the
    last persist (SNAPSHOT), on both sides alike; a gap of S_max or more
    forces every layer that drift did not select (Section 3.3), leaving
    every layer's age 0 after the decision."""
    spec = reduced_8b()
    assert spec.s_max == 8
    decisions = {1, 2, 5, 6, 7, 19, 20, 35}
    p = Pair(spec, mode, k0_for(spec, 0.01))
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        stats = {}
        for t in range(1, max(decisions) + 1):
            if t in decisions:
                mask, st = p.step(t)
                stats[t] = st
                log(f"  step {t}: selected {st['n_selected']}/{p.N} forced {st['n_forced']} "
                    f"max_age {st['max_age']}")
            else:
                p.advance(t)  # an iteration with no decision
        for t in (19, 35):  # 12 and 15 iterations since the previous decision
            assert stats[t]["n_selected"] == p.N and stats[t]["max_age"] == 0, (t, stats[t])
        assert any(st["n_forced"] > 0 for st in stats.values())
        p.check_arrays()
    finally:
        p.close()


@pytest.mark.parametrize("mode", [LC.LC_MODE_ACCUM, LC.LC_MODE_SNAPSHOT], ids=["accum", "snapshot"])
def test_rebase_mid_run_then_restore(mode):
    """A full base checkpoint in the middle of a run (Section 3.4's base,
    taken again after an unscored stretch): Delta and t_l reset, the shadow
    re-synchronised and every layer packed, both sides alike; the decisions
    after it agree, and a composite restore never reaches back past it."""
    spec = reduced_8b()
    p = Pair(spec, mode, k0_for(spec, 0.01))
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        run_steps(p, range(1, 4))
        p.advance(4)  # the weights move with no decision at step 4
        p.pack(4, p.rebase(4))
        run_steps(p, range(5, 9))
        chosen = _restore_and_compare(p, 7, "device")
        log(f"  restored from steps {sorted(set(chosen.tolist()))}")
        assert min(chosen.tolist()) >= 4
        p.adopt_restored()
        run_steps(p, range(8, 10))
    finally:
        p.close()


def _mean_scores(spec, steps):
    """Per-layer mean of u over the first ``steps`` steps of the synthetic
    trajectory, from an oracle-only dry run (no selection by drift)."""
    from tests.gpu_harness import to_numpy_weight
    g = I.SyntheticState(spec, device="cpu")
    hW = to_numpy_weight(g.weight)
    hS = np.zeros_like(hW)
    hM = None if g.master is None else g.master.numpy().copy()
    hm, hv = g.exp_avg.numpy().copy(), g.exp_avg_sq.numpy().copy()
    segs = [O.OSegment(s.layer, hW[s.offset:s.offset + s.numel], hS[s.offset:s.offset + s.numel],
                       None if hM is None else hM[s.offset:s.offset + s.numel],
                       hm[s.offset:s.offset + s.numel], hv[s.offset:s.offset + s.numel]) for s in g.segments]
    dt = O.DT_BF16 if spec.weight_dtype == "bf16" else O.DT_F32
    orc = O.LayerCheckOracle(segs, spec.n_layers, dt, spec.has_master, O.MODE_ACCUM,
                             [float("inf")] * spec.n_layers, 10 ** 9)
    us = []
    for t in range(1, steps + 1):
        g.step(t)
        hW[...] = to_numpy_weight(g.weight)
        orc.score(t)
        us.append(list(orc.u))
        orc.select(t, 1.0)
    return np.mean(us, axis=0)


def test_restore_five_timestamps():
    """A composite of five different timestamps (Section 3.5): per-layer
    thresholds give each layer its own persist period (every 1, 2, 3, 4 and 5
    steps; the final norm only by the S_max = 6 guard), twelve versions on
    the device, recovery at t_fail = 11 mixes steps 6, 8, 9, 10 and 11."""
    spec = reduced_qwen()
    names = [l.name for l in spec.layers]
    assert names == ["embed_tokens", "block_0", "block_1", "block_2", "norm", "lm_head"]
    u = _mean_scores(spec, 4)
    period = {"embed_tokens": 2, "block_0": 3, "block_1": 4, "block_2": 5, "lm_head": 1}
    k0 = [u[l] * (period[n] - 0.5) if n in period else 1e9 for l, n in enumerate(names)]
    p = Pair(spec, LC.LC_MODE_ACCUM, k0)
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        run_steps(p, range(1, 13))
        chosen = _restore_and_compare(p, 11, "device")
        assert sorted(set(chosen.tolist())) == [6, 8, 9, 10, 11], chosen
        assert chosen.tolist() == [10, 9, 8, 10, 6, 11]
    finally:
        p.close()


def test_restore_roundtrip_repack():
    """Restore, then re-pack every layer: each record equals the record it was
    restored from, bit for bit."""
    import torch
    spec = reduced_qwen()
    p = Pair(spec, LC.LC_MODE_SNAPSHOT, k0_for(spec, 0.01))
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        run_steps(p, range(1, 7))
        chosen = _restore_and_compare(p, 5, "device")
        lay2 = LC.LayoutDesc(p.lsegs, p.N, p.dtype, spec.has_master, LC.LC_MODE_SNAPSHOT, p.k0,
                             spec.s_max, stream=p.stream)
        ctx2 = LC.lc_init_layout(lay2)
        try:
            total = sum(p.R)
            st = torch.empty(total, dtype=torch.uint8, device="cuda")
            res = LC.lc_pack_selected(ctx2, st.data_ptr(), total, 0)
            assert res["done"] == 1 and res["bytes_written"] == total
            allrec = torch_bytes(st)
            pos = 0
            for l in range(p.N):
                v = [vv for vv in p.versions_host if vv[0] == chosen[l]][0]
                off = sum(p.R[j] for j in range(l) if v[1][j])
                assert np.array_equal(allrec[pos:pos + p.R[l]], v[2][off:off + p.R[l]]), l
                pos += p.R[l]
        finally:
            LC.lc_destroy(ctx2)
    finally:
        p.close()


def test_state_machine_errors():
    import torch
    spec = reduced_8b()
    p = Pair(spec, LC.LC_MODE_SNAPSHOT, k0_for(spec, 0.01))
    try:
        def expect(code, fn):
            with pytest.raises(LC.LCError) as e:
                fn()
            assert e.value.code == code, str(e.value)
        B, I_, C_, NV = LC.LC_ERR_BAD_STATE, LC.LC_ERR_INVALID_ARG, LC.LC_ERR_CAPACITY, LC.LC_ERR_NO_VERSION
        expect(B, lambda: LC.lc_score_layers(p.ctx, 1))        # base not packed (SNAPSHOT)
        expect(B, lambda: LC.lc_select(p.ctx, 1, 1.0, p.N))    # select before score
        st = torch.empty(max(p.R), dtype=torch.uint8, device="cuda")
        expect(C_, lambda: LC.lc_pack_selected(p.ctx, st.data_ptr(), min(p.R) - 1, 0))
        expect(I_, lambda: LC.lc_pack_selected(p.ctx, st.data_ptr() + 16, max(p.R), 0))  # misaligned staging
        expect(I_, lambda: LC.lc_pack_selected(p.ctx, st.data_ptr(), max(p.R), p.N + 1))
        p.pack(0, np.ones(p.N, np.uint8))
        p.advance(1)
        p.score(1)
        expect(B, lambda: LC.lc_pack_selected(p.ctx, st.data_ptr(), max(p.R), 0))  # nothing selected yet
        for bad in (0.0, -1.0, float("nan"), float("inf")):
            expect(I_, lambda: LC.lc_select(p.ctx, 1, bad, p.N))
        expect(B, lambda: LC.lc_select(p.ctx, 2, 1.0, p.N))
        expect(B, lambda: LC.lc_score_layers(p.ctx, 1))        # not increasing
        d, tl = LC.lc_read_state(p.ctx, p.N)[1:]
        mask, _ = p.select(1, 1.0, d, tl)
        expect(B, lambda: LC.lc_select(p.ctx, 1, 1.0, p.N))   # one select per score
        p.pack(1, mask)
        # restore errors
        full = np.ones(p.N, np.uint8)
        dev = p.versions_dev[0][2]
        v0 = {"step": 0, "mask": full, "payload": dev.data_ptr(), "payload_bytes": sum(p.R)}
        expect(NV, lambda: LC.lc_restore_composite(p.ctx, [v0], -1, p.N))
        expect(I_, lambda: LC.lc_restore_composite(p.ctx, [v0, dict(v0)], 3, p.N))
        expect(I_, lambda: LC.lc_restore_composite(p.ctx, [dict(v0, payload_bytes=sum(p.R) - 256)], 3, p.N))
        expect(I_, lambda: LC.lc_restore_composite(p.ctx, [], 3, p.N))
        expect(B, lambda: LC.lc_rebase(p.ctx, 0))              # a base before the last step
        p.check_arrays()  # failed calls changed nothing
    finally:
        p.close()


@pytest.mark.parametrize("mode", [LC.LC_MODE_ACCUM, LC.LC_MODE_SNAPSHOT], ids=["accum", "snapshot"])
def test_unpacked_selection_blocks_the_next_step(mode):
    """Eq. 4 resets Delta and t_l of a selected layer as if it were persisted,
    so a selection must be packed in full before the next score or optimizer
    step: both sides refuse (LC_ERR_BAD_STATE, state unchanged) while a record
    is missing, also after a base taken again with lc_rebase, and continue in
    parity once the rest is packed."""
    import torch
    spec = reduced_8b()
    p = Pair(spec, mode, k0_for(spec, 0.0))  # K0 = 0: every layer persists by drift every step
    try:
        def refused(fn_lib, fn_orc):
            with pytest.raises(LC.LCError) as e:
                fn_lib()
            assert e.value.code == LC.LC_ERR_BAD_STATE, str(e.value)
            with pytest.raises(O.OracleError) as e:
                fn_orc()
            assert e.value.code == O.LC_ERR_BAD_STATE

        p.pack(0, np.ones(p.N, np.uint8))
        p.advance(1)
        d, tl = p.score(1)
        mask, _ = p.select(1, 1.0, d, tl)
        assert mask.all()
        state = LC.lc_read_state(p.ctx, p.N)
        # one record packed, the rest not
        st = torch.empty(p.R[0], dtype=torch.uint8, device="cuda")
        res = LC.lc_pack_selected(p.ctx, st.data_ptr(), p.R[0], 0)
        pay_o, res_o = p.orc.pack(0, p.R[0])
        assert res == res_o and not res["done"]
        torch.cuda.synchronize()
        assert np.array_equal(torch_bytes(st), pay_o)
        p.advance(2)
        refused(lambda: LC.lc_score_layers(p.ctx, 2), lambda: p.orc.score(2))
        if mode == LC.LC_MODE_ACCUM:
            g = torch.zeros(spec.numel, dtype=torch.bfloat16, device="cuda")
            ptrs = [g[s.offset:s.offset + s.numel].data_ptr() for s in p.gen.segments]
            grads = [np.zeros(s.numel, np.float32) for s in p.gen.segments]
            refused(lambda: LC.lc_sgd_step_score(p.ctx, 2, ptrs, LC.LC_DT_BF16, 1e-3, 0.0),
                    lambda: p.orc.sgd_step_score(2, grads, 1e-3, 0.0))
        after = LC.lc_read_state(p.ctx, p.N)
        for a, b in zip(state, after):
            assert np.array_equal(a, b)
        # the rest of the selection, then the step goes ahead in parity
        total = sum(p.R[1:])
        st = torch.empty(total, dtype=torch.uint8, device="cuda")
        res = LC.lc_pack_selected(p.ctx, st.data_ptr(), total, 1)
        pay_o, res_o = p.orc.pack(1, total)
        assert res == res_o and res["done"]
        torch.cuda.synchronize()
        assert np.array_equal(torch_bytes(st), pay_o)
        p.check_arrays()
        d, tl = p.score(2)
        mask, _ = p.select(2, 1.0, d, tl)
        p.pack(2, mask)
        # a base taken again blocks the same way until it is packed
        p.rebase(2)
        p.advance(3)
        refused(lambda: LC.lc_score_layers(p.ctx, 3), lambda: p.orc.score(3))
        p.pack(2, np.ones(p.N, np.uint8))
        p.step(3)
    finally:
        p.close()


def test_scores_bitwise_reproducible_and_zero_change():
    """No floating-point atomics: two contexts over identical inputs give
    bit-identical scores; an unchanged state scores exactly zero."""
    spec = reduced_8b()
    pa = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 1e9))
    pb = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 1e9))
    try:
        for p in (pa, pb):
            p.pack(0, np.ones(p.N, np.uint8))
            p.score(1)  # no update since init: u == 0 exactly on both sides
            assert not LC.lc_read_state(p.ctx, p.N)[0].any()
            p.select(1, 1.0)
            p.advance(2)
            p.score(2)
        ua = LC.lc_read_state(pa.ctx, pa.N)[0]
        ub = LC.lc_read_state(pb.ctx, pb.N)[0]
        assert ua.any() and np.array_equal(ua.view(np.uint64), ub.view(np.uint64))
    finally:
        pa.close()
        pb.close()


def tied_spec():
    """Tied lm_head (Section 2.2): N = B + 2 layer groups, as for the paper's
    Qwen2.5-3B and Llama-3.2-1B; reduced width."""
    return I.ModelSpec(name="tied-reduced", layers=I._decoder_layers(192, 512, 3, 500, 6, 2, tied=True),
                       weight_dtype="bf16", has_master=True, scale_rule="loguniform_2dec_embed0.1",
                       target_fraction=0.2, s_max=4)


@pytest.mark.parametrize("mode", [LC.LC_MODE_ACCUM, LC.LC_MODE_SNAPSHOT], ids=["accum", "snapshot"])
def test_weights_only_records_sgd_variant(mode):
    """Records without Adam moments (Section 4.7), capacity-limited packs and a
    composite restore, against the oracle."""
    spec = reduced_8b()
    p = Pair(spec, mode, k0_for(spec, 0.01), moments=False)
    try:
        assert p.R == [O.record_bytes([t.numel for t in l.tensors], 2, True, has_moments=False)
                       for l in spec.layers]
        p.pack(0, np.ones(p.N, np.uint8))
        run_steps(p, range(1, 7), capacity=lambda t: max(p.R) if t % 2 else None)
        _restore_and_compare(p, 5, "device")
    finally:
        p.close()


def test_tied_embedding_layout():
    spec = tied_spec()
    assert spec.n_layers == 3 + 2
    p = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 0.01))
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        run_steps(p, range(1, 6))
        p.check_arrays()
    finally:
        p.close()
