"""GPU edge cases: odd tensor sizes (every later segment lands on a
misaligned address, so the element-wise paths of the score and copy kernels
run), tiny layouts, degenerate thresholds and a single segment larger than
4 GiB (64-bit offsets), checked against the oracle or against closed forms."""
import numpy as np
import pytest

from oracle import layercheck_oracle as O
from paper_2609_27193_amd import inputs as I
from paper_2609_27193_amd import layercheck as LC
from tests.conftest import gpu_available
from tests.gpu_harness import Pair, log
from tests.test_parity_gpu import assert_both_rules_fired

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not gpu_available():
        pytest.skip("needs an MI355X")
    LC.load_library()


def odd_spec(weight_dtype, has_master, s_max=3):
    T = I.TensorSpec
    layers = (
        I.LayerSpec("embed_tokens", (T("e", 4097, "embed"),)),
        I.LayerSpec("block_0", tuple(T(f"t{i}", n, "matrix") for i, n in enumerate((1, 3, 7, 8, 1023, 8193)))),
        I.LayerSpec("block_1", (T("a", 8191, "matrix"), T("b", 8192, "matrix"), T("n", 5, "norm"))),
        I.LayerSpec("norm", (T("n", 1, "norm"),)),
        I.LayerSpec("lm_head", (T("h", 3 * 8192 + 3, "embed"),)),
    )
    return I.ModelSpec(name=f"odd-{weight_dtype}-{int(has_master)}", layers=layers, weight_dtype=weight_dtype,
                       has_master=has_master, scale_rule="loguniform_0.01_1", target_fraction=0.3, s_max=s_max)


@pytest.mark.parametrize("dtype,master,mode", [("bf16", True, LC.LC_MODE_ACCUM), ("bf16", False, LC.LC_MODE_SNAPSHOT),
                                               ("f32", False, LC.LC_MODE_ACCUM), ("f32", True, LC.LC_MODE_SNAPSHOT)])
def test_odd_sizes_misaligned(dtype, master, mode):
    spec = odd_spec(dtype, master)
    p = Pair(spec, mode, [0.02] * spec.n_layers)  # both the threshold and the guard fire
    try:
        aligned = [seg.weight % 16 == 0 for seg in p.lsegs]
        assert not all(aligned), "layout should contain misaligned segments"
        p.pack(0, np.ones(p.N, np.uint8), capacity=max(p.R))
        stats = [p.step(t, capacity=max(p.R) if t % 2 else None)[1] for t in range(1, 8)]
        assert_both_rules_fired(stats)
        p.check_arrays()
    finally:
        p.close()


def test_single_layer_smax_one():
    T = I.TensorSpec
    spec = I.ModelSpec(name="one", layers=(I.LayerSpec("block_0", (T("w", 777, "matrix"),)),), weight_dtype="bf16",
                       has_master=True, scale_rule="constant_1", target_fraction=1.0, s_max=1)
    p = Pair(spec, LC.LC_MODE_ACCUM, [1e300])
    try:
        p.pack(0, np.ones(1, np.uint8))
        for t in range(1, 5):
            mask, st = p.step(t)
            assert mask.tolist() == [1] and st["n_forced"] == 1 and st["max_age"] == 0
    finally:
        p.close()


def test_all_zero_layer_with_eps_zero():
    """A layer whose weights are zero and stay zero while the others move.
    With eps_w = 0, Eq. 1 is 0/0 for it from the second step on: both sides
    give NaN, its accumulator stays NaN, the drift rule never fires for it and
    the staleness guard still persists it every S_max steps."""
    from tests.test_parity_gpu import reduced_8b
    spec = reduced_8b()
    z = 1  # block_0
    p = Pair(spec, LC.LC_MODE_ACCUM, [1e-30] * spec.n_layers, eps_w=0.0)
    try:
        a, b = p.gen.layer_range(z)

        def zero():
            p.dW[a:b].zero_()
            p.hW[a:b] = 0
            if p.dM is not None:
                p.dM[a:b].zero_()
                p.hM[a:b] = 0
            p.torch.cuda.synchronize()

        zero()  # the shadow still holds the initial weights: u = 1 at step 1
        p.pack(0, np.ones(p.N, np.uint8))
        for t in range(1, 2 * spec.s_max + 2):
            p.advance(t)
            zero()
            d, tl = p.score(t)
            u = LC.lc_read_state(p.ctx, p.N)[0]
            if t == 1:
                assert u[z] == 1.0
            else:
                assert np.isnan(u[z]) and np.isnan(d[z])
            mask, st = p.select(t, 1.0, d, tl)
            due = (t - 1) % spec.s_max == 0
            assert mask[z] == 1 if due else mask[z] == 0, (t, mask)
            if due and t > 1:  # z's accumulator is NaN: only the guard can have selected it
                assert st["n_forced"] >= 1
            p.pack(t, mask)
        p.check_arrays()
    finally:
        p.close()


def test_threshold_zero_selects_everything_and_no_change_scores_zero():
    spec = odd_spec("bf16", True, s_max=1000)
    p = Pair(spec, LC.LC_MODE_ACCUM, [0.0] * spec.n_layers)
    try:
        p.pack(0, np.ones(p.N, np.uint8))
        d, tl = p.score(1)  # no update since init: every score exactly zero
        assert not any(d)
        mask, st = p.select(1, 1.0, d, tl)
        assert mask.all() and st["n_forced"] == 0  # Delta = 0 >= K = 0
        p.pack(1, mask)
    finally:
        p.close()


def test_segment_larger_than_4gib_closed_form():
    """One layer, one segment of 2^31 + 4099 bf16 elements (its fp32 arrays
    are 8.6 GB each).  S = 0.5 and W = 0.5 + 2^-8 everywhere give
    u = 2^-7 exactly (Eq. 1 with eps_w = 0: every partial sum is exact); the
    record must hold the arrays' bytes at the offsets of the format, and a
    restore from it must reproduce them."""
    import torch
    n = (1 << 31) + 4099
    dev = torch.device("cuda")
    log(f"large segment: {n} elements")
    W = torch.full((n,), 0.5, dtype=torch.bfloat16, device=dev)
    S = torch.empty_like(W)
    idx = torch.arange(n, dtype=torch.int64, device=dev)  # distinct bit patterns per element
    M = (idx & 0x7FFFFFFF).to(torch.int32).view(torch.float32)
    m = ((n - idx) & 0x7FFFFFFF).to(torch.int32).view(torch.float32)
    v = ((idx * 2654435761) & 0x7FFFFFFF).to(torch.int32).view(torch.float32)
    del idx
    seg = LC.Segment(0, n, W.data_ptr(), S.data_ptr(), M.data_ptr(), m.data_ptr(), v.data_ptr())
    lay = LC.LayoutDesc([seg], 1, LC.LC_DT_BF16, True, LC.LC_MODE_ACCUM, [2.0 ** -7], s_max=100, eps_w=0.0,
                        stream=torch.cuda.current_stream().cuda_stream)
    ctx = LC.lc_init_layout(lay)
    try:
        R = LC.lc_record_bytes(ctx, 0)
        assert R == O.record_bytes([n], 2, True)
        W.fill_(0.5 + 2.0 ** -8)
        LC.lc_score_layers(ctx, 1)
        u, d, _ = LC.lc_read_state(ctx, 1)
        assert u[0] == 2.0 ** -7 and d[0] == 2.0 ** -7
        assert torch.equal(S, W)  # ACCUM refreshed the shadow in the same pass
        mask, st = LC.lc_select(ctx, 1, 1.0, 1)
        assert mask.tolist() == [1] and st["n_forced"] == 0 and st["payload_bytes"] == R  # Delta == K persists
        staging = torch.empty(R, dtype=torch.uint8, device=dev)
        res = LC.lc_pack_selected(ctx, staging.data_ptr(), R, 0)
        assert res == {"bytes_written": R, "n_packed": 1, "next_rank": 1, "done": 1}
        torch.cuda.synchronize()
        offs = [0]
        for nb in (2 * n, 4 * n, 4 * n, 4 * n):
            offs.append(offs[-1] + O.padded(nb))
        assert offs[-1] == R
        blocks = [(W, 2 * n), (M, 4 * n), (m, 4 * n), (v, 4 * n)]
        for (arr, nb), off in zip(blocks, offs):
            assert torch.equal(staging[off:off + nb], arr.view(torch.uint8)), off
            assert not staging[off + nb:O.padded(nb) + off].any()
        # fail-stop, then restore from the device-resident record
        saved = [a.clone() for a in (W, M, m, v)]
        for a in (W, S, M, m, v):
            a.zero_()
        chosen = LC.lc_restore_composite(ctx, [{"step": 1, "mask": np.ones(1, np.uint8),
                                                "payload": staging.data_ptr(), "payload_bytes": R}], 1, 1)
        assert chosen.tolist() == [1]
        for a, b in zip((W, M, m, v), saved):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))
        assert torch.equal(S, W)
    finally:
        LC.lc_destroy(ctx)


def test_delta_accumulates_in_fp64():
    """Eq. 2 in fp64 on the device: one fp32 layer of 1024 elements at 1.0,
    doubled at step 1 (u = 1 exactly), then one element moved by one ulp of
    2.0 at step 2 (u = 2^-33 exactly).  K0 = 1 + 2^-34 is crossed only by an
    fp64 accumulator; the same construction pins the oracle."""
    import torch
    n = 1024
    dev = torch.device("cuda")
    W = torch.ones(n, dtype=torch.float32, device=dev)
    S = torch.empty_like(W)
    m = torch.zeros_like(W)
    v = torch.zeros_like(W)
    seg = LC.Segment(0, n, W.data_ptr(), S.data_ptr(), None, m.data_ptr(), v.data_ptr())
    lay = LC.LayoutDesc([seg], 1, LC.LC_DT_F32, False, LC.LC_MODE_ACCUM, [1.0 + 2.0 ** -34], s_max=100, eps_w=0.0,
                        stream=torch.cuda.current_stream().cuda_stream)
    ctx = LC.lc_init_layout(lay)
    try:
        R = LC.lc_record_bytes(ctx, 0)
        staging = torch.empty(R, dtype=torch.uint8, device=dev)
        assert LC.lc_pack_selected(ctx, staging.data_ptr(), R, 0)["done"] == 1  # the base
        W.fill_(2.0)
        LC.lc_score_layers(ctx, 1)
        mask, _ = LC.lc_select(ctx, 1, 1.0, 1)
        u, d, _ = LC.lc_read_state(ctx, 1)
        assert u[0] == 1.0 and mask.tolist() == [0]
        W[0] = 2.0 + 2.0 ** -22
        LC.lc_score_layers(ctx, 2)
        u, d, _ = LC.lc_read_state(ctx, 1)
        assert u[0] == 2.0 ** -33 and d[0] == 1.0 + 2.0 ** -33, (u[0], d[0])
        mask, st = LC.lc_select(ctx, 2, 1.0, 1)
        assert mask.tolist() == [1] and st["n_forced"] == 0
        assert LC.lc_pack_selected(ctx, staging.data_ptr(), R, 0)["done"] == 1
    finally:
        LC.lc_destroy(ctx)


def many_layer_spec(n_layers=1500, seed=11):
    """Many tiny layers of 1-3 tensors (1..300 elements each): the select
    kernel's per-layer loops and prefix tables, and packs of hundreds of
    records, at a layer count far above any model's."""
    T = I.TensorSpec
    rng = np.random.default_rng(seed)
    layers = tuple(
        I.LayerSpec(f"block_{l}", tuple(T(f"t{k}", int(rng.integers(1, 301)), "matrix")
                                        for k in range(int(rng.integers(1, 4)))))
        for l in range(n_layers))
    return I.ModelSpec(name=f"many-{n_layers}", layers=layers, weight_dtype="bf16", has_master=True,
                       scale_rule="loguniform_0.01_1", target_fraction=0.3, s_max=5)


@pytest.mark.parametrize("mode", [LC.LC_MODE_ACCUM, LC.LC_MODE_SNAPSHOT], ids=["accum", "snapshot"])
def test_many_layers(mode):
    spec = many_layer_spec()
    rng = np.random.default_rng(3)
    p = Pair(spec, mode, list(10.0 ** rng.uniform(-2.5, -0.5, spec.n_layers)))
    try:
        p.pack(0, np.ones(p.N, np.uint8), capacity=64 * 1024)
        sel = []
        for t in range(1, 9):
            mask, st = p.step(t, capacity=64 * 1024 if t % 2 else None)
            sel.append(st["n_selected"])
        log(f"  {p.N} layers: selected per step {sel}")
        assert min(sel) > 0 and max(sel) < p.N
        p.check_arrays()
    finally:
        p.close()


def test_layer_of_64_segments_and_restore():
    """A layer of 64 tensors (1..5000 elements: 64 blocks per array in its
    record), a one-element layer and a plain layer, six steps, then a
    composite restore from device versions."""
    from tests.test_parity_gpu import _restore_and_compare
    T = I.TensorSpec
    rng = np.random.default_rng(64)
    layers = (I.LayerSpec("block_0", tuple(T(f"t{k}", int(rng.integers(1, 5001)), "matrix") for k in range(64))),
              I.LayerSpec("norm", (T("n", 1, "norm"),)),
              I.LayerSpec("block_1", (T("w", 20000, "matrix"),)))
    spec = I.ModelSpec(name="seg64", layers=layers, weight_dtype="bf16", has_master=True,
                       scale_rule="loguniform_0.01_1", target_fraction=0.5, s_max=3)
    p = Pair(spec, LC.LC_MODE_ACCUM, [0.02, 1e300, 0.02])
    try:
        assert len([s for s in p.lsegs if s.layer == 0]) == 64
        p.pack(0, np.ones(p.N, np.uint8))
        for t in range(1, 7):
            p.step(t)
        chosen = _restore_and_compare(p, 5, "device")
        log(f"  restored from steps {chosen.tolist()}")
    finally:
        p.close()
