"""GPU: draining device staging into the persistence store and composite
recovery from it (Section 3.5), against the oracle; the recovery runs after
the store has been compacted to what a recovery at t_fail can use.

One staging buffer is reused every step with no synchronisation between
lc_store_append and the next lc_pack_selected: the drain's copies must be
stream-ordered before the next pack overwrites the buffer.  The overlapped
variant alternates two staging buffers with lc_store_append_async, and the
caller's stream waits only on the reuse event of the buffer it packs next.
Small drain buffers force many chunks through the pinned ring."""
import os

import numpy as np
import pytest

from oracle import layercheck_oracle as O
from paper_2609_27193_amd import layercheck as LC
from tests.conftest import gpu_available
from tests.gpu_harness import Pair, log, torch_bytes
from tests.test_parity_gpu import k0_for, reduced_8b, reduced_qwen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not gpu_available():
        pytest.skip("needs an MI355X")
    LC.load_library()


@pytest.mark.parametrize("maker,mode,buf,overlapped", [(reduced_8b, LC.LC_MODE_ACCUM, 1 << 20, False),
                                                       (reduced_qwen, LC.LC_MODE_SNAPSHOT, 3 << 20, False),
                                                       (reduced_8b, LC.LC_MODE_ACCUM, 4 << 20, True),
                                                       (reduced_qwen, LC.LC_MODE_SNAPSHOT, 64 << 20, True)],
                         ids=["8b-accum", "qwen-snapshot", "8b-accum-overlapped", "qwen-snapshot-overlapped"])
def test_drain_and_restore_from_store(tmp_path, maker, mode, buf, overlapped):
    import torch
    spec = maker()
    p = Pair(spec, mode, k0_for(spec, 0.01))
    d = str(tmp_path / "store")
    store = LC.Store(d, p.R, buffer_bytes=buf)
    try:
        cur = torch.cuda.current_stream()
        stream = cur.cuda_stream
        cap = sum(p.R)
        stagings = [torch.empty(cap, dtype=torch.uint8, device="cuda") for _ in range(2 if overlapped else 1)]
        events = [torch.cuda.Event() for _ in stagings]
        for ev in events:
            ev.record(cur)  # creates the underlying event
        expected = []

        def pack_and_drain(t, mask):
            k = t % len(stagings)
            staging = stagings[k]
            if overlapped:
                cur.wait_event(events[k])  # the copies out of this buffer's previous payload are done
            res = LC.lc_pack_selected(p.ctx, staging.data_ptr(), cap, 0)
            pay_o, res_o = p.orc.pack(0, cap)
            assert res == res_o
            if overlapped:
                store.append_async(t, mask, staging.data_ptr(), res["bytes_written"], stream, events[k].cuda_event)
            else:
                store.append(t, mask, staging.data_ptr(), res["bytes_written"], stream)  # no sync afterwards
            expected.append({"step": t, "mask": mask.copy(), "payload": pay_o})

        pack_and_drain(0, np.ones(p.N, np.uint8))
        for t in range(1, 9):
            p.advance(t)
            dl, tl = p.score(t)
            mask, st = p.select(t, 1.0, dl, tl)
            pack_and_drain(t, mask)
        store.sync()
        # several versions were in flight on the writer pool; they become
        # visible in append order
        assert [e["step"] for e in store.entries()] == [e["step"] for e in expected]
        files = sorted(f for f in os.listdir(d) if f.endswith(".lcr"))
        assert len(files) == len(expected)
        for f, e in zip(files, expected):
            assert open(os.path.join(d, f), "rb").read() == bytes(e["payload"]), f
        store.close()
        store = LC.Store(d, p.R)
        t_fail = 6
        assert store.plan(t_fail).tolist() == [expected[i]["step"] for i in O.plan_versions(expected, p.N, t_fail)]
        # reclaiming space keeps every record a recovery at t_fail or later can choose
        before = len(store.entries())
        removed = store.compact(t_fail)
        assert removed > 0 and len(store.entries()) == before - removed
        assert store.plan(t_fail).tolist() == [expected[i]["step"] for i in O.plan_versions(expected, p.N, t_fail)]
        # fail-stop, then recover from the store
        for a in (p.dW, p.dS, p.dm, p.dv) + ((p.dM,) if p.dM is not None else ()):
            a.fill_(0)
        for a in (p.hW, p.hS, p.hm, p.hv) + ((p.hM,) if p.hM is not None else ()):
            a[...] = 0
        torch.cuda.synchronize()
        chosen = store.restore(p.ctx, t_fail)
        chosen_o = p.orc.restore(expected, t_fail)
        assert chosen.tolist() == chosen_o.tolist()
        log(f"  restored from steps {sorted(set(chosen.tolist()))}")
        p.check_arrays()
        # training continues after t_fail on both sides
        p.adopt_restored()
        for t in range(t_fail + 1, t_fail + 3):
            p.step(t)
    finally:
        store.close()
        p.close()


def test_async_append_needs_an_event_for_device_payloads(tmp_path):
    import torch
    spec = reduced_8b()
    p = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 0.01))
    store = LC.Store(str(tmp_path / "s"), p.R)
    try:
        staging = torch.empty(sum(p.R), dtype=torch.uint8, device="cuda")
        res = LC.lc_pack_selected(p.ctx, staging.data_ptr(), staging.numel(), 0)
        with pytest.raises(LC.LCError) as e:
            store.append_async(0, np.ones(p.N, np.uint8), staging.data_ptr(), res["bytes_written"],
                               torch.cuda.current_stream().cuda_stream, 0)
        assert e.value.code == LC.LC_ERR_INVALID_ARG
        store.sync()
        assert store.entries() == []  # refused before anything was written
    finally:
        store.close()
        p.close()


def test_store_rejects_other_layout(tmp_path):
    spec = reduced_8b()
    p = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 0.01))
    try:
        store = LC.Store(str(tmp_path / "s"), [r + 256 for r in p.R])
        with pytest.raises(LC.LCError) as e:
            store.restore(p.ctx, 0)
        assert e.value.code == LC.LC_ERR_INVALID_ARG
        store.close()
    finally:
        p.close()


def test_store_restore_pipeline_matches_device_restore(tmp_path):
    """Records of about 300 MB (five 64 MiB read pieces each) whose total
    exceeds the pinned restore ring, so the read pipeline wraps around it:
    the composite restored from the store's files must equal, byte for byte,
    the one the device restore (unpack kernel) builds from the same versions
    held in device memory."""
    import torch
    from paper_2609_27193_amd import inputs as I
    T = I.TensorSpec
    n = 21_000_000
    layers = tuple(I.LayerSpec(f"block_{l}", (T("w", n + 4097 * l, "matrix"),)) for l in range(6))
    spec = I.ModelSpec(name="store-ring", layers=layers, weight_dtype="bf16", has_master=True,
                       scale_rule="loguniform_0.01_1", target_fraction=0.4, s_max=3)
    state = I.SyntheticState(spec, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    segs = LC.segments_from_state(state)
    lay = LC.LayoutDesc(segs, spec.n_layers, LC.LC_DT_BF16, True, LC.LC_MODE_ACCUM, [0.005] * spec.n_layers,
                        spec.s_max, stream=stream)
    _, R = LC.lc_query_layout(lay)
    assert max(R) > (256 << 20) and sum(R) > max(2 * max(R), 1 << 30)
    ctx = LC.lc_init_layout(lay)
    store = LC.Store(str(tmp_path / "ring"), R)
    versions = []
    try:
        def pack_append(t, mask):
            nbytes = int(sum(R[l] for l in range(spec.n_layers) if mask[l]))
            buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")
            if nbytes:
                res = LC.lc_pack_selected(ctx, buf.data_ptr(), nbytes, 0)
                assert res["done"] == 1
            store.append(t, mask, buf.data_ptr() if nbytes else 0, nbytes, stream)
            versions.append({"step": t, "mask": mask.copy(), "payload": buf.data_ptr() if nbytes else 0,
                             "payload_bytes": nbytes, "buf": buf})

        pack_append(0, np.ones(spec.n_layers, np.uint8))
        for t in range(1, 4):
            state.step(t)
            LC.lc_score_layers(ctx, t)
            mask, _ = LC.lc_select(ctx, t, 1.0, spec.n_layers)
            pack_append(t, mask)
        store.sync()
        t_fail = 2
        arrays = [a for a in (state.weight, state.shadow, state.master, state.exp_avg, state.exp_avg_sq)]

        def wipe():
            for a in arrays:
                a.zero_()
            torch.cuda.synchronize()

        wipe()
        chosen_store = store.restore(ctx, t_fail)
        from_store = [a.clone() for a in arrays]
        wipe()
        chosen_dev = LC.lc_restore_composite(ctx, versions, t_fail, spec.n_layers)
        torch.cuda.synchronize()
        assert chosen_store.tolist() == chosen_dev.tolist()
        log(f"  restored from steps {chosen_store.tolist()}; record set {sum(R) / 1e9:.2f} GB")
        for a, b in zip(from_store, arrays):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))
    finally:
        store.close()
        LC.lc_destroy(ctx)
