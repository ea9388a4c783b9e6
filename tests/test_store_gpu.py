"""GPU: draining device staging into the persistence store and composite
recovery from it (Section 3.5), against the oracle.

One staging buffer is reused every step with no synchronisation between
lc_store_append and the next lc_pack_selected: the drain's copies must be
stream-ordered before the next pack overwrites the buffer.  Small drain
buffers force many chunks through the pinned ring."""
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


@pytest.mark.parametrize("maker,mode,buf", [(reduced_8b, LC.LC_MODE_ACCUM, 1 << 20),
                                            (reduced_qwen, LC.LC_MODE_SNAPSHOT, 3 << 20)],
                         ids=["8b-accum", "qwen-snapshot"])
def test_drain_and_restore_from_store(tmp_path, maker, mode, buf):
    import torch
    spec = maker()
    p = Pair(spec, mode, k0_for(spec, 0.01))
    d = str(tmp_path / "store")
    store = LC.Store(d, p.R, buffer_bytes=buf)
    try:
        stream = torch.cuda.current_stream().cuda_stream
        cap = sum(p.R)
        staging = torch.empty(cap, dtype=torch.uint8, device="cuda")
        expected = []

        def pack_and_drain(t, mask):
            res = LC.lc_pack_selected(p.ctx, staging.data_ptr(), cap, 0)
            pay_o, res_o = p.orc.pack(0, cap)
            assert res == res_o
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
