"""GPU: independent contexts.  Two contexts over different layouts, each on
its own HIP stream and driven from its own host thread at the same time,
must each agree with their oracle at every step and in a composite restore
(the library keeps no shared mutable state beyond the per-thread error
message)."""
import threading

import numpy as np
import pytest

from paper_2609_27193_amd import layercheck as LC
from tests.conftest import gpu_available
from tests.gpu_harness import Pair, log
from tests.test_parity_gpu import _restore_and_compare, k0_for, reduced_8b, reduced_qwen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not gpu_available():
        pytest.skip("needs an MI355X")
    LC.load_library()


def test_two_contexts_two_streams_two_threads():
    import torch
    jobs = [(reduced_8b(), LC.LC_MODE_ACCUM), (reduced_qwen(), LC.LC_MODE_SNAPSHOT)]
    errors = []
    done = []

    def run(spec, mode):
        try:
            stream = torch.cuda.Stream()
            with torch.cuda.stream(stream):
                p = Pair(spec, mode, k0_for(spec, 0.01))
                try:
                    assert p.stream == stream.cuda_stream
                    p.pack(0, np.ones(p.N, np.uint8))
                    for t in range(1, 9):
                        p.step(t, lr_scale=1.0 if t < 5 else 0.5)
                    chosen = _restore_and_compare(p, 7, "device")
                    log(f"  [{spec.name}] restored from steps {sorted(set(chosen.tolist()))}")
                    # an error on this thread leaves its message here, not on the other thread
                    with pytest.raises(LC.LCError):
                        LC.lc_select(p.ctx, 99, 1.0, p.N)
                    p.check_arrays()
                    done.append(spec.name)
                finally:
                    p.close()
        except BaseException as e:  # noqa: BLE001 - reported by the main thread
            errors.append((spec.name, repr(e)))

    threads = [threading.Thread(target=run, args=job) for job in jobs]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=240)
    assert not any(th.is_alive() for th in threads), "a worker did not finish"
    assert not errors, errors
    assert sorted(done) == sorted(s.name for s, _ in jobs)
    log(f"  both contexts agreed with their oracles: {done}")
