"""GPU: two contexts at once.

A context owns its device tables and is bound to the stream it was created
on, and the library keeps no other state (only the last error message, per
host thread).  Two contexts over two different states, each on its own
stream and driven from its own host thread at the same time, must each
match their own oracle exactly as when run alone: scores, masks, payloads,
shadows, and a composite restore (Sections 3.2-3.5).
"""
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
    LC.load_library()  # a missing build fails here, loudly


def _drive(name, p, stream, steps, t_fail, errors):
    import torch
    try:
        with torch.cuda.stream(stream):
            p.pack(0, np.ones(p.N, np.uint8))  # the base
            for t in steps:
                mask, st = p.step(t)
                log(f"  [{name}] step {t}: selected {st['n_selected']}/{p.N} forced {st['n_forced']}")
            chosen = _restore_and_compare(p, t_fail, "device")
            log(f"  [{name}] restored from steps {sorted(set(chosen.tolist()))}")
    except BaseException as e:  # re-raised by the main thread
        errors.append((name, e))


def test_two_contexts_two_streams_two_threads():
    import torch
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    spec_a, spec_b = reduced_8b(), reduced_qwen()
    with torch.cuda.stream(sa):
        a = Pair(spec_a, LC.LC_MODE_ACCUM, k0_for(spec_a, 0.02))
    with torch.cuda.stream(sb):
        b = Pair(spec_b, LC.LC_MODE_SNAPSHOT, k0_for(spec_b, 0.02))
    try:
        assert a.stream == sa.cuda_stream and b.stream == sb.cuda_stream and a.stream != b.stream
        errors = []
        threads = [threading.Thread(target=_drive, args=("8b-accum", a, sa, range(1, 11), 8, errors)),
                   threading.Thread(target=_drive, args=("qwen-snapshot", b, sb, range(1, 11), 7, errors))]
        for th in threads:
            th.start()
        for th in threads:
            th.join(timeout=300)
        assert not any(th.is_alive() for th in threads), "a driver thread did not finish"
        if errors:
            raise AssertionError(f"context {errors[0][0]} failed") from errors[0][1]
        # each side still agrees with its own oracle after the other's work
        a.check_arrays()
        b.check_arrays()
    finally:
        a.close()
        b.close()
