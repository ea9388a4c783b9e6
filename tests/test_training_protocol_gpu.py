"""GPU, end to end: the checkpointing protocol around a training run, against
the oracle at every step.

* Warm-up (Section 3.4): AdamW steps with the drift taken from the update but
  no selective persistence; the window ends with a full base checkpoint
  (lc_rebase), drained to the persistence store.
* Then every step: the fused AdamW step under a learning-rate schedule
  (linear warm-up, cosine decay), the threshold scaled with it,
  K(t) = K0 * lr(t) / lr_peak (Section 3.2), the staleness guard
  (Section 3.3), the pack of the selected layers and its drain into the store
  with no host synchronisation before the next step.
* A fail-stop at t_fail, the composite recovery from the store (Section 3.5),
  training resumed from the recovered state (the abandoned run's newer
  versions discarded from the store), and a second fail-stop recovered from
  a history that mixes both runs.

Optimizer state, weights and records are bit-exact against the oracle; the
scores agree within the harness tolerance."""
import math

import numpy as np
import pytest

from oracle import layercheck_oracle as O
from paper_2609_27193_amd import layercheck as LC
from tests.conftest import gpu_available
from tests.gpu_harness import Pair, log
from tests.test_parity_gpu import k0_for, reduced_8b, reduced_qwen

pytestmark = pytest.mark.gpu

LR_PEAK = 1e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not gpu_available():
        pytest.skip("needs an MI355X")
    LC.load_library()


def lr_at(t, warm, total):
    """Linear warm-up to LR_PEAK over ``warm`` steps, then cosine decay to a
    tenth of it at ``total``."""
    if t <= warm:
        return LR_PEAK * t / warm
    x = min(1.0, (t - warm) / max(1, total - warm))
    return LR_PEAK * (0.1 + 0.9 * 0.5 * (1.0 + math.cos(math.pi * x)))


@pytest.mark.parametrize("maker", [reduced_8b, reduced_qwen], ids=["8b", "qwen"])
def test_warmup_schedule_store_failure_recovery(tmp_path, maker):
    import torch
    spec = maker()
    warm, total = 4, 4 + 2 * spec.s_max
    p = Pair(spec, LC.LC_MODE_ACCUM, k0_for(spec, 0.08))
    store = LC.Store(str(tmp_path / "store"), p.R, buffer_bytes=2 << 20)
    stream = torch.cuda.current_stream().cuda_stream
    stored = []

    def drain(t, mask):
        _, _, dev = p.versions_dev[-1]
        nbytes = int(sum(p.R[l] for l in range(p.N) if mask[l]))
        store.append(t, mask, dev.data_ptr() if dev is not None else 0, nbytes, stream)
        stored.append({"step": t, "mask": mask.copy(), "payload": p.versions_host[-1][2]})

    try:
        # warm-up: optimizer steps, no selective persistence
        for t in range(1, warm + 1):
            p.fused_step(t, adam_t=t, lr=lr_at(t, warm, total), decide=False)
        mask = p.rebase(warm)
        p.pack(warm, mask)
        drain(warm, mask)
        with pytest.raises(LC.LCError) as e:
            LC.lc_rebase(p.ctx, warm - 1)
        assert e.value.code == LC.LC_ERR_BAD_STATE
        sel, forced = 0, 0
        for t in range(warm + 1, total + 1):
            lr = lr_at(t, warm, total)
            mask, st = p.fused_step(t, adam_t=t, lr=lr, lr_scale=lr / LR_PEAK)
            assert st["max_age"] <= spec.s_max - 1  # Eq. 5 after every decision
            sel += st["n_selected"]
            forced += st["n_forced"]
            drain(t, mask)
            log(f"  t={t} lr={lr:.2e}: selected {st['n_selected']}/{p.N} (forced {st['n_forced']}), "
                f"weighted staleness {st['weighted_age']:.2f}")
        assert 0 < sel - forced, "the threshold never fired"
        store.sync()
        assert [e["step"] for e in store.entries()] == [v["step"] for v in stored]
        # fail-stop after the last step that is not on a forced boundary
        t_fail = total - 1
        with pytest.raises(LC.LCError) as e:
            store.plan(warm - 1)  # before the base: nothing to recover from
        assert e.value.code == LC.LC_ERR_NO_VERSION
        for a in (p.dW, p.dS, p.dm, p.dv) + ((p.dM,) if p.dM is not None else ()):
            a.fill_(0)
        for a in (p.hW, p.hS, p.hm, p.hv) + ((p.hM,) if p.hM is not None else ()):
            a[...] = 0
        torch.cuda.synchronize()
        chosen = store.restore(p.ctx, t_fail)
        chosen_o = p.orc.restore(stored, t_fail)
        assert chosen.tolist() == chosen_o.tolist()
        assert min(chosen) >= t_fail - (spec.s_max - 1)  # the staleness bound holds at recovery
        p.check_arrays()
        log(f"  recovered at {t_fail} from steps {sorted(set(chosen.tolist()))}")
        # training resumes from the recovered state; the abandoned run's newer
        # versions leave the store, and the resumed run persists its own
        p.adopt_restored()
        removed = store.discard_after(t_fail)
        stored = [v for v in stored if v["step"] <= t_fail]
        assert removed >= 1 and [e["step"] for e in store.entries()] == [v["step"] for v in stored]
        for t in range(t_fail + 1, t_fail + 3):
            lr = lr_at(t, warm, total)
            mask, st = p.fused_step(t, adam_t=t, lr=lr, lr_scale=lr / LR_PEAK)
            assert st["max_age"] <= spec.s_max - 1
            drain(t, mask)
        store.sync()
        # a second fail-stop: the composite mixes the first run's records up
        # to its t_fail with the resumed run's
        t_fail2 = t_fail + 2
        for a in (p.dW, p.dS, p.dm, p.dv) + ((p.dM,) if p.dM is not None else ()):
            a.fill_(0)
        for a in (p.hW, p.hS, p.hm, p.hv) + ((p.hM,) if p.hM is not None else ()):
            a[...] = 0
        torch.cuda.synchronize()
        chosen = store.restore(p.ctx, t_fail2)
        assert chosen.tolist() == p.orc.restore(stored, t_fail2).tolist()
        assert min(chosen) >= t_fail2 - (spec.s_max - 1)
        assert min(chosen) <= t_fail < max(chosen), chosen  # records of both runs
        p.check_arrays()
        log(f"  second recovery at {t_fail2} from steps {sorted(set(chosen.tolist()))}")
        p.adopt_restored()
        lr = lr_at(t_fail2 + 1, warm, total)
        p.fused_step(t_fail2 + 1, adam_t=t_fail2 + 1, lr=lr, lr_scale=lr / LR_PEAK)
    finally:
        store.close()
        p.close()
