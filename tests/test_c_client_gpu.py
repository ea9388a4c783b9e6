"""GPU: the C interface driven from plain C (tests/c_client/lc_c_client.c,
no Python or torch in the process), against the oracle.

The test records a synthetic trajectory (the base state and every later
step's weights, master and moments) to a file; the client allocates the
arrays with hipMalloc (all segments of an array back to back in one
allocation, so odd-sized tensors leave later segments misaligned), runs
score, select and pack at every step into device version buffers, then
loses the live state and restores the composite at t_fail; every version
also goes through a persistence store (overlapped appends with a reuse
event), and the client checks that the composite rebuilt from the store's
files equals the device one byte for byte.  Scores are
compared within the harness tolerance, masks, stats, payloads and restored
arrays exactly (a layer whose accumulator sits inside the tolerance band of
its threshold takes the client's decision on the oracle side)."""
import os
import struct
import subprocess

import numpy as np
import pytest

from oracle import layercheck_oracle as O
from paper_2609_27193_amd import inputs as I
from paper_2609_27193_amd.build_lib import C_CLIENT
from paper_2609_27193_amd.inputs import to_numpy_weight
from tests.conftest import gpu_available
from tests.gpu_harness import REL, log, rel_ok
from tests.test_edges_gpu import odd_spec
from tests.test_parity_gpu import k0_for, reduced_8b, reduced_qwen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not gpu_available():
        pytest.skip("needs an MI355X")
    assert os.path.exists(C_CLIENT), "the C client is built by __graft_entry__.build()"


def _arrays(g):
    return (to_numpy_weight(g.weight).copy(), None if g.master is None else g.master.numpy().copy(),
            g.exp_avg.numpy().copy(), g.exp_avg_sq.numpy().copy())


class Reader:
    def __init__(self, data):
        self.d = data
        self.p = 0

    def take(self, dtype, n):
        a = np.frombuffer(self.d, dtype=dtype, count=n, offset=self.p).copy()
        self.p += a.nbytes
        return a

    def one(self, fmt):
        v = struct.unpack_from("<" + fmt, self.d, self.p)[0]
        self.p += struct.calcsize(fmt)
        return v


CASES = [("8b-accum-master", reduced_8b, O.MODE_ACCUM), ("qwen-snapshot-nomaster", reduced_qwen, O.MODE_SNAPSHOT),
         ("odd-f32-accum", lambda: odd_spec("f32", True), O.MODE_ACCUM)]


@pytest.mark.parametrize("name,maker,mode", CASES, ids=[c[0] for c in CASES])
def test_c_client_against_oracle(tmp_path, name, maker, mode):
    spec = maker()
    N, n_steps, t_base = spec.n_layers, 8, 0
    t_fail = n_steps - 1
    k0 = k0_for(spec, 0.01 if spec.weight_dtype == "bf16" else 0.05)
    lr_scale = [1.0 if k < 5 else 0.5 for k in range(n_steps + 1)]
    dt = O.DT_BF16 if spec.weight_dtype == "bf16" else O.DT_F32
    g = I.SyntheticState(spec, device="cpu")
    states = [_arrays(g)]
    for k in range(1, n_steps + 1):
        g.step(t_base + k)
        states.append(_arrays(g))
    fin = tmp_path / "in.bin"
    fout = tmp_path / "out.bin"
    with open(fin, "wb") as f:
        f.write(b"LCC1")
        f.write(struct.pack("<6I", N, len(g.segments), 1 if dt == O.DT_BF16 else 2, int(spec.has_master), mode,
                            n_steps))
        f.write(struct.pack("<3qd", spec.s_max, t_base, t_fail, 1e-8))
        f.write(np.asarray(k0, np.float64).tobytes())
        f.write(np.asarray(lr_scale, np.float64).tobytes())
        for s in g.segments:
            f.write(struct.pack("<IIQ", s.layer, 0, s.numel))
        for W, M, m, v in states:
            f.write(W.tobytes())
            if M is not None:
                f.write(M.tobytes())
            f.write(m.tobytes())
            f.write(v.tobytes())
    log(f"{name}: running the C client on {spec.numel} elements, {N} layers")
    r = subprocess.run([C_CLIENT, str(fin), str(fout), str(tmp_path / "store")], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 0, r.stderr
    rd = Reader(open(fout, "rb").read())

    # the oracle over the same trajectory
    W, M, m, v = (a.copy() if a is not None else None for a in states[0])
    S = np.zeros_like(W)
    osegs = [O.OSegment(s.layer, W[s.offset:s.offset + s.numel], S[s.offset:s.offset + s.numel],
                        None if M is None else M[s.offset:s.offset + s.numel],
                        m[s.offset:s.offset + s.numel], v[s.offset:s.offset + s.numel]) for s in g.segments]
    orc = O.LayerCheckOracle(osegs, N, dt, spec.has_master, mode, k0, spec.s_max, t_base=t_base)
    for l in range(N):
        assert rd.one("Q") == orc.n[l]
        assert rd.one("Q") == orc.R[l]
    versions = []

    def check_payload(step):
        nbytes = rd.one("Q")
        got = rd.take(np.uint8, nbytes)
        pay, res = orc.pack(0, 1 << 62)
        assert res["done"] == 1 and np.array_equal(got, pay), f"payload differs at step {step}"
        return got

    versions.append({"step": t_base, "mask": np.ones(N, np.uint8), "payload": check_payload(t_base)})
    resyncs = 0
    for k in range(1, n_steps + 1):
        t = t_base + k
        W[...], m[...], v[...] = states[k][0], states[k][2], states[k][3]
        if M is not None:
            M[...] = states[k][1]
        orc.score(t)
        u_c, d_c = rd.take(np.float64, N), rd.take(np.float64, N)
        tl_c, mask_c = rd.take(np.int64, N), rd.take(np.uint8, N)
        st_c = {"n_selected": rd.one("I"), "n_forced": rd.one("I"), "payload_bytes": rd.one("Q"),
                "max_age": rd.one("q"), "weighted_age": rd.one("d")}
        assert rel_ok(u_c, orc.u), (t, u_c, orc.u)
        mask_o, st_o = orc.select(t, lr_scale[k])
        for l in np.nonzero(mask_o != mask_c)[0]:
            K = k0[l] * lr_scale[k]
            assert abs(orc._pre_delta[l] - K) <= REL * K, f"step {t} layer {l}: mask differs outside the band"
            orc.resync(int(l), bool(mask_c[l]))
            resyncs += 1
        assert np.array_equal(orc.mask, mask_c)
        assert tl_c.tolist() == list(orc.t_last)
        if not resyncs:
            for key in ("n_selected", "n_forced", "payload_bytes", "max_age"):
                assert st_c[key] == st_o[key], (t, key)
            assert abs(st_c["weighted_age"] - st_o["weighted_age"]) <= 1e-12 * max(1.0, st_o["weighted_age"])
        versions.append({"step": t, "mask": mask_c.copy(), "payload": check_payload(t)})
        log(f"  t={t}: selected {int(mask_c.sum())}/{N}")
    chosen_c, tl_c = rd.take(np.int64, N), rd.take(np.int64, N)
    for a in (W, S, m, v) + ((M,) if M is not None else ()):
        a[...] = 0
    chosen_o = orc.restore(versions, t_fail)
    assert chosen_c.tolist() == chosen_o.tolist() == tl_c.tolist()
    log(f"  restored at {t_fail} from steps {sorted(set(chosen_c.tolist()))}")
    for name_, arr in (("W", W), ("S", S)) + ((("master", M),) if M is not None else ()) + (("m", m), ("v", v)):
        got = rd.take(np.uint8, arr.nbytes)
        assert np.array_equal(got, arr.view(np.uint8)), f"restored {name_} differs"
    assert rd.p == len(rd.d)
