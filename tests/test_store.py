"""The persistence store on the CPU (host payloads): versions written as
files plus an append-only manifest, read back after reopening, the
reconstruction plan against the oracle's (Section 3.5), and crash
consistency (torn or inconsistent manifest lines and files are ignored)."""
import os

import numpy as np
import pytest

from oracle import layercheck_oracle as O
from paper_2609_27193_amd import layercheck as LC
from tests._helpers import HostLayout


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LC.LIB_PATH):
        from paper_2609_27193_amd.build_lib import build
        build()
    return LC.load_library()


def oracle_history(steps=8, seed=0):
    """Payloads of an oracle run: the base at step 0, then every selection."""
    sizes = [[300, 7], [64], [129, 3, 3], [1], [500]]
    lay = HostLayout(sizes, seed=seed)
    N = len(sizes)
    orc = O.LayerCheckOracle(lay.segs, N, O.DT_BF16, True, O.MODE_ACCUM, [0.03] * N, s_max=3)
    versions = [{"step": 0, "mask": np.ones(N, np.uint8), "payload": orc.pack(0, 1 << 40)[0]}]
    for t in range(1, steps + 1):
        lay.step([4.0, 0.3, 1.0, 0.02, 2.0])
        orc.score(t)
        mask, _ = orc.select(t, 1.0)
        versions.append({"step": t, "mask": mask, "payload": orc.pack(0, 1 << 40)[0]})
    return orc, versions


def test_append_reopen_and_plan(lib, tmp_path):
    orc, versions = oracle_history()
    d = str(tmp_path / "store")
    st = LC.Store(d, orc.R)
    for v in versions:
        st.append(v["step"], v["mask"], v["payload"].ctypes.data if len(v["payload"]) else 0, len(v["payload"]))
    st.sync()
    st.close()
    st = LC.Store(d, orc.R)  # reopen: the manifest is the persistence history
    ent = st.entries()
    assert [e["step"] for e in ent] == [v["step"] for v in versions]
    for e, v in zip(ent, versions):
        assert np.array_equal(e["mask"], v["mask"]) and e["payload_bytes"] == len(v["payload"])
    files = sorted(f for f in os.listdir(d) if f.endswith(".lcr"))
    for f, v in zip(files, versions):
        assert open(os.path.join(d, f), "rb").read() == bytes(v["payload"])
    for t_fail in range(0, 10):
        expect = [versions[i]["step"] for i in O.plan_versions(versions, orc.N, t_fail)]
        assert st.plan(t_fail).tolist() == expect
    with pytest.raises(LC.LCError) as e:
        st.plan(-1)
    assert e.value.code == LC.LC_ERR_NO_VERSION
    st.close()


def test_append_validation(lib, tmp_path):
    orc, versions = oracle_history(steps=2)
    st = LC.Store(str(tmp_path / "s"), orc.R)
    v = versions[1]
    with pytest.raises(LC.LCError) as e:  # size does not match the mask
        st.append(v["step"], v["mask"], v["payload"].ctypes.data, len(v["payload"]) + 256)
    assert e.value.code == LC.LC_ERR_INVALID_ARG
    st.append(0, versions[0]["mask"], versions[0]["payload"].ctypes.data, len(versions[0]["payload"]))
    with pytest.raises(LC.LCError):  # a layer twice at one step
        st.append(0, versions[0]["mask"], versions[0]["payload"].ctypes.data, len(versions[0]["payload"]))
    # disjoint masks at one step are fine (a selection packed in several calls)
    m1 = np.zeros(orc.N, np.uint8)
    m1[0] = 1
    m2 = np.zeros(orc.N, np.uint8)
    m2[2] = 1
    p1 = np.zeros(orc.R[0], np.uint8)
    p2 = np.zeros(orc.R[2], np.uint8)
    st.append(5, m1, p1.ctypes.data, len(p1))
    st.append(5, m2, p2.ctypes.data, len(p2))
    assert st.plan(5).tolist() == [5, 0, 5, 0, 0]
    # the overlapped append takes host payloads the same way (no event needed:
    # the bytes are written before it returns), with the same validation
    st.append_async(6, m1, p1.ctypes.data, len(p1))
    with pytest.raises(LC.LCError):
        st.append_async(6, m1, p1.ctypes.data, len(p1))
    st.sync()
    assert st.plan(6).tolist() == [6, 0, 5, 0, 0]
    st.close()
    with pytest.raises(LC.LCError):
        LC.Store(str(tmp_path / "bad"), [100, 256])  # record sizes are 256-byte multiples


def test_crash_consistency(lib, tmp_path):
    orc, versions = oracle_history(steps=4)
    d = str(tmp_path / "c")
    st = LC.Store(d, orc.R)
    for v in versions:
        st.append(v["step"], v["mask"], v["payload"].ctypes.data if len(v["payload"]) else 0, len(v["payload"]))
    st.close()
    files = sorted(f for f in os.listdir(d) if f.endswith(".lcr"))
    sized = [f for f, v in zip(files, versions) if len(v["payload"])]
    # (1) a version whose file lost its tail is dropped
    victim = sized[-1]
    with open(os.path.join(d, victim), "r+b") as f:
        f.truncate(os.path.getsize(os.path.join(d, victim)) - 256)
    # (2) a garbage line, (3) a line for a file that does not exist,
    # (4) a line naming a file outside the directory (right size, right mask),
    # (5) a torn last line, (6) an orphan version file with no line
    outside = str(tmp_path / "v_outside.lcr")
    open(outside, "wb").write(b"\0" * orc.R[0])
    with open(os.path.join(d, "manifest.lcm"), "a") as f:
        f.write("not a manifest line\n")
        f.write("LCV1 9 256 v9999999999_s9.lcr " + "1" + "0" * (orc.N - 1) + "\n")
        f.write(f"LCV1 11 {orc.R[0]} ../v_outside.lcr " + "1" + "0" * (orc.N - 1) + "\n")
        f.write("LCV1 10 25")
    open(os.path.join(d, "v0000000777_s12.lcr"), "wb").write(b"\0" * 512)
    st = LC.Store(d, orc.R)
    kept = [e["step"] for e in st.entries()]
    dropped = versions[files.index(victim)]["step"]
    assert kept == [v["step"] for v in versions if v["step"] != dropped]
    # the plan falls back past the lost version
    survivors = [v for v in versions if v["step"] != dropped]
    for t_fail in range(0, 5):
        assert st.plan(t_fail).tolist() == [survivors[i]["step"] for i in O.plan_versions(survivors, orc.N, t_fail)]
    # appends continue after the recovered history
    v = versions[1]
    st.append(20, v["mask"], v["payload"].ctypes.data, len(v["payload"]))
    st.close()
    st = LC.Store(d, orc.R)
    assert st.entries()[-1]["step"] == 20
    # reclaiming space never reaches outside the store's directory
    st.compact(20)
    st.close()
    assert os.path.getsize(outside) == orc.R[0]


def test_large_host_payload_in_pieces(lib, tmp_path):
    """A host payload larger than one write piece is split over the writer
    threads; the file must hold it byte for byte, and versions appended one
    after another keep their order in the manifest."""
    R = [72 << 20, 256, 8 << 20]
    rng = np.random.default_rng(7)
    payload = rng.integers(0, 256, sum(R), dtype=np.uint8)
    d = str(tmp_path / "big")
    st = LC.Store(d, R)
    st.append(0, np.ones(3, np.uint8), payload.ctypes.data, payload.nbytes)
    part = payload[R[0]:R[0] + R[1] + R[2]]
    st.append(1, np.array([0, 1, 1], np.uint8), part.ctypes.data, part.nbytes)
    st.close()
    st = LC.Store(d, R)
    assert [e["step"] for e in st.entries()] == [0, 1]
    assert st.plan(1).tolist() == [0, 1, 1]
    st.close()
    files = sorted(f for f in os.listdir(d) if f.endswith(".lcr"))
    assert np.array_equal(np.fromfile(os.path.join(d, files[0]), np.uint8), payload)
    assert np.array_equal(np.fromfile(os.path.join(d, files[1]), np.uint8), part)


@pytest.mark.parametrize("t_keep", [0, 3, 5, 8, 100])
def test_compact_keeps_exactly_what_plans_can_choose(lib, tmp_path, t_keep):
    """After lc_store_compact(t_keep) the store holds exactly the union, over
    every t_fail >= t_keep, of the versions the oracle's plan chooses; those
    plans are unchanged; the removed files are gone and the history survives
    a reopen."""
    orc, versions = oracle_history(steps=8)
    d = str(tmp_path / "k")
    st = LC.Store(d, orc.R)
    for v in versions:
        st.append(v["step"], v["mask"], v["payload"].ctypes.data if len(v["payload"]) else 0, len(v["payload"]))
    st.sync()
    last = max(v["step"] for v in versions)
    t_fails = range(t_keep, max(t_keep, last) + 2)  # plans for t_fail >= last all agree
    chosen = set()
    plans_before = {}
    for t in t_fails:
        try:
            idx = O.plan_versions(versions, orc.N, t)
        except O.OracleError:
            continue
        chosen.update(idx)
        plans_before[t] = st.plan(t).tolist()
    removed = st.compact(t_keep)
    kept = [versions[i]["step"] for i in sorted(chosen)]
    assert [e["step"] for e in st.entries()] == kept
    assert removed == len(versions) - len(kept)
    for t, plan in plans_before.items():
        assert st.plan(t).tolist() == plan
    st.close()
    assert len([f for f in os.listdir(d) if f.endswith(".lcr")]) == len(kept)
    st = LC.Store(d, orc.R)
    assert [e["step"] for e in st.entries()] == kept
    assert st.compact(t_keep) == 0  # nothing more to reclaim
    st.close()


def test_compact_crash_leftovers(lib, tmp_path):
    """A crash during compaction leaves a stale temporary manifest or files the
    manifest no longer names; the next open ignores them and the next
    compaction removes the orphans."""
    orc, versions = oracle_history(steps=4)
    d = str(tmp_path / "c2")
    st = LC.Store(d, orc.R)
    for v in versions:
        st.append(v["step"], v["mask"], v["payload"].ctypes.data if len(v["payload"]) else 0, len(v["payload"]))
    st.close()
    open(os.path.join(d, "manifest.lcm.tmp"), "w").write("LCV1 garbage\n")
    open(os.path.join(d, "v0000000999_s3.lcr"), "wb").write(b"\0" * 256)
    st = LC.Store(d, orc.R)
    assert [e["step"] for e in st.entries()] == [v["step"] for v in versions]
    removed = st.compact(-1)  # keeps every non-empty version; removes the orphan
    assert removed >= 1
    assert "v0000000999_s3.lcr" not in os.listdir(d)
    st.close()


def test_store_context_manager(lib, tmp_path):
    orc, versions = oracle_history(steps=2)
    d = str(tmp_path / "cm")
    with LC.Store(d, orc.R) as st:
        v = versions[0]
        st.append(v["step"], v["mask"], v["payload"].ctypes.data, len(v["payload"]))
    assert st.h is None
    with LC.Store(d, orc.R) as st:
        assert [e["step"] for e in st.entries()] == [0]


def test_write_failure_drops_the_version(lib, tmp_path):
    """An I/O failure in the writers (here the file-size limit of a child
    process, so a write fails with EFBIG) drops the version being written,
    fails the call with LC_ERR_IO and every later append too; the
    manifest never names the failed version, and the earlier history stays
    restorable after reopening."""
    import subprocess
    import sys
    d = str(tmp_path / "efbig")
    child = f"""
import resource, signal, sys
import numpy as np
sys.path.insert(0, {os.path.dirname(os.path.dirname(os.path.abspath(__file__)))!r})
from paper_2609_27193_amd import layercheck as LC
signal.signal(signal.SIGXFSZ, signal.SIG_IGN)
R = [256 * 1024, 4 * 1024 * 1024]
st = LC.Store({d!r}, R)
small = np.arange(R[0], dtype=np.uint8)
st.append(0, np.array([1, 0], np.uint8), small.ctypes.data, small.nbytes)   # fits under the limit
resource.setrlimit(resource.RLIMIT_FSIZE, (1024 * 1024, 1024 * 1024))
big = np.ones(R[1], dtype=np.uint8)
codes = []
for step in (1, 2):
    try:
        st.append(step, np.array([0, 1], np.uint8), big.ctypes.data, big.nbytes)
        codes.append(0)
    except LC.LCError as e:
        codes.append(e.code)
print(codes)
"""
    r = subprocess.run([sys.executable, "-c", child], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == f"[{LC.LC_ERR_IO}, {LC.LC_ERR_IO}]", r.stdout
    st = LC.Store(d, [256 * 1024, 4 * 1024 * 1024])
    assert [e["step"] for e in st.entries()] == [0]
    assert "LCV1 1 " not in open(os.path.join(d, "manifest.lcm")).read()
    st.close()


def test_discard_after_for_a_resumed_run(lib, tmp_path):
    """After a restore at t_fail the versions newer than t_fail belong to the
    abandoned run: discarding them lets the resumed run append its own
    versions of those steps (a layer may be stored once per step), and plans
    then mix the old history up to t_fail with the new one."""
    orc, versions = oracle_history(steps=6)
    d = str(tmp_path / "tl")
    st = LC.Store(d, orc.R)
    for v in versions:
        st.append(v["step"], v["mask"], v["payload"].ctypes.data if len(v["payload"]) else 0, len(v["payload"]))
    st.sync()
    t_fail = 3
    new = [v for v in versions if v["step"] > t_fail and v["mask"].any()][0]
    with pytest.raises(LC.LCError):  # the abandoned run already stored these layers at this step
        st.append(new["step"], new["mask"], new["payload"].ctypes.data, len(new["payload"]))
    removed = st.discard_after(t_fail)
    assert removed == len([v for v in versions if v["step"] > t_fail])
    assert [e["step"] for e in st.entries()] == [v["step"] for v in versions if v["step"] <= t_fail]
    st.append(new["step"], new["mask"], new["payload"].ctypes.data, len(new["payload"]))
    st.close()
    st = LC.Store(d, orc.R)
    timeline = [v for v in versions if v["step"] <= t_fail] + [new]
    assert [e["step"] for e in st.entries()] == [v["step"] for v in timeline]
    for t in range(0, 8):
        assert st.plan(t).tolist() == [timeline[i]["step"] for i in O.plan_versions(timeline, orc.N, t)]
    st.close()


def test_one_store_per_directory(lib, tmp_path):
    """A directory is open in one store at a time: a second open, in this
    process or another, is refused until the first store is closed; the lock
    file survives compaction (only version files are ever removed)."""
    import subprocess
    import sys
    orc, versions = oracle_history(steps=3)
    d = str(tmp_path / "lk")
    a = LC.Store(d, orc.R)
    for v in versions:
        a.append(v["step"], v["mask"], v["payload"].ctypes.data if len(v["payload"]) else 0, len(v["payload"]))
    with pytest.raises(LC.LCError) as e:
        LC.Store(d, orc.R)
    assert e.value.code == LC.LC_ERR_BAD_STATE
    child = (f"import sys; sys.path.insert(0, {os.path.dirname(os.path.dirname(os.path.abspath(__file__)))!r})\n"
             "from paper_2609_27193_amd import layercheck as LC\n"
             f"try:\n    LC.Store({d!r}, {list(orc.R)!r})\n    print('opened')\n"
             "except LC.LCError as e:\n    print('refused', e.code)\n")
    r = subprocess.run([sys.executable, "-c", child], capture_output=True, text=True, timeout=120)
    assert r.stdout.strip() == f"refused {LC.LC_ERR_BAD_STATE}", (r.stdout, r.stderr)
    a.compact(versions[-1]["step"])
    assert os.path.exists(os.path.join(d, "store.lock"))
    a.close()
    b = LC.Store(d, orc.R)
    assert [e["step"] for e in b.entries()]
    b.close()


def test_file_failures_return_lc_err_io(lib, tmp_path):
    """Every failed file operation of the store returns LC_ERR_IO, whatever
    the call: opening a store under a missing parent, and, once the directory
    of an open store is gone, creating a version file and rewriting the
    manifest for a compaction or a discard.  Argument errors keep
    LC_ERR_INVALID_ARG."""
    import shutil
    orc, versions = oracle_history(steps=3)
    with pytest.raises(LC.LCError) as e:
        LC.Store(str(tmp_path / "missing" / "store"), orc.R)
    assert e.value.code == LC.LC_ERR_IO and "missing" in str(e.value)
    d = str(tmp_path / "gone")
    st = LC.Store(d, orc.R)
    for v in versions:
        st.append(v["step"], v["mask"], v["payload"].ctypes.data if len(v["payload"]) else 0, len(v["payload"]))
    st.sync()
    shutil.rmtree(d)
    v = [x for x in versions[1:] if x["mask"].any()][0]
    step = versions[-1]["step"] + 1
    for call in (lambda: st.append(step, v["mask"], v["payload"].ctypes.data, len(v["payload"])),
                 lambda: st.compact(versions[-1]["step"]),  # removes versions: rewrites the manifest
                 lambda: st.discard_after(0)):
        with pytest.raises(LC.LCError) as e:
            call()
        assert e.value.code == LC.LC_ERR_IO, str(e.value)
    with pytest.raises(LC.LCError) as e:
        st.append(step, v["mask"], v["payload"].ctypes.data, len(v["payload"]) - 256)
    assert e.value.code == LC.LC_ERR_INVALID_ARG
    st.close()
