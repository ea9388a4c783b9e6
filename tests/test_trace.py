"""Optional roctx ranges (CPU): the library does not link against roctx; with
LAYERCHECK_ROCTX=1 it loads the roctx library at run time on its first call,
without it never; calls that open a range and return early with an error keep
their status codes and leave no range open (no device work is issued by these
calls)."""
import os
import subprocess
import sys

import pytest

from paper_2609_27193_amd import layercheck as LC

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCTX = "librocprofiler-sdk-roctx.so"

CHILD = r"""
import ctypes as C, sys
sys.path.insert(0, sys.argv[1])
from paper_2609_27193_amd import layercheck as LC
lib = LC.load_library()
def mapped():
    return any(sys.argv[2] in line for line in open("/proc/self/maps"))
assert not mapped()
ctx = C.c_void_p()
assert lib.lc_init_layout(None, C.byref(ctx)) == LC.LC_ERR_INVALID_ARG
assert lib.lc_score_layers(None, 1) == LC.LC_ERR_INVALID_ARG
assert lib.lc_select(None, 1, 1.0, None, None) == LC.LC_ERR_INVALID_ARG
h = C.c_void_p()
assert lib.lc_store_open(None, 1, None, 0, C.byref(h)) == LC.LC_ERR_INVALID_ARG
for _ in range(1000):
    lib.lc_destroy(None)
print("mapped", int(mapped()))
if mapped():  # the same roctx instance the library loaded: no range left open
    path = [l.split()[-1] for l in open("/proc/self/maps") if sys.argv[2] in l][0]
    roctx = C.CDLL(path)
    roctx.roctxRangePushA.restype = C.c_int
    print("depth", roctx.roctxRangePushA(b"probe"))
"""


@pytest.fixture(scope="module")
def built():
    if not os.path.exists(LC.LIB_PATH):
        from paper_2609_27193_amd.build_lib import build
        build()


def test_no_link_time_roctx_dependency(built):
    out = subprocess.run(["readelf", "-d", LC.LIB_PATH], capture_output=True, text=True, check=True).stdout
    needed = [l for l in out.splitlines() if "(NEEDED)" in l]
    assert needed and not any("roctx" in l for l in needed), needed


def run_child(flag):
    env = dict(os.environ, LAYERCHECK_ROCTX=flag)
    r = subprocess.run([sys.executable, "-c", CHILD, ROOT, ROCTX], capture_output=True, text=True, env=env,
                       timeout=120)
    assert r.returncode == 0, r.stderr[-2000:]
    return r.stdout


def test_tracing_off_by_default(built):
    assert "mapped 0" in run_child("0")


def test_ranges_opened_and_closed_when_on(built):
    if not os.path.exists(f"/opt/rocm/lib/{ROCTX}.1"):
        pytest.skip("no roctx library in this ROCm")
    out = run_child("1")
    assert "mapped 1" in out and "depth 0" in out, out


GPU_CHILD = r"""
import sys
sys.path.insert(0, sys.argv[1])
import __graft_entry__ as g
g.smoke()
print("roctx mapped", int(any(sys.argv[2] in line for line in open("/proc/self/maps"))), flush=True)
"""


@pytest.mark.gpu
def test_traced_decision_steps_match_the_oracle():
    """Decision steps and a composite restore on cuda:0 with the ranges on
    (the smoke run: scores within 1e-5, masks, payloads, shadow and restore
    bit-exact against the oracle), in a process of its own."""
    from tests.conftest import gpu_available
    if not gpu_available():
        pytest.skip("needs an MI355X")
    if not os.path.exists(f"/opt/rocm/lib/{ROCTX}.1"):
        pytest.skip("no roctx library in this ROCm")
    env = dict(os.environ, LAYERCHECK_ROCTX="1")
    r = subprocess.run([sys.executable, "-u", "-c", GPU_CHILD, ROOT, ROCTX], capture_output=True, text=True,
                       env=env, timeout=240)
    print(r.stdout[-1500:], flush=True)
    assert r.returncode == 0, r.stderr[-2000:]
    assert "smoke OK" in r.stdout and "roctx mapped 1" in r.stdout
