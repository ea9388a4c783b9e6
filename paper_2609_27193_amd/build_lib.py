"""Build the HIP shared library ``liblayercheck.so`` for gfx950 in-tree.

Run as ``python -m paper_2609_27193_amd.build_lib``; every call recompiles.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "liblayercheck.so")
SOURCES = ["lc_runtime.cpp", "lc_store.cpp", "lc_kernels.hip", "lc_optim.hip", "lc_noalloc.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off",                      # keep the fp64 score formula unfused
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result", "-pthread",
    "-I", os.path.join(ROOT, "include"),
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


SANITIZED_LIB = os.path.join(HERE, "liblayercheck_hostsan.so")
# Test build: every grid capped at 40 blocks, so each kernel runs the form it
# takes beyond the 2^32 work-item dispatch limit (consecutive launches for the
# score and copy kernels, an in-kernel loop for the optimizer kernels).
GRID_CAPPED_LIB = os.path.join(HERE, "liblayercheck_gridcap.so")
GRID_CAP_DEFINES = ("LC_MAX_GRID_BLOCKS=40",)
# AddressSanitizer and UndefinedBehaviorSanitizer on the host code only (the
# validation, tables, state machine and store); device code is unchanged.
HOST_SANITIZER_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                        "-Xarch_host", "-fno-sanitize-recover=undefined", "-shared-libsan", "-g"]


def sanitizer_runtime() -> str:
    """The clang AddressSanitizer runtime the sanitized build needs preloaded."""
    import glob
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    hits = sorted(glob.glob(os.path.join(rocm, "lib", "llvm", "lib", "clang", "*", "lib", "linux",
                                         "libclang_rt.asan-x86_64.so")))
    return hits[-1] if hits else ""


def build(verbose: bool = False, out: str = LIB, defines=(), sanitize: bool = False) -> str:
    """Compile the library to ``out``; ``defines`` are extra -D macros
    (tile sizes LC_CHUNK_BYTES / LC_PIECE_BYTES for tuning builds);
    ``sanitize`` adds the host-side sanitizers (for CPU tests only)."""
    tmp = out + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, *(HOST_SANITIZER_FLAGS if sanitize else []), *[f"-D{d}" for d in defines],
           "-o", tmp, *[os.path.join(CSRC, s) for s in SOURCES]]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with exit code {res.returncode}")
    errs = [l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip()]
    if verbose and errs:
        sys.stderr.write("\n".join(errs) + "\n")
    os.replace(tmp, out)
    return out


HBM_PROBE = os.path.join(HERE, "lc_hbm_probe")
PROBE_LIB = os.path.join(HERE, "liblcprobe.so")


def build_hbm_probe(verbose: bool = False) -> str:
    """Compile the HBM ceiling probe twice: the stand-alone sweep
    (``bench.py --ceilings``) and the library that probes arrays the caller
    holds (``bench.py --placement-ceiling``)."""
    for out, extra in ((HBM_PROBE, ["-DLC_PROBE_MAIN"]), (PROBE_LIB, ["-fPIC", "-shared"])):
        cmd = [hipcc(), "--offload-arch=gfx950", "-O3", "-std=c++17", *extra,
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wall",
               "-o", out + ".tmp", os.path.join(CSRC, "hbm_probe.hip")]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            raise RuntimeError(f"hipcc failed with exit code {res.returncode}")
        os.replace(out + ".tmp", out)
    return HBM_PROBE


C_CLIENT_SRC = os.path.join(ROOT, "tests", "c_client", "lc_c_client.c")
C_CLIENT = os.path.join(ROOT, "tests", "c_client", "lc_c_client")


def build_c_client(verbose: bool = False, lib: str = LIB) -> str:
    """Compile the plain-C test client of the interface (gcc, C11, HIP host
    API only) against the in-tree library."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(rocm, "include"), "-I", os.path.join(ROOT, "include"),
           C_CLIENT_SRC, "-o", C_CLIENT + ".tmp",
           "-L", os.path.dirname(lib), "-l" + os.path.basename(lib)[3:-3],
           "-L", os.path.join(rocm, "lib"), "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/../../paper_2609_27193_amd", "-Wl,-rpath," + os.path.join(rocm, "lib")]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0 or res.stderr.strip():
        sys.stderr.write(res.stdout + res.stderr)
        if res.returncode != 0:
            raise RuntimeError(f"gcc failed with exit code {res.returncode}")
    os.replace(C_CLIENT + ".tmp", C_CLIENT)
    return C_CLIENT


def build_all(verbose: bool = False) -> None:
    """Everything the tests, smoke check and benchmark use: the library, then
    (in parallel) the plain-C client linked against it, the host-sanitized
    and grid-capped test builds, and the HBM probe."""
    from concurrent.futures import ThreadPoolExecutor
    build(verbose=verbose)
    jobs = [lambda: build_c_client(verbose=verbose),
            lambda: build(verbose=verbose, out=SANITIZED_LIB, sanitize=True),
            lambda: build(verbose=verbose, out=GRID_CAPPED_LIB, defines=GRID_CAP_DEFINES),
            lambda: build_hbm_probe(verbose=verbose)]
    with ThreadPoolExecutor(max_workers=len(jobs)) as pool:
        for f in [pool.submit(j) for j in jobs]:
            f.result()


if __name__ == "__main__":
    build_all(verbose=True)
