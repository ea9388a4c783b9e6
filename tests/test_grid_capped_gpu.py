"""GPU: work beyond one dispatch's grid.  Kernels take one work item per
block up to the 2^32 work-item dispatch limit; beyond it the score and copy
kernels are launched again over the next range of items and the optimizer
kernels loop.  The parity tests rarely reach the limit, so a build with
every grid capped at 40 blocks (`__graft_entry__.build()` makes it) runs the
parity, edge and optimizer tests again in a child process: the score and
copy kernels then run as many consecutive launches, the optimizer kernels
over many rounds."""
import os
import subprocess
import sys

import pytest

from paper_2609_27193_amd.build_lib import GRID_CAPPED_LIB
from tests.conftest import gpu_available

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_parity_with_capped_grids():
    if not gpu_available():
        pytest.skip("needs an MI355X")
    assert os.path.exists(GRID_CAPPED_LIB), "the grid-capped build is made by __graft_entry__.build()"
    env = dict(os.environ, LAYERCHECK_LIB=GRID_CAPPED_LIB)
    r = subprocess.run([sys.executable, "-u", "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "gpu",
                        "--timeout", "300", "--timeout-method", "thread",
                        "tests/test_parity_gpu.py", "tests/test_edges_gpu.py", "tests/test_adamw_gpu.py",
                        "-k", "not 4gib and not many_layers"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    print(tail.strip().splitlines()[-1], flush=True)
