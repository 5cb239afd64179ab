"""The range-checking build (DISCO_DEBUG_BOUNDS, libdisco_debug_bounds.so):
every kernel family runs through it in a process of its own
(tests/debug_bounds_run.py) with oracle parity and no failed psi-index
check."""
import os
import subprocess
import sys

import pytest

from paper_2209_13603_amd.build import DEBUG_BOUNDS_LIB_PATH

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


def test_kernels_keep_their_psi_indices_in_range():
    if not os.path.exists(DEBUG_BOUNDS_LIB_PATH):
        pytest.fail("libdisco_debug_bounds.so not built: python -m paper_2209_13603_amd.build --debug-bounds")
    env = dict(os.environ, DISCO_LIBRARY=DEBUG_BOUNDS_LIB_PATH)
    r = subprocess.run([sys.executable, "-u", os.path.join(HERE, "debug_bounds_run.py")], env=env,
                       capture_output=True, text=True, timeout=600)
    print(r.stdout[-4000:])
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert r.stdout.strip().endswith("OK")
