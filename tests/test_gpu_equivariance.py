"""The equivariance harness (App. D) run on the library's op on the GPU: its
errors equal the oracle's (the same op to fp32 rounding: rows the oracle
puts at rounding level, the rotations about z, are at fp32 rounding level on
the GPU) and have the shape of Table 5 at L = 64."""
import numpy as np
import pytest

import equivariance as E
from gpu_util import say

pytestmark = pytest.mark.gpu


def test_gpu_equivariance_errors_match_the_oracle():
    gpu = E.table(E.GpuOps(), [24], n_signals=2, n_rotations=2)
    cpu = E.table(E.OracleOps(), [24], n_signals=2, n_rotations=2)
    for g, c in zip(gpu, cpu):
        say("  %s %s %s: gpu %.5f%% oracle %.5f%%" % (g[1], g[2], g[3], g[4], c[4]))
        assert g[:4] == c[:4]
        assert abs(g[4] - c[4]) <= 1e-3 * c[4] + 1e-3     # percent: fp32 rounding is ~1e-5 relative


def test_gpu_equivariance_table_shape():
    rows = E.table(E.GpuOps(), [32, 64], n_signals=3, n_rotations=3)
    say(E.format_rows(rows))
    err = {(L, k, c, b): m for (L, k, c, b, m, *_) in rows}
    for L in (32, 64):
        assert err[(L, "axisym", "best", None)] < err[(L, "axisym", "worst", None)]
        for c in ("best", "worst"):
            assert err[(L, "directional", c, 0.0)] < err[(L, "directional", c, 5.0)] \
                < err[(L, "directional", c, 10.0)]
    # the axisymmetric errors do not grow with resolution (Table 5's flat column)
    a32, a64 = err[(32, "axisym", "best", None)], err[(64, "axisym", "best", None)]
    assert a64 <= 1.5 * a32
