"""GPU parity of the ring-sweep kernel over groups of input channels: with more
than eight input channels the fused schedule runs one sweep launch per group
of eight, the first storing y and the later ones adding their partial sums
(fp32 atomic adds; bf16 outputs through an fp32 workspace rounded at the
end).  Checked against the fp64 oracle (relative L2 <= 1e-5 fp32, <= 2e-2
bf16), for bitwise run-to-run determinism and for bitwise equivariance under
whole-pixel longitude shifts (spectral form switched off)."""
import math

import numpy as np
import pytest

from gpu_util import rel_l2, run_gpu, run_oracle, say
from paper_2209_13603_amd import disco, synth

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-5
BF16_TOL = 2e-2

CASES = [
    (64, 128, 64, 128),
    (64, 128, 32, 64),     # stride-2 downsampling (windows too wide for the sweep: the general kernel)
    (32, 64, 64, 128),     # forward that upsamples (two longitude phases)
    (33, 300, 33, 300),    # ragged tail over two tiles
]


def _case(case, op, chans, dtype, seed, algo="fused"):
    a, b, c, d = case
    tc = 3 * math.pi / min(a, c)
    Ci, Co = chans
    xs = (2, Ci, a, b) if op == "forward" else (2, Ci, c, d)
    ws = (Co, Ci, 9) if op == "forward" else (Ci, Co, 9)
    x, w = synth.random_inputs(seed, xs, ws, dtype=dtype)
    say("groups", case, op, chans, dtype, algo)
    y, plan = run_gpu((a, b, c, d, tc), x, w, op, dtype=dtype, algo=algo)
    info = plan.info()
    swept = info["sweep_patterns_forward" if op == "forward" else "sweep_patterns_transpose"]
    return x, w, y, plan, swept


@pytest.mark.parametrize("chans", [(9, 3), (16, 12), (20, 5), (33, 32)], ids=lambda c: "%dto%d" % c)
@pytest.mark.parametrize("op", ["forward", "transpose"])
@pytest.mark.parametrize("case", CASES, ids=lambda c: "%dx%d_%dx%d" % c)
def test_channel_groups_fp32(case, op, chans):
    x, w, y, plan, swept = _case(case, op, chans, "fp32", 81)
    if case[:2] == case[2:]:
        assert swept > 0, "the sweep kernel must cover some patterns here"
    ref = run_oracle(plan.grid_in + plan.grid_out + (plan.theta_c,), x, w, op)
    err = rel_l2(y, ref)
    say("  rel_l2 %.3e" % err)
    assert err <= FP32_TOL
    assert np.abs(y - ref).max() <= 1e-5 * np.abs(ref).max()
    plan.close()


@pytest.mark.parametrize("chans", [(12, 6), (64, 32)], ids=lambda c: "%dto%d" % c)
@pytest.mark.parametrize("op", ["forward", "transpose"])
@pytest.mark.parametrize("case", CASES[:3], ids=lambda c: "%dx%d_%dx%d" % c)
def test_channel_groups_bf16(case, op, chans):
    x, w, y, plan, swept = _case(case, op, chans, "bf16", 82)
    if case[:2] == case[2:]:
        assert swept > 0
    ref = run_oracle(plan.grid_in + plan.grid_out + (plan.theta_c,), x, w, op)
    err = rel_l2(y, ref)
    say("  rel_l2 %.3e" % err)
    assert err <= BF16_TOL
    plan.close()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_channel_groups_deterministic(dtype):
    case = CASES[0]
    x, w, y1, plan, _ = _case(case, "forward", (20, 7), dtype, 83)
    y2, _ = run_gpu(None, x, w, "forward", dtype=dtype, algo="fused", plan=plan)
    assert np.array_equal(y1, y2)
    plan.close()


def test_channel_groups_shift_equivariant_bitwise(monkeypatch):
    """Without the spectral form every ring is gathered directly, and each
    lane's order of accumulation (entries, then channel groups in launch
    order) does not depend on its longitude."""
    monkeypatch.setenv("DISCO_SPECTRAL_MIN_ENTRIES", "1000000")
    a, b = 64, 128
    plan = disco.Plan(a, b, a, b, 3 * math.pi / a)
    assert plan.info()["spectral_rings_forward"] == 0
    x, w = synth.random_inputs(84, (2, 12, a, b), (5, 12, 9))
    y, _ = run_gpu(None, x, w, "forward", algo="fused", plan=plan)
    ys, _ = run_gpu(None, np.roll(x, 7, axis=-1), w, "forward", algo="fused", plan=plan)
    assert np.array_equal(ys, np.roll(y, 7, axis=-1))
    plan.close()
