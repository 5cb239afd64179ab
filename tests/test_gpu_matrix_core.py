"""The bf16 matrix-core kernel (algo "matrix_core", and what "auto" and
"fused" run for bf16 storage where the op allows it) against the fp64
oracle on the stored bf16 inputs: element by element on small and mid-size
grids (forward and transposed ops, one and two longitude phases, strides 1
and 2, ragged longitude tiles, rings cut into several segments near the
poles, channel counts that are not multiples of the kernel's blocks), within
the bf16 tolerance (relative L2 <= 2e-2, largest error <= 3e-2 of the largest
output).  Also: determinism, bitwise equivariance under whole-pixel
longitude shifts, the refusal of ops the layout does not cover, and the
fallback of "auto" on them."""
import math

import numpy as np
import pytest

from gpu_util import rel_l2, run_gpu, run_oracle, say, torch_dev
from paper_2209_13603_amd import disco, synth

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2

CASES = [
    (8, 16, 8, 16),
    (16, 32, 8, 16),        # forward stride 2; transposed: two phases
    (8, 16, 16, 32),
    (40, 80, 40, 80),
    (33, 296, 33, 296),     # two longitude tiles, the second ragged
    (64, 128, 32, 64),      # polar rings cut into several segments
]
CHANS = [(3, 5), (8, 16), (24, 20), (9, 33)]


def _inputs(case, op, chans, seed, B=2):
    a, b, c, d = case
    Ci, Co = chans
    xs = (B, Ci, a, b) if op == "forward" else (B, Ci, c, d)
    ws = (Co, Ci, 9) if op == "forward" else (Ci, Co, 9)
    return synth.random_inputs(seed, xs, ws, dtype="bf16")


@pytest.mark.parametrize("chans", CHANS, ids=lambda c: "%dto%d" % c)
@pytest.mark.parametrize("case", CASES, ids=lambda c: "%dx%d_%dx%d" % c)
@pytest.mark.parametrize("op", ["forward", "transpose"])
def test_matrix_core_against_oracle(case, op, chans):
    a, b, c, d = case
    args = (a, b, c, d, 3 * math.pi / min(a, c))
    x, w = _inputs(case, op, chans, 91)
    say("matrix_core", case, op, chans)
    y, plan = run_gpu(args, x, w, op, dtype="bf16", algo="matrix_core")
    ref = run_oracle(args, x, w, op)
    err = rel_l2(y, ref)
    mx = float(np.abs(y - ref).max() / np.abs(ref).max())
    say("  rel_l2 %.3e max %.3e" % (err, mx))
    assert err <= BF16_TOL
    assert mx <= 3e-2
    plan.close()


@pytest.mark.parametrize("op", ["forward", "transpose"])
def test_auto_and_fused_take_the_matrix_cores_for_bf16(op):
    case, chans = (16, 32, 8, 16), (8, 16)
    a, b, c, d = case
    args = (a, b, c, d, 3 * math.pi / min(a, c))
    x, w = _inputs(case, op, chans, 92)
    plan = disco.Plan(*args)
    ys = {al: run_gpu(None, x, w, op, dtype="bf16", algo=al, plan=plan)[0]
          for al in ("matrix_core", "auto", "fused", "fused_direct")}
    assert np.array_equal(ys["auto"], ys["matrix_core"])
    assert np.array_equal(ys["fused"], ys["matrix_core"])
    for al in ("auto", "fused"):
        assert "mfma_gather_contract" in plan.kernel_work(op == "transpose", al, *chans, dtype="bf16")
    # the general kernel (bf16 Z, fp32 values) agrees within the bf16 tolerance
    assert rel_l2(ys["matrix_core"], ys["fused_direct"]) <= BF16_TOL
    plan.close()


def test_deterministic_and_shift_equivariant():
    """Two runs give the same bits; rolling the input by one longitude of
    the coarse grid rolls the two-phase output by two longitudes, bitwise."""
    import torch
    case, chans = (64, 128, 32, 64), (24, 20)
    a, b, c, d = case
    plan = disco.Plan(a, b, c, d, 3 * math.pi / c)
    x, w = _inputs(case, "transpose", chans, 93)
    xt, wt = torch_dev(x, "bf16"), torch_dev(w, "bf16")
    y1 = plan.transpose(xt, wt, algo="matrix_core")
    y2 = plan.transpose(xt, wt, algo="matrix_core")
    ys = plan.transpose(torch.roll(xt, 1, dims=3).contiguous(), wt, algo="matrix_core")
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    assert torch.equal(torch.roll(y1, 2, dims=3), ys)
    plan.close()


def test_uncovered_ops_are_refused_and_auto_falls_back():
    """nlon_in = 300 is not a multiple of 8: the explicit algo is refused,
    "auto" runs the general kernel and stays within the tolerance."""
    case, chans = (33, 300, 33, 300), (3, 5)
    a, b, c, d = case
    args = (a, b, c, d, 3 * math.pi / a)
    x, w = _inputs(case, "forward", chans, 94)
    plan = disco.Plan(*args)
    with pytest.raises(disco.DiscoError) as ei:
        run_gpu(None, x, w, "forward", dtype="bf16", algo="matrix_core", plan=plan)
    assert ei.value.status == disco.DISCO_ERR_UNSUPPORTED
    y, _ = run_gpu(None, x, w, "forward", dtype="bf16", algo="auto", plan=plan)
    assert rel_l2(y, run_oracle(args, x, w, "forward")) <= BF16_TOL
    assert "mfma_gather_contract" not in plan.kernel_work(False, "auto", *chans, dtype="bf16")
    plan.close()


def test_fp32_is_refused():
    case, chans = (16, 32, 8, 16), (3, 5)
    a, b, c, d = case
    plan = disco.Plan(a, b, c, d, 3 * math.pi / c)
    x, w = synth.random_inputs(95, (1, 3, a, b), (5, 3, 9))
    with pytest.raises(disco.DiscoError) as ei:
        run_gpu(None, x, w, "forward", algo="matrix_core", plan=plan)
    assert ei.value.status == disco.DISCO_ERR_UNSUPPORTED
    plan.close()
