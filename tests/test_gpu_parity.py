"""GPU parity: libdisco (through its C ABI) against the fp64 oracle.

Tolerances: relative L2 over all compared elements <= 1e-5 for fp32 storage,
<= 2e-2 for bf16 storage (fp32 accumulation); small grids are compared
element by element in full, the large workloads on sampled output pixels the
oracle computes one by one (rings next to both poles, a regular subset of
rings, longitudes including the 0 / 2 pi seam).
"""
import math

import numpy as np
import pytest

from gpu_util import rel_l2, run_gpu, run_oracle, sample_pixels, say
from paper_2209_13603_amd import disco, synth

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-5
BF16_TOL = 2e-2

SMALL = [
    (8, 16, 8, 16),
    (16, 32, 8, 16),
    (12, 24, 6, 12),
    (8, 16, 16, 32),
    (10, 20, 5, 20),
    (40, 80, 40, 80),       # not a multiple of the 256-lane tile
    (33, 300, 33, 300),     # ragged tail over two tiles
]
ALGOS = ["gather_then_contract", "contract_then_gather", "fused", "fused_direct"]


@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("case", SMALL, ids=lambda c: "%dx%d_%dx%d" % c)
@pytest.mark.parametrize("op", ["forward", "transpose"])
def test_small_grids_full(case, op, algo):
    a, b, c, d = case
    tc = 3 * math.pi / min(a, c)
    args = (a, b, c, d, tc)
    B, Ci, Co = 2, 3, 5
    xs = (B, Ci, a, b) if op == "forward" else (B, Ci, c, d)
    ws = (Co, Ci, 9) if op == "forward" else (Ci, Co, 9)
    x, w = synth.random_inputs(7, xs, ws)
    say("case", case, op, algo)
    y, plan = run_gpu(args, x, w, op, algo=algo)
    ref = run_oracle(args, x, w, op)
    err = rel_l2(y, ref)
    say("  rel_l2 %.3e" % err)
    assert err <= FP32_TOL
    assert np.abs(y - ref).max() <= 1e-5 * np.abs(ref).max()
    plan.close()


def _workload_check(name, pix_per_ring=6):
    wl = synth.WORKLOADS[name]
    say("workload", name)
    x, w = synth.make_inputs(wl)
    y, plan = run_gpu(wl.plan_args(), x, w, wl.op, wl.dtype)
    nlat, nlon = wl.y_shape[2], wl.y_shape[3]
    full = nlat * nlon <= 64 * 128
    pix = None if full else sample_pixels(nlat, nlon, pix_per_ring)
    ref = run_oracle(wl.plan_args(), x, w, wl.op, pix=pix)
    got = y if full else y.reshape(y.shape[0], y.shape[1], -1)[:, :, pix]
    err = rel_l2(got, ref)
    tol = BF16_TOL if wl.dtype == "bf16" else FP32_TOL
    say("  %s rel_l2 %.3e (tol %.0e) over %d outputs" % (name, err, tol, ref.size))
    assert err <= tol
    assert np.isfinite(y).all()
    plan.close()
    return err


def test_workload_sphere32x64():
    _workload_check("sphere32x64")


def test_workload_down128x256_to_64x128():
    _workload_check("down128x256_to_64x128")


def test_workload_sphere512x1024():
    _workload_check("sphere512x1024")


def test_workload_up256x512_to_512x1024_bf16():
    _workload_check("up256x512_to_512x1024_bf16", pix_per_ring=3)


def test_workload_sphere2048x4096():
    _workload_check("sphere2048x4096", pix_per_ring=4)


SPECTRAL = [(32, 64, 32, 64), (64, 128, 64, 128), (48, 128, 48, 128), (20, 256, 20, 256)]


@pytest.mark.parametrize("case", SPECTRAL, ids=lambda c: "%dx%d" % c[:2])
@pytest.mark.parametrize("op", ["forward", "transpose"])
def test_spectral_path_small_grids(case, op, monkeypatch):
    """Rings on the spectral (DFT) path, forced down to 8 entries so that most
    rings of these small grids take it, against the oracle in full."""
    monkeypatch.setenv("DISCO_SPECTRAL_MIN_ENTRIES", "8")
    a, b, c, d = case
    tc = 3 * math.pi / min(a, c)
    plan = disco.Plan(a, b, c, d, tc)
    info = plan.info()
    key = "spectral_rings_forward" if op == "forward" else "spectral_rings_transpose"
    assert info[key] > 0
    B, Ci, Co = 2, 3, 5
    xs = (B, Ci, a, b) if op == "forward" else (B, Ci, c, d)
    ws = (Co, Ci, 9) if op == "forward" else (Ci, Co, 9)
    x, w = synth.random_inputs(8, xs, ws)
    say("spectral", case, op, info[key], "rings")
    y, _ = run_gpu(None, x, w, op, algo="fused", plan=plan)
    ref = run_oracle((a, b, c, d, tc), x, w, op)
    err = rel_l2(y, ref)
    say("  rel_l2 %.3e" % err)
    assert err <= FP32_TOL
    assert np.abs(y - ref).max() <= 1e-5 * np.abs(ref).max()
    plan.close()


@pytest.mark.parametrize("algo", ["auto", "fused_direct", "gather_then_contract"])
@pytest.mark.parametrize("op", ["forward", "transpose"])
def test_sphere2048x4096_both_ops(op, algo):
    """Forward and transpose on the 2048 x 4096 sphere (8 -> 8 channels), every
    kernel schedule, on sampled output pixels against the oracle."""
    wl = synth.WORKLOADS["sphere2048x4096"]
    a, b = wl.nlat_in, wl.nlon_in
    x, w = synth.random_inputs(21 if op == "forward" else 22, (1, 8, a, b), (8, 8, 9))
    say("2048x4096", op, algo)
    y, plan = run_gpu(wl.plan_args(), x, w, op, algo=algo)
    pix = sample_pixels(a, b, 3, seed=5)
    ref = run_oracle(wl.plan_args(), x, w, op, pix=pix)
    got = y.reshape(1, 8, -1)[:, :, pix]
    err = rel_l2(got, ref)
    say("  rel_l2 %.3e over %d outputs" % (err, ref.size))
    assert err <= FP32_TOL
    assert np.isfinite(y).all()
    plan.close()


@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("op", ["forward", "transpose"])
@pytest.mark.parametrize("chans", [(3, 5), (12, 6), (20, 9)], ids=lambda c: "%dto%d" % c)
def test_bf16_small_grids(chans, op, algo):
    """bf16 storage (fp32 accumulation; the general kernel contracts with bf16
    matrix instructions): element-wise against the oracle on the stored
    bf16 inputs, within the bf16 tolerance."""
    a, b, c, d = 16, 32, 8, 16
    tc = 3 * math.pi / c
    Ci, Co = chans
    xs = (2, Ci, a, b) if op == "forward" else (2, Ci, c, d)
    ws = (Co, Ci, 9) if op == "forward" else (Ci, Co, 9)
    x, w = synth.random_inputs(9, xs, ws, dtype="bf16")
    say("bf16", chans, op, algo)
    y, plan = run_gpu((a, b, c, d, tc), x, w, op, dtype="bf16", algo=algo)
    ref = run_oracle((a, b, c, d, tc), x, w, op)
    err = rel_l2(y, ref)
    say("  rel_l2 %.3e" % err)
    assert err <= BF16_TOL
    assert np.abs(y - ref).max() <= 3e-2 * np.abs(ref).max()
    plan.close()
