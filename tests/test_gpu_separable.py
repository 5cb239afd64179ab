"""GPU parity of the separable basis (Sec. 3.4: four nodes along theta times
four periodic nodes along the direction, K = 16) and of depthwise channels
(Sec. 4.2: each channel filtered by its own filter) through the C ABI
against the fp64 oracle.

Tolerances as the other parity tests: relative L2 <= 1e-5 for fp32 storage,
<= 2e-2 for bf16.  Small grids are compared in full (several 256-lane tiles
and ragged tails among them); the 2048 x 4096 workload on sampled outputs.
"""
import math

import numpy as np
import pytest

from gpu_util import rel_l2, run_gpu, run_oracle, sample_pixels, say, to_numpy, torch_dev
import oracle
from paper_2209_13603_amd import disco, synth

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-5
BF16_TOL = 2e-2
BASES = {"bilinear3x3": (0, 9), "axisym4": (1, 4), "separable4x4": (2, 16)}

CASES = [
    # (nlat_in, nlon_in, nlat_out, nlon_out, sampling)
    (9, 16, 9, 16, "poles"),
    (17, 32, 9, 16, "poles"),
    (9, 16, 17, 32, "poles"),
    (151, 300, 151, 300, "poles"),    # ragged tail over two tiles
    (16, 32, 8, 16, "cell_centred"),
    (8, 16, 16, 32, "cell_centred"),
    (33, 300, 33, 300, "cell_centred"),
    (64, 1100, 64, 1100, "cell_centred"),  # two 1024-longitude tiles of the blocked kernel
]


def _tc(case):
    a, b, c, d, smp = case
    return 3 * math.pi / (min(a, c) - (1 if smp == "poles" else 0))


def _ids(c):
    return "%dx%d_%dx%d_%s" % c


def _sep_case(case, op, chans, dtype, seed):
    a, b, c, d, smp = case
    tc = _tc(case)
    Ci, Co = chans
    xs = (2, Ci, a, b) if op == "forward" else (2, Ci, c, d)
    ws = (Co, Ci, 16) if op == "forward" else (Ci, Co, 16)
    x, w = synth.random_inputs(seed, xs, ws, dtype=dtype)
    say("separable", case, op, chans, dtype)
    y, plan = run_gpu((a, b, c, d, tc), x, w, op, dtype=dtype,
                      plan_kw={"basis": "separable4x4", "sampling": smp})
    assert plan.info()["K"] == 16
    ref = run_oracle((a, b, c, d, tc), x, w, op, basis=2, sampling=1 if smp == "poles" else 0)
    err = rel_l2(y, ref)
    say("  rel_l2 %.3e" % err)
    plan.close()
    return y, ref, err


@pytest.mark.parametrize("chans", [(1, 1), (3, 1), (2, 3), (3, 5), (9, 12)], ids=lambda c: "%dto%d" % c)
@pytest.mark.parametrize("op", ["forward", "transpose"])
@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_separable_small_grids_full(case, op, chans):
    y, ref, err = _sep_case(case, op, chans, "fp32", 41)
    assert err <= FP32_TOL
    assert np.abs(y - ref).max() <= 1e-5 * np.abs(ref).max()


@pytest.mark.parametrize("op", ["forward", "transpose"])
@pytest.mark.parametrize("case", CASES[:3] + CASES[4:6], ids=_ids)
def test_separable_bf16(case, op):
    y, ref, err = _sep_case(case, op, (3, 5), "bf16", 42)
    assert err <= BF16_TOL


def test_separable_with_equal_phi_nodes_is_the_axisymmetric_op():
    """W_sep[., ., 4a + b] = W_ax[., ., a] for every b: the phi hats sum to one
    in every direction, so the GPU's separable op equals its axisymmetric op."""
    a, b = 41, 80
    tc = 3 * math.pi / 40
    x, w4 = synth.random_inputs(43, (2, 3, a, b), (2, 3, 4))
    w16 = np.repeat(w4, 4, axis=2)
    y4, p4 = run_gpu((a, b, a, b, tc), x, w4, "forward", plan_kw={"basis": "axisym4", "sampling": "poles"})
    y16, p16 = run_gpu((a, b, a, b, tc), x, w16, "forward",
                       plan_kw={"basis": "separable4x4", "sampling": "poles"})
    err = rel_l2(y16, y4)
    say("separable vs axisymmetric rel_l2 %.3e" % err)
    assert err <= 1e-6
    p4.close()
    p16.close()


# --------------------------------------------------------------------------- #
# Depthwise channels, every basis.
# --------------------------------------------------------------------------- #
def _run_dw(plan, x, w, op, dtype="fp32"):
    import torch
    xt, wt = torch_dev(x, dtype), torch_dev(w, dtype)
    y = plan.forward_depthwise(xt, wt) if op == "forward" else plan.transpose_depthwise(xt, wt)
    torch.cuda.synchronize()
    return to_numpy(y)


def _dw_case(case, op, basis, C, dtype, seed):
    a, b, c, d, smp = case
    tc = _tc(case)
    code, K = BASES[basis]
    xs = (2, C, a, b) if op == "forward" else (2, C, c, d)
    x, w = synth.random_inputs(seed, xs, (C, K), dtype=dtype, c_in=1)
    say("depthwise", case, op, basis, C, dtype)
    plan = disco.Plan(a, b, c, d, tc, basis=basis, sampling=smp)
    y = _run_dw(plan, x, w, op, dtype)
    ref = run_oracle((a, b, c, d, tc), x, oracle.depthwise_weights(w.astype(np.float64)), op,
                     basis=code, sampling=1 if smp == "poles" else 0)
    err = rel_l2(y, ref)
    say("  rel_l2 %.3e" % err)
    return plan, x, w, y, ref, err


@pytest.mark.parametrize("C", [1, 3, 8])
@pytest.mark.parametrize("basis", list(BASES))
@pytest.mark.parametrize("op", ["forward", "transpose"])
@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_depthwise_small_grids_full(case, op, basis, C):
    plan, x, w, y, ref, err = _dw_case(case, op, basis, C, "fp32", 51)
    plan.close()
    assert err <= FP32_TOL
    assert np.abs(y - ref).max() <= 1e-5 * np.abs(ref).max()


@pytest.mark.parametrize("basis", list(BASES))
@pytest.mark.parametrize("op", ["forward", "transpose"])
@pytest.mark.parametrize("case", [CASES[1], CASES[4], CASES[6]], ids=_ids)
def test_depthwise_bf16(case, op, basis):
    plan, x, w, y, ref, err = _dw_case(case, op, basis, 5, "bf16", 52)
    plan.close()
    assert err <= BF16_TOL


@pytest.mark.parametrize("basis", ["axisym4", "separable4x4"])
@pytest.mark.parametrize("op", ["forward", "transpose"])
@pytest.mark.parametrize("case", [CASES[1], CASES[3], CASES[6]], ids=_ids)
def test_depthwise_equals_one_channel_ops_bitwise(case, op, basis):
    """Channel c of a depthwise call equals the full op run on channel c alone
    with W = w[c] (both fold W into psi in the same kernels and order)."""
    plan, x, w, y, ref, err = _dw_case(case, op, basis, 4, "fp32", 53)
    for c in range(4):
        yc, _ = run_gpu(None, np.ascontiguousarray(x[:, c:c + 1]), np.ascontiguousarray(w[c][None, None, :]),
                        op, plan=plan)
        assert np.array_equal(yc[:, 0], y[:, c]), c
    plan.close()


def test_depthwise_argument_errors():
    a, b = 16, 32
    plan = disco.Plan(a, b, a, b, 3 * math.pi / 16, basis="separable4x4")
    import torch
    x = torch.zeros((2, 3, a, b), device="cuda:0")
    y = torch.zeros((2, 3, a, b), device="cuda:0")
    cases = [
        (x, torch.zeros((3, 9), device="cuda:0"), y, disco.DISCO_ERR_SHAPE),       # K of another basis
        (x, torch.zeros((4, 16), device="cuda:0"), y, disco.DISCO_ERR_SHAPE),      # C mismatch
        (x, torch.zeros((3, 3, 16), device="cuda:0"), y, disco.DISCO_ERR_SHAPE),   # full W
        (x, torch.zeros((3, 16), device="cuda:0"), torch.zeros((2, 4, a, b), device="cuda:0"),
         disco.DISCO_ERR_SHAPE),                                                      # y channels
        (x, torch.zeros((3, 16), device="cuda:0", dtype=torch.bfloat16), y, disco.DISCO_ERR_DTYPE),
    ]
    for xx, ww, yy, st in cases:
        with pytest.raises(disco.DiscoError) as ei:
            plan.forward_depthwise(xx, ww, yy)
        assert ei.value.status == st, (tuple(ww.shape), ei.value)
    with pytest.raises(disco.DiscoError) as ei:
        plan.forward_depthwise(x, torch.zeros((3, 16), device="cuda:0"), x)  # y aliases x
    assert ei.value.status == disco.DISCO_ERR_INVALID_ARGUMENT
    # an empty batch enqueues nothing and succeeds
    plan.forward_depthwise(torch.zeros((0, 3, a, b), device="cuda:0"), torch.zeros((3, 16), device="cuda:0"),
                           torch.zeros((0, 3, a, b), device="cuda:0"))
    plan.close()


@pytest.mark.parametrize("name", ["sphere2048x4096_separable_dw", "up256x512_to_512x1024_separable_dw"])
def test_workload_separable_depthwise(name):
    """The separable depthwise workloads at full size, on sampled outputs
    (rings next to both poles and the seam included)."""
    wl = synth.WORKLOADS[name]
    x, w = synth.make_inputs(wl)
    say("workload", name)
    plan = disco.Plan(*wl.plan_args(), **wl.plan_kwargs())
    y = _run_dw(plan, x, w, wl.op)
    nlat, nlon = wl.y_shape[2], wl.y_shape[3]
    pix = sample_pixels(nlat, nlon, 3)
    ref = run_oracle(wl.plan_args(), x, oracle.depthwise_weights(w.astype(np.float64)), wl.op, pix=pix,
                     **wl.oracle_kwargs())
    got = y.reshape(y.shape[0], y.shape[1], -1)[:, :, pix]
    err = rel_l2(got, ref)
    say("  %s rel_l2 %.3e over %d outputs" % (name, err, ref.size))
    assert err <= FP32_TOL
    assert np.isfinite(y).all()
    plan.close()


# --------------------------------------------------------------------------- #
# Gradients of the depthwise ops (App. C per channel): dx through the adjoint
# run depthwise, dw the diagonal blocks of the full weight gradient.
# --------------------------------------------------------------------------- #
GRAD_CASES = [
    (16, 32, 8, 16, "cell_centred"),
    (33, 300, 33, 300, "cell_centred"),
    (17, 32, 9, 16, "poles"),
    (41, 80, 41, 80, "poles"),
]


def _dw_grad(case, transpose, basis, C, dtype, seed):
    import torch
    a, b, c, d, smp = case
    tc = _tc(case)
    code, K = BASES[basis]
    xs = (2, C, c, d) if transpose else (2, C, a, b)
    ys = (2, C, a, b) if transpose else (2, C, c, d)
    r = np.random.default_rng(seed)
    x = synth.to_storage(r.standard_normal(xs), dtype)
    w = synth.to_storage(r.standard_normal((C, K)) / math.sqrt(K), dtype)
    dy = synth.to_storage(r.standard_normal(ys), dtype)
    say("depthwise backward", case, "transpose" if transpose else "forward", basis, C, dtype)
    plan = disco.Plan(a, b, c, d, tc, basis=basis, sampling=smp, backward=True)
    fn = disco.transpose_depthwise_backward if transpose else disco.forward_depthwise_backward
    dx, dw = fn(plan, torch_dev(x, dtype), torch_dev(w, dtype), torch_dev(dy, dtype))
    torch.cuda.synchronize()
    o = oracle.default()
    kw = {"sampling": 1 if smp == "poles" else 0, "basis": code}
    wfull = oracle.depthwise_weights(w.astype(np.float64))
    ref_dx = o.input_grad(a, b, c, d, tc, dy.astype(np.float64), wfull, transpose=transpose, **kw)
    ref_full = o.weight_grad(a, b, c, d, tc, x.astype(np.float64), dy.astype(np.float64), transpose=transpose, **kw)
    ref_dw = np.stack([ref_full[ch, ch] for ch in range(C)])
    plan.close()
    return to_numpy(dx), to_numpy(dw), ref_dx, ref_dw


@pytest.mark.parametrize("basis", list(BASES))
@pytest.mark.parametrize("transpose", [False, True], ids=["forward", "transpose"])
@pytest.mark.parametrize("case", GRAD_CASES, ids=_ids)
def test_depthwise_gradients(case, transpose, basis):
    dx, dw, rdx, rdw = _dw_grad(case, transpose, basis, 3, "fp32", 61)
    ex, ew = rel_l2(dx, rdx), rel_l2(dw, rdw)
    say("  dx rel_l2 %.3e  dw rel_l2 %.3e" % (ex, ew))
    assert ex <= FP32_TOL and ew <= FP32_TOL


@pytest.mark.parametrize("basis", list(BASES))
@pytest.mark.parametrize("transpose", [False, True], ids=["forward", "transpose"])
def test_depthwise_gradients_bf16(transpose, basis):
    dx, dw, rdx, rdw = _dw_grad(GRAD_CASES[0], transpose, basis, 5, "bf16", 62)
    ex, ew = rel_l2(dx, rdx), rel_l2(dw, rdw)
    say("  bf16 dx %.3e dw %.3e" % (ex, ew))
    assert ex <= BF16_TOL and ew <= BF16_TOL


def test_depthwise_gradients_match_the_full_op():
    """On the GPU: the depthwise gradients equal the full-W gradients of the
    diagonal W (dx to rounding, dw the diagonal blocks)."""
    import torch
    a, b = 33, 300
    tc = 3 * math.pi / 33
    plan = disco.Plan(a, b, a, b, tc, basis="separable4x4", backward=True)
    r = np.random.default_rng(63)
    C = 4
    x = r.standard_normal((2, C, a, b)).astype(np.float32)
    dy = r.standard_normal((2, C, a, b)).astype(np.float32)
    w = (r.standard_normal((C, 16)) / 4).astype(np.float32)
    dx, dw = disco.forward_depthwise_backward(plan, torch_dev(x), torch_dev(w), torch_dev(dy))
    wf = oracle.depthwise_weights(w.astype(np.float64)).astype(np.float32)
    dxf, dwf = disco.forward_backward(plan, torch_dev(x), torch_dev(wf), torch_dev(dy))
    torch.cuda.synchronize()
    assert rel_l2(to_numpy(dx), to_numpy(dxf)) <= 1e-6
    full = to_numpy(dwf)
    assert rel_l2(to_numpy(dw), np.stack([full[c, c] for c in range(C)])) <= 1e-6
    plan.close()


def test_depthwise_gradient_errors():
    import torch
    a, b = 16, 32
    plan = disco.Plan(a, b, a, b, 3 * math.pi / 16, basis="axisym4", backward=True)
    x = torch.zeros((2, 3, a, b), device="cuda:0")
    dy = torch.zeros((2, 3, a, b), device="cuda:0")
    w = torch.zeros((3, 4), device="cuda:0")
    with pytest.raises(disco.DiscoError) as ei:       # dw of the full layout
        disco._backward(plan, "disco_forward_depthwise_backward", x, w, dy, None,
                        torch.zeros((3, 3, 4), device="cuda:0"), None)
    assert ei.value.status == disco.DISCO_ERR_SHAPE
    with pytest.raises(disco.DiscoError) as ei:       # dy with other channels
        disco.forward_depthwise_backward(plan, x, w, torch.zeros((2, 4, a, b), device="cuda:0"))
    assert ei.value.status == disco.DISCO_ERR_SHAPE
    plan2 = disco.Plan(a, b, a, b, 3 * math.pi / 16, basis="axisym4")
    with pytest.raises(disco.DiscoError) as ei:       # plan without the backward flag
        disco.forward_depthwise_backward(plan2, x, w, dy)
    assert ei.value.status == disco.DISCO_ERR_UNSUPPORTED
    plan.close()
    plan2.close()
