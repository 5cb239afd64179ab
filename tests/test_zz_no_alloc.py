"""disco_forward_noalloc (the forward op with its scratch memory in the
library's fixed per-GPU array) against disco_forward on the same inputs,
through the C ABI: several calls in a row on one GPU, each smaller than the
one before (so every call runs on what the previous one left in the array),
to the fp32 parity bar; a call that needs more scratch than the array holds
is rejected before anything is enqueued."""
import math

import numpy as np
import pytest

from gpu_util import rel_l2, say, to_numpy, torch_dev
import oracle
from paper_2209_13603_amd import disco, synth

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-5

# (plan args, batch, c_in, c_out), largest scratch first.
CALLS = [
    ((2048, 4096, 2048, 4096, 3 * math.pi / 2048), 1, 8, 8),   # spectral + sweep + general kernel
    ((512, 1024, 512, 1024, 3 * math.pi / 512), 2, 32, 32),    # sweep channel groups
    ((128, 256, 64, 128, 3 * math.pi / 64), 4, 16, 16),        # one general-kernel launch
    ((32, 64, 32, 64, 3 * math.pi / 32), 1, 4, 4),             # split patterns, partial slots
]


def _inputs(seed, args, B, Ci, Co):
    import torch
    g = torch.Generator(device="cuda:0").manual_seed(seed)
    x = torch.randn((B, Ci, args[0], args[1]), generator=g, device="cuda:0")
    w = torch.randn((Co, Ci, 9), generator=g, device="cuda:0") / math.sqrt(Ci * 9)
    return x, w


def test_noalloc_matches_forward_on_successive_calls():
    import torch
    for i, (args, B, Ci, Co) in enumerate(CALLS):
        say("noalloc call", i, args[:4], "B", B, "channels", Ci, Co)
        plan = disco.Plan(*args)
        x, w = _inputs(100 + i, args, B, Ci, Co)
        ref = plan.forward(x, w)
        y = torch.full_like(ref, float("nan"))
        plan.forward_noalloc(x, w, y)
        torch.cuda.synchronize()
        got, want = to_numpy(y), to_numpy(ref)
        err = rel_l2(got, want)
        mx = float(np.abs(got - want).max())
        say("  rel_l2 %.3e max abs diff %.3e" % (err, mx))
        assert np.isfinite(got).all()
        assert err <= FP32_TOL
        assert mx <= FP32_TOL * float(np.abs(want).max())
        plan.close()


def test_noalloc_small_against_oracle():
    """The smallest call also against the oracle itself."""
    import torch
    wl = synth.WORKLOADS["sphere32x64"]
    x, w = synth.make_inputs(wl)
    plan = disco.Plan(*wl.plan_args())
    y = torch.empty((1, 4, 32, 64), device="cuda:0")
    plan.forward_noalloc(torch_dev(x), torch_dev(w), y)
    torch.cuda.synchronize()
    ref = oracle.default().forward(*wl.plan_args(), x.astype(np.float64), w.astype(np.float64))
    err = rel_l2(to_numpy(y), ref)
    say("noalloc sphere32x64 vs oracle rel_l2 %.3e" % err)
    assert err <= FP32_TOL
    plan.close()


def test_noalloc_rejects_scratch_beyond_its_array():
    """bf16 storage with 32 input channels on 512 x 1024 accumulates fp32
    partial outputs of 2 x 32 x 512 x 1024 floats (134 MB): more than the
    array holds, so the call fails before writing anything."""
    import torch
    args = (512, 1024, 512, 1024, 3 * math.pi / 512)
    plan = disco.Plan(*args)
    x = torch.ones((2, 32, 512, 1024), device="cuda:0", dtype=torch.bfloat16)
    w = torch.ones((32, 32, 9), device="cuda:0", dtype=torch.bfloat16)
    y = torch.full((2, 32, 512, 1024), 7.0, device="cuda:0", dtype=torch.bfloat16)
    with pytest.raises(disco.DiscoError) as ei:
        plan.forward_noalloc(x, w, y)
    assert ei.value.status == disco.DISCO_ERR_UNSUPPORTED
    assert "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())
    plan.close()
