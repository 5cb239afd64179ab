"""Runs every kernel family of the library once through the range-checking
build (DISCO_LIBRARY names it; run by tests/test_gpu_debug_bounds.py in a
process of its own) and checks each output against the oracle and that no
psi-index range check failed.  Prints one line per case and a final "OK"."""
import math
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)
sys.path.insert(0, os.path.dirname(HERE))

import numpy as np  # noqa: E402
import torch  # noqa: E402

import oracle  # noqa: E402
from gpu_util import rel_l2, run_gpu, run_oracle, say, to_numpy, torch_dev  # noqa: E402
from paper_2209_13603_amd import disco, synth  # noqa: E402


def check(name, err, tol):
    say("%-58s rel_l2 %.3e" % (name, err))
    assert err <= tol, name


def main():
    torch.zeros(1, device="cuda:0")
    assert disco.debug_bounds_violations() == 0, "flags set before any call"
    # 3x3 basis, fp32, forward: the sweep, the spectral rings and the general
    # kernel (algo fused), then the general kernel alone on 64- and 128-lane
    # tiles (lane groups), and a stride-2 op with two channel passes.
    a, b = 64, 128
    args = (a, b, a, b, 3 * math.pi / a)
    x, w = synth.random_inputs(11, (2, 4, a, b), (5, 4, 9))
    for algo in ("fused", "fused_direct", "gather_then_contract"):
        y, plan = run_gpu(args, x, w, "forward", algo=algo)
        check("3x3 fp32 64x128 forward %s" % algo, rel_l2(y, run_oracle(args, x, w, "forward")), 1e-5)
        plan.close()
    for case, chans in (((32, 64, 32, 64), (4, 4)), ((128, 256, 64, 128), (16, 16)), ((64, 128, 32, 64), (3, 20))):
        a2, b2, c2, d2 = case
        args2 = (a2, b2, c2, d2, 3 * math.pi / min(a2, c2))
        x2, w2 = synth.random_inputs(12, (2, chans[0], a2, b2), (chans[1], chans[0], 9))
        y, plan = run_gpu(args2, x2, w2, "forward")
        check("3x3 fp32 %dx%d->%dx%d %d->%d auto" % (case + chans), rel_l2(y, run_oracle(args2, x2, w2, "forward")),
              1e-5)
        plan.close()
    # Transposed op, bf16: the matrix-core kernel.
    args3 = (64, 128, 32, 64, 3 * math.pi / 32)
    x3, w3 = synth.random_inputs(13, (2, 24, 32, 64), (24, 20, 9), dtype="bf16")
    y, plan = run_gpu(args3, x3, w3, "transpose", dtype="bf16", algo="matrix_core")
    check("3x3 bf16 32x64->64x128 transpose matrix_core", rel_l2(y, run_oracle(args3, x3, w3, "transpose")), 2e-2)
    plan.close()
    # Axisymmetric basis on the pole grid: the blocked stencil; with several
    # output channels the general stencil.
    for chans in ((1, 1), (3, 5)):
        a4, b4 = 41, 80
        args4 = (a4, b4, a4, b4, 3 * math.pi / (a4 - 1))
        x4, w4 = synth.random_inputs(14, (2, chans[0], a4, b4), (chans[1], chans[0], 4))
        y, plan = run_gpu(args4, x4, w4, "forward", plan_kw={"basis": "axisym4", "sampling": "poles"})
        check("axisym poles 41x80 %d->%d" % chans,
              rel_l2(y, run_oracle(args4, x4, w4, "forward", basis=1, sampling=1)), 1e-5)
        plan.close()
    # Separable basis, depthwise channels.
    a5, b5 = 32, 64
    args5 = (a5, b5, a5, b5, 3 * math.pi / a5)
    x5, w5 = synth.random_inputs(15, (2, 3, a5, b5), (3, 16), c_in=1)
    plan = disco.Plan(*args5, basis="separable4x4")
    y = to_numpy(plan.forward_depthwise(torch_dev(x5), torch_dev(w5)))
    ref = run_oracle(args5, x5, oracle.depthwise_weights(w5.astype(np.float64)), "forward", basis=2)
    check("separable depthwise 32x64 C=3", rel_l2(y, ref), 1e-5)
    plan.close()
    n = disco.debug_bounds_violations()
    say("range-check failures: %d kernel files" % n)
    assert n == 0
    say("OK")


if __name__ == "__main__":
    main()
