"""Benchmark of the DISCO forward op on the 2048 x 4096 sphere (one MI355X).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--algo A]

One step = one full forward op (psi gather + channel contraction) over one
batch of synthetic input already resident in HBM.  Prints ONE JSON line on
stdout; diagnostics go to stderr.  `roofline` describes the step's dominant
kernel from HIP events recorded around every kernel launch inside the timed
steps; `cpu_baseline` times the fp64 oracle on a bounded random sample of the
same workload's output pixels on this host's cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "DISCO fwd output pix*chan/s at 2048x4096; achieved HBM GB/s vs peak"
UNIT = "pix*chan/s"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP32_VALU_PEAK_TFLOPS = 157.3  # MI355X fp32 vector (published)
FP32_MFMA_PEAK_TFLOPS = 157.3
BF16_MFMA_PEAK_TFLOPS = 2500.0
KERNEL_SOURCE = os.path.join(ROOT, "paper_2209_13603_amd", "csrc", "disco_kernels.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_digest() -> str:
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def kernel_model(name, wl, info, es):
    """Algorithmic (bytes, flops, bound) of one launch of kernel `name`.

    Per unit figures (one unit = one output pixel x one channel of the
    kernel's output): gather_z reads x once and writes 9 fp32 Z planes;
    contract_z reads Z and writes y; contract_x reads x and writes 9 fp32
    planes per output channel; gather_y reads those planes and writes y; a
    fused kernel reads x once and writes y once.
    """
    B = wl.batch
    Ci, Co = wl.c_in, wl.c_out
    if wl.op == "forward":
        n_in, n_out = wl.nlat_in * wl.nlon_in, wl.nlat_out * wl.nlon_out
    else:
        n_in, n_out = wl.nlat_out * wl.nlon_out, wl.nlat_in * wl.nlon_in
    pairs = info["nnz_pairs_total"] if wl.op == "forward" else None
    if pairs is None:
        # The transposed op visits the same (pixel, pixel, k) triples.
        pairs = info["nnz_pairs_total"]
    if name == "gather_z":
        return (B * Ci * n_in * es + B * Ci * 9 * n_out * 4, 2.0 * pairs * B * Ci, "hbm")
    if name == "contract_z":
        return (B * Ci * 9 * n_out * 4 + B * Co * n_out * es, 2.0 * B * Ci * 9 * Co * n_out, "hbm")
    if name == "contract_x":
        return (B * Ci * n_in * es + B * Co * 9 * n_in * 4, 2.0 * B * Ci * 9 * Co * n_in, "hbm")
    if name == "gather_y":
        return (B * Co * 9 * n_in * 4 + B * Co * n_out * es, 2.0 * pairs * B * Co, "hbm")
    # fused kernels: x in, y out
    fl = 2.0 * pairs * B * min(Ci, Co) + 2.0 * B * Ci * 9 * Co * min(n_in, n_out)
    return (B * Ci * n_in * es + B * Co * n_out * es, fl, "alu")


def load_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic_%s_%s.json" % (kernel, workload))
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_sha256_16") != kernel_source_digest():
        return None
    return float(t["hbm_bytes_per_launch"])


def cpu_baseline(wl, x, w, seconds=15.0):
    """Time the oracle (as it stands) on a bounded random sample of output pixels."""
    import numpy as np
    import oracle
    o = oracle.default()
    nlat, nlon = wl.y_shape[2], wl.y_shape[3]
    rng = np.random.default_rng(12345)
    args = wl.plan_args()
    fn = o.forward if wl.op == "forward" else o.transpose
    x64, w64 = x.astype(np.float64), w.astype(np.float64)
    n = 64
    pix = rng.choice(nlat * nlon, size=n, replace=False)
    t0 = time.perf_counter()
    fn(*args, x64, w64, pix=pix)
    t_cal = time.perf_counter() - t0
    n = int(min(nlat * nlon, max(64, n * seconds / max(t_cal, 1e-6))))
    pix = rng.choice(nlat * nlon, size=n, replace=False)
    t0 = time.perf_counter()
    fn(*args, x64, w64, pix=pix)
    dt = time.perf_counter() - t0
    return {"value": n * wl.batch * wl.c_out / dt, "unit": UNIT, "cores": o.max_threads(),
            "kind": "oracle", "seconds": round(dt, 3),
            "sample": "%d output pixels drawn uniformly (seed 12345) of %s, all %d batch x %d "
                      "channels, fp64 ring-window mode" % (n, wl.name, wl.batch, wl.c_out)}


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--algo", default="auto")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_2209_13603_amd import disco, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    wl = synth.WORKLOADS[args.workload or synth.HEADLINE]
    es = 2 if wl.dtype == "bf16" else 4
    log("workload", wl)
    t0 = time.time()
    x_np, w_np = synth.make_inputs(wl)
    log("inputs generated in %.1fs" % (time.time() - t0))
    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    x = torch.from_numpy(x_np).to(dev).to(tdt)
    w = torch.from_numpy(w_np).to(dev).to(tdt)
    y = torch.empty(wl.y_shape, dtype=tdt, device=dev)
    t0 = time.time()
    plan = disco.Plan(*wl.plan_args())
    plan_s = time.time() - t0
    info = plan.info()
    log("plan built in %.2fs: %s" % (plan_s, info))
    step = (lambda: plan.forward(x, w, y, algo=args.algo)) if wl.op == "forward" else \
        (lambda: plan.transpose(x, w, y, algo=args.algo))

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    disco.kernel_timing(True)
    disco.kernel_timing_read()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        step()
    end.record()
    torch.cuda.synchronize()
    kt = disco.kernel_timing_read()
    disco.kernel_timing(False)
    ms_total = start.elapsed_time(end)
    # Step time without the event bracketing: a second, untimed-kernel pass.
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        step()
    end.record()
    torch.cuda.synchronize()
    ms_plain = start.elapsed_time(end)
    ms_per_step = ms_plain / args.steps
    value = wl.out_pix_chan / (ms_per_step / 1e3)
    log("step %.4f ms (with kernel events %.4f ms); kernels: %s"
        % (ms_per_step, ms_total / args.steps, kt))

    dom = max(kt.items(), key=lambda kv: kv[1][1])
    name, (launches, tot_ms) = dom
    avg_ms = tot_ms / launches
    bytes_, flops, bound = kernel_model(name, wl, info, es)
    if bound == "hbm":
        achieved = bytes_ / (avg_ms / 1e3) / 1e9
        peak, unit = HBM_PEAK_GBS, "GB/s"
    else:
        achieved = flops / (avg_ms / 1e3) / 1e12
        peak, unit = FP32_VALU_PEAK_TFLOPS, "TFLOP/s"
    traffic = load_traffic(name, wl.name)
    roof = {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": traffic, "kernel": name,
            "kernel_avg_us": round(avg_ms * 1e3, 2), "algorithmic_bytes": int(bytes_),
            "algorithmic_flops": flops}
    per_kernel = {k: {"launches": v[0], "avg_us": round(v[1] / v[0] * 1e3, 2)} for k, v in kt.items()}
    op_bytes = wl.batch * (wl.c_in * (wl.nlat_in * wl.nlon_in if wl.op == "forward" else
                                      wl.nlat_out * wl.nlon_out)
                           + wl.c_out * wl.y_shape[2] * wl.y_shape[3]) * es
    out = {
        "metric": METRIC, "value": value, "unit": UNIT, "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32" if wl.dtype == "fp32" else "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "op": wl.op, "nlat_in": wl.nlat_in, "nlon_in": wl.nlon_in,
                   "nlat_out": wl.nlat_out, "nlon_out": wl.nlon_out, "theta_c": wl.theta_c,
                   "batch": wl.batch, "c_in": wl.c_in, "c_out": wl.c_out, "basis": "bilinear3x3",
                   "algo": args.algo, "storage": wl.dtype},
        "op_algorithmic_gbs": round(op_bytes / (ms_per_step / 1e3) / 1e9, 2),
        "kernels": per_kernel,
        "roofline": roof,
        "plan_seconds": round(plan_s, 3),
    }
    if not args.no_cpu_baseline:
        log("timing the oracle on a bounded sample ...")
        out["cpu_baseline"] = cpu_baseline(wl, x_np, w_np, args.cpu_seconds)
    else:
        out["cpu_baseline"] = None
    plan.close()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
