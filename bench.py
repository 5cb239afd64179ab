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
SOURCE_DIRS = [os.path.join(ROOT, "paper_2209_13603_amd", "csrc"), os.path.join(ROOT, "include")]
# Library kernel name (as the kernel timing reports it) -> device function name.
DEVICE_KERNEL = {"gather_z": "k_gather_z", "contract_z": "k_contract_z", "contract_x": "k_contract_x",
                 "gather_y": "k_gather_y", "fused_gather_contract": "k_fused",
                 "reduce_partials": "k_reduce_partials", "sweep_gather_contract": "k_sweep",
                 "sweep_gather_z": "k_sweep",
                 "spectral_rfft": "k_rfft_rings", "spectral_mac": "k_spectral",
                 "spectral_irfft": "k_irfft_rings", "stencil": "k_stencil",
                 "stencil_blocked": "k_stencil_blocked", "mfma_gather_contract": "k_mfma",
                 "mfma_weights": "k_mfma_wop"}
# The paper's wall-clock for its timed layer (App. B: one channel, batch 1,
# axisymmetric four-node filter, theta_c = 3 pi / L, (L + 1) x 2L pixels; NVIDIA
# RTX 3090, TensorFlow sparse-dense products, mean of 10 runs), in seconds.
PAPER_SECONDS = {"poles_axisym_L1024": 0.0302, "poles_axisym_L2048": 0.0898,
                 "poles_axisym_L4096": 0.3255}
# Template argument that tells two schedules' launches of one device function apart.
KERNEL_VARIANT = {"sweep_gather_contract": ", false, ", "sweep_gather_z": ", true, "}
COPY_PROBE_BYTES = 256 << 20   # per direction, fp32 negation used as the plain copy kernel
EVICT_BYTES = 512 << 20       # larger than the 256 MB last-level cache (MALL)
COPY_KERNEL_BYTES = 1 << 30   # per direction, torch copy_ timed as the achievable streaming rate
COPY_PROBE_KERNEL = "neg"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_digest() -> str:
    """Digest of every library source with comments and blank space removed:
    counter figures go stale when any code changes, not when comments do."""
    import re
    strip = re.compile(r"//[^\n]*|/\*.*?\*/", re.S)
    h = hashlib.sha256()
    for d in SOURCE_DIRS:
        for fn in sorted(os.listdir(d)):
            if fn.endswith((".hip", ".cpp", ".h")):
                with open(os.path.join(d, fn)) as f:
                    code = " ".join(strip.sub(" ", f.read()).split())
                h.update(fn.encode() + b"\0" + code.encode())
    return h.hexdigest()[:16]


PEAK_TFLOPS = {"valu": FP32_VALU_PEAK_TFLOPS, "mfma_f32": FP32_MFMA_PEAK_TFLOPS,
               "mfma_bf16": BF16_MFMA_PEAK_TFLOPS}


def fft_flops(n):
    """Flops of one real n-point FFT (half the 5 n log2 n of a complex one)."""
    return 2.5 * n * math.log2(n) if n > 1 else 0.0


def kernel_model(name, wl, work, es, spec=None):
    """Algorithmic work of one launch of kernel `name`: a dict with `bytes`,
    the flops per execution unit (`valu`: fp32 vector FMAs; `mfma_f32` /
    `mfma_bf16`: matrix-core products of that input type), and `bound`.

    `work` = (out_pixels, in_pixels, pairs) per batch item and channel, as
    the library reports it for this kernel.  Per unit figures: every output
    pixel x channel written costs es bytes, every input pixel x channel read
    es bytes; the sparse gather costs 2 flop per non-zero (pixel pair, k) per
    gathered channel (VALU), the channel contraction 2 * 9 * Cin flop per
    output pixel x output channel (matrix cores: fp32 in the ring sweep,
    bf16 in the general kernel with bf16 storage).  The two-kernel path also
    moves its fp32 intermediate (9 planes per channel), which its kernels must
    write and read.  The spectral kernels count their own work: a real FFT of
    each ring (2.5 N log2 N flop) and, per (ring pair, frequency), 36 flop per
    input channel for the three basis rows plus 36 per (input, output
    channel) pair and output frequency for the weights; `spec` gives the op's
    spectral structure from the plan ({"rings", "pairs", "slots"}: output
    rings, (output ring, input ring) pairs, input rings transformed).
    """
    B, Ci, Co = wl.batch, wl.c_in, wl.c_out
    if getattr(wl, "depthwise", False):
        # B x C one-channel items, each filtered by its channel's own filter.
        B, Ci, Co = B * Ci, 1, 1
    outp, inp, pairs = work
    fwd = getattr(wl, "op", "forward") == "forward"
    n_in = wl.nlon_in if fwd else wl.nlon_out     # ring length of the op's input grid
    n_out = wl.nlon_out if fwd else wl.nlon_in
    m = dict(bytes=0.0, valu=0.0, mfma_f32=0.0, mfma_bf16=0.0, bound="alu")
    if name in ("stencil", "stencil_blocked"):
        # W folded into psi: 2 flop per stored (output pixel, input pixel)
        # pair per channel pair; bound by whichever roof is lower.
        m["bytes"] = B * Ci * inp * es + B * Co * outp * es
        m["valu"] = 2.0 * pairs * B * Ci * Co
        m["bound"] = "hbm" if m["bytes"] / (HBM_PEAK_GBS * 1e9) > m["valu"] / (FP32_VALU_PEAK_TFLOPS * 1e12) \
            else "alu"
    elif name == "convert_y":
        # fp32 partial sums read, bf16 output written, per covered pixel.
        m.update(bytes=B * Co * outp * (4 + es), bound="hbm")
    elif name in ("gather_z", "sweep_gather_z"):
        m.update(bytes=B * Ci * inp * es + B * Ci * 9 * outp * 4, valu=2.0 * pairs * B * Ci, bound="hbm")
    elif name == "contract_z":
        m.update(bytes=B * Ci * 9 * outp * 4 + B * Co * outp * es, valu=2.0 * B * Ci * 9 * Co * outp, bound="hbm")
    elif name == "contract_x":
        m.update(bytes=B * Ci * inp * es + B * Co * 9 * inp * 4, valu=2.0 * B * Ci * 9 * Co * inp, bound="hbm")
    elif name == "gather_y":
        m.update(bytes=B * Co * 9 * inp * 4 + B * Co * outp * es, valu=2.0 * pairs * B * Co, bound="hbm")
    elif name.startswith("spectral_"):
        if not spec:
            raise SystemExit("kernel %s needs the plan's spectral structure" % name)
        mi, mo = n_in // 2 + 1, n_out // 2 + 1
        if name == "spectral_rfft":
            m["bytes"] = B * Ci * spec["slots"] * (n_in * es + mi * 8)
            m["valu"] = B * Ci * spec["slots"] * fft_flops(n_in)
        elif name == "spectral_mac":
            # per (ring pair, frequency): the input transform of each input
            # channel read; per (psi table, frequency) its 9 values (pairs
            # mirrored about the equator share a table); per output bin: Yhat
            # written
            m["bytes"] = (B * Ci * 8 * spec["pairs"] + 9 * 4 * spec.get("tables", spec["pairs"])) * mi \
                + B * Co * spec["rings"] * mi * 8
            m["valu"] = 36.0 * B * Ci * spec["pairs"] * mi
            if not spec.get("z_mode"):
                # the contraction with W per output bin (the weight gradient's
                # pass writes the planes of Z instead: Co = Ci * 9, no W)
                m["valu"] += 36.0 * B * Ci * Co * spec["rings"] * mi
        else:
            m["bytes"] = B * Co * spec["rings"] * (mo * 8 + n_out * es)
            m["valu"] = B * Co * spec["rings"] * fft_flops(n_out)
    elif name in ("fused_gather_contract", "sweep_gather_contract"):
        # x in, y out, gather over the input channels (VALU), contraction per
        # output (matrix cores).
        m["bytes"] = B * Ci * inp * es + B * Co * outp * es
        m["valu"] = 2.0 * pairs * B * Ci
        dt = "mfma_bf16" if (name == "fused_gather_contract" and es == 2) else "mfma_f32"
        m[dt] = 2.0 * B * Ci * 9 * Co * outp
    elif name == "mfma_gather_contract":
        # x in, y out; the gather and the contraction both on bf16 matrix
        # cores (counted at their algorithmic size: the non-zero triples and
        # 9 basis functions, not the padded instruction shapes).
        m["bytes"] = B * Ci * inp * es + B * Co * outp * es
        m["mfma_bf16"] = 2.0 * pairs * B * Ci + 2.0 * B * Ci * 9 * Co * outp
    elif name == "mfma_weights":
        # W read, its operand table (8 bf16 per lane, 16 k per 9) written.
        m.update(bytes=Ci * Co * 9 * es + Ci * Co * 16 * 2, bound="hbm")
    elif name == "reduce_partials":
        m.update(bound="hbm")
    else:
        raise SystemExit("no work model for kernel %s" % name)
    m["flops"] = m["valu"] + m["mfma_f32"] + m["mfma_bf16"]
    return m


def spectral_spec(plan, transpose):
    """The op's spectral structure from the plan's info."""
    info = plan.info()
    sfx = "transpose" if transpose else "forward"
    return {"rings": info["spectral_rings_" + sfx], "pairs": info["spectral_pairs_" + sfx],
            "slots": info["spectral_slots_" + sfx],
            "tables": info.get("spectral_tables_" + sfx, info["spectral_pairs_" + sfx])}


def model_roof(m, avg_s):
    """Achieved rate of one launch of modelled work `m` lasting avg_s seconds,
    against the bound: HBM bytes at the HBM peak, or the arithmetic at each
    unit's own peak (VALU fp32, fp32 and bf16 matrix cores), the unit times
    added (they share one issue port).  `peak` is then the rate the kernel's
    mix of work would reach with every unit at its peak."""
    if m["bound"] == "hbm":
        ach = m["bytes"] / avg_s / 1e9
        return {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS}
    t_bound = sum(m[u] / (PEAK_TFLOPS[u] * 1e12) for u in PEAK_TFLOPS)
    ach = m["flops"] / avg_s / 1e12
    peak = m["flops"] / t_bound / 1e12 if t_bound > 0 else FP32_VALU_PEAK_TFLOPS
    bound = "mfma" if m["flops"] > 0 and m["valu"] == 0 else "alu"
    return {"bound": bound, "achieved": ach, "peak": peak, "unit": "TFLOP/s",
            "frac": (t_bound / avg_s) if t_bound > 0 else 0.0}


def traffic_path(kernel, workload):
    return os.path.join(ROOT, "profiles", "traffic_%s_%s.txt" % (kernel, workload))


def load_traffic(kernel, workload):
    """Calibrated HBM bytes per launch from the committed counter summary, or
    None when absent or taken on different library sources."""
    path = traffic_path(kernel, workload)
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith((" ", "#", "-")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("library_source_sha256_16") != kernel_source_digest():
        return None
    return float(kv["hbm_bytes_per_launch"])


COUNTER_SET = ("MfmaUtil", "VALUBusy", "SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_WAIT_ANY", "SQ_WAVE_CYCLES",
               "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_VALU_MFMA_COEXEC_CYCLES")


def counters_path(kernel, workload):
    return os.path.join(ROOT, "profiles", "counters_%s_%s.txt" % (kernel, workload))


def load_counters(kernel, workload):
    """Matrix-core and VALU busy fractions of `kernel` from the committed
    counter summary (None when absent or taken on different library sources)."""
    out = {"mfma_busy": None, "valu_busy": None, "wait_frac": None}
    path = counters_path(kernel, workload)
    if not os.path.exists(path):
        return out
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith((" ", "#", "-")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip().split()[0] if v.strip() else ""
    if kv.get("library_source_sha256_16") != kernel_source_digest():
        return out
    for k in out:
        out[k] = float(kv[k]) if k in kv else None
    return out


def counter_summary(csv_path, kernel, workload, commands):
    """Write profiles/counters_<kernel>_<workload>.txt from one rocprofv3
    --pmc run of COUNTER_SET: MfmaUtil and VALUBusy are rocprofv3's derived
    metrics (matrix-core busy cycles per SIMD, VALU-active cycles per CU, as
    percentages of the GPU's busy cycles), averaged over the kernel's
    dispatches."""
    dev = DEVICE_KERNEL[kernel]
    sel = KERNEL_VARIANT.get(kernel, "")
    rows = _pmc_rows(csv_path)
    ks = [cs for n, cs in rows.values() if ((dev + "<") in n or n.split("(")[0].endswith(dev)) and sel in n]
    if not ks:
        raise SystemExit("%s: no %s dispatch" % (csv_path, dev))
    avg = {c: sum(k.get(c, 0.0) for k in ks) / len(ks) for c in COUNTER_SET}
    lines = ["# Counters of %s (%s) on %s, rocprofv3 --pmc, mean of %d dispatches" % (kernel, dev, workload, len(ks)),
             "# mfma_busy = MfmaUtil / 100: SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE x SIMDs)",
             "# valu_busy = VALUBusy / 100: SQ_ACTIVE_INST_VALU / (GRBM_GUI_ACTIVE x CUs)",
             "# wait_frac = SQ_WAIT_ANY / SQ_WAVE_CYCLES: share of wave cycles spent waiting",
             "# mfma_valu_coexec = SQ_VALU_MFMA_COEXEC_CYCLES / SQ_VALU_MFMA_BUSY_CYCLES: share of the",
             "#   matrix cores' busy cycles in which a VALU instruction issued beside them",
             "kernel: %s" % kernel, "workload: %s" % workload,
             "library_source_sha256_16: %s" % kernel_source_digest(),
             "mfma_busy: %.4f" % (avg["MfmaUtil"] / 100.0),
             "valu_busy: %.4f" % (avg["VALUBusy"] / 100.0),
             "wait_frac: %.4f" % (avg["SQ_WAIT_ANY"] / max(avg["SQ_WAVE_CYCLES"], 1.0)),
             "mfma_valu_coexec: %.4f" % (avg["SQ_VALU_MFMA_COEXEC_CYCLES"] / max(avg["SQ_VALU_MFMA_BUSY_CYCLES"], 1.0)),
             "SQ_INSTS_VALU_per_dispatch: %.0f" % avg["SQ_INSTS_VALU"],
             "SQ_INSTS_MFMA_per_dispatch: %.0f" % avg["SQ_INSTS_MFMA"],
             "commands:"] + ["    " + c for c in commands]
    path = counters_path(kernel, workload)
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(path)
    print("\n".join(lines))


def _pmc_rows(path):
    """{dispatch id: (kernel name, {counter: value})} from a rocprofv3 counter CSV."""
    import csv
    per = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            d = int(r["Dispatch_Id"])
            name, cs = per.setdefault(d, (r["Kernel_Name"], {}))
            cs[r["Counter_Name"]] = cs.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return per


def traffic_summary(fetch_csv, write_csv, kernel, workload, commands):
    """Write the calibrated traffic summary of `kernel` from two counter runs
    (FETCH_SIZE, then WRITE_SIZE) that each also ran the copy probe."""
    dev = DEVICE_KERNEL[kernel]
    sel = KERNEL_VARIANT.get(kernel, "")
    out = {}
    for ctr, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = _pmc_rows(path)
        kv = [cs[ctr] for n, cs in rows.values()
              if ((dev + "<") in n or n.split("(")[0].endswith(dev)) and sel in n]
        cp = [cs[ctr] for n, cs in rows.values() if COPY_PROBE_KERNEL in n.split("(")[0]]
        if not kv or not cp:
            raise SystemExit("%s: no %s dispatch (%d) or copy probe (%d)" % (path, dev, len(kv), len(cp)))
        kib = sum(kv) / len(kv)
        cal = (sum(cp) / len(cp)) * 1024.0 / COPY_PROBE_BYTES
        out[ctr] = (kib, len(kv), sum(cp) / len(cp), cal)
    fetch = out["FETCH_SIZE"][0] * 1024.0 / out["FETCH_SIZE"][3]
    write = out["WRITE_SIZE"][0] * 1024.0 / out["WRITE_SIZE"][3]
    lines = ["# HBM traffic of %s (%s) on %s, from rocprofv3 counters" % (kernel, dev, workload),
             "# Each counter is scaled by what it reads for a plain copy kernel (fp32 negation)",
             "# moving %d bytes each way in the same process." % COPY_PROBE_BYTES,
             "kernel: %s" % kernel, "workload: %s" % workload,
             "library_source_sha256_16: %s" % kernel_source_digest()]
    for ctr in ("FETCH_SIZE", "WRITE_SIZE"):
        kib, n, ckib, cal = out[ctr]
        lines.append("%s_kib_per_dispatch: %.1f   (mean of %d dispatches)" % (ctr, kib, n))
        lines.append("%s_copy_probe_kib: %.1f   (calibration factor %.4f)" % (ctr, ckib, cal))
    lines += ["fetch_bytes_per_launch: %.0f" % fetch, "write_bytes_per_launch: %.0f" % write,
              "hbm_bytes_per_launch: %.0f" % (fetch + write), "commands:"]
    lines += ["    " + c for c in commands]
    path = traffic_path(kernel, workload)
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(path)
    print("\n".join(lines))


def copy_probe(torch, dev, reps=3):
    """A plain streaming kernel of known size, for counter calibration."""
    n = COPY_PROBE_BYTES // 4
    a = torch.ones(n, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    for _ in range(reps):
        torch.neg(a, out=b)
    torch.cuda.synchronize()
    del a, b


def cpu_baseline(wl, x, w, seconds=15.0, y=None):
    """Time the oracle (as it stands) on a bounded random sample of output
    pixels; with ``y`` (the GPU output on the same inputs) also report the
    parity of that output at the sampled pixels."""
    import numpy as np
    import oracle
    o = oracle.default()
    nlat, nlon = wl.y_shape[2], wl.y_shape[3]
    rng = np.random.default_rng(12345)
    args = wl.plan_args()
    fn = o.forward if wl.op == "forward" else o.transpose
    kw = wl.oracle_kwargs()
    x64, w64 = x.astype(np.float64), w.astype(np.float64)
    if wl.depthwise:
        w64 = oracle.depthwise_weights(w64)
    # Grow the sample until one timed call takes at least half the budget
    # (the first calls also pay thread start-up, so one calibration is short).
    n, dt = 256, 0.0
    for _ in range(6):
        pix = rng.choice(nlat * nlon, size=n, replace=False)
        t0 = time.perf_counter()
        ref = fn(*args, x64, w64, pix=pix, **kw)
        dt = time.perf_counter() - t0
        if dt >= 0.5 * seconds or n == nlat * nlon:
            break
        n = int(min(nlat * nlon, max(2 * n, n * seconds / max(dt, 1e-6))))
    out = {"value": n * wl.batch * wl.c_out / dt, "unit": UNIT, "cores": o.max_threads(),
           "kind": "oracle", "seconds": round(dt, 3),
            "sample": "%d output pixels drawn uniformly (seed 12345) of %s, all %d batch x %d "
                      "channels, fp64 ring-window mode" % (n, wl.name, wl.batch, wl.c_out)}
    if nlat * nlon * wl.nlat_in * wl.nlon_in <= (128 * 256) ** 2:
        # Small grids: the same sample without the ring window (every input
        # pixel against every sampled output pixel), the cost the window saves.
        t0 = time.perf_counter()
        full = fn(*args, x64, w64, pix=pix, window=False, **kw)
        out["all_pairs_seconds"] = round(time.perf_counter() - t0, 3)
        out["all_pairs_max_diff"] = float(np.abs(full - ref).max())
    out["host_cpu"] = host_cpu()
    out["nproc"] = os.cpu_count()
    if y is not None:
        out["parity"] = sample_parity(y, ref, pix, wl.dtype)
    return out


def host_cpu():
    """The host's CPU model as /proc/cpuinfo names it (None elsewhere)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def step_percentiles(torch, step, reps, evict=None):
    """Per-step GPU times (events on the calling stream around each step):
    median, p10 and p90 in microseconds.  With ``evict`` (a byte tensor
    larger than the last-level cache) every step is preceded by an untimed
    fill of it, so the step starts with its inputs out of the caches."""
    import numpy as np
    if reps <= 0:
        return None
    times = []
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    for r in range(reps):
        if evict is not None:
            evict.fill_(r & 0xFF)
        ev[0].record()
        step()
        ev[1].record()
        ev[1].synchronize()
        times.append(ev[0].elapsed_time(ev[1]) * 1e3)
    t = np.asarray(times)
    return {"reps": reps, "time_us_median": round(float(np.median(t)), 2),
            "p10": round(float(np.percentile(t, 10)), 2), "p90": round(float(np.percentile(t, 90)), 2)}


def sample_parity(y, ref, pix, dtype):
    """Relative L2 and largest error (relative to the sample's largest
    reference value) of the GPU output at the oracle's sampled pixels, and
    per output ring the largest error relative to that ring's largest
    reference value (the worst ring reported)."""
    import numpy as np
    got = y.reshape(y.shape[0], y.shape[1], -1)[:, :, pix].astype(np.float64)
    err = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))
    mx = float(np.abs(got - ref).max() / max(np.abs(ref).max(), 1e-300))
    ring = np.asarray(pix) // y.shape[-1]
    d = np.abs(got - ref).max(axis=(0, 1))
    r = np.abs(ref).max(axis=(0, 1))
    worst, worst_ring = 0.0, -1
    for t in np.unique(ring):
        sel = ring == t
        v = float(d[sel].max() / max(r[sel].max(), 1e-300))
        if v > worst:
            worst, worst_ring = v, int(t)
    return {"rel_l2": err, "max_rel": mx, "max_rel_worst_ring": worst, "worst_ring": worst_ring,
            "rings": int(len(np.unique(ring))), "pixels": int(len(pix)),
            "tol_rel_l2": 1e-5 if dtype == "fp32" else 2e-2,
            "pass": err <= (1e-5 if dtype == "fp32" else 2e-2)}


def copy_kernel_gbs(torch, dev, nbytes=COPY_KERNEL_BYTES, reps=5):
    """Bandwidth of a plain device copy (torch's copy_ of nbytes of fp32 into
    another buffer: nbytes read and nbytes written), the best of reps timed
    launches: what a streaming kernel reaches on this GPU, beside the HBM
    peak."""
    a = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    b.copy_(a)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    best = None
    for _ in range(reps):
        ev[0].record()
        b.copy_(a)
        ev[1].record()
        ev[1].synchronize()
        ms = ev[0].elapsed_time(ev[1])
        best = ms if best is None else min(best, ms)
    del a, b
    return {"gbs": round(2 * nbytes / (best / 1e3) / 1e9, 1), "bytes_per_launch": 2 * nbytes,
            "kernel": "torch copy_ of %d MiB fp32 (read + write), best of %d" % (nbytes >> 20, reps)}


def add_copy_fracs(obj, copy_gbs):
    """Every HBM-bound kernel row and roofline in obj gains copy_frac: its
    algorithmic GB/s over the copy kernel's."""
    if isinstance(obj, dict):
        if obj.get("bound") == "hbm":
            gbs = obj.get("alg_gbs", obj.get("achieved") if obj.get("unit") == "GB/s" else None)
            if gbs is not None:
                obj["copy_frac"] = round(gbs / copy_gbs, 4)
        for v in obj.values():
            add_copy_fracs(v, copy_gbs)


def kernel_report(plan, kt, wl, transpose, algo, es, steps):
    """Per-kernel figures of one timed pass and the roofline object of the
    kernel with the largest total time, or of the sparse gather in the
    all-HBM schedule (achieved against HBM peak for HBM-bound kernels,
    against each unit's own peak otherwise).  A kernel launched
    several times per step (the sweep over groups of eight input channels)
    shares the step's algorithmic work equally between its launches."""
    cin, cout = (1, 1) if wl.depthwise else (wl.c_in, wl.c_out)
    work = plan.kernel_work(transpose, algo, cin, cout, wl.dtype)
    spec = spectral_spec(plan, transpose)
    missing = sorted(set(kt) - set(work))
    if missing:
        raise SystemExit("no work figures for kernels %s" % missing)
    per_kernel = {}
    def model(k):
        m = kernel_model(k, wl, work[k], es, spec)
        per_step = max(1, round(kt[k][0] / steps))
        return {u: (v if u == "bound" else v / per_step) for u, v in m.items()}

    for k, (launches, tot_ms) in kt.items():
        avg_ms = tot_ms / launches
        m = model(k)
        r = model_roof(m, avg_ms / 1e3)
        per_kernel[k] = {"launches": launches, "avg_us": round(avg_ms * 1e3, 2),
                         "alg_bytes": int(m["bytes"]), "alg_flops": m["flops"], "bound": m["bound"],
                         "alg_gbs": round(m["bytes"] / (avg_ms / 1e3) / 1e9, 1),
                         "alg_tflops": round(m["flops"] / (avg_ms / 1e3) / 1e12, 2),
                         "frac": round(r["frac"], 4)}
        if m["bound"] == "hbm":
            per_kernel[k]["hbm_frac"] = round(r["frac"], 4)
    # The roofline names the direct kernel with the largest total time: the
    # spectral kernels share the GPU with the sweep from the helper stream,
    # which stretches their event-timed spans over the sweep's.
    direct = [k for k in kt if not k.startswith("spectral_")] or list(kt)
    name = max(direct, key=lambda k: kt[k][1])
    # The all-HBM schedule is reported on its sparse gather (the ring sweep's
    # Z mode), the kernel the gather-bandwidth figure is about.
    if "sweep_gather_z" in kt:
        name = "sweep_gather_z"
    launches, tot_ms = kt[name]
    avg_ms = tot_ms / launches
    m = model(name)
    r = model_roof(m, avg_ms / 1e3)
    traffic = load_traffic(name, wl.name)
    roof = {"bound": r["bound"], "achieved": round(r["achieved"], 2), "peak": round(r["peak"], 2),
            "unit": r["unit"], "frac": round(r["frac"], 4), "traffic": traffic, "kernel": name,
            "kernel_avg_us": round(avg_ms * 1e3, 2), "algorithmic_bytes": int(m["bytes"]),
            "algorithmic_flops": m["flops"],
            "flops_by_unit": {u: m[u] for u in PEAK_TFLOPS if m[u] > 0},
            "algorithmic_gbs": round(m["bytes"] / (avg_ms / 1e3) / 1e9, 1),
            "work_per_launch": dict(zip(("out_pixels", "in_pixels", "pairs"), work[name]))}
    roof.update(load_counters(name, wl.name))
    return per_kernel, roof


def _timed(torch, fn, steps):
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s.record()
    for _ in range(steps):
        fn()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / steps


def _events(torch, disco, fn, steps):
    disco.kernel_timing(True)
    disco.kernel_timing_read()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    kt = disco.kernel_timing_read()
    disco.kernel_timing(False)
    return kt


def bench_backward(args, wl, plan, x, w, es, torch, disco):
    """Gradient step of the workload's op (App. C): dx through the adjoint op
    and dW from the gathered sums.  value = output pix x chan of the op per
    second of one gradient step (dx and dW).  Kernel figures from two passes
    with kernel events, dx alone and dW alone (their kernels share names)."""
    from types import SimpleNamespace
    transpose = wl.op != "forward"
    fb = disco.transpose_backward if transpose else disco.forward_backward
    dy = torch.randn(wl.y_shape, device=x.device).to(x.dtype)
    both = lambda: fb(plan, x, w, dy)
    for _ in range(args.warmup):
        both()
    ms = _timed(torch, both, args.steps)
    kt_dx = _events(torch, disco, lambda: fb(plan, x, w, dy, want_dw=False), args.steps)
    kt_dw = _events(torch, disco, lambda: fb(plan, x, w, dy, want_dx=False), args.steps)
    log("backward step %.4f ms; dx kernels %s; dW kernels %s" % (ms, kt_dx, kt_dw))
    B, Ci, Co, K = wl.batch, wl.c_in, wl.c_out, wl.K
    P = wl.y_shape[2] * wl.y_shape[3]
    kernels, cands = {}, []

    def add(tag, kt, work, model_wl, spec):
        for k, (launches, tot_ms) in kt.items():
            avg = tot_ms / launches
            if k == "weight_grad":
                b_ = B * Ci * K * P * (4 if (wl.dtype == "fp32" and wl.basis == "bilinear3x3") else es) + B * Co * P * es
                f_, bd = 2.0 * B * Co * Ci * K * P, "hbm"
            elif k == "weight_grad_reduce":
                b_, f_, bd = 0, 0.0, "hbm"
            elif k == "spectral_rfft_dy":
                # dy's transform on the op's spectral output rings (the
                # weight gradient's frequency-domain share): dy read, the
                # half spectrum written
                n_o = wl.nlon_out if wl.op == "forward" else wl.nlon_in
                rings = spec["rings"]
                b_ = B * Co * rings * (n_o * 4 + (n_o // 2 + 1) * 8)
                f_, bd = B * Co * rings * fft_flops(n_o), "alu"
            else:
                if k not in work:
                    raise SystemExit("no work figures for kernel %s" % k)
                mm = kernel_model(k, model_wl, work[k], es, spec)
                b_, f_, bd = mm["bytes"], mm["flops"], mm["bound"]
            row = {"launches": launches, "avg_us": round(avg * 1e3, 2), "alg_bytes": int(b_), "alg_flops": f_,
                   "bound": bd, "alg_gbs": round(b_ / (avg / 1e3) / 1e9, 1),
                   "alg_tflops": round(f_ / (avg / 1e3) / 1e12, 2)}
            if bd == "hbm":
                row["hbm_frac"] = round(b_ / (avg / 1e3) / 1e9 / HBM_PEAK_GBS, 4)
            kernels["%s:%s" % (tag, k)] = row
            if not k.startswith("spectral_") and k != "weight_grad_reduce":
                cands.append(("%s:%s" % (tag, k), tot_ms, b_, f_, bd, avg))

    # dx: the adjoint op has the other op's filter pairs (its work figures).
    work_dx = plan.kernel_work(not transpose, "auto", Co, Ci, wl.dtype)
    grids = dict(nlon_in=wl.nlon_in, nlon_out=wl.nlon_out)
    # (the adjoint op's spectral rings are those of the other op's filter pairs)
    add("dx", kt_dx, work_dx, SimpleNamespace(batch=B, c_in=Co, c_out=Ci, op="forward" if transpose else "transpose",
                                              **grids), spectral_spec(plan, not transpose))
    # dW: one-pass gathered sums (fp32, 3x3 basis) or the op's kernels per channel.
    if wl.dtype == "fp32" and wl.basis == "bilinear3x3":
        work_dw = plan.kernel_work(transpose, "gather_then_contract", Ci, Ci * K, wl.dtype)
        mwl = SimpleNamespace(batch=B, c_in=Ci, c_out=Ci * K, op=wl.op, **grids)
        spec_dw = dict(spectral_spec(plan, transpose), z_mode=True)
    else:
        work_dw = plan.kernel_work(transpose, "auto", 1, K, wl.dtype)
        mwl = SimpleNamespace(batch=B * Ci, c_in=1, c_out=K, op=wl.op, **grids)
        spec_dw = spectral_spec(plan, transpose)
    add("dw", kt_dw, work_dw, mwl, spec_dw)
    name, tot, b_, f_, bd, avg = max(cands, key=lambda c: c[1])
    if bd == "hbm":
        achieved, peak, unit = b_ / (avg / 1e3) / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        achieved, peak, unit = f_ / (avg / 1e3) / 1e12, FP32_VALU_PEAK_TFLOPS, "TFLOP/s"
    roof = {"bound": bd, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": load_traffic(name.split(":")[1], wl.name + "_backward"),
            "kernel": name, "kernel_avg_us": round(avg * 1e3, 2), "algorithmic_bytes": int(b_),
            "algorithmic_flops": f_}
    return ms, kernels, roof


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--algo", default="auto")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--reps", type=int, default=50,
                    help="steps timed one by one for the median / p10 / p90")
    ap.add_argument("--cold-reps", type=int, default=20,
                    help="steps timed after a 512 MiB cache-evicting fill (0: skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="after the timed steps, run a plain copy kernel of known size "
                         "(counter calibration for the traffic summary)")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/traffic_<kernel>_<workload>.txt from two rocprofv3 "
                         "counter runs (FETCH_SIZE, then WRITE_SIZE) of --copy-probe benches; "
                         "no GPU needed")
    ap.add_argument("--counter-summary", metavar="CSV",
                    help="write profiles/counters_<kernel>_<workload>.txt from a rocprofv3 --pmc run "
                         "of %s; no GPU needed" % " ".join(COUNTER_SET))
    ap.add_argument("--kernel", default="sweep_gather_contract",
                    help="library kernel name for --traffic-summary and --counter-summary")
    ap.add_argument("--command", action="append", default=[],
                    help="the command that produced each counter run (recorded verbatim)")
    ap.add_argument("--backward", action="store_true",
                    help="time the op's gradient step (input and weight gradients) instead")
    ap.add_argument("--no-hbm-schedule", action="store_true",
                    help="skip the extra pass over the gather-then-contract schedule (whose "
                         "kernels are HBM-bound) that the JSON line reports as hbm_schedule")
    args = ap.parse_args(argv)

    if args.traffic_summary or args.counter_summary:
        from paper_2209_13603_amd import synth
        wl = synth.WORKLOADS[args.workload or synth.HEADLINE]
        if args.traffic_summary:
            traffic_summary(*args.traffic_summary, args.kernel, wl.name, args.command)
        else:
            counter_summary(args.counter_summary, args.kernel, wl.name, args.command)
        return 0

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
    plan = disco.Plan(*wl.plan_args(), **wl.plan_kwargs(), backward=args.backward)
    plan_s = time.time() - t0
    info = plan.info()
    log("plan built in %.2fs: %s" % (plan_s, info))
    if args.backward and wl.depthwise:
        print("--backward: the depthwise calls have no gradient entry points", file=sys.stderr)
        return 2
    if args.backward:
        ms, kernels, roof = bench_backward(args, wl, plan, x, w, es, torch, disco)
        out = {
            "metric": "DISCO %s gradient (dx and dW) output pix*chan/s on %s" % (wl.op, wl.name),
            "value": wl.out_pix_chan / (ms / 1e3), "unit": UNIT, "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "f32" if wl.dtype == "fp32" else "bf16", "data": "synthetic",
            "config": {"workload": wl.name, "op": wl.op + "_backward", "nlat_in": wl.nlat_in,
                       "nlon_in": wl.nlon_in, "nlat_out": wl.nlat_out, "nlon_out": wl.nlon_out,
                       "theta_c": wl.theta_c, "batch": wl.batch, "c_in": wl.c_in, "c_out": wl.c_out,
                       "basis": wl.basis, "sampling": wl.sampling, "storage": wl.dtype},
            "kernels": kernels, "roofline": roof, "plan_seconds": round(plan_s, 3), "cpu_baseline": None,
        }
        plan.close()
        print(json.dumps(out), flush=True)
        return 0
    if wl.depthwise:
        step = (lambda: plan.forward_depthwise(x, w, y)) if wl.op == "forward" else \
            (lambda: plan.transpose_depthwise(x, w, y))
    else:
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

    dist = step_percentiles(torch, step, args.reps)
    cold = None
    if args.cold_reps > 0 and dist is not None:
        evict = torch.empty(EVICT_BYTES, dtype=torch.uint8, device=dev)
        cold = step_percentiles(torch, step, args.cold_reps, evict)
        cold["evict_bytes"] = EVICT_BYTES
        del evict
    log("per step: warm %s; cold %s" % (dist, cold))

    if args.copy_probe:
        copy_probe(torch, dev)

    transpose = wl.op != "forward"
    per_kernel, roof = kernel_report(plan, kt, wl, transpose, args.algo, es, args.steps)

    # The same op through the gather-then-contract schedule, whose kernels
    # move the gathered sums through HBM: their achieved GB/s against the
    # HBM peak (the default schedule's kernels are bound by arithmetic).
    hbm = None
    if not args.no_hbm_schedule and args.algo != "gather_then_contract" and wl.basis == "bilinear3x3" \
            and not wl.depthwise:
        step2 = (lambda: plan.forward(x, w, y, algo="gather_then_contract")) if wl.op == "forward" else \
            (lambda: plan.transpose(x, w, y, algo="gather_then_contract"))
        for _ in range(2):
            step2()
        torch.cuda.synchronize()
        start.record()
        for _ in range(args.steps):
            step2()
        end.record()
        torch.cuda.synchronize()
        ms2 = start.elapsed_time(end) / args.steps
        disco.kernel_timing(True)
        disco.kernel_timing_read()
        for _ in range(args.steps):
            step2()
        torch.cuda.synchronize()
        kt2 = disco.kernel_timing_read()
        disco.kernel_timing(False)
        log("gather-then-contract step %.4f ms; kernels: %s" % (ms2, kt2))
        pk2, roof2 = kernel_report(plan, kt2, wl, transpose, "gather_then_contract", es, args.steps)
        hbm = {"algo": "gather_then_contract", "ms_per_step": ms2,
               "value": wl.out_pix_chan / (ms2 / 1e3), "kernels": pk2, "roofline": roof2}
    # The dominant kernel alone: the same schedule through the entry point
    # that allocates nothing, which runs the spectral rings on the caller's
    # stream before the ring sweep instead of beside it, so the sweep's event
    # span is its own (the default dispatch's includes the time it shares the
    # GPU with the helper stream's kernels).
    alone, step3 = None, None
    if roof.get("kernel") == "sweep_gather_contract" and not args.no_hbm_schedule and wl.op == "forward":
        step3 = lambda: plan.forward_noalloc(x, w, y)
        try:
            step3()
        except disco.DiscoError as err:  # scratch too small for this workload
            step3 = None
            log("dominant kernel alone: not measured (%s)" % err)
    if alone is None and roof.get("kernel") == "sweep_gather_contract" and not args.no_hbm_schedule \
            and wl.op == "forward" and step3 is not None:
        step3()
        torch.cuda.synchronize()
        disco.kernel_timing(True)
        disco.kernel_timing_read()
        for _ in range(args.steps):
            step3()
        torch.cuda.synchronize()
        kt3 = disco.kernel_timing_read()
        disco.kernel_timing(False)
        pk3, _ = kernel_report(plan, kt3, wl, transpose, args.algo, es, args.steps)
        if "sweep_gather_contract" in pk3:
            r3 = pk3["sweep_gather_contract"]
            alone = {"kernel": "sweep_gather_contract", "entry": "disco_forward_noalloc", "avg_us": r3["avg_us"],
                     "bound": r3["bound"], "achieved": r3["alg_tflops"], "unit": "TFLOP/s",
                     "peak": roof["peak"], "frac": r3["frac"]}
        log("dominant kernel alone (spectral rings before it on one stream): %s" % alone)
    op_bytes = wl.batch * (wl.c_in * (wl.nlat_in * wl.nlon_in if wl.op == "forward" else
                                      wl.nlat_out * wl.nlon_out)
                           + wl.c_out * wl.y_shape[2] * wl.y_shape[3]) * es
    metric = METRIC if wl.name == synth.HEADLINE else \
        "DISCO %s output pix*chan/s on %s" % ("fwd" if wl.op == "forward" else "transpose", wl.name)
    vs_baseline, baseline = None, None
    if wl.name in PAPER_SECONDS:
        paper = wl.out_pix_chan / PAPER_SECONDS[wl.name]
        vs_baseline = value / paper
        baseline = {"value": paper, "unit": UNIT, "seconds": PAPER_SECONDS[wl.name],
                    "hardware": "NVIDIA RTX 3090 (the paper's App. B; other hardware, context)"}
    copy_k = copy_kernel_gbs(torch, dev)
    add_copy_fracs(per_kernel, copy_k["gbs"])
    add_copy_fracs(roof, copy_k["gbs"])
    if hbm:
        add_copy_fracs(hbm, copy_k["gbs"])
    out = {
        "metric": metric, "value": value, "unit": UNIT, "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": vs_baseline,
        "dtype": "f32" if wl.dtype == "fp32" else "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "op": wl.op, "nlat_in": wl.nlat_in, "nlon_in": wl.nlon_in,
                   "nlat_out": wl.nlat_out, "nlon_out": wl.nlon_out, "theta_c": wl.theta_c,
                   "batch": wl.batch, "c_in": wl.c_in, "c_out": wl.c_out, "basis": wl.basis,
                   "sampling": wl.sampling, "channels": wl.channels,
                   "algo": "depthwise" if wl.depthwise else args.algo, "storage": wl.dtype},
        "paper_baseline": baseline,
        "op_algorithmic_gbs": round(op_bytes / (ms_per_step / 1e3) / 1e9, 2),
        "copy_kernel": copy_k,
        "kernels": per_kernel,
        "roofline": roof,
        "dominant_kernel_alone": alone,
        "step_distribution": dist,
        "cold_cache": cold,
        "hbm_schedule": hbm,
        "plan_seconds": round(plan_s, 3),
    }
    if not args.no_cpu_baseline:
        log("timing the oracle on a bounded sample ...")
        # The oracle reads the values the GPU holds (bf16-rounded for bf16
        # storage), so the sample also checks the timed output.
        step()
        torch.cuda.synchronize()
        xs = x.float().cpu().numpy()
        ws = w.float().cpu().numpy()
        ys = y.float().cpu().numpy()
        out["cpu_baseline"] = cpu_baseline(wl, xs, ws, args.cpu_seconds, ys)
    else:
        out["cpu_baseline"] = None
    plan.close()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
