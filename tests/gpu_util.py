"""Helpers shared by the GPU tests: run the library on cuda:0 and compare with
the oracle on the same seeded inputs."""
from __future__ import annotations

import sys

import numpy as np

import oracle
from paper_2209_13603_amd import disco, synth


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def torch_dev(a: np.ndarray, dtype: str = "fp32"):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda:0")
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def to_numpy(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def rel_l2(got: np.ndarray, ref: np.ndarray) -> float:
    den = float(np.linalg.norm(ref.ravel()))
    return float(np.linalg.norm((got - ref).ravel())) / (den if den > 0 else 1.0)


def sample_pixels(nlat: int, nlon: int, per_ring: int = 6, seed: int = 0, extra_rings=()) -> np.ndarray:
    """Flat pixel indices: the 6 rings next to each pole, every (nlat/12)-th ring,
    the extra rings asked for, and on each a few longitudes including the
    seam (0, nlon - 1)."""
    rings = set(range(min(6, nlat))) | set(range(max(0, nlat - 6), nlat))
    rings |= set(range(0, nlat, max(1, nlat // 12)))
    rings |= set(int(t) for t in extra_rings if 0 <= t < nlat)
    r = np.random.default_rng(seed)
    pix = []
    for t in sorted(rings):
        lons = {0, nlon - 1, nlon // 2} | set(int(v) for v in r.integers(0, nlon, per_ring))
        pix += [t * nlon + p for p in sorted(lons)]
    return np.array(pix, dtype=np.int64)


def run_gpu(wl_or_args, x: np.ndarray, w: np.ndarray, op: str, dtype: str = "fp32",
            algo="auto", plan=None, plan_kw=None):
    """Run forward/transpose through the C ABI; returns (y as float64 numpy, plan)."""
    import torch
    if plan is None:
        plan = disco.Plan(*wl_or_args, **(plan_kw or {}))
    xt, wt = torch_dev(x, dtype), torch_dev(w, dtype)
    y = plan.forward(xt, wt, algo=algo) if op == "forward" else plan.transpose(xt, wt, algo=algo)
    torch.cuda.synchronize()
    return to_numpy(y), plan


def run_oracle(args, x, w, op, pix=None, **kw):
    """kw: the oracle's ``sampling`` and ``basis`` codes."""
    o = oracle.default()
    fn = o.forward if op == "forward" else o.transpose
    return fn(*args, x.astype(np.float64), w.astype(np.float64), pix=pix, **kw)


def kernel_boundary_rings(plan_args, transpose: bool, plan_kw=None, min_entries: int = 128) -> list:
    """Output rings on both sides of every change of kernel along latitude:
    the op's rings with at least `min_entries` stored entries take the
    spectral path (the library's default threshold), the others the direct
    kernels; from the host-side export of the op's entries."""
    kw = {k: v for k, v in (plan_kw or {}).items() if k in ("node_spacing", "quadrature", "basis", "sampling")}
    e = disco.psi_entries(*plan_args, transpose=transpose, **kw)
    nlat_o = plan_args[0] if transpose else plan_args[2]
    counts = np.zeros((nlat_o, e["phases"]), dtype=np.int64)
    np.add.at(counts, (e["out_ring"], e["phase"]), 1)
    heavy = (counts >= min_entries).any(axis=1)
    out = []
    for t in range(1, nlat_o):
        if heavy[t] != heavy[t - 1]:
            out += [t - 1, t]
    return out


def per_ring_max_error(got: np.ndarray, ref: np.ndarray, pix: np.ndarray, nlon: int):
    """Largest |got - ref| on each sampled ring relative to that ring's largest
    |ref| (over batch and channels): (worst ratio, its ring, rings checked).
    got and ref are [B, C, n] at the flat pixels pix."""
    rings = pix // nlon
    worst, worst_ring = 0.0, -1
    for t in np.unique(rings):
        sel = rings == t
        scale = float(np.abs(ref[:, :, sel]).max())
        err = float(np.abs(got[:, :, sel] - ref[:, :, sel]).max())
        r = err / scale if scale > 0 else err
        if r > worst:
            worst, worst_ring = r, int(t)
    return worst, worst_ring, int(np.unique(rings).size)
