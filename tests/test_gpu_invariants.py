"""Exact invariants of the GPU path and its error handling (Sec. 3.3 exact
equivariance to rotations about z; Sec. 3.5 adjointness; the ABI contract)."""
import ctypes
import math
import os

import numpy as np
import pytest

import oracle
from gpu_util import run_gpu, say, torch_dev, to_numpy
from paper_2209_13603_amd import disco, synth

pytestmark = pytest.mark.gpu

ALGOS = ["gather_then_contract", "contract_then_gather", "fused", "fused_direct"]


def _same(got, ref, algo):
    """Direct gathers commute with whole-pixel shifts bitwise; the spectral
    (DFT) form of the fused path does so in exact arithmetic, to fp32 rounding."""
    if algo == "fused":
        return np.abs(got - ref).max() <= 1e-6 * np.abs(ref).max()
    return np.array_equal(got, ref)


@pytest.mark.parametrize("algo", ALGOS)
@pytest.mark.parametrize("case", [(32, 64, 32, 64), (64, 128, 32, 64), (32, 64, 64, 128)])
def test_shift_equivariance_bitwise(case, algo, monkeypatch):
    monkeypatch.setenv("DISCO_SPECTRAL_MIN_ENTRIES", "8")
    a, b, c, d = case
    tc = 3 * math.pi / min(a, c)
    plan = disco.Plan(a, b, c, d, tc)
    x, w = synth.random_inputs(21, (2, 3, a, b), (4, 3, 9))
    say("shift", case, algo)
    y, _ = run_gpu(None, x, w, "forward", algo=algo, plan=plan)
    if b % d == 0:
        s, m_in, m_out = b // d, (b // d) * 3, 3
    else:
        s, m_in, m_out = d // b, 3, 3 * (d // b)
    ys, _ = run_gpu(None, np.roll(x, m_in, axis=-1), w, "forward", algo=algo, plan=plan)
    assert _same(ys, np.roll(y, m_out, axis=-1), algo)
    # Transposed op: a shift of its input by m shifts its output by the ratio.
    xT, wT = synth.random_inputs(22, (2, 4, c, d), (4, 3, 9))
    yT, _ = run_gpu(None, xT, wT, "transpose", algo=algo, plan=plan)
    m_in = 2 if b % d == 0 else 2 * (d // b)
    m_out = 2 * (b // d) if b % d == 0 else 2
    ysT, _ = run_gpu(None, np.roll(xT, m_in, axis=-1), wT, "transpose", algo=algo, plan=plan)
    assert _same(ysT, np.roll(yT, m_out, axis=-1), algo)
    plan.close()


@pytest.mark.parametrize("algo", ALGOS)
def test_determinism_bitwise(algo):
    wl = synth.WORKLOADS["down128x256_to_64x128"]
    x, w = synth.make_inputs(wl)
    plan = disco.Plan(*wl.plan_args())
    y1, _ = run_gpu(None, x, w, "forward", algo=algo, plan=plan)
    y2, _ = run_gpu(None, x, w, "forward", algo=algo, plan=plan)
    assert np.array_equal(y1, y2)
    plan.close()


@pytest.mark.parametrize("case", [(32, 64, 32, 64), (64, 128, 32, 64), (24, 48, 12, 24)])
def test_adjoint_identity(case):
    """<A x, g>_q_out = <x, B g>_q_in in fp32 (Sec. 3.5, R11)."""
    a, b, c, d = case
    tc = 3 * math.pi / min(a, c)
    plan = disco.Plan(a, b, c, d, tc)
    r = np.random.default_rng(23)
    x = r.standard_normal((2, 3, a, b)).astype(np.float32)
    g = r.standard_normal((2, 4, c, d)).astype(np.float32)
    w = (r.standard_normal((4, 3, 9)) / 6).astype(np.float32)
    Ax, _ = run_gpu(None, x, w, "forward", plan=plan)
    Bg, _ = run_gpu(None, g, w, "transpose", plan=plan)
    o = oracle.default()
    qo = o.quadrature(c, d)[None, None, :, None]
    qi = o.quadrature(a, b)[None, None, :, None]
    lhs = float((Ax * g * qo).sum())
    rhs = float((x * Bg * qi).sum())
    scale = float(np.sqrt((Ax ** 2 * qo).sum() * (g ** 2 * qo).sum()))
    say("adjoint", case, lhs, rhs)
    assert abs(lhs - rhs) <= 1e-6 * scale
    plan.close()


def test_empty_batch_and_plan_info():
    import torch
    plan = disco.Plan(32, 64, 32, 64, 3 * math.pi / 32)
    x = torch.empty((0, 2, 32, 64), device="cuda:0")
    w = torch.zeros((3, 2, 9), device="cuda:0")
    y = plan.forward(x, w)
    assert y.shape == (0, 3, 32, 64)
    info = plan.info()
    assert info["K"] == 9 and info["nnz_entries"] > 0 and info["psi_bytes"] > 0
    assert abs(info["h"] - math.pi / 32) < 1e-15
    plan.close()


def test_plan_memory_2048x4096():
    """The 2048 x 4096 plan as created: the spectral pairs of the southern cap
    read the northern tables (one table per mirrored pair), and the device
    holds a small multiple of the compressed psi."""
    wl = synth.WORKLOADS["sphere2048x4096"]
    plan = disco.Plan(*wl.plan_args())
    info = plan.info()
    say("plan bytes %d, compressed %d, spectral pairs %d tables %d" % (
        info["psi_bytes"], info["psi_compressed_bytes"], info["spectral_pairs_forward"],
        info["spectral_tables_forward"]))
    assert info["spectral_pairs_forward"] > 0
    assert 2 * info["spectral_tables_forward"] == info["spectral_pairs_forward"]
    assert 2 * info["spectral_tables_transpose"] == info["spectral_pairs_transpose"]
    assert info["psi_bytes"] < 4 * info["psi_compressed_bytes"]
    plan.close()


def test_error_paths():
    import torch
    plan = disco.Plan(16, 32, 8, 16, 3 * math.pi / 8)
    dev = "cuda:0"
    x = torch.zeros((1, 2, 16, 32), device=dev)
    w = torch.zeros((3, 2, 9), device=dev)
    y = torch.zeros((1, 3, 8, 16), device=dev)
    plan.forward(x, w, y)
    with pytest.raises(disco.DiscoError) as e:
        plan.forward(x, w, torch.zeros((1, 3, 8, 15), device=dev))
    assert e.value.status == disco.DISCO_ERR_SHAPE
    with pytest.raises(disco.DiscoError) as e:
        plan.forward(x, torch.zeros((3, 2, 8), device=dev), y)
    assert e.value.status == disco.DISCO_ERR_SHAPE
    with pytest.raises(disco.DiscoError) as e:
        plan.forward(x, w.to(torch.bfloat16), y)
    assert e.value.status == disco.DISCO_ERR_DTYPE
    with pytest.raises(disco.DiscoError) as e:
        plan.forward(x.double(), w.double(), y.double())
    assert e.value.status == disco.DISCO_ERR_DTYPE
    # The transposed op shares the forward W buffer: [CinT=3, CoutT=2, 9] is valid,
    # [2, 3, 9] is not.
    plan.transpose(y, w, torch.zeros((1, 2, 16, 32), device=dev))
    with pytest.raises(disco.DiscoError) as e:
        plan.transpose(y, torch.zeros((2, 3, 9), device=dev), torch.zeros((1, 2, 16, 32), device=dev))
    assert e.value.status == disco.DISCO_ERR_SHAPE
    # y overlapping x.
    buf = torch.zeros(2 * 16 * 32 * 2, device=dev)
    xo = buf[: 2 * 16 * 32].view(1, 2, 16, 32)
    yo = buf[100: 100 + 3 * 8 * 16].view(1, 3, 8, 16)
    with pytest.raises(disco.DiscoError) as e:
        plan.forward(xo, w, yo)
    assert e.value.status == disco.DISCO_ERR_INVALID_ARGUMENT
    # Host memory is refused.
    with pytest.raises(disco.DiscoError) as e:
        plan.forward(x.cpu(), w, y)
    assert e.value.status == disco.DISCO_ERR_DEVICE
    torch.cuda.synchronize()
    plan.close()


def test_fault_injection_alloc(monkeypatch):
    import torch
    plan = disco.Plan(16, 32, 8, 16, 3 * math.pi / 8)
    x = torch.zeros((1, 2, 16, 32), device="cuda:0")
    w = torch.zeros((3, 2, 9), device="cuda:0")
    y = torch.full((1, 3, 8, 16), 7.0, device="cuda:0")
    monkeypatch.setenv("DISCO_FAULT_INJECT", "alloc")
    with pytest.raises(disco.DiscoError) as e:
        plan.forward(x, w, y, algo="gather_then_contract")
    assert e.value.status == disco.DISCO_ERR_OUT_OF_MEMORY
    with pytest.raises(disco.DiscoError) as e:
        disco.Plan(16, 32, 8, 16, 3 * math.pi / 8)
    assert e.value.status == disco.DISCO_ERR_OUT_OF_MEMORY
    monkeypatch.delenv("DISCO_FAULT_INJECT")
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())   # a failed call writes nothing
    plan.close()


@pytest.mark.parametrize("name", ["sphere32x64", "down128x256_to_64x128", "sphere512x1024",
                                  "up256x512_to_512x1024_bf16", "sphere2048x4096"])
def test_kernel_work_covers_the_op(name):
    """The per-kernel work the library reports for the timing tools splits
    the op exactly: every output pixel written once, every non-zero triple
    of psi counted once, whichever kernels the dispatch picks."""
    wl = synth.WORKLOADS[name]
    plan = disco.Plan(*wl.plan_args())
    info = plan.info()
    for transpose in (False, True):
        # The transposed op visits the same triples, up to fp64 rounding of
        # its own geometry exactly at the cutoff.
        total = plan.kernel_work(transpose, "fused_direct", 1, 1)["fused_gather_contract"][2]
        if not transpose:
            assert total == info["nnz_pairs_total"]
        assert abs(total - info["nnz_pairs_total"]) <= 1e-4 * info["nnz_pairs_total"]
        n_out = (wl.nlat_in * wl.nlon_in) if transpose else (wl.nlat_out * wl.nlon_out)
        n_in = (wl.nlat_out * wl.nlon_out) if transpose else (wl.nlat_in * wl.nlon_in)
        for algo in ("gather_then_contract", "contract_then_gather", "fused", "fused_direct", "auto"):
            for ci, co, dt in ((wl.c_in, wl.c_out, wl.dtype), (32, 8, "fp32"), (4, 64, "fp32"), (4, 4, "bf16")):
                work = plan.kernel_work(transpose, algo, ci, co, dt)
                say(name, transpose, algo, ci, co, dt, work)
                gather = [k for k in work if k in ("gather_z", "gather_y", "spectral_mac", "sweep_gather_z",
                                                    "sweep_gather_contract", "fused_gather_contract",
                                                    "mfma_gather_contract")]
                assert sum(work[k][2] for k in gather) == total
                writers = [k for k in work if k in ("contract_z", "gather_y", "spectral_irfft",
                                                     "sweep_gather_contract", "fused_gather_contract",
                                                     "mfma_gather_contract")]
                assert sum(work[k][0] for k in writers) == n_out
                for k, (o, i, p) in work.items():
                    assert 0 <= o <= n_out and 0 <= i <= n_in and p >= 0
                # bf16 storage with auto / fused: the matrix-core kernel over every ring
                assert ("mfma_gather_contract" in work) == (dt == "bf16" and algo in ("auto", "fused"))
                if algo == "fused" and dt != "bf16":
                    assert ("spectral_mac" in work) == (info["spectral_rings_transpose" if transpose
                                                              else "spectral_rings_forward"] > 0)
                    # the sweep takes any channel count on single-phase ops (one
                    # launch per group of eight), at most eight otherwise
                    phases = info["phases_transpose" if transpose else "phases_forward"]
                    assert ("sweep_gather_contract" in work) == (
                        info["sweep_patterns_transpose" if transpose else "sweep_patterns_forward"] > 0
                        and (ci <= 8 or phases == 1))
                    assert ("convert_y" in work) == ("sweep_gather_contract" in work and ci > 8 and dt == "bf16")
    plan.close()


def test_kernel_work_names_match_timing():
    """Every kernel the timing records for a call has a work row."""
    import torch
    a, b = 32, 64
    plan = disco.Plan(a, b, a, b, 3 * math.pi / a)
    dev = torch.device("cuda:0")
    for algo in ("gather_then_contract", "contract_then_gather", "fused", "fused_direct"):
        x = torch.randn(1, 4, a, b, device=dev)
        w = torch.randn(4, 4, 9, device=dev)
        disco.kernel_timing(True)
        disco.kernel_timing_read()
        plan.forward(x, w, algo=algo)
        kt = disco.kernel_timing_read()
        disco.kernel_timing(False)
        work = plan.kernel_work(False, algo, 4, 4)
        say(algo, sorted(kt), sorted(work))
        assert set(kt) <= set(work) and kt
    plan.close()


def test_batch_times_channels_limit():
    """(Batch item, channel) pairs index a 16-bit grid dimension: a call with
    more than 65535 of them is rejected with a shape error before launch."""
    import torch
    a, b = 8, 16
    plan = disco.Plan(a, b, a, b, 3 * math.pi / a, backward=True)
    x = torch.zeros((16385, 1, a, b), device="cuda:0")
    y = torch.zeros((16385, 4, a, b), device="cuda:0")
    w = torch.zeros((4, 1, 9), device="cuda:0")
    with pytest.raises(disco.DiscoError) as ei:
        plan.forward(x, w, y)
    assert ei.value.status == disco.DISCO_ERR_SHAPE
    # the weight gradient's gathered sums: B * Cin * K pairs
    x2 = torch.zeros((8000, 1, a, b), device="cuda:0")
    dy2 = torch.zeros((8000, 1, a, b), device="cuda:0")
    w2 = torch.zeros((1, 1, 9), device="cuda:0")
    with pytest.raises(disco.DiscoError) as ei:
        disco.forward_backward(plan, x2, w2, dy2, want_dx=False)
    assert ei.value.status == disco.DISCO_ERR_SHAPE
    plan.close()
