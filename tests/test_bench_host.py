"""Host-side checks of bench.py's measurement logic (no GPU): the algorithmic
work model per kernel, the sharing of a step's work between the launches of a
kernel that runs several times per step, the counter-summary writer and
reader, and the refusal of more than one GPU."""
import os
import subprocess
import sys

import pytest

import bench
from paper_2209_13603_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_fused_model_counts_gather_and_contraction():
    wl = synth.WORKLOADS["sphere2048x4096"]
    outp, inp, pairs = 1000, 900, 50000
    m = bench.kernel_model("sweep_gather_contract", wl, (outp, inp, pairs), 4)
    assert m["bound"] == "alu"
    assert m["bytes"] == wl.batch * (wl.c_in * inp + wl.c_out * outp) * 4
    assert m["valu"] == 2.0 * pairs * wl.batch * wl.c_in
    assert m["mfma_f32"] == 2.0 * wl.batch * wl.c_in * 9 * wl.c_out * outp and m["mfma_bf16"] == 0.0
    assert m["flops"] == m["valu"] + m["mfma_f32"]


def test_bf16_general_kernel_contracts_on_bf16_matrix_cores():
    """The general kernel with bf16 storage contracts on bf16 matrix cores:
    those flops count against 2.5 PFLOP/s, the gather against the fp32 VALU
    peak, and the bound is the sum of the two times."""
    wl = synth.WORKLOADS["up256x512_to_512x1024_bf16"]
    m = bench.kernel_model("fused_gather_contract", wl, (1000, 900, 50000), 2)
    assert m["mfma_f32"] == 0.0 and m["mfma_bf16"] == 2.0 * wl.batch * wl.c_in * 9 * wl.c_out * 1000
    t = m["valu"] / 157.3e12 + m["mfma_bf16"] / 2500e12
    r = bench.model_roof(m, 2 * t)
    assert r["frac"] == pytest.approx(0.5)
    assert r["peak"] == pytest.approx(m["flops"] / t / 1e12)
    assert r["achieved"] == pytest.approx(r["frac"] * r["peak"])


def test_spectral_models_count_their_own_work():
    """rfft / irfft: 2.5 N log2 N flop per ring transform; the products: 36
    flop per (ring pair, frequency, input channel) and 36 per (output
    frequency, input channel, output channel).  No spectral row claims the
    direct sum it replaces, so none exceeds its unit's peak by construction."""
    wl = synth.WORKLOADS["sphere2048x4096"]
    N = wl.nlon_in
    spec = {"rings": 162, "pairs": 1000, "slots": 170}
    B, Ci, Co = wl.batch, wl.c_in, wl.c_out
    m = bench.kernel_model("spectral_rfft", wl, (0, 170 * N, 0), 4, spec)
    assert m["valu"] == pytest.approx(B * Ci * 170 * 2.5 * N * 12)
    m = bench.kernel_model("spectral_irfft", wl, (162 * N, 0, 0), 4, spec)
    assert m["valu"] == pytest.approx(B * Co * 162 * 2.5 * N * 12)
    m = bench.kernel_model("spectral_mac", wl, (0, 0, 10 ** 9), 4, spec)
    bins = N // 2 + 1
    assert m["valu"] == 36.0 * B * Ci * 1000 * bins + 36.0 * B * Ci * Co * 162 * bins
    assert m["mfma_f32"] == 0.0
    # psi tables are read once per table, input transforms once per pair
    m2 = bench.kernel_model("spectral_mac", wl, (0, 0, 10 ** 9), 4, dict(spec, tables=500))
    assert m2["bytes"] == (B * Ci * 8 * 1000 + 36 * 500) * bins + B * Co * 162 * bins * 8
    assert m["bytes"] - m2["bytes"] == 36 * 500 * bins
    # the weight gradient's pass: the planes of Z, no contraction with W
    m3 = bench.kernel_model("spectral_mac", wl, (0, 0, 10 ** 9), 4, dict(spec, z_mode=True))
    assert m3["valu"] == 36.0 * B * Ci * 1000 * bins
    with pytest.raises(SystemExit):
        bench.kernel_model("spectral_mac", wl, (0, 0, 10 ** 9), 4)


def test_depthwise_stencil_model_is_one_channel_per_item():
    wl = synth.WORKLOADS["sphere2048x4096_separable_dw"]
    outp, inp, pairs = 4096, 4096, 100000
    m = bench.kernel_model("stencil_blocked", wl, (outp, inp, pairs), 4)
    items = wl.batch * wl.c_in
    assert m["bytes"] == items * (inp + outp) * 4
    assert m["flops"] == 2.0 * pairs * items


def test_convert_model_is_hbm():
    wl = synth.WORKLOADS["up256x512_to_512x1024_bf16"]
    m = bench.kernel_model("convert_y", wl, (777, 0, 0), 2)
    assert m["bound"] == "hbm" and m["flops"] == 0.0
    assert m["bytes"] == wl.batch * wl.c_out * 777 * (4 + 2)


class _FakePlan:
    def __init__(self, work):
        self.work = work

    def kernel_work(self, transpose, algo, cin, cout, dtype):
        return self.work

    def info(self):
        return {"spectral_%s_%s" % (k, op): n for k, n in (("rings", 40), ("pairs", 300), ("slots", 44))
                for op in ("forward", "transpose")}


def test_multi_launch_kernel_shares_the_step():
    """A kernel launched four times per step reports a quarter of the step's
    work per launch; the time per launch is the total over launches."""
    wl = synth.WORKLOADS["sphere512x1024"]
    work = {"sweep_gather_contract": (1000, 1000, 20000), "spectral_mac": (0, 0, 5000)}
    steps = 10
    kt = {"sweep_gather_contract": (4 * steps, 40.0), "spectral_mac": (steps, 5.0)}
    per, roof = bench.kernel_report(_FakePlan(work), kt, wl, False, "auto", 4, steps)
    m_full = bench.kernel_model("sweep_gather_contract", wl, work["sweep_gather_contract"], 4)
    b_full, f_full = m_full["bytes"], m_full["flops"]
    assert per["sweep_gather_contract"]["alg_bytes"] == int(b_full / 4)
    assert per["sweep_gather_contract"]["alg_flops"] == pytest.approx(f_full / 4)
    assert per["sweep_gather_contract"]["avg_us"] == pytest.approx(1000.0)
    assert roof["kernel"] == "sweep_gather_contract"
    assert roof["achieved"] == pytest.approx(round(f_full / 4 / 1e-3 / 1e12, 2))


def _write_csv(path, rows):
    with open(path, "w") as f:
        f.write("Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value\n")
        for r in rows:
            f.write('%d,"%s",%s,%s\n' % r)


def test_traffic_summary_round_trip(tmp_path, monkeypatch):
    """Counters scaled by the copy probe: FETCH_SIZE reads half the moved
    bytes, WRITE_SIZE all of them; the summary carries the source digest and
    load_traffic returns its per-launch bytes."""
    monkeypatch.setattr(bench, "traffic_path", lambda k, w: str(tmp_path / ("t_%s_%s.txt" % (k, w))))
    probe_kib = bench.COPY_PROBE_BYTES / 1024.0
    sweep = "void disco::k_sweep<float, 8, false, 0>(int)"
    fetch = [(1, sweep, "FETCH_SIZE", 1000.0), (2, sweep, "FETCH_SIZE", 1200.0),
             (3, "neg_kernel(float)", "FETCH_SIZE", probe_kib / 2)]
    write = [(1, sweep, "WRITE_SIZE", 3000.0), (2, sweep, "WRITE_SIZE", 3000.0),
             (3, "neg_kernel(float)", "WRITE_SIZE", probe_kib)]
    fc, wc = tmp_path / "f.csv", tmp_path / "w.csv"
    _write_csv(fc, fetch)
    _write_csv(wc, write)
    bench.traffic_summary(str(fc), str(wc), "sweep_gather_contract", "sphere2048x4096", ["cmd"])
    got = bench.load_traffic("sweep_gather_contract", "sphere2048x4096")
    assert got == pytest.approx((1100.0 * 2 + 3000.0) * 1024.0)


def test_counter_summary_round_trip(tmp_path, monkeypatch):
    """Derived metrics averaged over the kernel's dispatches (other kernels
    ignored), written with the source digest and read back as fractions."""
    monkeypatch.setattr(bench, "counters_path", lambda k, w: str(tmp_path / ("c_%s_%s.txt" % (k, w))))
    sweep = "void disco::k_sweep<float, 8, false, 0>(int)"
    rows = []
    for d, (mf, vb) in enumerate([(30.0, 40.0), (34.0, 44.0)]):
        rows += [(d, sweep, "MfmaUtil", mf), (d, sweep, "VALUBusy", vb), (d, sweep, "SQ_INSTS_VALU", 1e6),
                 (d, sweep, "SQ_INSTS_MFMA", 2e5), (d, sweep, "SQ_WAIT_ANY", 25.0), (d, sweep, "SQ_WAVE_CYCLES", 100.0)]
    rows += [(9, "void disco::k_spectral<float, 8>(int)", "MfmaUtil", 99.0)]
    c = tmp_path / "c.csv"
    _write_csv(c, rows)
    bench.counter_summary(str(c), "sweep_gather_contract", "sphere2048x4096", ["cmd"])
    got = bench.load_counters("sweep_gather_contract", "sphere2048x4096")
    assert got == {"mfma_busy": pytest.approx(0.32), "valu_busy": pytest.approx(0.42), "wait_frac": pytest.approx(0.25)}


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_sample_parity_reads_the_sampled_pixels():
    """The GPU output is compared at the flat pixels the oracle evaluated, in
    the oracle's (batch, channel, pixel) order; a planted error at one of them
    is seen, one at an unsampled pixel is not."""
    import numpy as np
    rng = np.random.default_rng(0)
    y = rng.standard_normal((2, 3, 4, 8)).astype(np.float32)
    pix = np.array([5, 0, 31, 17])
    ref = y.reshape(2, 3, 32)[:, :, pix].astype(np.float64)
    assert bench.sample_parity(y, ref, pix, "fp32")["rel_l2"] < 1e-7
    bad = y.copy()
    bad[1, 2, 3, 7] += 1.0                     # flat pixel 31: sampled
    p = bench.sample_parity(bad, ref, pix, "fp32")
    assert p["rel_l2"] > 1e-3 and not p["pass"]
    ok = y.copy()
    ok[0, 0, 0, 1] += 1.0                      # flat pixel 1: not sampled
    assert bench.sample_parity(ok, ref, pix, "fp32")["pass"]
    # per ring (8 longitudes per ring here): the planted error sits in ring 3
    assert p["worst_ring"] == 3 and p["rings"] == 3
    r3 = np.abs(ref[:, :, 2]).max()            # ring 3's only sampled pixel is 31
    assert p["max_rel_worst_ring"] == pytest.approx(1.0 / r3)


def test_copy_fraction_marks_hbm_rows_only():
    rows = {"a": {"bound": "hbm", "alg_gbs": 4000.0}, "b": {"bound": "alu", "alg_gbs": 100.0},
            "roof": {"bound": "hbm", "achieved": 3000.0, "unit": "GB/s"}}
    bench.add_copy_fracs(rows, 5000.0)
    assert rows["a"]["copy_frac"] == 0.8 and "copy_frac" not in rows["b"]
    assert rows["roof"]["copy_frac"] == 0.6


class _FakeEvent:
    clock = [0.0]

    def __init__(self, enable_timing=True):
        self.t = None

    def record(self):
        self.t = _FakeEvent.clock[0]

    def synchronize(self):
        pass

    def elapsed_time(self, other):
        return other.t - self.t


class _FakeTorch:
    class cuda:
        Event = _FakeEvent

        @staticmethod
        def synchronize():
            pass


def test_step_percentiles_and_eviction():
    """Steps of 1..10 ms give median 5.5 ms, p10 1.9 ms, p90 9.1 ms; the
    eviction buffer is filled before every step, outside the timed span."""
    durations = iter(range(1, 11))
    fills = []

    def step():
        _FakeEvent.clock[0] += next(durations)

    class Evict:
        def fill_(self, v):
            fills.append(v)
            _FakeEvent.clock[0] += 100.0

    d = bench.step_percentiles(_FakeTorch, step, 10, Evict())
    assert d["reps"] == 10 and fills == list(range(10))
    assert d["time_us_median"] == pytest.approx(5500.0)
    assert d["p10"] == pytest.approx(1900.0) and d["p90"] == pytest.approx(9100.0)
