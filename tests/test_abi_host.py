"""Host-side checks of libdisco.so that need no GPU: the library loads, exports
every function include/disco.h declares, validates arguments, and its plan
builder's psi entries equal the oracle's dense Psi entry by entry."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle
from paper_2209_13603_amd import disco

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    with open(os.path.join(ROOT, "include", "disco.h")) as f:
        src = f.read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(disco_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    lib = disco.library()
    declared = _declared_functions()
    assert declared, "no declarations parsed"
    assert set(declared) == set(disco.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def test_status_strings():
    lib = disco.library()
    for s in range(7):
        assert lib.disco_status_string(s).decode() == disco._status_name(s)
    assert lib.disco_status_string(99).decode() == "DISCO_ERR_UNKNOWN"


def _create(*args, basis=None):
    lib = disco.library()
    h = ctypes.c_void_p()
    b = ctypes.byref(basis) if basis is not None else None
    return lib.disco_plan_create(*args, b, ctypes.byref(h)), h


@pytest.mark.parametrize("args,status", [
    ((0, 64, 32, 64, 0.3), disco.DISCO_ERR_INVALID_ARGUMENT),
    ((32, 1, 32, 64, 0.3), disco.DISCO_ERR_INVALID_ARGUMENT),
    ((32, 64, 32, 64, 0.0), disco.DISCO_ERR_INVALID_ARGUMENT),
    ((32, 64, 32, 64, -1.0), disco.DISCO_ERR_INVALID_ARGUMENT),
    ((32, 64, 32, 64, 3.5), disco.DISCO_ERR_INVALID_ARGUMENT),
    ((32, 64, 32, 64, float("nan")), disco.DISCO_ERR_INVALID_ARGUMENT),
    ((32, 64, 32, 48, 0.3), disco.DISCO_ERR_UNSUPPORTED),
])
def test_plan_create_validation(args, status):
    rc, h = _create(*args)
    assert rc == status
    assert not h.value
    assert disco.library().disco_last_error().decode()


def test_basis_validation():
    rc, _ = _create(32, 64, 32, 64, 0.3, basis=disco.Basis(7, 0, 0.0))
    assert rc == disco.DISCO_ERR_UNSUPPORTED
    rc, _ = _create(32, 64, 32, 64, 0.3, basis=disco.Basis(0, 5, 0.0))
    assert rc == disco.DISCO_ERR_UNSUPPORTED
    rc, _ = _create(32, 64, 32, 64, 0.3, basis=disco.Basis(0, 0, -0.1))
    assert rc == disco.DISCO_ERR_INVALID_ARGUMENT
    lib = disco.library()
    assert lib.disco_plan_create(32, 64, 32, 64, 0.3, None, None) == disco.DISCO_ERR_INVALID_ARGUMENT


def test_null_plan_calls():
    lib = disco.library()
    t = disco.Tensor()
    assert lib.disco_forward(None, ctypes.byref(t), ctypes.byref(t), ctypes.byref(t), None) == \
        disco.DISCO_ERR_INVALID_ARGUMENT
    assert lib.disco_transpose(None, ctypes.byref(t), ctypes.byref(t), ctypes.byref(t), None) == \
        disco.DISCO_ERR_INVALID_ARGUMENT
    assert lib.disco_plan_query(None, None) == disco.DISCO_ERR_INVALID_ARGUMENT
    assert lib.disco_plan_destroy(None) == disco.DISCO_OK


# --------------------------------------------------------------------------- #
# Plan entries against the oracle's dense Psi (fp64 oracle, fp32 entries).
# --------------------------------------------------------------------------- #
PLAN_CASES = [
    (8, 16, 8, 16),       # same grid
    (16, 32, 8, 16),      # stride-2 downsampling forward
    (12, 24, 6, 12),      # odd ring counts
    (8, 16, 16, 32),      # forward that upsamples (2 longitude phases)
    (32, 64, 32, 64),     # the 32 x 64 workload
    (10, 20, 5, 20),      # latitude-only change
]


def _dense_check(case, transpose, sampling=0, basis=0, quad=0, h_scale=None):
    """h_scale: node spacing as a multiple of theta_c (None: the default)."""
    a, b, c, d = case
    K = {1: 4, 2: 16}.get(basis, 9)
    # theta_c = 3 pixels of the coarser grid (the pole-including grid has
    # nlat - 1 ring spacings).
    tc = 3 * math.pi / (min(a, c) - (1 if sampling == 1 else 0))
    h = 0.0 if h_scale is None else h_scale * tc
    o = oracle.default()
    psi = o.psi_dense(a, b, c, d, tc, h=h or None, sampling=sampling, basis=basis)  # [Nout_plan, Nin_plan, K]
    if not transpose:
        nlat_o, nlon_o, nlat_i, nlon_i = c, d, a, b
        q = o.quadrature(a, b, kind=quad, sampling=sampling)
        dense = psi                           # [op out pixel, op in pixel, K]
    else:
        nlat_o, nlon_o, nlat_i, nlon_i = a, b, c, d
        q = o.quadrature(c, d, kind=quad, sampling=sampling)
        dense = psi.transpose(1, 0, 2)        # filter centred at the op's input points
    ent = disco.psi_entries(a, b, c, d, tc, transpose=transpose, basis=basis, sampling=sampling,
                            quadrature=quad, node_spacing=h)
    assert not ent["values"][:, K:].any()
    P, s = ent["phases"], ent["stride"]
    assert (P, s) == ((1, nlon_i // nlon_o) if nlon_i % nlon_o == 0 else (nlon_o // nlon_i, 1))
    n = ent["values"].shape[0]
    assert n > 0
    seen = set()
    for e in range(n):
        to, r, ti, dd = (int(ent[k][e]) for k in ("out_ring", "phase", "in_ring", "offset"))
        key = (to, r, ti, dd)
        assert key not in seen
        seen.add(key)
        jo = to * nlon_o + r                  # output pixel q = 0 of the pattern
        ii = ti * nlon_i + dd % nlon_i        # input pixel (stride * 0 + d) mod nlon
        ref = dense[jo, ii] * q[ti]
        got = ent["values"][e, :K].astype(np.float64)
        assert np.abs(got - ref).max() <= 2e-7 * abs(q[ti]) + 1e-30, (key, got, ref)
    # Completeness: every non-zero dense element of the q = 0 outputs is stored
    # (the two geometry routes may disagree on exact zeros at hat edges by
    # ~1e-16, a difference the continuity of the basis keeps harmless).
    for to in range(nlat_o):
        for r in range(P):
            jo = to * nlon_o + r
            nz = np.nonzero(np.abs(dense[jo]).sum(axis=1) > 1e-12)[0]
            for ii in nz:
                assert (to, r, int(ii // nlon_i), int(ii % nlon_i)) in seen, (to, r, ii)
    # Shift structure (Sec. 4.2): output q > 0 of the pattern reads pixel
    # (stride q + d) mod nlon with the same values.
    for to in range(nlat_o):
        for r in range(P):
            for qq in (1, nlon_o // P - 1):
                jo = to * nlon_o + P * qq + r
                jr = to * nlon_o + r
                shifted = np.roll(dense[jr].reshape(nlat_i, nlon_i, K), s * qq, axis=1)
                assert np.abs(dense[jo] - shifted.reshape(-1, K)).max() <= 1e-13


@pytest.mark.parametrize("case", PLAN_CASES)
def test_plan_entries_forward_match_dense_psi(case):
    _dense_check(case, False)


@pytest.mark.parametrize("case", PLAN_CASES)
def test_plan_entries_transpose_match_dense_psi(case):
    _dense_check(case, True)


# The paper's own pole-including (L + 1) x 2L grid (Sec. 4.2) and the
# axisymmetric basis (Sec. 3.4), on either grid.
POLE_CASES = [
    (9, 16, 9, 16),       # L = 8
    (17, 32, 9, 16),      # 2x downsampling L = 16 -> 8
    (9, 16, 17, 32),      # forward that upsamples (2 longitude phases)
    (13, 24, 13, 24),     # L = 12
]


@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("case", POLE_CASES)
def test_plan_entries_poles_axisym_match_dense_psi(case, transpose):
    _dense_check(case, transpose, sampling=1, basis=1)


@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("case", POLE_CASES[:2])
def test_plan_entries_poles_bilinear_match_dense_psi(case, transpose):
    _dense_check(case, transpose, sampling=1, basis=0)


@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("case", PLAN_CASES[:3])
def test_plan_entries_axisym_cell_centred_match_dense_psi(case, transpose):
    _dense_check(case, transpose, sampling=0, basis=1)


# Cell-area quadrature and node spacings other than the default (the
# options disco_basis_t carries).  No spacing puts a node or a hat edge exactly
# at the cutoff, where fp64 rounding of the two geometry routes decides.
@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("case", PLAN_CASES[:3])
@pytest.mark.parametrize("basis", [0, 1])
def test_plan_entries_cell_area_match_dense_psi(case, transpose, basis):
    _dense_check(case, transpose, sampling=0, basis=basis, quad=1)


@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("case", PLAN_CASES[:3])
@pytest.mark.parametrize("basis,h_scale", [(0, 0.5), (0, 0.25), (1, 0.22), (2, 0.2)])
def test_plan_entries_node_spacing_match_dense_psi(case, transpose, basis, h_scale):
    _dense_check(case, transpose, sampling=0, basis=basis, h_scale=h_scale)


# The separable basis (Sec. 3.4: four nodes along theta times four periodic
# nodes along the direction), both grids.
@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("case", PLAN_CASES[:4])
def test_plan_entries_separable_cell_centred_match_dense_psi(case, transpose):
    _dense_check(case, transpose, sampling=0, basis=2)


@pytest.mark.parametrize("transpose", [False, True])
@pytest.mark.parametrize("case", POLE_CASES[:3])
def test_plan_entries_separable_poles_match_dense_psi(case, transpose):
    _dense_check(case, transpose, sampling=1, basis=2)


def test_separable_entries_stay_in_their_cell():
    """Every stored separable entry has at most four non-zero values, on at
    most two neighbouring theta nodes and two neighbouring (periodic) phi
    nodes, and its values sum to q times one minus the missing fifth theta
    node's share (the theta hats are a partition of unity on [0, 3h])."""
    a, b = 16, 32
    tc = 3 * math.pi / a
    ent = disco.psi_entries(a, b, a, b, tc, basis=2)
    q = oracle.default().quadrature(a, b)
    v = ent["values"].astype(np.float64).reshape(-1, 4, 4)
    for e in range(v.shape[0]):
        nz = np.argwhere(v[e] != 0)
        assert 1 <= len(nz) <= 4
        ta = sorted(set(nz[:, 0]))
        pb = sorted(set(nz[:, 1]))
        assert len(ta) <= 2 and (len(ta) < 2 or ta[1] == ta[0] + 1)
        assert len(pb) <= 2 and (len(pb) < 2 or (pb[1] - pb[0]) in (1, 3))
        s = v[e].sum() / q[int(ent["in_ring"][e])]
        assert s <= 1.0 + 1e-6
        if v[e, 3].sum() == 0.0:
            assert abs(s - 1.0) <= 1e-6


def test_pole_grid_validation():
    B = disco.Basis
    # nlon must be 2 (nlat - 1); cell areas are not offered there; unknown flag bits.
    rc, _ = _create(9, 18, 9, 18, 0.3, basis=B(1, 0, 0.0, 1, 0))
    assert rc == disco.DISCO_ERR_INVALID_ARGUMENT
    rc, _ = _create(9, 16, 9, 16, 0.3, basis=B(1, 1, 0.0, 1, 0))
    assert rc == disco.DISCO_ERR_UNSUPPORTED
    rc, _ = _create(9, 16, 9, 16, 0.3, basis=B(1, 0, 0.0, 2, 0))
    assert rc == disco.DISCO_ERR_UNSUPPORTED
    rc, _ = _create(9, 16, 9, 16, 0.3, basis=B(1, 0, 0.0, 1, 6))
    assert rc == disco.DISCO_ERR_INVALID_ARGUMENT


def test_psi_entries_validation():
    lib = disco.library()
    cnt = ctypes.c_int64()
    null = ctypes.POINTER(ctypes.c_int32)()
    nullf = ctypes.POINTER(ctypes.c_float)()
    rc = lib.disco_psi_entries(0, 16, 8, 16, 0.3, None, 0, 0, null, null, null, null, nullf,
                               ctypes.byref(cnt), None, None)
    assert rc == disco.DISCO_ERR_INVALID_ARGUMENT
    rc = lib.disco_psi_entries(8, 16, 8, 12, 0.3, None, 0, 0, null, null, null, null, nullf,
                               ctypes.byref(cnt), None, None)
    assert rc == disco.DISCO_ERR_UNSUPPORTED
    rc = lib.disco_psi_entries(8, 16, 8, 16, 0.3, None, 0, 0, null, null, null, null, nullf,
                               None, None, None)
    assert rc == disco.DISCO_ERR_INVALID_ARGUMENT


def test_pattern_count_limit():
    """Kernels index (output ring, longitude phase) patterns in a 16-bit grid
    dimension: ops with more are rejected before any device work."""
    lib = disco.library()
    b = disco._basis()
    count = ctypes.c_int64()
    null_i = ctypes.POINTER(ctypes.c_int32)()
    null_f = ctypes.POINTER(ctypes.c_float)()
    def entries(a, bb, c, d):
        return lib.disco_psi_entries(a, bb, c, d, 0.01, ctypes.byref(b), 0, 0, null_i, null_i, null_i, null_i,
                                     null_f, ctypes.byref(count), None, None)
    assert entries(65536, 2, 65536, 2) == disco.DISCO_ERR_UNSUPPORTED
    assert entries(40000, 2, 40000, 4) == disco.DISCO_ERR_UNSUPPORTED   # forward op: 2 phases x 40000 rings
    assert "65535" in lib.disco_last_error().decode()


def _plan_stderr(env_log):
    """stderr of a fresh process that creates a 32 x 64 plan (without a
    device the creation stops after the host build)."""
    import subprocess
    import sys
    env = dict(os.environ)
    env.pop("DISCO_LOG", None)
    if env_log is not None:
        env["DISCO_LOG"] = env_log
    code = ("import ctypes; from paper_2209_13603_amd import disco; lib = disco.library(); "
            "h = ctypes.c_void_p(); rc = lib.disco_plan_create(32, 64, 32, 64, 3 * 3.141592653589793 / 32, None, "
            "ctypes.byref(h)); print(rc); rc == 0 and lib.disco_plan_destroy(h)")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    return r.stderr


def test_plan_statistics_are_logged_with_disco_log():
    err = _plan_stderr("1")
    fwd = [l for l in err.splitlines() if l.startswith("disco: forward op 32x64 -> 32x64")]
    assert len(fwd) == 1, err
    m = re.search(r"(\d+) stored entries, (\d+) non-zero .*largest window (\d+) entries, (\d+) full-ring windows, "
                  r"compressed psi ([0-9.]+) MB", fwd[0])
    assert m, fwd[0]
    entries, pairs, window, full, mb = int(m.group(1)), int(m.group(2)), int(m.group(3)), int(m.group(4)), \
        float(m.group(5))
    assert entries > 0 and pairs >= entries and 0 < window <= entries and 0 <= full <= 32
    assert abs(mb - (entries * (8 + 4 * 9) + 4 * 33) / 1e6) < 0.01
    assert any(l.startswith("disco: transpose op") for l in err.splitlines())


def test_plan_log_is_off_by_default():
    assert "disco:" not in _plan_stderr(None)
    assert "disco:" not in _plan_stderr("0")


def test_default_build_has_no_range_checks():
    """The production library compiles the psi-index range checks out."""
    assert disco.library().disco_debug_bounds_violations() == -1
