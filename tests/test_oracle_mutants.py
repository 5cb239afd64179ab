"""Planted mistakes in a copy of the oracle must each fail at least one pin.

Every mutant is a textual edit of ``oracle/disco_oracle.c`` compiled on the
CPU into a temporary library; the real oracle is untouched.  The mistakes are
the plausible ones: a wrong sign, a dropped term, a transposed operand, a
wrong index or constant.
"""
import pytest

import oracle
import oracle_pins

MUTANTS = {
    "v_sign": ("*v = th * yr / rho;", "*v = -th * yr / rho;"),
    "u_sign": ("*u = th * xr / rho;", "*u = -th * xr / rho;"),
    "rotation_y_sign": ("mat_y(-theta, my);", "mat_y(theta, my);"),
    "rotation_order": ("mat_mul(my, mz, m);", "mat_mul(mz, my, m);"),
    "fejer_denominator": ("(4.0 * (double)m * (double)m - 1.0)",
                          "(4.0 * (double)m * (double)m + 1.0)"),
    "fejer_last_term": ("m <= nlat / 2;", "m < nlat / 2;"),
    "cell_area_full_step": ("w = 2.0 * sin(th) * sin(0.5 * M_PI / nlat);",
                            "w = 2.0 * sin(th) * sin(M_PI / nlat);"),
    "cell_area_cosine": ("w = 2.0 * sin(th) * sin(0.5 * M_PI / nlat);",
                         "w = 2.0 * cos(th) * sin(0.5 * M_PI / nlat);"),
    "quadrature_kind_ignored": ("oracle_quadrature_s(g_in.nlat, g_in.nlon, smp, cfg.quad_kind, q_in)",
                                "oracle_quadrature_s(g_in.nlat, g_in.nlon, smp, 0, q_in)"),
    "colatitude_scale": ("(t + 0.5) * M_PI / (double)nlat", "(t + 0.5) * M_PI / (double)(nlat + 1)"),
    "longitude_direction": ("2.0 * M_PI * (double)p / (double)nlon",
                            "-2.0 * M_PI * (double)p / (double)nlon"),
    "drop_quadrature": ("zc[k] += val[k] * qw * xv;", "zc[k] += val[k] * xv;"),
    "transpose_drops_quadrature": ("double qw = q_in[t];", "double qw = transpose ? 1.0 : q_in[t];"),
    "forward_w_transposed": (": w[((int64_t)co * Cin + ci) * K + k];",
                             ": w[((int64_t)ci * Cout + co) * K + k];"),
    "transpose_w_not_transposed": ("double wv = transpose ? w[((int64_t)ci * Cout + co) * K + k]",
                                   "double wv = transpose ? w[((int64_t)co * Cin + ci) * K + k]"),
    "basis_index_order": ("psi[3 * a + b] = hat", "psi[3 * b + a] = hat"),
    "node_spacing_ignored": ("        oracle_basis(u, v, h, psi);", "        oracle_basis(u, v, theta_c / 3.0, psi);"),
    "axisym_node_spacing_ignored": ("        oracle_basis_axisym(Th, h, psi);",
                                    "        oracle_basis_axisym(Th, theta_c / 4.0, psi);"),
    "hat_shape": ("return a < 1.0 ? 1.0 - a : 0.0;", "return a < 1.0 ? 1.0 - a * a : 0.0;"),
    "cutoff_too_small": ("if (Th > theta_c) return 0;", "if (Th > 0.5 * theta_c) return 0;"),
    "window_too_narrow": ("if (window && fabs(th_i - th_o) > theta_c) continue;",
                          "if (window && fabs(th_i - th_o) > 0.5 * theta_c) continue;"),
    "transpose_centre_swapped": ("nz = filter_values(cfg.basis, m_i, e_o, theta_c, h, val);",
                                 "nz = filter_values(cfg.basis, m_o, e_i_t, theta_c, h, val);"),
    "basis_drops_corner": ("psi[3 * a + b] = hat(u / h - (a - 1)) * hat(v / h - (b - 1));",
                           "psi[3 * a + b] = (a != 1 && b != 1) ? 0.0 : "
                           "hat(u / h - (a - 1)) * hat(v / h - (b - 1));"),
    # The pole-including grid, App. A's quadrature and the axisymmetric basis.
    "mw_colatitude": ("return M_PI * (double)t / (double)(nlat - 1);",
                      "return M_PI * (double)t / (double)nlat;"),
    "mw_fold_dropped": ("if (t != 0 && t != L) s += band_limited_sin",
                        "if (0) s += band_limited_sin"),
    "mw_fold_at_poles": ("if (t != 0 && t != L) s += band_limited_sin",
                         "s += band_limited_sin"),
    "mw_sum_range": ("for (int m = -L; m <= L - 1; ++m)", "for (int m = -L + 1; m <= L - 1; ++m)"),
    "mw_even_coefficient": ("*re = 2.0 / (1.0 - (double)m * (double)m);",
                            "*re = 2.0 / (1.0 + (double)m * (double)m);"),
    "mw_normalisation": ("2.0 * M_PI / ((2.0 * L) * (2.0 * L))",
                         "2.0 * M_PI / ((2.0 * L) * (2.0 * L + 1.0))"),
    "axisym_node_shift": ("psi[k] = hat(Theta / h - k);", "psi[k] = hat(Theta / h - k - 1);"),
    "axisym_signed_coordinate": ("oracle_basis_axisym(Th, h, psi);", "oracle_basis_axisym(u, h, psi);"),
    "axisym_drops_last_node": ("return basis == 1 ? 4 : basis", "return basis == 1 ? 3 : basis"),
    "separable_phi_node_offset": ("double d = fmod(fabs(Phi - b * 0.5 * M_PI), 2.0 * M_PI);",
                                  "double d = fmod(fabs(Phi + b * 0.5 * M_PI), 2.0 * M_PI);"),
    "separable_phi_not_periodic": ("if (d > M_PI) d = 2.0 * M_PI - d;", "if (d > 4.0 * M_PI) d = 2.0 * M_PI - d;"),
    "separable_index_order": ("psi[4 * a + b] = la * hat(d / (0.5 * M_PI));",
                              "psi[4 * b + a] = la * hat(d / (0.5 * M_PI));"),
    "separable_centre_direction": ("if (Theta <= 1e-12) Phi = 0.0;", "if (Theta <= 1e-12) Phi = 0.5 * M_PI;"),
    # Gradients (App. C).
    "adjoint_quadrature_of_source": ("            double qw = q[td];", "            double qw = q[td] * 0.0 + 1.0;"),
    "adjoint_w_not_transposed": (": w[((int64_t)cy * C_dx + cx) * K + k];",
                                 ": w[((int64_t)(cy % C_dx) * C_dy + (cx % C_dy)) * K + k];"),
    "adjoint_centre_swapped": ("nz = filter_values(cfg.basis, m_s, e_d, theta_c, h, val);",
                               "nz = filter_values(cfg.basis, m_d, e_s_t, theta_c, h, val);"),
    "weight_grad_first_batch_only": ("        for (int b = 0; b < B; ++b)\n            for (int cx = 0; cx < C_x; ++cx)\n                for (int cy = 0; cy < C_dy; ++cy)",
                                     "        for (int b = 0; b < 1; ++b)\n            for (int cx = 0; cx < C_x; ++cx)\n                for (int cy = 0; cy < C_dy; ++cy)"),
    "weight_grad_layout_swapped": ("int64_t at = transpose ? ((int64_t)cx * C_dy + cy) * K + k : ((int64_t)cy * C_x + cx) * K + k;",
                                   "int64_t at = transpose ? ((int64_t)cy * C_x + cx) * K + k : ((int64_t)cx * C_dy + cy) * K + k;"),
}


def _mutant_source(name):
    with open(oracle.SOURCE) as f:
        src = f.read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, (name, src.count(old))
    src = src.replace(old, new)
    if name == "adjoint_centre_swapped":
        src = src.replace("double m_s[9];", "double m_s[9], e_s_t[3]; unit_vector(th_s, ph_s, e_s_t);")
    if name == "transpose_centre_swapped":
        # Evaluate the transposed op's filter centred at the output point.
        src = src.replace("double m_i[9];", "double m_i[9], e_i_t[3]; unit_vector(th_i, ph_i, e_i_t);")
    return src


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    src = tmp_path / "mutant.c"
    src.write_text(_mutant_source(name))
    lib = oracle.build(out=str(tmp_path / ("lib_%s.so" % name)), source=str(src))
    o = oracle.Oracle(lib)
    failed = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(o)
        except AssertionError:
            failed.append(pin.__name__)
            break
    assert failed, "mutant %s passed every pin" % name
