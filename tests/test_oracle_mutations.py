"""Planted mistakes in the oracle must fail its pins (CPU only).

Each mutation below is a plausible slip in the C oracle (an off-by-one, a
wrong index, a swapped weight, a dropped term).  The test compiles a mutated
copy of ``oracle/logo_oracle.c`` into a temporary library, runs the pin suite
against it in a subprocess and requires that suite to fail.  The real oracle
is never modified.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "logo_oracle.c")

MUTATIONS = {
    "window_w_plus_1_keys": ("pos - window + 1 > 0 ? pos - window + 1 : 0",
                             "pos - window > 0 ? pos - window : 0"),
    "gate_ge_instead_of_gt": ("if (gate[t] > thr[b])", "if (gate[t] >= thr[b])"),
    "threshold_index_off_by_one": ("float thr = s[T - k - 1];", "float thr = s[T - k];"),
    "ratio_ceil": ("(int64_t)floor(ratio * (double)T)", "(int64_t)ceil(ratio * (double)T)"),
    "gqa_modulo_mapping": ("int hk = h / G;", "int hk = h % Hkv;"),
    "scale_dropped": ("s[j] = scale * dot;", "s[j] = dot;"),
    "values_read_from_keys": ("const uint16_t *vr = v + ", "const uint16_t *vr = k + "),
    "softmax_not_normalised": ("o[c] = acc[c] / den;", "o[c] = acc[c] / (double)nk;"),
    "norm_eps_outside_sqrt": ("1.0 / sqrt(ss / (double)d + eps)", "1.0 / (sqrt(ss / (double)d) + eps)"),
    "norm_sum_not_mean": ("1.0 / sqrt(ss / (double)d + eps)", "1.0 / sqrt(ss + eps)"),
    "norm_gain_ignores_head": ("gain[h * d + c]", "gain[c]"),
    "fusion_weights_swapped": ("o[e] = (1.0 - p) * l[e] + p * g[e];",
                               "o[e] = p * l[e] + (1.0 - p) * g[e];"),
    "unselected_not_normalised": ("oracle_contextnorm(nl, N, Hq, d, gain_local, eps);", ""),
    "global_branch_reads_local_tensors": (
        "oracle_attn_rows(q_g, k_g, v_g, Hq, Hkv, d, cu, B, sel_idx",
        "oracle_attn_rows(q, k, v, Hq, Hkv, d, cu, B, sel_idx"),
    "global_branch_windowed": ("sel_idx, n_sel, 0, scale, o_global", "sel_idx, n_sel, window, scale, o_global"),
    "varlen_leak_into_previous_sequence": (
        "int64_t lo = (window >= 1) ? (pos - window + 1 > 0 ? pos - window + 1 : 0) : 0;",
        "int64_t lo = (window >= 1) ? (pos - window + 1 > 0 ? pos - window + 1 : 0) : -base;"),
    "tok2sel_rank_off_by_one": ("tok2sel[t] = (int32_t)n;", "tok2sel[t] = (int32_t)n + 1;"),
    "cu_sel_not_prefix": ("cu_sel[b] = (int32_t)n;", "cu_sel[b] = 0;"),
    "controller_sign_flipped": ("        return b_th + gamma;\n    if (f < rho)\n        return b_th - gamma;",
                                "        return b_th - gamma;\n    if (f < rho)\n        return b_th + gamma;"),
    "controller_moves_on_equality": ("    if (f > rho)\n        return b_th + gamma;",
                                     "    if (f >= rho)\n        return b_th + gamma;"),
    "realized_ratio_inverted": ("(double)n_selected / (double)n_valid", "(double)n_valid / (double)n_selected"),
    "pmask_start_sign": ("(float)(0.5 - (double)gamma * (double)pmask_steps)",
                         "(float)(0.5 + (double)gamma * (double)pmask_steps)"),
    "decode_window_w_plus_1_keys": ("(branch == 0 && L > window) ? L - window : 0",
                                    "(branch == 0 && L > window) ? L - window - 1 : 0"),
    "decode_gate_ge_instead_of_gt": ("z_out[b] = gate_new[b] > threshold ? 1 : 0;",
                                     "z_out[b] = gate_new[b] >= threshold ? 1 : 0;"),
    "decode_global_reads_local_query": ("(branch == 0 ? q_new : q_g_new)", "q_new"),
    "decode_global_windowed": ("(branch == 0 && L > window)", "(L > window)"),
    "decode_gqa_modulo_mapping": ("const int kvh = h / G;", "const int kvh = h % Hkv;"),
    "decode_fusion_weights_swapped": ("? (1.0 - p) * l + p * ng[b * row + e] : l",
                                      "? p * l + (1.0 - p) * ng[b * row + e] : l"),
    "decode_unselected_fused": ("z_out[b] ? (1.0 - p) * l + p * ng[b * row + e] : l",
                                "(1.0 - p) * l + p * ng[b * row + e]"),
    "decode_cache_offset_dropped": ("const int64_t base = cu[b];\n            const int64_t L",
                                    "const int64_t base = 0;\n            const int64_t L"),
    "gate_sigmoid_sign": ("p_out[t] = (float)(1.0 / (1.0 + exp(-dot)));",
                          "p_out[t] = (float)(1.0 / (1.0 + exp(dot)));"),
    "gate_weight_index": ("* bf16_to_double(w_g[c]);", "* bf16_to_double(w_g[0]);"),
    "lp_matrix_transposed": ("A[((int64_t)h * d + c) * d + j]", "A[((int64_t)h * d + j) * d + c]"),
    "lp_matrix_ignores_head": ("A[((int64_t)h * d + c) * d + j]", "A[((int64_t)0 * d + c) * d + j]"),
    "so_offset_sign": ("+ (double)b[h * d + j];", "- (double)b[h * d + j];"),
    "transform_rows_ignored": ("const int64_t t = rows ? rows[r] : r;", "const int64_t t = r;"),
    "bwd_norm_missing_cubic_term": (
        "dO[c] = gc * dy[c] / r - o[c] * gdo / ((double)d * r * r * r);", "dO[c] = gc * dy[c] / r;"),
    "bwd_softmax_delta_dropped": ("const double ds = P[j] * (dP[j] - delta);",
                                  "const double ds = P[j] * dP[j];"),
    "bwd_dk_missing_scale": ("dkr[c] += scale * ds * qd[c];", "dkr[c] += ds * qd[c];"),
    "bwd_dv_before_norm": ("dvr[c] += P[j] * dO[c];", "dvr[c] += P[j] * dy[c];"),
    "bwd_local_weight_ignores_gate": ("const double wgt = branch ? p : (z ? 1.0 - p : 1.0);",
                                      "const double wgt = branch ? p : 1.0;"),
    "bwd_dgate_sign": ("(yg[t * row + e] - yl[t * row + e])", "(yl[t * row + e] - yg[t * row + e])"),
    "bwd_gain_grad_unnormalised": ("dG[h * d + c] += dy[c] * o[c] / r;",
                                   "dG[h * d + c] += dy[c] * o[c];"),
    "bwd_window_w_plus_1_keys": ("(branch == 0 && i - window + 1 > 0) ? i - window + 1 : 0",
                                 "(branch == 0 && i - window > 0) ? i - window : 0"),
    "fusion_bwd_projection_ignores_weight": ("proj += gc * wgt * dr[c] * o[c];",
                                             "proj += gc * dr[c] * o[c];"),
    "fusion_bwd_dgate_sign": ("side += (branch ? 1.0 : -1.0) * dr[c] * y;",
                              "side += (branch ? -1.0 : 1.0) * dr[c] * y;"),
    "fusion_bwd_delta_uses_dout": ("dl += dO[c] * o[c];", "dl += dr[c] * o[c];"),
    "attn_bwd_rowdot_dropped": ("const double g_s = w_p[j] * (w_dp[j] - rowdot);",
                                "const double g_s = w_p[j] * w_dp[j];"),
    "attn_bwd_dv_unweighted": ("dv[ko + c] += w_p[j] * go[c];", "dv[ko + c] += go[c];"),
    "bwd_sample_key_rows_short": ("(window >= 1 && i + window < T) ? i + window : T",
                                  "(window >= 1 && i + window - 1 < T) ? i + window - 1 : T"),
    "bwd_sample_global_rows_unselected": ("                    if (tok2sel[base + r] >= 0)\n                        need[2 * (base + r) + 1] = 1;",
                                          "                    need[2 * (base + r) + 1] = 0;"),
    "attn_bwd_window_w_plus_1_keys": ("(window >= 1 && i - window + 1 > 0) ? i - window + 1 : 0",
                                      "(window >= 1 && i - window > 0) ? i - window : 0"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_fails_pins(name, tmp_path):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique/present: {old!r}"
    mutated = tmp_path / "mut.c"
    mutated.write_text(src.replace(old, new))
    lib = tmp_path / "libmut.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                    "-ffp-contract=off", "-o", str(lib), str(mutated), "-lm"], check=True)
    env = dict(os.environ, LOGO_ORACLE_LIB=str(lib), OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"pins did not catch mutation {name}:\n{r.stdout[-2000:]}"
