"""The oracle's pins catch plausible mistakes (CPU only).

Each case plants one mistake in a copy of the oracle's C source (never in the
oracle itself), builds it with gcc into a temporary directory, swaps it in for
the real build and runs the pins of ``test_oracle_pins.py``: at least one pin
must fail for every planted mistake.
"""
import os
import subprocess

import pytest

from oracle import oracle as O
import test_oracle_pins as P

SRC = os.path.join(os.path.dirname(O.__file__), "wavernn_oracle.c")

MUTANTS = {
    "u_reads_r_gate": ("float au = G[0 * H + i] + (ix[0] + add[0 * H + i]);",
                       "float au = G[1 * H + i] + (ix[1] + add[1 * H + i]);"),
    "reset_gate_dropped": ("orc_tanh(fmaf(r, G[2 * H + i],", "orc_tanh(fmaf(1.0f, G[2 * H + i],"),
    "interpolation_swapped": ("fmaf(u, h_prev[i], (1.0f - u) * e)", "fmaf(1.0f - u, h_prev[i], u * e)"),
    "R_transposed": ("for (int row = 0; row < 3 * H; ++row) G[row] = dot(m->R + (size_t)row * H, hs, H);",
                     "for (int row = 0; row < 3 * H; ++row) { float acc = 0.0f; int g = row / H, q = row % H;"
                     " for (int j = 0; j < H; ++j) acc = fmaf(m->R[((size_t)g * H + j) * H + q], hs[j], acc);"
                     " G[row] = acc; }"),
    "mask_ignored": ("ix[g] = dot(Ig, x, i < Hh ? 2 : 3);", "ix[g] = dot(Ig, x, 3);",
                     "float x[3] = {orc_scale(cprev[st]), orc_scale(fprev[st]), 0.0f};",
                     "float x[3] = {orc_scale(cprev[st]), orc_scale(fprev[st]), tgt ? orc_scale(tgt[local] >> 8) : 0.0f};"),
    "gate_bias_dropped": ("float a = m->b[row];", "float a = 0.0f;",
                          "feat_frame, m->Dc) + m->b[row];", "feat_frame, m->Dc);"),
    "conditioning_dropped": ("if (m->Dc > 0) a = dot(", "if (0) a = dot("),
    "frame_off_by_one": ("int64_t fr = n / m->frame_len;", "int64_t fr = (n + 1) / m->frame_len;"),
    "heads_read_wrong_half": ("head(m, m->O1, m->b1, m->O2, m->b2, hn, zc);",
                              "head(m, m->O1, m->b1, m->O2, m->b2, hn + Hh, zc);"),
    "relu_dropped": ("hid[k] = relu(dot(Oa + (size_t)k * Hh, y, Hh) + ba[k]);",
                     "hid[k] = dot(Oa + (size_t)k * Hh, y, Hh) + ba[k];"),
    "head_bias_dropped": ("z[v] = dot(Ob + (size_t)v * Hh, hid, Hh) + bb[v];", "z[v] = dot(Ob + (size_t)v * Hh, hid, Hh);"),
    "philox_words_swapped": ("*uc = (float)(w[0] >> 40)", "*uc = (float)(w[1] >> 40)",
                             "*uf = (float)(w[1] >> 40)", "*uf = (float)(w[0] >> 40)"),
    "philox_counter_layout": ("uint64_t ctr[4] = {(uint64_t)t, stream, 0, 0}", "uint64_t ctr[4] = {stream, (uint64_t)t, 0, 0}"),
    "philox_no_key_bump": ("if (round > 0) { k0 += W0; k1 += W1; }", "if (0) { k0 += W0; k1 += W1; }"),
    "draw_strict_compare": ("count += (c[k] <= thr);", "count += (c[k] < thr);"),
    "draw_without_max_shift": ("w[k] = orc_exp(z[k] - m);", "w[k] = orc_exp(z[k]);"),
    "scale_formula": ("return (float)(2 * v - 255) / 255.0f;", "return (float)v / 128.0f - 1.0f;"),
    "sigmoid_sign": ("return 1.0f / (1.0f + orc_exp(-x));", "return 1.0f / (1.0f + orc_exp(x));"),
    "tanh_as_sigmoid": ("float t = (1.0f - q) / (1.0f + q);", "float t = 1.0f / (1.0f + q);"),
    "nll_fine_term_dropped": ("neg_log_prob(zc, ORC_MAX_CLASSES, c) + neg_log_prob(zf, ORC_MAX_CLASSES, f)",
                              "neg_log_prob(zc, ORC_MAX_CLASSES, c)"),
    "nll_coarse_fine_swapped": ("neg_log_prob(zc, ORC_MAX_CLASSES, c) + neg_log_prob(zf, ORC_MAX_CLASSES, f)",
                                "neg_log_prob(zc, ORC_MAX_CLASSES, f) + neg_log_prob(zf, ORC_MAX_CLASSES, c)"),
    "sample_bytes_swapped": ("if (!tgt) seq[local] = (uint16_t)(256 * c + f);", "if (!tgt) seq[local] = (uint16_t)(256 * f + c);"),
    "fused_nll_coarse_nibbles_swapped": ("neg_log_prob(zc[s], 16, c[s] >> 4) + neg_log_prob(zc[s] + 16, 16, c[s] & 15)",
                                         "neg_log_prob(zc[s], 16, c[s] & 15) + neg_log_prob(zc[s] + 16, 16, c[s] >> 4)"),
    "fused_nll_fine_nibbles_swapped": ("neg_log_prob(zf[s], 16, f[s] >> 4) + neg_log_prob(zf[s] + 16, 16, f[s] & 15)",
                                       "neg_log_prob(zf[s], 16, f[s] & 15) + neg_log_prob(zf[s] + 16, 16, f[s] >> 4)"),
    "fused_nll_levels_swapped": ("neg_log_prob(zc[s], 16, c[s] >> 4) + neg_log_prob(zc[s] + 16, 16, c[s] & 15) +\n"
                                 "                       neg_log_prob(zf[s], 16, f[s] >> 4) + neg_log_prob(zf[s] + 16, 16, f[s] & 15)",
                                 "neg_log_prob(zc[s], 16, f[s] >> 4) + neg_log_prob(zc[s] + 16, 16, f[s] & 15) +\n"
                                 "                       neg_log_prob(zf[s], 16, c[s] >> 4) + neg_log_prob(zf[s] + 16, 16, c[s] & 15)"),
    "subscale_no_row_mask": ("seen = q >= 0 && q < (int64_t)B * i;", "seen = q >= 0 && q < n;"),
    "subscale_horizon_plus_one": ("return z < s && k <= i + F;", "return z < s && k <= i + F + 1;"),
    "subscale_sees_own_sub_tensor": ("return z < s && k <= i + F;", "return z <= s && k <= i + F;"),
    "subscale_sees_own_past": ("return z < s && k <= i + F;", "return (z < s && k <= i + F) || (z == s && k < i);"),
    "subscale_window_includes_n": ("n + 1 + (j - P / 2)", "n + (j - P / 2)"),
    "subscale_lane_order": ("const int64_t n = (B == 1) ? t0 + i : B * i + lane;",
                            "const int64_t n = (B == 1) ? t0 + i : rows * lane + i;"),
    "fused_lag_short_by_one": ("const int64_t p[2] = {t, t - (m->F + 1)};", "const int64_t p[2] = {t, t - m->F};"),
    "fused_fine_sees_other_coarse": ("      x[4] = 0.0f;\n", "      x[4] = orc_scale(c[0]);\n"),
    "fused_nibble_words_swapped": ("return 16 * orc_draw(z, 16, u[0]) + orc_draw(z + 16, 16, u[1]);",
                                   "return 16 * orc_draw(z, 16, u[1]) + orc_draw(z + 16, 16, u[0]);"),
    "fused_heads_read_other_quarter": ("fused_head(m, s, hn + s * Q, zc[s]);", "fused_head(m, s, hn + (1 - s) * Q, zc[s]);"),
    "fused_idle_coarse_input_reset": ("act[s] ? fused_nibbles(zc[s], u[s], tgt ? tgt[2 * p[s] + s] >> 8 : -1) : cl[s];",
                                      "act[s] ? fused_nibbles(zc[s], u[s], tgt ? tgt[2 * p[s] + s] >> 8 : -1) : 128;"),
    "fused_stream_index": ("(uint64_t)(2 * ut + s), 0, 0}", "(uint64_t)(ut + s), 0, 0}"),
    "fused_coarse_sees_current_bytes": ("fused_units(m, G, add, x, 4, h, hn, 0, 2 * Q);",
                                        "x[4] = 1.0f; fused_units(m, G, add, x, 6, h, hn, 0, 2 * Q);"),
    "cnn_context_of_previous_sub_tensor": ("if (m->cnn) orc_ctx_cnn(m->cnn, tgt ? tgt : seq, T, (int32_t)o, ctab);",
                                           "if (m->cnn) orc_ctx_cnn(m->cnn, tgt ? tgt : seq, T, (int32_t)(o > 0 ? o - 1 : 0), ctab);"),
    "cnn_context_row_ahead": ("if (m->cnn) memcpy(ctx, ctab + (size_t)i * m->Dx,",
                              "if (m->cnn) memcpy(ctx, ctab + (size_t)(i + 1 < rows ? i + 1 : i) * m->Dx,"),
    "cnn_past_taps": ("const int64_t kk = k + (int64_t)tap * d;", "const int64_t kk = k - (int64_t)tap * d;"),
    "cnn_dilation_stages_4": ("const int d = 1 << (l % 5);", "const int d = 1 << (l % 4);"),
    "cnn_sees_own_sub_tensor": ("const int seen = z < s;", "const int seen = z <= s;"),
    "cnn_no_residual": ("rn[k * Rc + o] = r[k * Rc + o] + (dot(", "rn[k * Rc + o] = 0.0f * r[k * Rc + o] + (dot("),
    "cnn_relu_dropped": ("        a[c] = relu(acc);", "        a[c] = acc;"),
    "exp_low_coeffs_off": ("g_inv_fact[i] = (float)(1.0 / f);", "g_inv_fact[i] = (float)(1.0 / (f + (i == 2)));"),
}

PINS = [
    "test_philox_matches_numpy", "test_exp_accuracy_and_specials", "test_sigmoid_tanh_accuracy",
    "test_scale_is_correctly_rounded", "test_draw_uniform_logits_is_floor_256u",
    "test_draw_point_mass_and_zero_probability_classes",
    "test_zero_model_samples_are_floor_256u_and_nll_is_2ln256", "test_zero_model_streams_use_their_own_philox_stream",
    "test_nll_and_samples_at_point_mass_logits", "test_nll_at_unequal_coarse_and_fine_distributions",
    "test_fused_nll_at_point_mass_nibbles",
    "test_update_gate_saturated_at_one_keeps_state", "test_hand_case_input_mask_and_heads",
    "test_hand_case_reset_gate_placement_and_R_orientation", "test_hand_case_update_gate_interpolates",
    "test_hand_case_conditioning_frames", "test_coarse_logits_do_not_depend_on_current_coarse_byte",
    "test_chunked_sampling_equals_one_call", "test_subscale_without_context_is_interleaved_plain_streams",
    "test_subscale_context_masks_samples_of_the_current_row", "test_subscale_horizon_context_hand_cases",
    "test_subscale_horizon_dependencies_precede_in_the_lagged_schedule",
    "test_fused_zero_model_nibbles_are_floor_16u_and_nll_is_4ln16", "test_fused_state_reduces_to_the_plain_oracle",
    "test_fused_heads_read_their_own_quarter", "test_fused_dependencies_follow_the_fused_order",
    "test_cnn_shift_layers_sum_the_future_rows", "test_cnn_sees_only_previous_sub_tensors_within_124_rows_ahead",
    "test_cnn_first_sub_tensor_sees_nothing", "test_cnn_relu_clips_a_negative_layer",
    "test_cnn_conditioned_subscale_dependencies", "test_cnn_with_zero_output_is_the_plain_subscale_model",
]

_PARAMS = {"test_philox_matches_numpy": [dict(seed=7, stream=3, t=123456), dict(seed=1, stream=0, t=5)],
           "test_subscale_context_masks_samples_of_the_current_row": [dict(j=0), dict(j=5)],
           "test_subscale_horizon_context_hand_cases": [
               dict(zip(("B", "F", "Dx", "s", "i", "idx"), c))
               for c in P.test_subscale_horizon_context_hand_cases.pytestmark[0].args[1]],
           "test_subscale_horizon_dependencies_precede_in_the_lagged_schedule": [dict(F=1)],
           "test_fused_state_reduces_to_the_plain_oracle": [dict(s=0), dict(s=1)],
           "test_fused_heads_read_their_own_quarter": [dict(k=k) for k in range(4)],
           "test_fused_dependencies_follow_the_fused_order": [dict(F=2)],
           "test_cnn_shift_layers_sum_the_future_rows": [dict(layers=l) for l in (1, 2, 5, 10)]}


def _failures(tmp_path, name):
    src = open(SRC).read()
    edits = MUTANTS[name]
    for a, b in zip(edits[::2], edits[1::2]):
        assert src.count(a) == 1, (name, a)
        src = src.replace(a, b)
    d = tmp_path / name
    d.mkdir()
    (d / "m.c").write_text(src)
    (d / "wavernn_oracle.h").write_text(open(os.path.join(os.path.dirname(SRC), "wavernn_oracle.h")).read())
    so = str(d / "libm.so")
    subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fPIC", "-shared", "-std=c11", "-I", str(d),
                           "-o", so, str(d / "m.c"), "-lm"])
    saved = O._lib
    O._lib = O.load(so)
    failed = []
    try:
        for pin in PINS:
            for kw in _PARAMS.get(pin, [dict()]):
                try:
                    getattr(P, pin)(**kw)
                except (AssertionError, ValueError):
                    failed.append(pin)
                    break
    finally:
        O._lib = saved
    return failed


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    assert _failures(tmp_path, name), f"no pin caught the planted mistake {name}"
