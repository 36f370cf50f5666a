"""Planted mistakes in the oracle must each fail at least one pin.

Every mutant is the oracle's C source with one plausible slip (a dropped term, a
wrong sign, index or pitch, a transposed operand), compiled into a temporary
directory on the CPU. None of them touches memory outside the arrays, so they run
safely; the test asserts that the pin suite rejects each one, which is what makes
the pins worth trusting.
"""
import pytest

import oracle
from oracle_pins import ALL_PINS

MUTANTS = {
    "filter_flipped": ("const int iy = y * stride + r - pad;", "const int iy = y * stride + (R - 1 - r) - pad;"),
    "stride_on_tap": ("const int ix = xo * stride + s - pad;", "const int ix = xo + s * stride - pad;"),
    "stride_dropped_y": ("const int iy = y * stride + r - pad;", "const int iy = y + r - pad;"),
    "taps_transposed": ("const int iy = y * stride + r - pad;", "const int iy = y * stride + s - pad;"),
    "bias_dropped": ("const double b = bias ? (double)bias[k] : 0.0;", "const double b = 0.0;"),
    "bias_wrong_row": ("const double b = bias ? (double)bias[k] : 0.0;", "const double b = bias ? (double)bias[0] : 0.0;"),
    "accumulate_overwrites": ("acc[y * Wo + xo] += coeff * v;", "acc[y * Wo + xo] = coeff * v;"),
    "batch_ignored": ("const float *plane = x + ((size_t)n * C + c) * H * W;", "const float *plane = x + ((size_t)c) * H * W;"),
    "left_border_dropped": ("ix >= 0 && ix < W", "ix > 0 && ix < W"),
    "relu_inverted": ("acc[i] = acc[i] > 0.0 ? acc[i] : 0.0;", "acc[i] = acc[i] < 0.0 ? acc[i] : 0.0;"),
    "pool_window_narrow": ("const double v = acc[(2 * i + di) * Wo + 2 * j + dj];",
                           "const double v = acc[(2 * i + di) * Wo + 2 * j];"),
    "absacc_signed": ("ab[y * Wo + xo] += fabs(coeff * v);", "ab[y * Wo + xo] += coeff * v;"),
    "mask_ignored": ("if (mask) return mask[i] != 0;", "(void)mask;"),
    "mask_drops_explicit_zero": ("if (mask) return mask[i] != 0;", "if (mask) return mask[i] != 0 && w[i] != 0.0f;"),
    "offset_row_pitch": ("offset[nnz] = (int32_t)(c * Hp * Wp + r * Wp + s);",
                         "offset[nnz] = (int32_t)(c * Hp * Wp + r * Hp + s);"),
    "offset_plane_pitch": ("offset[nnz] = (int32_t)(c * Hp * Wp + r * Wp + s);",
                           "offset[nnz] = (int32_t)(c * Wp * Wp + r * Wp + s);"),
    "colidx_transposed": ("colidx[nnz] = (int32_t)((c * R + r) * S + s);",
                          "colidx[nnz] = (int32_t)((c * S + s) * R + r);"),
    "residual_dropped": ("acc[i] += (double)rp[i];", "(void)rp[i];"),
    "residual_after_relu": ("    if (res) {\n        const float *rp", "    if (relu)\n        for (int i = 0; i < Ho * Wo; ++i) acc[i] = acc[i] > 0.0 ? acc[i] : 0.0;\n    if (res) {\n        const float *rp"),
    "residual_batch_ignored": ("const float *rp = res + ((size_t)n * K + k) * Ho * Wo;", "const float *rp = res + ((size_t)k) * Ho * Wo;"),
    "residual_sign": ("acc[i] += (double)rp[i];", "acc[i] -= (double)rp[i];"),
    "resize_no_half_pixel": ("long long ny = (2LL * y + 1) * Hin - H;", "long long ny = 2LL * y * Hin;"),
    "resize_no_clamp": ("            if (ny < 0) ny = 0;\n", "\n"),
    "resize_weights_swapped": ("const double w00 = (1 - ty) * (1 - tx), w01 = (1 - ty) * tx,",
                               "const double w00 = (1 - ty) * tx, w01 = (1 - ty) * (1 - tx),"),
    "resize_x_fraction_from_height": ("const double tx = (double)(nx - x0 * 2LL * W) / (2.0 * W);",
                                      "const double tx = (double)(nx - x0 * 2LL * W) / (2.0 * H);"),
    "pack_last_row_dropped": ("for (int k = 0; k < K; ++k) {\n        for (int c = 0; c < C; ++c)\n            for (int r = 0; r < R; ++r)\n                for (int s = 0; s < S; ++s) {\n                    size_t i",
                              "for (int k = 0; k < K - 1; ++k) {\n        for (int c = 0; c < C; ++c)\n            for (int r = 0; r < R; ++r)\n                for (int s = 0; s < S; ++s) {\n                    size_t i"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = oracle.SOURCE.read_text()
    assert src.count(old) >= 1, f"mutation site for {name} not found in the oracle source"
    mutated = src.replace(old, new, 1)
    path = tmp_path / "mutant.c"
    path.write_text(mutated)
    lib = oracle.build(path, tmp_path / f"lib_{name}.so")
    orc = oracle.Oracle(lib)
    failed = []
    for pin in ALL_PINS:
        try:
            pin(orc)
        except Exception:  # an assertion, or a pin that cannot even digest the output
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
