"""The oracle's pins must catch plausible slips.

Each case below plants one mistake in a copy of the oracle's C source (on the
CPU, in a temporary directory), builds it, and runs the pins of test_oracle.py
against it: at least one pin has to fail.  The unmodified oracle passes all of
them (test_oracle.py).
"""
import os
import subprocess

import numpy as np
import pytest

import oracle
from oracle import oracle as oracle_mod
import test_oracle as pins

SRC = os.path.join(os.path.dirname(oracle_mod.__file__), "lapattn_oracle.c")

MUTANTS = {
    "scale gradient dropped": ("dW[a * m + bs] += dc * ninf", "dW[a * m + bs] += 0 * dc * ninf"),
    "X0 without transpose": ("Xs[a * m + b] = W[b * m + a] / c", "Xs[a * m + b] = W[a * m + b] / c"),
    "landmark-key gradient sign": ("dkt[l * d + c] -= t;", "dkt[l * d + c] += t;"),
    "centring term halved": ("o = y + (1.0 - si) * s->vbar[c];", "o = y + (1.0 - si) * s->vbar[c] * 0.5;"),
    "segments rounded up": ("starts[l] = (int)(((long long)l * n) / m);",
                            "starts[l] = (int)(((long long)l * n + m - 1) / m);"),
    "row norm used twice": ("double c = n1 * ninf;", "double c = ninf * ninf;"),
    "mean-value gradient dropped": ("tv + dvbar[c] / n", "tv"),
    "NS factors swapped": ("matmul(X, WX, Xn, m, m, m);", "matmul(WX, X, Xn, m, m, m);"),
    "kernel gradient sign": ("s->M[l * dv + c];\n                dD[(size_t)i * m + l] = -s->A",
                             "s->M[l * dv + c];\n                dD[(size_t)i * m + l] = s->A"),
    "K_LL backward dropped": ("dqt[a * d + c] += g * sg;", "dqt[a * d + c] += 0 * g * sg;"),
    "rowsum backward power": ("dYi[d] = -t / (si * si);", "dYi[d] = -t / si;"),
    "ones column wrong": ("(c < d ? v[(size_t)j * d + c] : 1.0)", "(c < d ? v[(size_t)j * d + c] : 0.5)"),
    "l2 instead of l1": ("dist += fabs(x[c] - y[c]);", "dist += (x[c] - y[c]) * (x[c] - y[c]);"),
    "eps ignored": ("for (int a = 0; a < m; ++a) W[a * m + a] += eps;", "(void)eps;"),
    "window rows and columns swapped": ("const int wy = l / mw, wx = l % mw;", "const int wy = l % mw, wx = l / mw;"),
    "window row stride r instead of the map width": (
        "members[l * r * r + t] = (wy * r + t / r) * grid_w + wx * r + t % r;",
        "members[l * r * r + t] = (wy * r + t / r) * r + wx * r + t % r;"),
    "window backward spread to segments": ("const int i = s->members[t];\n                dq[", "const int i = t;\n                dq["),
    "DWC filter flipped": ("if (j >= 0) acc += w[u * k + t] * v[(size_t)j * d + c];",
                           "if (j >= 0) acc += w[(k - 1 - u) * k + (k - 1 - t)] * v[(size_t)j * d + c];"),
    "DWC map rows and columns swapped": ("return y * gw + x;", "return x * gh + y;"),
    "DWC padding off by one": ("const int j = map_token(y + u - p, x + t - p, gh, gw);\n                                if (j >= 0) acc",
                               "const int j = map_token(y + u - p - 1, x + t - p, gh, gw);\n                                if (j >= 0) acc"),
    "DWC bias dropped": ("double acc = bias ? bias[h * d + c] : 0.0;", "double acc = 0.0;"),
    "DWC value gradient not flipped": ("map_token(y - (u - p), x - (t - p), gh, gw)", "map_token(y + (u - p), x + (t - p), gh, gw)"),
    "DWC bias gradient misses the batch": ("dbias[h * d + c] += gi;", "dbias[h * d + c] = gi;"),
    "DWC filter gradient misses the batch": ("for (size_t e = 0; e < (size_t)H * d * k * k; ++e) dWt[e] = 0.0;\n    for (size_t e = 0; e < (size_t)H * d; ++e) dbias[e] = 0.0;\n    for (int b = 0; b < B; ++b)\n        for (int h = 0; h < H; ++h) {",
        "for (size_t e = 0; e < (size_t)H * d; ++e) dbias[e] = 0.0;\n    for (int b = 0; b < B; ++b)\n        for (int h = 0; h < H; ++h) {\n            for (size_t e = (size_t)h * d * k * k; e < (size_t)(h + 1) * d * k * k; ++e) dWt[e] = 0.0;"),
    "m-space centring dropped": (
        "const double z = (wl ? wl[l] : 1.0) * (s->A[(size_t)i * m + l] - abar) + 1.0 / m;\n                    o += z",
        "const double z = (wl ? wl[l] : 1.0) * (s->A[(size_t)i * m + l]) + 1.0 / m;\n                    o += z"),
    "m-space offset 1/n": (
        "const double z = (wl ? wl[l] : 1.0) * (s->A[(size_t)i * m + l] - abar) + 1.0 / m;\n                    o += z",
        "const double z = (wl ? wl[l] : 1.0) * (s->A[(size_t)i * m + l] - abar) + 1.0 / n;\n                    o += z"),
    "m-space whitening misses the mean": (
        "const double z = (wl ? wl[l] : 1.0) * (s->A[(size_t)i * m + l] - abar) + 1.0 / m;\n                    o += z",
        "const double z = (wl ? wl[l] : 1.0) * s->A[(size_t)i * m + l] - abar + 1.0 / m;\n                    o += z"),
    "m-space backward mean term dropped": ("const double da = (wl ? wl[l] : 1.0) * dz[l] - t / m;",
                                           "const double da = (wl ? wl[l] : 1.0) * dz[l];"),
    "m-space dM from the kernel values": ("t += z * dO[(size_t)i * d + c];",
                                          "t += s->A[(size_t)i * m + l] * dO[(size_t)i * d + c];"),
    "query/key landmarks swapped in K_LL": (
        "s->Wk[a * m + b] = lapattn_oracle_kernel(s->qt + a * d, s->kt + b * d, d, lambda);",
        "s->Wk[a * m + b] = lapattn_oracle_kernel(s->kt + a * d, s->qt + b * d, d, lambda);"),
}

PIN_CALLS = [
    lambda: pins.test_kernel_identity_and_unit_distance(None),
    lambda: pins.test_kernel_gradient_norm_appendix_a(None),
    lambda: pins.test_segments_golden(None),
    lambda: pins.test_ns_golden_examples(None),
    lambda: pins.test_ns_x0_uses_transpose_and_induced_norms(None),
    lambda: pins.test_ns_residual_identity(None, 16, 6),
    lambda: pins.test_ns_special_cases(None),
    lambda: pins.test_forward_golden_examples(None),
    lambda: pins.test_forward_landmarks_equal_tokens_is_dense_attention(None, oracle.NORM_INLINE, 16, 8, 8 ** 0.5),
    lambda: pins.test_forward_one_landmark_closed_form(None),
    lambda: pins.test_forward_inline_rows_sum_to_one(None),
    lambda: pins.test_forward_permutation_within_hand_stated_segments(None),
    lambda: pins.test_forward_factored_equals_explicit_nystrom(None),
    lambda: pins.test_backward_matches_finite_differences(None, oracle.NORM_ROWSUM, 13, 3, 5, 4, 1.5),
    lambda: pins.test_backward_matches_finite_differences(None, oracle.NORM_INLINE, 17, 4, 4, 6, 4.0),
    lambda: pins.test_backward_with_perturbation_and_two_heads(None),
    lambda: pins.test_windows_landmarks_are_average_pooling(None, 4, 6, 2),
    lambda: pins.test_windows_equal_segments_of_the_window_ordered_tokens(None, oracle.NORM_INLINE),
    lambda: pins.test_windows_special_cases_and_rejections(None),
    lambda: pins.test_dwc_is_library_cross_correlation(None, 5, 7, 3),
    lambda: pins.test_dwc_one_hot_filters_shift_the_map(None),
    lambda: pins.test_dwc_backward_matches_finite_differences(None),
    lambda: pins.test_mspace_landmarks_equal_tokens_is_dense_whitened_attention(None, 16, 8, 8 ** 0.5),
    lambda: pins.test_mspace_zero_whitening_gives_the_mean_landmark_row(None),
    lambda: pins.test_mspace_backward_matches_finite_differences(None, 13, 3, 5, 4, 1.5),
]


def _count_failures():
    fails = 0
    for call in PIN_CALLS:
        try:
            call()
        except (AssertionError, ValueError):
            fails += 1
    return fails


def test_unmodified_oracle_passes_the_pin_subset(oracle_lib):
    assert _count_failures() == 0


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(oracle_lib, tmp_path, name):
    a, b = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(a) == 1, "mutation anchor not found: %s" % name
    mpath = tmp_path / "mut.c"
    mpath.write_text(src.replace(a, b))
    so = tmp_path / "libmut.so"
    subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                           "-I", os.path.dirname(SRC), "-o", str(so), str(mpath), "-lm"])
    with oracle_mod.using(str(so)):
        assert _count_failures() >= 1, "no pin caught the mutant '%s'" % name
