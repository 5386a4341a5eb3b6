"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake in a copy of the oracle source, builds it on the
CPU with the same compiler flags, and checks that at least one pin of
``test_oracle_pins`` fails against the mutant.  The committed oracle itself
is untouched.
"""
import os
import shutil

import pytest

import oracle
from tests import test_oracle_pins as pins

# (name, original, replacement[, original, replacement ...]) -- each original
# text must occur exactly once in the source
MUTANTS = [
    ("transposed histogram", "Hv[b * bins_w + a] += (uint64_t)qx[a] * (uint64_t)qy[b];",
     "Hv[(a * bins_h + b) % (bins_w * bins_h)] += (uint64_t)qx[a] * (uint64_t)qy[b];"),
    ("dropped channel", "for (int32_t ch = 0; ch < twoF; ch++) {\n            int64_t diff",
     "for (int32_t ch = 1; ch < twoF; ch++) {\n            int64_t diff"),
    ("wrong sign in distance", "(int64_t)X[ch] - (int64_t)pal[a * twoF + ch]", "(int64_t)X[ch] + (int64_t)pal[a * twoF + ch]"),
    ("bin centre off by one", "double centre = ((double)(a + 1) * (double)extent) / (double)(n + 1);\n        for (int32_t k = 0; k < F; k++) {\n            double phase",
     "double centre = ((double)(a) * (double)extent) / (double)(n + 1);\n        for (int32_t k = 0; k < F; k++) {\n            double phase"),
    ("sin/cos swapped", "pal[a * 2 * F + 2 * k] = (int16_t)rint(4096.0 * sin(phase));",
     "pal[a * 2 * F + 2 * k] = (int16_t)rint(4096.0 * cos(phase));"),
    ("y block read from x channels", "Y[c] = to_fixed(load_value(emb, dtype, p * (size_t)D + (size_t)(yoff + c)));\n        }\n        axis_profile(X, Pw, bins_w, twoF, wt, qx, NULL);",
     "Y[c] = to_fixed(load_value(emb, dtype, p * (size_t)D + (size_t)(c)));\n        }\n        axis_profile(X, Pw, bins_w, twoF, wt, qx, NULL);"),
    ("y block taken right after the decoded x channels",
     "twoF = 2 * n_freq, yoff = D / 2;\n    const size_t npix = (size_t)H * (size_t)W;\n    const int32_t nbins = bins_w * bins_h;\n\n    int16_t *Pw",
     "twoF = 2 * n_freq, yoff = twoF;\n    const size_t npix = (size_t)H * (size_t)W;\n    const int32_t nbins = bins_w * bins_h;\n\n    int16_t *Pw"),
    ("x palette used for y", "axis_profile(Y, Ph, bins_h, twoF, wt, qy, NULL);", "axis_profile(Y, Pw, bins_h, twoF, wt, qy, NULL);"),
    ("weight e^-2d", "wt[key] = (uint16_t)rint(32768.0 * exp(-key_distance(key, W_MANT)));",
     "wt[key] = (uint16_t)rint(32768.0 * exp(-2.0 * key_distance(key, W_MANT)));"),
    ("weight scale", "wt[key] = (uint16_t)rint(32768.0 * exp(", "wt[key] = (uint16_t)rint(32767.0 * exp("),
    ("distance squared, not rooted", "if (r) r[a] = sqrtf((float)(uint32_t)s);", "if (r) r[a] = (float)(uint32_t)s;"),
    ("distance of S+1", "if (r) r[a] = sqrtf((float)(uint32_t)s);", "if (r) r[a] = sqrtf((float)(uint32_t)(s + 1u));"),
    ("distance sum rounded to a half unit",
     "double dk = (double)rx[peak_a[k]] + (double)ry[peak_b[k]];",
     "double dk = 0.5 * rint(2.0 * ((double)rx[peak_a[k]] + (double)ry[peak_b[k]]));",
     "double best_d = (double)rx[peak_a[0]] + (double)ry[peak_b[0]];",
     "double best_d = 0.5 * rint(2.0 * ((double)rx[peak_a[0]] + (double)ry[peak_b[0]]));"),
    ("NaN not clamped", "if (isnan(c) || c < -V_CLAMP) c = -V_CLAMP;", "if (c < -V_CLAMP) c = -V_CLAMP;"),
    ("non-strict local max", "if (!(v > h[nb * bw + na])) return 0;\n        }\n    return 1;\n}\n\nstatic int is_peak_f64",
     "if (!(v >= h[nb * bw + na])) return 0;\n        }\n    return 1;\n}\n\nstatic int is_peak_f64"),
    ("4-neighbourhood", "if (!da && !db) continue;\n            int32_t nb = b + db, na = a + da;\n            if (nb < 0 || nb >= bh || na < 0 || na >= bw) continue;\n            if (!(v > h[nb * bw + na])) return 0;\n        }\n    return 1;\n}\n\nstatic int is_peak_f64",
     "if (!da == !db) continue;\n            int32_t nb = b + db, na = a + da;\n            if (nb < 0 || nb >= bh || na < 0 || na >= bw) continue;\n            if (!(v > h[nb * bw + na])) return 0;\n        }\n    return 1;\n}\n\nstatic int is_peak_f64"),
    ("threshold not strict", "if (v > cut && is_peak_u64", "if (v >= cut - 1000000 && is_peak_u64"),
    ("tie goes to the last candidate", "if (dk < best_d) {\n                best_d = dk;\n                best = k;\n            }\n        }\n        /* Eq8",
     "if (dk <= best_d) {\n                best_d = dk;\n                best = k;\n            }\n        }\n        /* Eq8"),
    ("assignment ignores the y axis", "double dk = (double)rx[peak_a[k]] + (double)ry[peak_b[k]];", "double dk = (double)rx[peak_a[k]];",
     "double best_d = (double)rx[peak_a[0]] + (double)ry[peak_b[0]];", "double best_d = (double)rx[peak_a[0]];"),
    ("background pixels vote", "if (!participates(fg, dtype, p, fg_threshold)) continue;\n        for (int32_t c = 0; c < twoF; c++) {\n            X[c]",
     "if (!participates(fg, dtype, p, -1e30f)) continue;\n        for (int32_t c = 0; c < twoF; c++) {\n            X[c]"),
    ("no-fg mode votes nothing", "return !fg || load_value(fg, dtype, p) > fg_threshold;", "return fg && load_value(fg, dtype, p) > fg_threshold;"),
    ("mask threshold not strict", "if (!(best_d < 4096.0 * tau)) continue;", "if (!(best_d <= 4096.0 * tau)) continue;"),
    ("mask threshold on a wrong scale", "if (!(best_d < 4096.0 * tau)) continue;", "if (!(best_d < 256.0 * tau)) continue;"),
    ("mask threshold on the x distance only", "if (!(best_d < 4096.0 * tau)) continue;",
     "if (!((double)rx[peak_a[best]] < 4096.0 * tau)) continue;"),
    ("pixel over the mask threshold still counted", "if (!(best_d < 4096.0 * tau)) continue;\n        labels[p] = best + 1;\n        centroids[best].npix += 1;",
     "if (!(best_d < 4096.0 * tau)) { centroids[best].npix += 1; continue; }\n        labels[p] = best + 1;\n        centroids[best].npix += 1;"),
    ("clamp too wide", "if (c > V_CLAMP) c = V_CLAMP;", "if (c > 1.6f) c = 1.6f;"),
    ("input read on a 1/256 grid", "return (int32_t)rintf(FIX_SCALE * c);", "return 16 * (int32_t)rintf(256.0f * c);"),
    ("input truncated instead of rounded", "return (int32_t)rintf(FIX_SCALE * c);", "return (int32_t)truncf(FIX_SCALE * c);"),
    ("real mode: weight e^-2d", "hist[b * bins_w + a] += exp(-dx[a]) * exp(-dy[b]);",
     "hist[b * bins_w + a] += exp(-2.0 * dx[a]) * exp(-dy[b]);"),
    ("real mode: y block read from the x channels",
     "vy[c] = (double)load_value(emb, dtype, p * (size_t)D + (size_t)(yoff + c));\n        }\n        real_distances(vx, Pw, bins_w, twoF, dx);\n        real_distances(vy, Ph, bins_h, twoF, dy);\n        for (int32_t b = 0;",
     "vy[c] = (double)load_value(emb, dtype, p * (size_t)D + (size_t)(c));\n        }\n        real_distances(vx, Pw, bins_w, twoF, dx);\n        real_distances(vy, Ph, bins_h, twoF, dy);\n        for (int32_t b = 0;"),
    ("real mode: assignment ignores the y axis", "double d = dx[pk[k] % bins_w] + dy[pk[k] / bins_w];", "double d = dx[pk[k] % bins_w];",
     "double best_d = dx[pk[0] % bins_w] + dy[pk[0] / bins_w];", "double best_d = dx[pk[0] % bins_w];"),
]

PIN_CASES = [
    (pins.test_weight_buckets_bound_e_minus_d_over_each_bucket, ()),
    (pins.test_palette_is_gamma_at_bin_centres, ()),
    (pins.test_distance_of_exact_offsets_from_a_palette_entry, ()),
    (pins.test_palette_unit_circle_and_mirror, ()),
    (pins.test_histogram_matches_eq11_within_quantisation_bound, (pins.np.float32, 4, 12)),
    (pins.test_histogram_matches_eq11_within_quantisation_bound, (pins.np.float16, 16, 32)),
    (pins.test_histogram_catches_axis_swap, ()),
    (pins.test_peaks_match_library_local_max, (0,)),
    (pins.test_oracle_equals_exhaustive_search, (0, pins.np.float32, 2, 5, 4, 6)),
    (pins.test_oracle_equals_exhaustive_search, (1, pins.np.float16, 3, 6, 6, 2)),
    (pins.test_noise_free_decodes_generating_centroids_and_labels, (0,)),
    (pins.test_invariants, (0,)),
    (pins.test_clamp_saturates, ()),
    (pins.test_plateau_gives_no_peak_and_single_bin_is_a_peak, ()),
    (pins.test_threshold_is_strict, ()),
    (pins.test_exact_tie_goes_to_lowest_index, ()),
    (pins.test_assignment_agrees_with_eq7_in_fp64, (1,)),
    (pins.test_far_pixels_take_the_exact_argmin, ()),
    (pins.test_real_mode_equals_matrix_form_library_maxima_and_argmin, ("tiny1",)),
    (pins.test_real_mode_equals_matrix_form_library_maxima_and_argmin, ("cfg0",)),
    (pins.test_mask_threshold_and_all_pixels_equal_exhaustive_search, (5, pins.np.float16, 3, 6, 6, 3, False, (0.7, 0.5))),
    (pins.test_mask_threshold_and_all_pixels_equal_exhaustive_search, (6, pins.np.float32, 1, 4, 7, 8, False, (0.5, 0))),
    (pins.test_mask_threshold_on_noise_free_frame_with_all_pixels, ()),
    (pins.test_mask_threshold_nests, ()),
    (pins.test_low_harmonics_equal_decoding_the_sliced_encoding, (0, 4)),
]


def _fails(fn, args):
    try:
        fn(*args)
    except (AssertionError, ValueError, IndexError):
        return True
    return False


@pytest.mark.parametrize("mutant", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, mutant):
    name, edits = mutant[0], mutant[1:]
    src = open(oracle.SRC).read()
    for old, new in zip(edits[0::2], edits[1::2]):
        assert src.count(old) == 1, f"mutation site for '{name}' not unique"
        src = src.replace(old, new)
    path = tmp_path / "cpe_oracle.c"
    path.write_text(src)
    shutil.copy(os.path.join(oracle.HERE, "cpe_oracle.h"), tmp_path / "cpe_oracle.h")
    lib = oracle.build(src=str(path), out=str(tmp_path / "libmutant.so"))
    with oracle.using_library(lib):
        caught = [fn.__name__ for fn, args in PIN_CASES if _fails(fn, args)]
    assert caught, f"no pin catches the planted mistake '{name}'"


def test_unmutated_passes_all_pins():
    assert not [fn.__name__ for fn, args in PIN_CASES if _fails(fn, args)]
