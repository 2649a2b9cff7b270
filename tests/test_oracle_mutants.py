"""Planted mistakes in copies of the oracle must each fail at least one pin.

Each mutant is a plausible slip (a dropped term, a wrong sign, index, bound or
operand, an accumulator of the wrong width, a reordered rule).  The test
applies it to a temporary copy of oracle/nfo.cpp, builds that copy, and runs
the pins of oracle_pins.py against it.  The real oracle is never modified.
"""
import os
import shutil
import tempfile

import pytest

import oracle as nfo
from oracle import build as obuild
from tests import oracle_pins

SRC = os.path.join(os.path.dirname(obuild.__file__), "nfo.cpp")
HDR = os.path.join(os.path.dirname(obuild.__file__), "nfo.h")

# (name, original text, replacement) - the original must occur exactly once
MUTANTS = [
    ("pack_sign_of_zero", "mask_bit(mask, i) && row[i] > 0.0f", "mask_bit(mask, i) && row[i] >= 0.0f"),
    ("pack_ignores_mask", "mask_bit(mask, i) && row[i] > 0.0f", "row[i] > 0.0f"),
    ("pack_msb_first", "        brow[i / 64] |= (uint64_t)1 << (i % 64);",
     "        brow[i / 64] |= (uint64_t)1 << (63 - i % 64);"),
    ("counts_wrong_stride", "bits[(int64_t)w * bits_stride + i / 64]",
     "bits[(int64_t)w * ((n + 63) / 64) + i / 64]"),
    ("counts_drop_last_worker", "    for (int32_t w = 0; w < W; ++w)\n      c += ",
     "    for (int32_t w = 0; w + 1 < W; ++w)\n      c += "),
    ("fp32_drops_first_term", "    float s = g[i];", "    float s = 0.0f;"),
    ("fp32_mean_by_reciprocal", "s = s / (float)W;", "s = s * (1.0f / (float)W);"),
    ("fp32_reversed_order", "    for (int32_t w = 1; w < W; ++w) s = s + g[(int64_t)w * stride + i];",
     "    s = g[(int64_t)(W - 1) * stride + i];\n"
     "    for (int32_t w = W - 2; w >= 0; --w) s = s + g[(int64_t)w * stride + i];"),
    ("ssq_eligible_only", "      xsum_add(&ssq, m * m, 2 * p);", "      if (elig) xsum_add(&ssq, m * m, 2 * p);"),
    ("ssq_exponent_not_doubled", "xsum_add(&ssq, m * m, 2 * p);", "xsum_add(&ssq, m * m, p);"),
    ("sabs_all_elements", "      if (elig) xsum_add(&sabs, m, p);", "      xsum_add(&sabs, m, p);"),
    ("sabs_no_implicit_bit", "(e ? 0x800000u : 0u)", "0u"),
    ("sabs_subnormal_exponent", "int p = (int)(e ? e : 1) - 1;", "int p = (int)e;"),
    ("sum_truncated", "    if (half && (below || (m & 1u))) m += 1;", ""),
    ("sum_ties_away", "if (half && (below || (m & 1u))) m += 1;", "if (half) m += 1;"),
    ("sum_ignores_sticky", "if (half && (below || (m & 1u))) m += 1;", "if (half && (m & 1u)) m += 1;"),
    ("sum_drops_carry", "    a->d[i + 1] += a->d[i] >> 32;\n", ""),
    ("sum_drops_third_digit", "  a->d[i + 2] += (uint64_t)(t >> 64);\n", ""),
    ("sum_inf_before_nan", "abs_nan ? NAN : abs_inf ? INFINITY", "abs_inf ? INFINITY : abs_nan ? NAN"),
    ("sum_nonfinite_any_position", "        if (elig) {\n          abs_nan |= nan;", "        if (1) {\n          abs_nan |= nan;"),
    ("nonfinite_nan_only", "return ((u >> 23) & 0xffu) == 0xffu;", "return isnan(x);"),
    ("scale_over_n", "d->scale = nfo_scale(stats, W, n_eligible);", "d->scale = nfo_scale(stats, W, n);"),
    ("scale_missing_mean_over_workers", "return (float)(acc / (double)W);", "return (float)acc;"),
    ("scale_fp32_accumulator", "  double acc = 0.0;\n  for (int32_t w = 0; w < W; ++w)\n    acc +=",
     "  float acc = 0.0f;\n  for (int32_t w = 0; w < W; ++w)\n    acc +="),
    ("decode_by_reciprocal", "q[c] = (float)margin / (float)W;", "q[c] = (float)margin * (1.0f / (float)W);"),
    ("decode_sign_flipped", "int32_t margin = 2 * c - W;", "int32_t margin = W - 2 * c;"),
    ("decode_margin_halved", "int32_t margin = 2 * c - W;", "int32_t margin = c - W / 2;"),
    ("majority_tie_positive", "q[c] = margin > 0 ? 1.0f", "q[c] = margin >= 0 ? 1.0f"),
    ("median_upper", "double m = fin[(k - 1) / 2];", "double m = fin[k / 2];"),
    ("spike_ge", "if (fin[i] > thr) r |= NFO_R_NORM_SPIKE;", "if (fin[i] >= thr) r |= NFO_R_NORM_SPIKE;"),
    ("spike_kappa_not_squared", "double thr = (p->kappa * p->kappa) * m;", "double thr = p->kappa * m;"),
    ("spike_needs_three", "  if (k >= 2) {", "  if (k >= 3) {"),
    ("spike_counts_nonfinite", "    if (!isfinite(v)) continue;\n", ""),
    ("zero_worker_without_eligible", "  if (n_eligible > 0)\n    for (int32_t w = 0; w < W; ++w)\n      if",
     "  if (n_eligible >= 0)\n    for (int32_t w = 0; w < W; ++w)\n      if"),
    ("route_forced_before_plain", "  if (r & (NFO_R_NOT_ADMITTED | NFO_R_NO_ELIGIBLE)) {",
     "  if (!p->force_lowbit && (r & (NFO_R_NOT_ADMITTED | NFO_R_NO_ELIGIBLE))) {"),
    ("route_ignores_no_eligible", "  if (r & (NFO_R_NOT_ADMITTED | NFO_R_NO_ELIGIBLE)) {",
     "  if (r & NFO_R_NOT_ADMITTED) {"),
    ("route_ignores_veto", "  } else if (r & (NFO_R_VETO | NFO_R_GUARD |", "  } else if (r & (NFO_R_GUARD |"),
    ("route_ignores_guard", "  } else if (r & (NFO_R_VETO | NFO_R_GUARD |", "  } else if (r & (NFO_R_VETO |"),
    ("forced_reason_missing", "    r |= NFO_R_FORCED;\n", ""),
    ("bytes_without_scale", "(double)n_eligible / 8.0 + 4.0 +", "(double)n_eligible / 8.0 +"),
    ("bytes_bits_not_bytes", "(double)n_eligible / 8.0 + 4.0 +", "(double)n_eligible + 4.0 +"),
    ("output_decodes_routed", "    if (route == NFO_ROUTE_L && mask_bit(mask, i))\n      out[i] = scale * q[counts[i]];",
     "    if (route == NFO_ROUTE_L)\n      out[i] = scale * q[counts[i]];"),
    ("output_count_off_by_one", "out[i] = scale * q[counts[i]];", "out[i] = scale * q[counts[i] ? counts[i] - 1 : 0];"),
    ("output_ignores_route", "    if (route == NFO_ROUTE_L && mask_bit(mask, i))\n      out[i] = scale * q[counts[i]];",
     "    if (mask_bit(mask, i))\n      out[i] = scale * q[counts[i]];"),
    ("tern_output_decodes_routed",
     "    if (route == NFO_ROUTE_L && mask_bit(mask, i))\n      out[i] = scale * q[(int32_t)cpos[i]",
     "    if (route == NFO_ROUTE_L)\n      out[i] = scale * q[(int32_t)cpos[i]"),
    ("mask_ignores_eligibility", "    if (!eligible[s]) continue;  /* FP32-only segment: bits stay 0 */\n", ""),
    ("mask_short_segment", "for (int64_t i = off[s]; i < off[s] + len[s]; ++i)",
     "for (int64_t i = off[s]; i + 1 < off[s] + len[s]; ++i)"),
    ("mask_no_bounds_check", "    if (off[s] < 0 || len[s] < 0 || off[s] + len[s] > n) return -1;\n", ""),
    ("count_eligible_all", "  for (int64_t i = 0; i < n; ++i) c += mask_bit(mask, i);",
     "  for (int64_t i = 0; i < n; ++i) c += 1;"),
    ("health_skips_last_element", "    for (int64_t i = 0; i < n; ++i) {\n      float x",
     "    for (int64_t i = 0; i + 1 < n; ++i) {\n      float x"),
    # G-Ternary (R18-R21)
    ("tern_gate_le", "if (fabsf(x) < theta[w]) continue;", "if (fabsf(x) <= theta[w]) continue;"),
    ("tern_gate_signed", "if (fabsf(x) < theta[w]) continue;", "if (x < theta[w]) continue;"),
    ("tern_neg_includes_zero", "if (x < 0.0f) nrow[i / 64]", "if (x <= 0.0f) nrow[i / 64]"),
    ("tern_ignores_mask", "      if (!mask_bit(mask, i)) continue;\n      float x = row[i];", "      float x = row[i];"),
    ("tern_vote_reversed", "q[(int32_t)cpos[i] - (int32_t)cneg[i] + W]", "q[(int32_t)cneg[i] - (int32_t)cpos[i] + W]"),
    ("tern_threshold_rounded_once",
     "  float mean_abs = (float)(st->sum_abs_elig / (double)n_eligible);\n  return tau * mean_abs;",
     "  return (float)((double)tau * (st->sum_abs_elig / (double)n_eligible));"),
    ("tern_threshold_sum_not_mean", "(float)(st->sum_abs_elig / (double)n_eligible)", "(float)(st->sum_abs_elig)"),
    ("tern_bytes_one_plane", "(p->format == NFO_FORMAT_TERNARY ? 2.0 : 1.0)", "1.0"),
    ("tern_majority_tie", "q[d + W] = d > 0 ? 1.0f", "q[d + W] = d >= 0 ? 1.0f"),
    ("tern_counts_neg_from_pos", "nfo_counts(neg, bits_stride, W, n, cneg);", "nfo_counts(pos, bits_stride, W, n, cneg);"),
    ("tern_decode_by_reciprocal", "q[d + W] = (float)d / (float)W;", "q[d + W] = (float)d * (1.0f / (float)W);"),
    # compacted payload and per-slice scales (R29-R33)
    ("compact_positional_rank", "      if (!mask_bit(mask, i)) continue;\n      if (row[i] > 0.0f) crow[r / 64]",
     "      if (row[i] > 0.0f && mask_bit(mask, i)) crow[r / 64]"),
    ("compact_sign_ge", "if (row[i] > 0.0f) crow[r / 64]", "if (row[i] >= 0.0f) crow[r / 64]"),
    ("compact_msb_first", "crow[r / 64] |= (uint64_t)1 << (r % 64);", "crow[r / 64] |= (uint64_t)1 << (63 - r % 64);"),
    ("slice_sum_signed", "for (int64_t j = 0; j < len[s]; ++j) t += fabs((double)row[j]);",
     "for (int64_t j = 0; j < len[s]; ++j) t += (double)row[j];"),
    ("slice_mean_missing", "acc += t / (double)len[s];", "acc += t;"),
    ("slice_workers_not_averaged", "scales[s] = (float)(acc / (double)W);", "scales[s] = (float)acc;"),
    ("slice_skips_last", "for (int64_t j = 0; j < len[s]; ++j) t +=", "for (int64_t j = 0; j + 1 < len[s]; ++j) t +="),
    ("sliced_boundary_off_by_one", "while (s < S && i >= off[s] + len[s]) ++s;", "while (s < S && i > off[s] + len[s]) ++s;"),
    ("sliced_first_scale_only", "out[i] = scales[s] * q[counts[i]];", "out[i] = scales[0] * q[counts[i]];"),
]


def test_mutant_table_applies():
    src = open(SRC).read()
    for name, old, new in MUTANTS:
        assert src.count(old) == 1, f"{name}: target occurs {src.count(old)} times"
        assert old != new, name


@pytest.fixture(scope="module")
def tmpdir_mut():
    d = tempfile.mkdtemp(prefix="nfo_mut_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmpdir_mut, name, old, new):
    src = open(SRC).read()
    d = os.path.join(tmpdir_mut, name)
    os.makedirs(d, exist_ok=True)
    shutil.copy(HDR, d)
    with open(os.path.join(d, "nfo.cpp"), "w") as f:
        f.write(src.replace(old, new))
    lib_path = obuild.build(out=os.path.join(d, "libnfo_mut.so"),
                            src=os.path.join(d, "nfo.cpp"), extra=("-w",))
    lib = nfo.load(lib_path)
    failures = oracle_pins.run_all(lib)
    assert failures, f"mutant {name} passed every pin"
