/*
 * nfo.cpp - reference oracle for the NEURON-Fabric bucket reducer.
 *
 * TEST INFRASTRUCTURE ONLY (see nfo.h).  Plain single-threaded C++: every
 * loop visits elements in ascending order and workers in ascending order,
 * and nothing is blocked, fused or reordered.  Build with -ffp-contract=off
 * so that no multiply-add is contracted.
 *
 * Readings fixed here where the paper is silent or ambiguous:
 *   R1  One eligibility mask per bucket, shared by all W workers: the binding
 *       is per model and identical on every replica (§5.1, §5.3).  A
 *       parameter absent from the binding is FP32-only (§5.1).
 *   R2  Sign payloads are positional bitmaps, LSB-first uint64: bit j of word
 *       k is element 64k+j; elements that are not eligible, and padding past
 *       n, hold 0.  §6.1 speaks of bit-packed updates without a layout.
 *   R3  The sign indicator is (g > 0): +0, -0 and NaN give 0.  §5.2 names
 *       positive-sign indicators.
 *   R4  Counts are uint8, so 1 <= W <= 255.
 *   R5  One scale per bucket: the mean over workers of each worker's mean
 *       |g| over eligible elements (§5.2 records a mean-absolute scale).
 *       The per-worker sums are those of R8; the combination divides each
 *       worker sum by n_E, adds in worker order in FP64, divides by W, and
 *       rounds to FP32 once.
 *   R6  Decode: SOFT q_c = (2c - W) / W, the vote margin (default); MAJORITY
 *       q_c = sign(2c - W) with a tie giving 0 (§5.2's majority voting).
 *       Both are FP32 correctly-rounded quotients of exact integers.  The
 *       decoded value is fl32(scale * q_c).
 *   R7  FP32 path (§2.1 sums or averages): s = g_0, then s = fl32(s + g_w)
 *       for w = 1..W-1 (worker order, no contraction).  SUM returns s, MEAN
 *       returns fl32(s / W) by IEEE division.
 *   R8  Health per worker: nonfinite count over all n; sum |g| over eligible
 *       elements; sum g*g over all n.  Both sums are the exact real sums of
 *       their terms, rounded once to FP64 (to nearest, ties to even), so they
 *       depend on no summation order.  A NaN term makes a sum NaN; otherwise
 *       an infinite term makes it +Inf (as IEEE addition of non-negative
 *       terms does).  The paper fixes no precision for these statistics; the
 *       exact sum is the one every correct implementation can reproduce bit
 *       for bit, which the G-Ternary threshold (R18) needs.
 *   R9  Reason bits are all evaluated every time (nfo.h lists them).
 *   R10 Any non-finite input value in any worker sends the bucket to FP32.
 *   R11 A worker whose eligible |g| sum is exactly 0 (n_E > 0) sends the
 *       bucket to FP32: under R3 it would vote -1 everywhere.
 *   R12 Norm spike: over the workers whose sum g*g is finite (at least two),
 *       m = the lower median (sorted ascending, index floor((k-1)/2)); the
 *       bucket spikes if some such worker has sum g*g > (kappa*kappa) * m.
 *   R13 Route precedence: P (not admitted, or no eligible element) before
 *       forced L, before F (veto, guard, non-finite, zero worker, spike),
 *       before L.
 *   R14 Modeled bytes per worker (§3.2 MGTR): FP32 = 4n; the selected route
 *       is n_E/8 + 4 (one FP32 scale) + 4 n_F for L and 4n for F and P.
 *
 * G-Ternary (§2.2 adds a zero-gating rule to the sign route; §5.2 applies
 * the gating pattern around the vote; the paper fixes neither the rule nor
 * its point):
 *   R18 Gating is on the write side, before aggregation (§2.2), per worker:
 *       theta_w = fl32(tau * fl32(S_w / n_E)), S_w the worker's |g| sum over
 *       eligible elements (R8, exact and rounded once), tau >= 0 a policy
 *       input (default 0.5).
 *       An eligible element with |g| < theta_w (FP32 comparison) is gated to
 *       0.  NaN compares false, so it is never gated and never votes.
 *   R19 The payload is two positional planes per worker (R2 layout): pos =
 *       eligible, not gated and g > 0; neg = eligible, not gated and g < 0.
 *   R20 Counts c+ and c- per coordinate; d = c+ - c-; SOFT q_d = fl32(d / W),
 *       MAJORITY q_d = sign(d) (0 at d = 0); the output is fl32(scale * q_d)
 *       with the scale of R5.  Routes, reasons and FP32 positions as above.
 *   R21 MGTR for the ternary L route: 2 n_E / 8 + 4 + 4 n_F bytes per worker.
 *
 * Per-slice scales and a compacted payload (§5.2 records a mean-absolute
 * scale per eligible slice; §6.1 counts bit-packed updates; the paper fixes
 * neither the scale's granularity nor the payload's layout):
 *   R29 The eligible slices of a bucket are S intervals [off_s, off_s +
 *       len_s), sorted, disjoint, len_s >= 1; the mask is their union.
 *   R30 Compacted payload: bit r of worker w's row is (g > 0) of the r-th
 *       eligible element in element order (r = 0 .. n_E - 1), LSB-first
 *       uint64 words, ceil(n_E / 64) words, padding bits 0.
 *   R31 Slice scale: scale_s = fl32((sum_w S_sw / len_s) / W), S_sw the FP64
 *       sum of |g| over the slice in element order, workers in order (R5 on
 *       one slice).
 *   R32 Sliced decode: out_i = fl32(scale_s(i) * q[c_i]) at eligible i (c_i
 *       the count over the compacted rows at i's rank, equal to the
 *       positional count), the FP32 path elsewhere.
 *   R33 MGTR for this route: n_E / 8 + 4 S + 4 n_F bytes per worker.
 */
#include "nfo.h"

#include <math.h>
#include <string.h>

/* element i of the mask: R1, R2 */
static int mask_bit(const uint64_t* mask, int64_t i) {
  return (int)((mask[i / 64] >> (i % 64)) & 1u);
}

/* An FP32 value is non-finite when its exponent field is all ones. */
static int is_nonfinite(float x) {
  uint32_t u;
  memcpy(&u, &x, sizeof u);
  return ((u >> 23) & 0xffu) == 0xffu;
}

/* ---- a1: mask from the binding's segments (§5.1, R1, R2) ---------------- */
int nfo_mask_from_segments(const int64_t* off, const int64_t* len,
                           const uint8_t* eligible, int64_t nseg, int64_t n,
                           uint64_t* mask) {
  int64_t nwords = (n + 63) / 64;
  for (int64_t k = 0; k < nwords; ++k) mask[k] = 0;
  for (int64_t s = 0; s < nseg; ++s) {
    if (off[s] < 0 || len[s] < 0 || off[s] + len[s] > n) return -1;
    if (!eligible[s]) continue;  /* FP32-only segment: bits stay 0 */
    for (int64_t i = off[s]; i < off[s] + len[s]; ++i)
      mask[i / 64] |= (uint64_t)1 << (i % 64);
  }
  return 0;
}

int64_t nfo_count_eligible(const uint64_t* mask, int64_t n) {
  int64_t c = 0;
  for (int64_t i = 0; i < n; ++i) c += mask_bit(mask, i);
  return c;
}

/* ---- a2: per-worker health (R8) ----------------------------------------- */

/* Exact sums.  A finite FP32 value is m * 2^(e - 150) with a 24-bit integer
 * significand m and e = max(biased exponent, 1), so |g| is an integer number
 * of units 2^-149 and g*g (m*m < 2^48) an integer number of units 2^-298.  A
 * sum of such terms is kept exactly as an unsigned integer in base-2^32
 * digits (least significant first); 20 digits hold any sum of fewer than
 * 2^40 terms of either kind.  Carries are propagated lazily: a term adds
 * less than 2^32 to each of three digits, so a digit stays below 2^63 for
 * 2^31 terms between propagations. */
#define NFO_XDIG 20
typedef struct {
  uint64_t d[NFO_XDIG];
  uint32_t pending; /* terms added since the last carry propagation */
} nfo_xsum;

static void xsum_carry(nfo_xsum* a) {
  for (int i = 0; i + 1 < NFO_XDIG; ++i) {
    a->d[i + 1] += a->d[i] >> 32;
    a->d[i] &= 0xffffffffu;
  }
  a->pending = 0;
}

/* a += v * 2^p (v < 2^48, 0 <= p <= 506). */
static void xsum_add(nfo_xsum* a, uint64_t v, int p) {
  unsigned __int128 t = (unsigned __int128)v << (p % 32); /* < 2^80 */
  int i = p / 32;
  a->d[i] += (uint64_t)(t & 0xffffffffu);
  a->d[i + 1] += (uint64_t)((t >> 32) & 0xffffffffu);
  a->d[i + 2] += (uint64_t)(t >> 64);
  if (++a->pending == (1u << 31)) xsum_carry(a);
}

static int xsum_bit(const nfo_xsum* a, int i) {
  return (int)((a->d[i / 32] >> (i % 32)) & 1u);
}

/* The integer a times 2^unit_exp, rounded once to FP64, to nearest with ties
 * to even.  The results here are far inside FP64's normal range. */
static double xsum_round(nfo_xsum* a, int unit_exp) {
  xsum_carry(a);
  int top = -1; /* index of the highest set bit */
  for (int i = 32 * NFO_XDIG - 1; i >= 0; --i)
    if (xsum_bit(a, i)) {
      top = i;
      break;
    }
  if (top < 0) return 0.0;
  int low = top - 52; /* lowest bit kept in a 53-bit significand */
  if (low < 0) low = 0;
  uint64_t m = 0;
  for (int i = top; i >= low; --i) m = (m << 1) | (uint64_t)xsum_bit(a, i);
  if (low > 0) {
    int half = xsum_bit(a, low - 1); /* the first bit dropped */
    int below = 0;                   /* any later bit dropped */
    for (int i = low - 2; i >= 0; --i) below |= xsum_bit(a, i);
    if (half && (below || (m & 1u))) m += 1; /* may carry to 2^53: still exact */
  }
  return ldexp((double)m, low + unit_exp);
}

void nfo_health(const float* g, int64_t stride, int32_t W, int64_t n,
                const uint64_t* mask, nfo_stats* stats) {
  for (int32_t w = 0; w < W; ++w) {
    const float* row = g + (int64_t)w * stride;
    nfo_xsum sabs, ssq;
    memset(&sabs, 0, sizeof sabs);
    memset(&ssq, 0, sizeof ssq);
    int abs_nan = 0, abs_inf = 0, sq_nan = 0, sq_inf = 0;
    stats[w].nonfinite = 0;
    for (int64_t i = 0; i < n; ++i) {
      float x = row[i];
      int elig = mask_bit(mask, i);
      if (is_nonfinite(x)) {
        stats[w].nonfinite += 1;
        int nan = x != x;
        sq_nan |= nan;
        sq_inf |= !nan;
        if (elig) {
          abs_nan |= nan;
          abs_inf |= !nan;
        }
        continue;
      }
      uint32_t u;
      memcpy(&u, &x, sizeof u);
      uint32_t e = (u >> 23) & 0xffu;
      uint64_t m = (u & 0x7fffffu) | (e ? 0x800000u : 0u);
      int p = (int)(e ? e : 1) - 1; /* |x| = m * 2^p units of 2^-149 */
      xsum_add(&ssq, m * m, 2 * p); /* x*x = m*m * 2^2p units of 2^-298 */
      if (elig) xsum_add(&sabs, m, p);
    }
    stats[w].sum_abs_elig = abs_nan ? NAN : abs_inf ? INFINITY : xsum_round(&sabs, -149);
    stats[w].sum_sq = sq_nan ? NAN : sq_inf ? INFINITY : xsum_round(&ssq, -298);
  }
}

/* ---- a5 part 1: bucket scale (§5.2, R5) --------------------------------- */
float nfo_scale(const nfo_stats* stats, int32_t W, int64_t n_eligible) {
  if (n_eligible <= 0) return 0.0f;
  double acc = 0.0;
  for (int32_t w = 0; w < W; ++w)
    acc += stats[w].sum_abs_elig / (double)n_eligible;
  return (float)(acc / (double)W);
}

/* ---- a5 part 2: reasons, route and modeled bytes (§3.2, §6.4, R9-R14) --- */
void nfo_decide(const nfo_stats* stats, int32_t W, int64_t n,
                int64_t n_eligible, const nfo_policy* p, nfo_decision* d) {
  uint32_t r = 0;
  if (!p->admitted) r |= NFO_R_NOT_ADMITTED;
  if (n_eligible == 0) r |= NFO_R_NO_ELIGIBLE;
  if (p->veto) r |= NFO_R_VETO;
  if (!p->guard_ok) r |= NFO_R_GUARD;

  uint64_t nonfinite = 0;
  for (int32_t w = 0; w < W; ++w) nonfinite += stats[w].nonfinite;
  if (nonfinite > 0) r |= NFO_R_NONFINITE;

  if (n_eligible > 0)
    for (int32_t w = 0; w < W; ++w)
      if (stats[w].sum_abs_elig == 0.0) r |= NFO_R_ZERO_WORKER;

  /* R12: lower median of the finite sums of squares, by insertion sort. */
  double fin[256];
  int k = 0;
  for (int32_t w = 0; w < W; ++w) {
    double v = stats[w].sum_sq;
    if (!isfinite(v)) continue;
    int j = k++;
    while (j > 0 && fin[j - 1] > v) {
      fin[j] = fin[j - 1];
      --j;
    }
    fin[j] = v;
  }
  if (k >= 2) {
    double m = fin[(k - 1) / 2];
    double thr = (p->kappa * p->kappa) * m;
    for (int i = 0; i < k; ++i)
      if (fin[i] > thr) r |= NFO_R_NORM_SPIKE;
  }

  int32_t route;
  if (r & (NFO_R_NOT_ADMITTED | NFO_R_NO_ELIGIBLE)) {
    route = NFO_ROUTE_P;
  } else if (p->force_lowbit) {
    route = NFO_ROUTE_L;
    r |= NFO_R_FORCED;
  } else if (r & (NFO_R_VETO | NFO_R_GUARD | NFO_R_NONFINITE |
                  NFO_R_ZERO_WORKER | NFO_R_NORM_SPIKE)) {
    route = NFO_ROUTE_F;
  } else {
    route = NFO_ROUTE_L;
  }

  d->route = route;
  d->reasons = r;
  d->scale = nfo_scale(stats, W, n_eligible);
  d->n_eligible = n_eligible;
  d->bytes_fp32 = 4.0 * (double)n;
  if (route == NFO_ROUTE_L)  /* one bit (R14) or two planes (R21) per element */
    d->bytes_route = (p->format == NFO_FORMAT_TERNARY ? 2.0 : 1.0) *
                         (double)n_eligible / 8.0 + 4.0 +
                     4.0 * (double)(n - n_eligible);
  else
    d->bytes_route = 4.0 * (double)n;
}

/* ---- a3: write-side sign payload (§5.2, §6.1, R2, R3) ------------------- */
void nfo_pack(const float* g, int64_t stride, int32_t W, int64_t n,
              const uint64_t* mask, uint64_t* bits, int64_t bits_stride) {
  int64_t nwords = (n + 63) / 64;
  for (int32_t w = 0; w < W; ++w) {
    const float* row = g + (int64_t)w * stride;
    uint64_t* brow = bits + (int64_t)w * bits_stride;
    for (int64_t k = 0; k < nwords; ++k) brow[k] = 0;
    for (int64_t i = 0; i < n; ++i)
      if (mask_bit(mask, i) && row[i] > 0.0f)
        brow[i / 64] |= (uint64_t)1 << (i % 64);
  }
}

/* ---- a6 part 1: per-coordinate sign counts (§6.1, R4) ------------------- */
void nfo_counts(const uint64_t* bits, int64_t bits_stride, int32_t W,
                int64_t n, uint8_t* counts) {
  for (int64_t i = 0; i < n; ++i) {
    int c = 0;
    for (int32_t w = 0; w < W; ++w)
      c += (int)((bits[(int64_t)w * bits_stride + i / 64] >> (i % 64)) & 1u);
    counts[i] = (uint8_t)c;
  }
}

/* ---- a4 / a7: full-precision path (§2.1, §6.1 FP32 reference, R7) ------- */
void nfo_fp32_path(const float* g, int64_t stride, int32_t W, int64_t n,
                   int32_t op, float* y) {
  for (int64_t i = 0; i < n; ++i) {
    float s = g[i];
    for (int32_t w = 1; w < W; ++w) s = s + g[(int64_t)w * stride + i];
    if (op == NFO_OP_MEAN) s = s / (float)W;
    y[i] = s;
  }
}

/* ---- a6 part 2: decode table (§5.2, R6) --------------------------------- */
void nfo_decode_table(int32_t W, int32_t mode, float* q) {
  for (int32_t c = 0; c <= W; ++c) {
    int32_t margin = 2 * c - W;
    if (mode == NFO_DECODE_MAJORITY)
      q[c] = margin > 0 ? 1.0f : (margin < 0 ? -1.0f : 0.0f);
    else
      q[c] = (float)margin / (float)W;
  }
}

/* ---- output assembly (§3.3 step 7, §5.2 write-back, R6) ----------------- */
void nfo_output(const uint64_t* mask, int64_t n, const uint8_t* counts,
                const float* y, const float* q, float scale, int32_t route,
                float* out) {
  for (int64_t i = 0; i < n; ++i) {
    if (route == NFO_ROUTE_L && mask_bit(mask, i))
      out[i] = scale * q[counts[i]];
    else
      out[i] = y[i];
  }
}

/* ---- the whole bucket (§3.3 steps 3-7) ---------------------------------- */
int nfo_reduce_bucket(const float* g, int64_t stride, int32_t W, int64_t n,
                      const uint64_t* mask, const nfo_policy* p,
                      uint64_t* bits, int64_t bits_stride, uint8_t* counts,
                      float* out, nfo_stats* stats, nfo_decision* d) {
  if (W < 1 || W > 255 || n < 0 || stride < n || bits_stride < (n + 63) / 64 ||
      p->format != NFO_FORMAT_BINARY)
    return -1;
  int64_t n_eligible = nfo_count_eligible(mask, n);          /* step 3 */
  nfo_health(g, stride, W, n, mask, stats);
  nfo_decide(stats, W, n, n_eligible, p, d);                 /* steps 4, 6 */
  nfo_pack(g, stride, W, n, mask, bits, bits_stride);        /* step 5 */
  nfo_counts(bits, bits_stride, W, n, counts);               /* step 7 */
  float q[256];
  nfo_decode_table(W, p->decode_mode, q);
  /* The FP32 path is needed at every position: at routed positions for any
   * route, and at eligible positions when the route is F or P.  It is taken
   * in ascending chunks whose starts are multiples of 64. */
  for (int64_t i0 = 0; i0 < n; i0 += 4096) {
    int64_t m = n - i0 < 4096 ? n - i0 : 4096;
    float y[4096];
    nfo_fp32_path(g + i0, stride, W, m, p->fp32_op, y);
    nfo_output(mask + i0 / 64, m, counts + i0, y, q, d->scale, d->route,
               out + i0);
  }
  return 0;
}

/* ---- G-Ternary: gate threshold (§2.2, R18) ------------------------------ */
float nfo_ternary_threshold(const nfo_stats* st, int64_t n_eligible, float tau) {
  if (n_eligible <= 0) return 0.0f;
  float mean_abs = (float)(st->sum_abs_elig / (double)n_eligible);
  return tau * mean_abs;
}

/* ---- G-Ternary: write-side payload (§2.2, R18, R19) --------------------- */
void nfo_pack_ternary(const float* g, int64_t stride, int32_t W, int64_t n,
                      const uint64_t* mask, const float* theta, uint64_t* pos,
                      uint64_t* neg, int64_t bits_stride) {
  int64_t nwords = (n + 63) / 64;
  for (int32_t w = 0; w < W; ++w) {
    const float* row = g + (int64_t)w * stride;
    uint64_t* prow = pos + (int64_t)w * bits_stride;
    uint64_t* nrow = neg + (int64_t)w * bits_stride;
    for (int64_t k = 0; k < nwords; ++k) {
      prow[k] = 0;
      nrow[k] = 0;
    }
    for (int64_t i = 0; i < n; ++i) {
      if (!mask_bit(mask, i)) continue;
      float x = row[i];
      if (fabsf(x) < theta[w]) continue;  /* gated to 0 */
      if (x > 0.0f) prow[i / 64] |= (uint64_t)1 << (i % 64);
      if (x < 0.0f) nrow[i / 64] |= (uint64_t)1 << (i % 64);
    }
  }
}

/* ---- G-Ternary: decode table over the vote difference (§5.2, R20) ------- */
void nfo_ternary_decode_table(int32_t W, int32_t mode, float* q) {
  for (int32_t d = -W; d <= W; ++d) {
    if (mode == NFO_DECODE_MAJORITY)
      q[d + W] = d > 0 ? 1.0f : (d < 0 ? -1.0f : 0.0f);
    else
      q[d + W] = (float)d / (float)W;
  }
}

void nfo_ternary_output(const uint64_t* mask, int64_t n, const uint8_t* cpos,
                        const uint8_t* cneg, const float* y, const float* q,
                        float scale, int32_t W, int32_t route, float* out) {
  for (int64_t i = 0; i < n; ++i) {
    if (route == NFO_ROUTE_L && mask_bit(mask, i))
      out[i] = scale * q[(int32_t)cpos[i] - (int32_t)cneg[i] + W];
    else
      out[i] = y[i];
  }
}

/* ---- the whole bucket, G-Ternary payload (§3.3 steps 3-7, R18-R21) ------ */
int nfo_reduce_bucket_ternary(const float* g, int64_t stride, int32_t W,
                              int64_t n, const uint64_t* mask,
                              const nfo_policy* p, uint64_t* pos, uint64_t* neg,
                              int64_t bits_stride, uint8_t* cpos, uint8_t* cneg,
                              float* out, nfo_stats* stats, nfo_decision* d) {
  if (W < 1 || W > 255 || n < 0 || stride < n || bits_stride < (n + 63) / 64 ||
      p->format != NFO_FORMAT_TERNARY || !(p->tau >= 0.0f))
    return -1;
  int64_t n_eligible = nfo_count_eligible(mask, n);          /* step 3 */
  nfo_health(g, stride, W, n, mask, stats);
  nfo_decide(stats, W, n, n_eligible, p, d);                 /* steps 4, 6 */
  float theta[256];
  for (int32_t w = 0; w < W; ++w)
    theta[w] = nfo_ternary_threshold(&stats[w], n_eligible, p->tau);
  nfo_pack_ternary(g, stride, W, n, mask, theta, pos, neg, bits_stride); /* 5 */
  nfo_counts(pos, bits_stride, W, n, cpos);                  /* step 7 */
  nfo_counts(neg, bits_stride, W, n, cneg);
  float q[511];
  nfo_ternary_decode_table(W, p->decode_mode, q);
  for (int64_t i0 = 0; i0 < n; i0 += 4096) {
    int64_t m = n - i0 < 4096 ? n - i0 : 4096;
    float y[4096];
    nfo_fp32_path(g + i0, stride, W, m, p->fp32_op, y);
    nfo_ternary_output(mask + i0 / 64, m, cpos + i0, cneg + i0, y, q, d->scale,
                       W, d->route, out + i0);
  }
  return 0;
}

/* ---- compacted payload (R30) --------------------------------------------- */
void nfo_pack_compact(const float* g, int64_t stride, int32_t W, int64_t n,
                      const uint64_t* mask, uint64_t* cbits, int64_t cstride) {
  int64_t n_eligible = nfo_count_eligible(mask, n);
  int64_t cwords = (n_eligible + 63) / 64;
  for (int32_t w = 0; w < W; ++w) {
    const float* row = g + (int64_t)w * stride;
    uint64_t* crow = cbits + (int64_t)w * cstride;
    for (int64_t k = 0; k < cwords; ++k) crow[k] = 0;
    int64_t r = 0; /* rank of the next eligible element */
    for (int64_t i = 0; i < n; ++i) {
      if (!mask_bit(mask, i)) continue;
      if (row[i] > 0.0f) crow[r / 64] |= (uint64_t)1 << (r % 64);
      ++r;
    }
  }
}

/* ---- per-slice scales (R29, R31) ----------------------------------------- */
void nfo_slice_scales(const float* g, int64_t stride, int32_t W,
                      const int64_t* off, const int64_t* len, int64_t S,
                      double* sums /* [S][W] */, float* scales /* [S] */) {
  for (int64_t s = 0; s < S; ++s) {
    double acc = 0.0;
    for (int32_t w = 0; w < W; ++w) {
      const float* row = g + (int64_t)w * stride + off[s];
      double t = 0.0;
      for (int64_t j = 0; j < len[s]; ++j) t += fabs((double)row[j]);
      sums[s * W + w] = t;
      acc += t / (double)len[s];
    }
    scales[s] = (float)(acc / (double)W);
  }
}

/* ---- sliced decode (R32) ------------------------------------------------- */
void nfo_sliced_output(const uint64_t* mask, int64_t n, const uint8_t* counts,
                       const float* y, const float* q, const int64_t* off,
                       const int64_t* len, int64_t S, const float* scales,
                       int32_t route, float* out) {
  int64_t s = 0;
  for (int64_t i = 0; i < n; ++i) {
    if (route == NFO_ROUTE_L && mask_bit(mask, i)) {
      while (s < S && i >= off[s] + len[s]) ++s; /* the slice holding i */
      out[i] = scales[s] * q[counts[i]];
    } else {
      out[i] = y[i];
    }
  }
}
