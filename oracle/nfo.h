/*
 * nfo.h - reference oracle for the NEURON-Fabric bucket reducer.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, single-threaded CPU
 * statement of what the bucket reducer computes.  Only the test suite, the
 * smoke entry point and the benchmark's CPU-baseline leg may load it.  It
 * shares no code, header, table or helper with the GPU library; the two are
 * compared element by element.
 *
 * Sources (NEURON-Fabric, arXiv 2606.25759):
 *   - §2.2 (Low-bit gradient aggregation): G-Binary is a one-bit sign-count
 *     route; workers send a compact direction payload and the reducer
 *     returns an aggregate direction.  G-Ternary adds a zero-gating rule
 *     that suppresses selected entries before aggregation.
 *   - §3.2 (Calibration-to-runtime interface): route states L / F / P and the
 *     modeled gradient-communication traffic ratio (MGTR) equation.
 *   - §3.3 (Runtime execution), steps 3-7: classify bucket contents, encode
 *     admitted eligible slices, leave sensitive slices on FP32, aggregate,
 *     write back.
 *   - §5.1 (Binding schema): per-parameter eligibility; an absent parameter
 *     is FP32-only.
 *   - §5.2 (DDP hook prototype semantics): a mean-absolute scale is recorded
 *     per eligible slice, gradients become positive-sign indicators, the
 *     indicators are summed over workers, a vote is applied and the scaled
 *     aggregate direction is written back.
 *   - §6.1 (Reducer model): per-coordinate sign counts over bit-packed
 *     updates.
 *   - §6.4 (Endpoint-capacity guard): the guard outcome is a comparison the
 *     caller supplies; a rejected bucket stays on FP32.
 *
 * Readings where the paper is silent are fixed in nfo.cpp and numbered
 * R1..R21; each function names the readings it applies.
 *
 * Layouts: gradients are W rows of FP32, row w starting at g + w*stride.
 * Masks and sign bitmaps are little-endian uint64 words, LSB-first: bit j of
 * word k is element 64k+j.  Bits at or beyond n are zero.
 */
#ifndef NFO_H
#define NFO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Route states of §3.2: low-bit, FP32 fallback of an admitted route, plain FP32. */
enum { NFO_ROUTE_L = 0, NFO_ROUTE_F = 1, NFO_ROUTE_P = 2 };

/* Reason bits (R9).  Every bit is always evaluated. */
enum {
  NFO_R_NOT_ADMITTED = 1,
  NFO_R_NO_ELIGIBLE = 2,
  NFO_R_VETO = 4,
  NFO_R_GUARD = 8,
  NFO_R_NONFINITE = 16,
  NFO_R_ZERO_WORKER = 32,
  NFO_R_NORM_SPIKE = 64,
  NFO_R_FORCED = 128
};

enum { NFO_DECODE_SOFT = 0, NFO_DECODE_MAJORITY = 1 };
enum { NFO_OP_SUM = 0, NFO_OP_MEAN = 1 };
/* Payload formats of §2.2: G-Binary (sign counts), G-Ternary (zero gating). */
enum { NFO_FORMAT_BINARY = 0, NFO_FORMAT_TERNARY = 1 };

typedef struct {
  uint64_t nonfinite;   /* count of non-finite values of worker w over all n   */
  double sum_abs_elig;  /* sum of |g| over eligible elements: exact, rounded
                           once to FP64 (R8)                                  */
  double sum_sq;        /* sum of g*g over all n elements: exact, rounded once
                           to FP64 (R8)                                       */
} nfo_stats;

typedef struct {
  int admitted;      /* Commander admission (§4.2)                     */
  int veto;          /* Supervisor veto (§4.3)                         */
  int guard_ok;      /* endpoint-capacity guard outcome (§6.4)         */
  int force_lowbit;  /* guard disabled, low-bit forced (§6.4, panel C) */
  int decode_mode;   /* NFO_DECODE_SOFT or NFO_DECODE_MAJORITY         */
  int fp32_op;       /* NFO_OP_SUM or NFO_OP_MEAN                      */
  double kappa;      /* norm-spike ratio on L2 norms (R12)             */
  int format;        /* NFO_FORMAT_BINARY or NFO_FORMAT_TERNARY        */
  float tau;         /* G-Ternary gate, in units of the worker's mean
                        |g| over eligible elements (R18)              */
} nfo_policy;

typedef struct {
  int32_t route;       /* NFO_ROUTE_*                                  */
  uint32_t reasons;    /* NFO_R_* bitmask                              */
  float scale;         /* bucket scale (R5)                            */
  int64_t n_eligible;  /* popcount of the mask over [0, n)             */
  double bytes_route;  /* modeled payload bytes per worker (§3.2)      */
  double bytes_fp32;   /* matched FP32 payload bytes per worker (§3.2) */
} nfo_decision;

/* Binding -> mask (§5.1).  Returns 0, or -1 on a segment outside [0, n). */
int nfo_mask_from_segments(const int64_t* off, const int64_t* len,
                           const uint8_t* eligible, int64_t nseg, int64_t n,
                           uint64_t* mask);
int64_t nfo_count_eligible(const uint64_t* mask, int64_t n);

/* Health (R8): non-finite counts and the two exact sums of each worker. */
void nfo_health(const float* g, int64_t stride, int32_t W, int64_t n,
                const uint64_t* mask, nfo_stats* stats);

float nfo_scale(const nfo_stats* stats, int32_t W, int64_t n_eligible);
void nfo_decide(const nfo_stats* stats, int32_t W, int64_t n,
                int64_t n_eligible, const nfo_policy* p, nfo_decision* d);

void nfo_pack(const float* g, int64_t stride, int32_t W, int64_t n,
              const uint64_t* mask, uint64_t* bits, int64_t bits_stride);
void nfo_counts(const uint64_t* bits, int64_t bits_stride, int32_t W,
                int64_t n, uint8_t* counts);
void nfo_fp32_path(const float* g, int64_t stride, int32_t W, int64_t n,
                   int32_t op, float* y);
void nfo_decode_table(int32_t W, int32_t mode, float* q /* W+1 */);
void nfo_output(const uint64_t* mask, int64_t n, const uint8_t* counts,
                const float* y, const float* q, float scale, int32_t route,
                float* out);

/* The whole bucket, steps in the order of §3.3.  bits, counts, out and
 * stats are always written (bits and counts are computed for every route).
 * Returns 0, or -1 on invalid arguments or a format other than binary. */
int nfo_reduce_bucket(const float* g, int64_t stride, int32_t W, int64_t n,
                      const uint64_t* mask, const nfo_policy* p,
                      uint64_t* bits, int64_t bits_stride, uint8_t* counts,
                      float* out, nfo_stats* stats, nfo_decision* d);

/* ---- G-Ternary (§2.2 zero gating; readings R18-R21) ---------------------
 * A worker's gate threshold from its statistics: fl32(tau * fl32(S / n_E))
 * with S its |g| sum over eligible elements; 0 when n_E = 0 (R18). */
float nfo_ternary_threshold(const nfo_stats* st, int64_t n_eligible, float tau);
/* Two planes per worker (R19): pos bit = eligible, not gated, g > 0; neg
 * bit = eligible, not gated, g < 0; gated means |g| < theta[w]. */
void nfo_pack_ternary(const float* g, int64_t stride, int32_t W, int64_t n,
                      const uint64_t* mask, const float* theta, uint64_t* pos,
                      uint64_t* neg, int64_t bits_stride);
/* q[d + W] for d = c+ - c- in [-W, W] (R20). */
void nfo_ternary_decode_table(int32_t W, int32_t mode, float* q /* 2W+1 */);
void nfo_ternary_output(const uint64_t* mask, int64_t n, const uint8_t* cpos,
                        const uint8_t* cneg, const float* y, const float* q,
                        float scale, int32_t W, int32_t route, float* out);
/* The whole bucket with the G-Ternary payload: pos and neg planes, c+ and c-
 * counts, out, stats and the decision (the MGTR bytes of R21).  Returns 0,
 * or -1 on invalid arguments or a format other than ternary. */
int nfo_reduce_bucket_ternary(const float* g, int64_t stride, int32_t W,
                              int64_t n, const uint64_t* mask,
                              const nfo_policy* p, uint64_t* pos, uint64_t* neg,
                              int64_t bits_stride, uint8_t* cpos, uint8_t* cneg,
                              float* out, nfo_stats* stats, nfo_decision* d);

/* Per-slice scales and the compacted payload (R29-R33). */
void nfo_pack_compact(const float* g, int64_t stride, int32_t W, int64_t n,
                      const uint64_t* mask, uint64_t* cbits, int64_t cstride);
void nfo_slice_scales(const float* g, int64_t stride, int32_t W,
                      const int64_t* off, const int64_t* len, int64_t S,
                      double* sums, float* scales);
void nfo_sliced_output(const uint64_t* mask, int64_t n, const uint8_t* counts,
                       const float* y, const float* q, const int64_t* off,
                       const int64_t* len, int64_t S, const float* scales,
                       int32_t route, float* out);

#ifdef __cplusplus
}
#endif
#endif
