/*
 * nf.h - C ABI of the NEURON-Fabric bucket reducer for AMD MI355X (gfx950).
 *
 * The reducer is the data-parallel hot path of controlled low-bit gradient
 * aggregation (NEURON-Fabric, arXiv 2606.25759).  It takes the FP32 gradient
 * buckets of W data-parallel workers and the bucket's per-element
 * eligibility mask, and
 *   - packs the signs of the low-bit-eligible elements (write side, §3.3
 *     step 5, §5.2),
 *   - sums the FP32-routed elements in full precision (§2.1, §3.3 step 5),
 *   - computes per-worker health statistics and the bucket's route
 *     decision L / F / P with its modeled traffic (§3.2, §6.4),
 *   - counts the packed signs per coordinate and decodes the scaled aggregate
 *     direction (read side, §3.3 step 7, §5.2, §6.1), or, on fallback, sums
 *     the eligible elements in FP32 as well.
 *
 * The W workers are W rows of one device buffer: row w of a bucket starts at
 * grads + w * worker_stride.
 *
 * Conventions shared by every function:
 *   - Every function returns nf_status.  On an error nothing is launched and
 *     nf_last_error() (thread-local) describes the failing argument.
 *   - Pointers named *_host are host memory.  Every other pointer is device
 *     memory owned by the caller; the library never allocates.  Scratch
 *     space comes from a caller-provided workspace `ws` of at least the size
 *     the matching nf_*workspace_bytes function returns.
 *   - Device work is enqueued asynchronously on `stream` (a hipStream_t passed
 *     as void*; NULL is the null stream).  Results are valid after the stream
 *     is synchronised.  A launch failure returns NF_ERR_HIP.
 *   - Requirements checked before any launch (NF_ERR_INVALID_ARG unless
 *     stated): 1 <= W <= 255 (counts are uint8); n >= 0;
 *     worker_stride >= n; grads 16-byte aligned and worker_stride a multiple
 *     of 4 (NF_ERR_ALIGNMENT); mask and bits 8-byte aligned, out 4-byte
 *     aligned (NF_ERR_ALIGNMENT); bits_stride_words >= ceil(n / 64).  Inputs
 *     and outputs must not overlap (not checked).
 *   - Layouts: masks and sign bitmaps are little-endian uint64 words,
 *     LSB-first: bit j of word k is element 64k + j.  Mask bits at or past n
 *     are ignored.  One mask is shared by all W workers (the binding is per
 *     model, §5.1).  Bitmap row w starts at bits + w * bits_stride_words.
 *   - Floating point: FP32 sums add workers in order w = 0..W-1 in FP32
 *     without contraction, so they are bit-reproducible.  Per-worker health
 *     sums are FP64 in a fixed order (deterministic, within 1e-12 relative
 *     of the exact sum); where a pass builds no sign payload
 *     (nf_bucket_health, the G-Ternary route, and routes the policy fixes
 *     before reading) each worker's sum of |g| over eligible elements is
 *     the exact sum rounded once to FP64 (ties to even), because the
 *     G-Ternary gate derives from it (§2.2).  No floating-point atomics are
 *     used, so two calls on the same inputs give bitwise identical results.
 *   - Calls on different streams with different workspaces may run
 *     concurrently.  The library keeps no mutable state besides the
 *     thread-local error string and the thread-local profiling events of
 *     nf_set_phase_events.
 */
#ifndef NF_H
#define NF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define NF_ABI_VERSION 2

typedef enum {
  NF_OK = 0,
  NF_ERR_INVALID_ARG = 1,
  NF_ERR_ALIGNMENT = 2,
  NF_ERR_UNSUPPORTED = 3,
  NF_ERR_HIP = 4,
  NF_ERR_WORKSPACE = 5
} nf_status;

/* Route states (§3.2): low-bit; FP32 fallback of an admitted route; plain FP32. */
enum { NF_ROUTE_LOWBIT = 0, NF_ROUTE_FALLBACK = 1, NF_ROUTE_PLAIN = 2 };

/* Reason bits of a route decision; every bit is evaluated on every call. */
enum {
  NF_REASON_NOT_ADMITTED = 1,  /* policy.admitted == 0 (Commander, §4.2)      */
  NF_REASON_NO_ELIGIBLE = 2,   /* no mask bit set in [0, n) (§5.1)            */
  NF_REASON_VETO = 4,          /* policy.veto != 0 (Supervisor, §4.3)         */
  NF_REASON_GUARD = 8,         /* policy.guard_ok == 0 (endpoint guard, §6.4) */
  NF_REASON_NONFINITE = 16,    /* some worker holds a NaN or an infinity      */
  NF_REASON_ZERO_WORKER = 32,  /* n_E > 0 and a worker's eligible |g| sum is 0 */
  NF_REASON_NORM_SPIKE = 64,   /* a finite sum g^2 > kappa^2 * lower median    */
  NF_REASON_FORCED = 128       /* low-bit taken because force_lowbit was set  */
};

enum { NF_DECODE_SOFT = 0, NF_DECODE_MAJORITY = 1 };
enum { NF_FP32_SUM = 0, NF_FP32_MEAN = 1 };
enum { NF_SEL_ROUTED = 0, NF_SEL_ELIGIBLE = 1, NF_SEL_ALL = 2 };
/* Low-bit payload formats (§2.2): G-Binary sign counts; G-Ternary adds
 * write-side zero gating and a second (negative) plane. */
enum { NF_FORMAT_BINARY = 0, NF_FORMAT_TERNARY = 1 };

/* Per-worker health of one bucket. */
typedef struct {
  uint64_t nonfinite;   /* count of NaN / +-Inf values over all n elements    */
  double sum_abs_elig;  /* sum of |g| over eligible elements (FP64)           */
  double sum_sq;        /* sum of g*g over all n elements (FP64)              */
} nf_worker_stats;

/* Controller and guard inputs of a route decision. */
typedef struct {
  int32_t admitted;      /* Commander has admitted the low-bit mode (§4.2)     */
  int32_t veto;          /* Supervisor veto is active (§4.3)                   */
  int32_t guard_ok;      /* endpoint-capacity guard admits low-bit (§6.4)      */
  int32_t force_lowbit;  /* guard disabled: take low-bit despite F reasons     */
  int32_t decode_mode;   /* NF_DECODE_SOFT (default) or NF_DECODE_MAJORITY     */
  int32_t fp32_op;       /* NF_FP32_SUM (default) or NF_FP32_MEAN              */
  double kappa;          /* norm-spike ratio on L2 norms, > 0 (default 4.0)    */
  int32_t format;        /* NF_FORMAT_BINARY (default) or NF_FORMAT_TERNARY    */
  float tau;             /* G-Ternary gate in units of each worker's mean |g|
                            over eligible elements, finite and >= 0 (default
                            0.5; see nf_ternary_threshold)                     */
} nf_route_policy;

/* Route decision of one bucket (40 bytes). */
typedef struct {
  int32_t route;        /* NF_ROUTE_*                                          */
  uint32_t reasons;     /* NF_REASON_* bitmask                                 */
  float scale;          /* mean over workers of the mean |g| over eligible
                           elements, rounded once to FP32; 0 if n_E == 0      */
  uint32_t resummed;    /* workers whose |g| sum was re-summed exactly from
                           the gradients because its carried error bound
                           could not certify the rounding (diagnostic; 0
                           from nf_route_decide and with sign words)          */
  int64_t n_eligible;   /* n_E: mask bits set in [0, n)                        */
  double bytes_route;   /* modeled payload bytes per worker of this route:
                           b*n_E/8 + 4 + 4(n - n_E) for L with b = 1 bit per
                           element (binary) or 2 (ternary's two planes);
                           4n for F and P                                      */
  double bytes_fp32;    /* matched FP32 payload bytes per worker: 4n (§3.2)    */
} nf_route_decision;

int nf_abi_version(void);
const char* nf_last_error(void);

/*
 * Binding -> eligibility mask (§5.1: per-parameter eligibility; an element
 * not covered by an eligible segment is FP32).  Host helper: segment s covers
 * [off_host[s], off_host[s] + len_host[s]) and is eligible when
 * eligible_host[s] != 0.  Writes ceil(n/64) words to mask_host (padding bits
 * zero).  NF_ERR_INVALID_ARG if a segment leaves [0, n).
 */
nf_status nf_mask_from_segments(const int64_t* off_host, const int64_t* len_host,
                                const uint8_t* eligible_host, int64_t nseg, int64_t n,
                                uint64_t* mask_host);

/* Workspace bytes for one bucket of n elements (nf_bucket_health,
 * nf_pack_signs, nf_route_bucket). */
size_t nf_workspace_bytes(int32_t W, int64_t n);

/*
 * Per-worker health of one bucket (write-side statistics behind the fallback
 * decision; the paper's Supervisor and guard act on health, §4.3, §6.4).
 * Writes stats[0..W) (device).  Reads 4*W*n bytes once.
 */
nf_status nf_bucket_health(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                           const uint64_t* mask, nf_worker_stats* stats, void* ws,
                           size_t ws_bytes, void* stream);

/*
 * Write-side sign payload (§3.3 step 5, §5.2 positive-sign indicators, §6.1
 * bit-packed updates): bit j of bits[w][k] = mask(64k+j) && g_w[64k+j] > 0
 * (+0, -0 and NaN give 0).  Writes all ceil(n/64) words of each of the W rows,
 * with zero padding.  When stats is not NULL the same single read also
 * produces the per-worker health of nf_bucket_health.
 */
nf_status nf_pack_signs(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                        const uint64_t* mask, uint64_t* bits, int64_t bits_stride_words,
                        nf_worker_stats* stats, void* ws, size_t ws_bytes, void* stream);

/*
 * Full-precision path (§2.1 sum or average; §6.1 FP32 reference path):
 * out[i] = g_0[i] + g_1[i] + ... + g_{W-1}[i] in FP32, workers in order;
 * NF_FP32_MEAN divides the sum by W (IEEE division).  Written only at the
 * selected positions: NF_SEL_ROUTED mask = 0, NF_SEL_ELIGIBLE mask = 1,
 * NF_SEL_ALL every position (mask may then be NULL).  No workspace.
 */
nf_status nf_fp32_reduce(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                         const uint64_t* mask, int32_t select, int32_t fp32_op, float* out,
                         void* stream);

/*
 * Read side of the sign-count route (§3.3 step 7, §5.2 vote and scaled
 * write-back, §6.1 per-coordinate counts): c_i = sum_w bit_w(i) in [0, W];
 * when counts is not NULL it receives all n counts.  When out is not NULL,
 * out[i] = fl32(scale * q[c_i]) at positions with mask = 1 (others untouched),
 * with scale = *scale_dev (device, one float) and
 * q[c] = fl32((2c - W) / W) (NF_DECODE_SOFT) or sign(2c - W) with a tie giving
 * 0 (NF_DECODE_MAJORITY).  No workspace.
 */
nf_status nf_signcount_reduce(const uint64_t* bits, int64_t bits_stride_words, int32_t W,
                              int64_t n, const uint64_t* mask, const float* scale_dev,
                              int32_t decode_mode, uint8_t* counts, float* out, void* stream);

/*
 * Node-local counting of the hierarchical sign-count reducer (§6.1: counting
 * at the node, then an exchange of partial counts between nodes, then the
 * aggregate's return; §6.3 contrasts this with stock packed-sign transport,
 * where every worker counts every stream itself).  The W rows of bits form
 * G = W / P groups of P consecutive workers, a group standing for one node's
 * P GPUs.  partial[g][i] = the number of rows of group g whose bit i is set,
 * in [0, P]: G rows of n bytes, row g at partial + g * partial_stride
 * (device).  Requires 1 <= P <= W, W a multiple of P, partial_stride >= n.
 * The sum over g of partial[g][i] is the count c_i of nf_signcount_reduce.
 * No workspace.
 */
nf_status nf_partial_counts(const uint64_t* bits, int64_t bits_stride_words, int32_t W, int32_t P,
                            int64_t n, uint8_t* partial, int64_t partial_stride, void* stream);

/*
 * Partial-count exchange and aggregate return of the hierarchical reducer
 * (§6.1), on one device: c_i = sum of the G rows of partial (row g at
 * partial + g * partial_stride; G divides W), then counts (nullable, n
 * bytes) and out (nullable, at mask = 1) exactly as nf_signcount_reduce with
 * W workers, scale *scale_dev and decode_mode.  partial must be 16-byte
 * aligned and partial_stride a multiple of 16 (NF_ERR_ALIGNMENT).  No
 * workspace.
 */
nf_status nf_partial_count_reduce(const uint8_t* partial, int64_t partial_stride, int32_t G,
                                  int32_t W, int64_t n, const uint64_t* mask,
                                  const float* scale_dev, int32_t decode_mode, uint8_t* counts,
                                  float* out, void* stream);

/*
 * Stock packed-sign baseline (§6.3): after an all-gather of the packed signs,
 * every worker counts all W rows and decodes the aggregate itself.  On one
 * device: `replicas` (1..65535) independent count-and-decode passes of
 * nf_signcount_reduce, replica r writing counts + r * replica_stride
 * (nullable) and out + r * replica_stride (nullable; at mask = 1);
 * replica_stride >= n elements.  Every replica equals nf_signcount_reduce's
 * result.  No workspace.
 */
nf_status nf_stock_signcount(const uint64_t* bits, int64_t bits_stride_words, int32_t W, int64_t n,
                             const uint64_t* mask, const float* scale_dev, int32_t decode_mode,
                             int32_t replicas, uint8_t* counts, float* out, int64_t replica_stride,
                             void* stream);

/* ------------------------------------------------------------------------
 * Per-slice scales and the compacted eligible-only payload.  §5.2 records a
 * mean-absolute scale for the eligible slices and §6.1 counts bit-packed
 * updates; the paper fixes neither the scale's granularity nor the
 * payload's layout.  Here:
 *   - the bucket's eligible slices are S intervals [off[s], off[s] +
 *     len[s]), sorted, disjoint and non-empty (one per eligible parameter
 *     slice of the binding, §5.1); the mask is their union;
 *   - the compacted payload of worker w holds bit r = (g > 0) of the r-th
 *     eligible element in element order, r = 0 .. n_E - 1 (ceil(n_E / 64)
 *     LSB-first words, padding 0): exactly n_E payload bits per worker;
 *   - scale_s = fl32((sum over workers, in order, of S_sw / len[s]) / W),
 *     S_sw the FP64 sum of |g| of worker w over slice s (the bucket scale's
 *     rule on one slice); the decoded value at an eligible element i of
 *     slice s is fl32(scale_s * q[c_i]).
 * ------------------------------------------------------------------------ */

/* Sizes of a slice table (host): n_E = sum of len[s]; segments = the number
 * of statistics segments, sum of ceil(len[s] / 65536). */
nf_status nf_sliced_layout_sizes(const int64_t* len_host, int64_t S, int64_t* n_eligible_host,
                                 int64_t* segments_host);

/*
 * Layout tables of a slice table over n elements (host; built once per
 * binding, like the mask).  Slices outside [0, n), unsorted, overlapping or
 * empty give NF_ERR_INVALID_ARG.  Writes, into caller-allocated host arrays
 * (nw = ceil(n / 64), nwc = ceil(n_E / 64)):
 *   mask_host[nw]       the eligibility mask, the union of the slices
 *   prefix_host[nw + 1] eligible elements before word k (prefix[nw] = n_E)
 *   start_host[nwc]     the word holding compacted rank 64 o
 *   wslice_host[nw]     the slice holding word k's first eligible element
 *                       (S when the word has none)
 *   rstart_host[S + 1]  compacted rank of slice s's first element
 *                       (rstart[S] = n_E)
 *   segp_host[S + 1]    first statistics segment of slice s
 */
nf_status nf_sliced_layout(const int64_t* off_host, const int64_t* len_host, int64_t S, int64_t n,
                           uint64_t* mask_host, uint64_t* prefix_host, int64_t* start_host,
                           int32_t* wslice_host, int64_t* rstart_host, int64_t* segp_host);

/*
 * Compaction of the positional sign payload (rows of nf_pack_signs) into
 * the compacted payload: for each of the W rows, cbits row w (at cbits + w *
 * cbits_stride_words, cbits_stride_words >= ceil(n_E / 64)) receives the
 * bits of the eligible positions in order.  mask, prefix and start: device
 * copies of the layout tables; n_eligible = prefix[nw].  No workspace.
 */
nf_status nf_compact_signs(const uint64_t* bits, int64_t bits_stride_words, int32_t W, int64_t n,
                           const uint64_t* mask, const uint64_t* prefix, const int64_t* start,
                           int64_t n_eligible, uint64_t* cbits, int64_t cbits_stride_words,
                           void* stream);

/* Workspace bytes of nf_slice_scales for W workers and `segments`. */
size_t nf_slice_workspace_bytes(int32_t W, int64_t segments);

/*
 * Per-slice statistics and scales: sums[s * W + w] = S_sw (FP64, in a fixed
 * order: per 65,536-element segment, then the segments in order; within
 * 1e-12 relative of a sequential sum) and scales[s] = scale_s (device
 * arrays).  off, len, segp: device copies of the slice table and of
 * segp_host; grads as for nf_bucket_health (4-byte alignment suffices).
 * Reads the eligible elements once.
 */
nf_status nf_slice_scales(const float* grads, int64_t worker_stride, int32_t W, const int64_t* off,
                          const int64_t* len, const int64_t* segp, int64_t S, int64_t segments,
                          double* sums, float* scales, void* ws, size_t ws_bytes, void* stream);

/*
 * Per-slice statistics and scales as nf_slice_scales computes them (§5.2's
 * mean-absolute scale per eligible slice), without a second read of the
 * gradients: taken from the per-chunk partial statistics that pass 1 leaves
 * in its workspace.  Call it after nf_pack_signs (with or without stats),
 * nf_bucket_health or nf_route_bucket over the same grads, worker_stride,
 * W and n, with a mask that is exactly the union of the slices, on the same
 * stream and with the same workspace ws (ws_bytes >= nf_workspace_bytes(W,
 * n); read only), before anything else writes to it.  Only the parts of
 * the slices in pass-1 chunks that two slices share are read again (at most
 * two chunks per slice).  off, len: device copies of the slice table (S
 * slices, sorted, disjoint, non-empty, within [0, n)).  sums[s * W + w]
 * (FP64; the chunks' partials in a fixed order, within 1e-12 relative of a
 * sequential sum) and scales[s]: device arrays.  S = 0 is a no-op.
 */
nf_status nf_slice_scales_from_pass1(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                                     const int64_t* off, const int64_t* len, int64_t S, double* sums,
                                     float* scales, const void* ws, size_t ws_bytes, void* stream);

/*
 * Read side over the compacted payload (§3.3 step 7 with per-slice scales):
 * counts_c[r] = sum over the W compacted rows of bit r (n_E bytes, in
 * compacted order; required, 4-byte aligned), then, when out is not NULL, out[i] =
 * fl32(scales[s] * q[c]) at every eligible element i (slice s, count c of
 * its rank), other positions untouched; q as nf_signcount_reduce's.  mask,
 * prefix, wslice, rstart: device copies of the layout tables.  No workspace.
 */
nf_status nf_compact_signcount_reduce(const uint64_t* cbits, int64_t cbits_stride_words, int32_t W,
                                      int64_t n, const uint64_t* mask, const uint64_t* prefix,
                                      const int32_t* wslice, const int64_t* rstart, int64_t S,
                                      int64_t n_eligible, const float* scales, int32_t decode_mode,
                                      uint8_t* counts_c, float* out, void* stream);

/*
 * G-Ternary write-side threshold (§2.2's zero gating, applied before
 * aggregation; host, pure function): for each worker w,
 * theta[w] = fl32(tau * fl32(stats[w].sum_abs_elig / n_eligible)), i.e. tau
 * times the worker's mean |g| over eligible elements; 0 when n_eligible = 0.
 */
nf_status nf_ternary_threshold(const nf_worker_stats* stats_host, int32_t W, int64_t n_eligible,
                               float tau, float* theta_host);

/*
 * G-Ternary write-side payload (§2.2, §3.3 step 5): two positional planes
 * per worker in the layout of the sign bitmaps.  Row w (0 <= w < W) is the
 * positive plane, row W + w the negative plane of worker w: bit j of word k
 * is set when element 64k+j is eligible, not gated (|g| < theta[w] gates it
 * to 0, an FP32 comparison) and g > 0 (positive) or g < 0 (negative).  NaN
 * is never gated and never set.  theta_dev: W floats (device), e.g. from
 * nf_ternary_threshold.  bits holds 2W rows of bits_stride_words words; all
 * ceil(n/64) words of each row are written, zero padded.  No workspace.
 */
nf_status nf_pack_ternary(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                          const uint64_t* mask, const float* theta_dev, uint64_t* bits,
                          int64_t bits_stride_words, void* stream);

/*
 * G-Ternary read side (§3.3 step 7, §5.2 vote and scaled write-back):
 * c+_i and c-_i are the per-coordinate counts of the positive rows (0..W-1)
 * and negative rows (W..2W-1) of bits; d_i = c+_i - c-_i.  counts (nullable)
 * receives 2n bytes: c+ in [0, n), c- in [n, 2n).  out (nullable) receives
 * fl32(scale * q[d_i]) at mask = 1 (others untouched) with scale =
 * *scale_dev and q[d] = fl32(d / W) (NF_DECODE_SOFT) or sign(d)
 * (NF_DECODE_MAJORITY).  No workspace.
 */
nf_status nf_ternary_reduce(const uint64_t* bits, int64_t bits_stride_words, int32_t W, int64_t n,
                            const uint64_t* mask, const float* scale_dev, int32_t decode_mode,
                            uint8_t* counts, float* out, void* stream);

/*
 * Route decision from statistics (host, pure function; the rules the device
 * path applies).  Reasons as listed above; route by precedence P (not
 * admitted, or no eligible element) > forced L > F (veto, guard, non-finite,
 * zero worker, norm spike) > L.  The norm-spike rule takes the workers whose
 * sum_sq is finite (at least two), their lower median m (index
 * floor((k-1)/2) in ascending order), and flags sum_sq > (kappa*kappa)*m.
 */
nf_status nf_route_decide(const nf_worker_stats* stats_host, int32_t W, int64_t n,
                          int64_t n_eligible, const nf_route_policy* policy_host,
                          nf_route_decision* decision_host);

/*
 * One bucket end to end (§3.3 steps 3-7), with no host synchronisation:
 * pass 1 reads the gradients once and produces the sign payload, the health
 * statistics and the FP32 sums at mask = 0; a one-block decision kernel
 * writes *decision (device); pass 2 then counts and decodes at mask = 1
 * (route L), sums the eligible elements in FP32 (route F), or does nothing
 * (route P).  When the policy fixes the route before any data is read (not
 * admitted, veto or guard without force_lowbit), pass 1 writes FP32 sums at
 * every position instead and bits are not written.
 * Always written: out[0..n), stats[0..W), *decision.  bits: written unless
 * the policy fixed the route before reading.  counts (nullable): written
 * when the route is L.
 * With policy format NF_FORMAT_TERNARY the low-bit route carries the
 * G-Ternary payload instead: pass 1 builds no sign payload; for route L the
 * per-worker thresholds come from the statistics (nf_ternary_threshold with
 * policy tau), a second read of the eligible elements writes the two planes
 * into bits (2W rows, as nf_pack_ternary), and the count and decode of
 * nf_ternary_reduce follow; counts (nullable) then receives 2n bytes.
 */
nf_status nf_route_bucket(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                          const uint64_t* mask, const nf_route_policy* policy_host,
                          uint64_t* bits, int64_t bits_stride_words, uint8_t* counts,
                          float* out, nf_worker_stats* stats, nf_route_decision* decision,
                          void* ws, size_t ws_bytes, void* stream);

/*
 * Many buckets of one flat gradient buffer in one call: pass 1 over all of
 * them, every bucket's decision, then pass 2, each phase a few launches on
 * `stream` (DDP cuts a model's flat gradient into fixed-capacity buckets,
 * §2.1).  Bucket b covers
 * elements [b*bucket_n, min((b+1)*bucket_n, n_total)) of every worker row,
 * of the mask, of the bitmap rows (from word b*bucket_n/64), of counts and of
 * out; nb = ceil(n_total / bucket_n).  bucket_n must be a multiple of 64
 * unless bucket_n >= n_total.  stats is [nb][W], decisions is [nb] (device).
 * Per bucket, the results equal those of nf_route_bucket on that bucket (with
 * the ternary format, c- of bucket b starts at counts + n_total + b*bucket_n).
 * At most NF_MAX_BUCKETS buckets per call (NF_ERR_INVALID_ARG beyond: the
 * read side runs a launch-grid row per bucket).
 */
#define NF_MAX_BUCKETS 65535
size_t nf_workspace_bytes_buckets(int32_t W, int64_t n_total, int64_t bucket_n);
nf_status nf_route_buckets(const float* grads, int64_t worker_stride, int32_t W,
                           int64_t n_total, int64_t bucket_n, const uint64_t* mask,
                           const nf_route_policy* policy_host, uint64_t* bits,
                           int64_t bits_stride_words, uint8_t* counts, float* out,
                           nf_worker_stats* stats, nf_route_decision* decisions, void* ws,
                           size_t ws_bytes, void* stream);

/*
 * nf_route_buckets without a workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments (less ws and ws_bytes), semantics
 * and results as nf_route_buckets.  The partial statistics go to a static
 * device array of NF_STATIC_SCRATCH_BYTES that the library holds on every
 * GPU it runs on until the process ends; the call allocates nothing.  A size
 * whose workspace (nf_workspace_bytes_buckets) exceeds that array returns
 * NF_ERR_WORKSPACE before anything is launched (64 MiB covers, e.g., 201
 * buckets of 16 x 6,553,600 elements, or one bucket of 64 x 100M).  Every
 * call on one GPU uses that GPU's one array, whose contents the next call
 * overwrites: calls that may overlap in time on one GPU (other streams or
 * threads without ordering between them) race, and must not be made.
 */
#define NF_STATIC_SCRATCH_BYTES (64ull << 20)
nf_status nf_route_buckets_noalloc(const float* grads, int64_t worker_stride, int32_t W,
                                   int64_t n_total, int64_t bucket_n, const uint64_t* mask,
                                   const nf_route_policy* policy_host, uint64_t* bits,
                                   int64_t bits_stride_words, uint8_t* counts, float* out,
                                   nf_worker_stats* stats, nf_route_decision* decisions,
                                   void* stream);

/*
 * Buckets of different sizes in one flat buffer (§2.1, §2.3: DDP fills a
 * bucket with whole parameters up to its capacity, so buckets end at
 * parameter boundaries and differ in size).  Bucket b covers elements
 * [bucket_offsets[b], bucket_offsets[b+1]) of every worker row, of the mask,
 * of the bitmap rows (from word bucket_offsets[b] / 64), of counts and of out;
 * n_total = bucket_offsets[nb].  bucket_offsets (host, nb + 1 values):
 * offsets[0] = 0, strictly increasing (no empty bucket), every bucket start
 * offsets[b] (b < nb) a multiple of 64.  stats is [nb][W], decisions [nb].
 * Per bucket, the results equal those of nf_route_bucket on that bucket
 * (with the ternary format, c- of bucket b starts at counts + n_total +
 * offsets[b]).
 *
 * The kernels find a bucket through a device table built once per bucket
 * layout and worker count (the layout is fixed for a training run):
 *   nf_bucket_table_bytes   size of the table (0 for invalid offsets or W)
 *   nf_bucket_table_init    builds it on the host and copies it into
 *                           `table` (device, caller-owned, 256-byte aligned,
 *                           at least nf_bucket_table_bytes), then
 *                           synchronises `stream`: a set-up call, not for
 *                           the step loop
 *   nf_workspace_bytes_table  workspace of nf_route_bucket_table
 * nf_route_bucket_table reads the table and needs the same W and offsets it
 * was built with (not checked on the device: another table gives wrong
 * results or invalid accesses).  Errors as nf_route_buckets, and
 * NF_ERR_INVALID_ARG for invalid offsets or nb above NF_MAX_BUCKETS,
 * NF_ERR_WORKSPACE for a short table.
 */
size_t nf_bucket_table_bytes(int32_t W, const int64_t* bucket_offsets, int32_t nb);
nf_status nf_bucket_table_init(int32_t W, const int64_t* bucket_offsets, int32_t nb, void* table,
                               size_t table_bytes, void* stream);
size_t nf_workspace_bytes_table(int32_t W, const int64_t* bucket_offsets, int32_t nb);
/* Profiling query (no paper counterpart): nf_pass1_launches for a bucket
 * table; 0 for invalid offsets or W.  Pure host function. */
int64_t nf_pass1_launches_table(int32_t W, const int64_t* bucket_offsets, int32_t nb, int32_t sign_words);
nf_status nf_route_bucket_table(const float* grads, int64_t worker_stride, int32_t W,
                                const int64_t* bucket_offsets, int32_t nb, const void* table,
                                const uint64_t* mask, const nf_route_policy* policy_host, uint64_t* bits,
                                int64_t bits_stride_words, uint8_t* counts, float* out,
                                nf_worker_stats* stats, nf_route_decision* decisions, void* ws,
                                size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Controller inputs on the host (§4.3 Supervisor recovery, §4.4 online
 * control, §6.4 endpoint-capacity guard).  These functions produce the
 * admitted / veto / guard_ok fields of nf_route_policy from an operating
 * profile, the training loss and the route decisions of earlier steps.
 * Pure host functions; every pointer is host memory.
 *
 * Supervisor per step t (the paper gives the mechanisms, not formulas; the
 * readings are stated here):
 *   - health signal: s_0 = loss_0, s_t = s_{t-1} + ema_alpha (loss_t - s_{t-1});
 *   - detector, Page's one-sided CUSUM on the per-step increase of s with the
 *     profile's slack and threshold (§4.1): S_t = max(0, S_{t-1} + (s_t -
 *     s_{t-1}) - slack), on steps run with low-bit admitted and not vetoed
 *     only; alarm when S_t > threshold (threshold * guard_scale during a
 *     readmission guard);
 *   - an alarm starts an FP32 cooldown (veto) of cooldown_steps steps and
 *     resets S; a near-threshold alarm (S_t <= threshold_eff * (1 +
 *     near_band)) with a small loss movement (|loss_t - loss_{t-1}| <=
 *     small_move) gets short_cooldown_steps instead when that is > 0 (the
 *     noise-aware short recovery);
 *   - after the cooldown low-bit is readmitted under a guard of guard_steps
 *     low-bit steps with the stricter threshold (0: readmitted directly);
 *   - Commander admits low-bit from step admit_step on (earlier steps: plain
 *     FP32, not admitted);
 *   - route-use budget guard: when the realized low-bit share L / (L + F + P)
 *     of the route events recorded so far exceeds target_share + share_margin,
 *     the next step is vetoed (target_share >= 1 disables it).
 * ------------------------------------------------------------------------ */
enum { NF_SUP_WARMUP = 0, NF_SUP_LOWBIT = 1, NF_SUP_COOLDOWN = 2, NF_SUP_GUARD = 3 };

/* Operating-profile settings of Commander and Supervisor (§4.1, Table 2). */
typedef struct {
  int32_t admit_step;            /* first step with low-bit admitted, >= 0         */
  int32_t cooldown_steps;        /* FP32 fallback length after an alarm, >= 0     */
  int32_t guard_steps;           /* readmission guard length, >= 0                 */
  int32_t short_cooldown_steps;  /* noise-aware short recovery, >= 0 (0: off)      */
  double ema_alpha;              /* smoothing of the loss, in (0, 1]               */
  double slack;                  /* CUSUM slack (tolerated increase per step)      */
  double threshold;              /* CUSUM threshold, > 0                           */
  double guard_scale;            /* threshold factor in the guard, in (0, 1]       */
  double near_band;              /* near-threshold band, >= 0                      */
  double small_move;             /* small loss movement, >= 0                      */
  double target_share;           /* route-use budget: target low-bit share         */
  double share_margin;           /* guard band over the target, >= 0               */
} nf_supervisor_profile;

/* Supervisor state and the run's route evidence (caller-owned, host). */
typedef struct {
  int64_t step;                  /* steps recorded so far                           */
  int32_t state;                 /* NF_SUP_*                                        */
  int32_t has_prev;              /* a loss has been recorded                        */
  int32_t cooldown_left, guard_left;
  double smoothed, cusum, prev_loss;
  int64_t alarms, short_recoveries, readmissions, budget_vetoes;
  int64_t events_l, events_f, events_p;  /* route events (buckets) by route (§3.2) */
  double bytes_route, bytes_fp32;        /* MGTR = bytes_route / bytes_fp32 (§3.2)  */
} nf_supervisor_state;

/* Validates the profile and starts a run (state WARMUP, or LOWBIT when
 * admit_step is 0).  NF_ERR_INVALID_ARG on an invalid profile. */
nf_status nf_supervisor_init(const nf_supervisor_profile* profile_host, nf_supervisor_state* state_host);

/* Controller inputs for the next step: sets policy->admitted and
 * policy->veto (cooldown or route-use budget); other fields untouched. */
nf_status nf_supervisor_policy(const nf_supervisor_profile* profile_host,
                               const nf_supervisor_state* state_host, nf_route_policy* policy_host);

/* Records the step just run: its nb route decisions (events and modeled
 * bytes) and its loss (finite), then advances the detector and the state.
 * The decisions are those made under nf_supervisor_policy for this step. */
nf_status nf_supervisor_update(const nf_supervisor_profile* profile_host,
                               nf_supervisor_state* state_host,
                               const nf_route_decision* decisions_host, int64_t nb, double loss);

/* Endpoint-capacity guard (§6.4): reducer-path measurements and topology. */
typedef struct {
  int32_t nodes, gpus_per_node;  /* N nodes x P GPUs, W = N P workers, >= 1        */
  int32_t bits_per_element;      /* payload bits per eligible element: 1 (G-Binary)
                                    or 2 (G-Ternary)                                */
  int32_t reserved;
  double net_bytes_per_s;        /* per-link network bandwidth B, > 0               */
  double endpoint_bytes_per_s;   /* endpoint counting service rate R (payload bytes
                                    per second), > 0                                */
  double latency_fp32_s, latency_lowbit_s;  /* fixed costs, >= 0                     */
} nf_endpoint_model;

/*
 * Estimated bucket communication time of the hierarchical low-bit reducer
 * and of the matched FP32 ring all-reduce, for a bucket of n elements of
 * which n_eligible are eligible; *guard_ok = (t_lowbit < t_fp32):
 *   t_fp32   = latency_fp32 + 2 (W-1)/W * 4 n / B
 *   t_lowbit = latency_lowbit + b n_E/8 / B       payload to the node endpoint
 *            + P b n_E/8 / R                      node-local counting
 *            + 2 (N-1)/N * n_E / B                uint8 partial-count exchange
 *            + n_E / B                            aggregate return
 *            + 2 (W-1)/W * 4 (n - n_E) / B        routed elements in FP32
 */
nf_status nf_endpoint_guard(const nf_endpoint_model* model_host, int64_t n, int64_t n_eligible,
                            double* t_fp32_host, double* t_lowbit_host, int32_t* guard_ok_host);

/*
 * Profiling hook (no paper counterpart).  When set on the calling thread,
 * nf_route_bucket and nf_route_buckets record these hipEvent_t handles (each
 * passed as void*) on their stream: before pass 1, after pass 1, after the
 * decision kernel and after pass 2 (the last one also when pass 2 is not
 * needed).  The caller owns the events; passing four NULLs turns recording
 * off.  Events are recorded, never synchronised, so calls stay asynchronous.
 */
nf_status nf_set_phase_events(void* before_pass1, void* after_pass1, void* after_decide,
                              void* after_pass2);

/*
 * Profiling query (no paper counterpart): the number of pass-1 kernel
 * launches that one nf_route_buckets call with these sizes makes (pass 1
 * runs as one launch for a problem of at most 4,096 element chunks, else in
 * launches of a fixed number of chunks, and above 32 workers once per row
 * group).  sign_words = 1
 * for a pass 1 that packs sign words (G-Binary), 0 for one that does not
 * (G-Ternary's first pass, nf_bucket_health), which runs in bigger
 * launches.  0 for n_total = 0 or invalid sizes.  Pure host function.
 */
int64_t nf_pass1_launches(int32_t W, int64_t n_total, int64_t bucket_n, int32_t sign_words);

/*
 * Geometry query (no paper counterpart): the number of elements of every
 * pass-1 chunk (a block's share of one bucket, the unit of its partial
 * statistics; a bucket's last chunk may be shorter) for these sizes, and in
 * *chunks_per_bucket (nullable) the chunks of a full bucket.  Pass 1 takes a
 * chunk with no eligible element, or with every element eligible, by a loop
 * of its own; tests use this to build such chunks.  0 for n_total = 0 or
 * invalid sizes.  Pure host function.
 */
int64_t nf_pass1_chunk_elems(int32_t W, int64_t n_total, int64_t bucket_n, int64_t* chunks_per_bucket);

#ifdef __cplusplus
}
#endif
#endif /* NF_H */
