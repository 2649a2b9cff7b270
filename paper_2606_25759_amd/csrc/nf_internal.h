// nf_internal.h - launch geometry, kernel argument blocks and the route rules
// shared by the host decision function and the device decision kernel.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "nf.h"

#define NF_HD __host__ __device__

namespace nf {

// ---------------------------------------------------------------- geometry
//
// Pass 1 is worker-major: a block is 16 wavefronts; wavefront v serves
// worker group wg = v % WG and element group eg = v / WG.  With W <= 16 each
// wavefront owns one worker (WG = W) and the spare wavefronts take further
// element groups (EG = 16 / W); with 16 < W <= 32 each wavefront owns
// ceil(W / 16) workers.  Above 32 workers the rows go in groups of
// near-equal size, one after another (a launch sequence per group, all
// with the geometry of the largest): two groups up to 64 workers, then
// ceil(W / 64).  Sixteen workers per wavefront held 32 FP64 health sums per
// lane and spilled (W = 255: pass 1 at 2.9 TB/s); at W = 64, two groups of
// 32 (two workers per wavefront, eight wavefronts per SIMD, two blocks per
// compute unit) ran the stress bucket's G-Ternary step 4% faster than one
// group of 64, while at W = 255 groups of 32 ran 26% slower than groups of
// 64.  Every group has at least 16 rows, so each of the 16 wavefronts'
// first worker exists in every group.  The groups share the chunk slots
// (each writes its own workers' partials) and carry the FP32 sums at routed
// positions from one to the next through the output, so the workers are
// still added in order.  A tile is EG * T consecutive elements of all W
// rows; staging one tile of all workers in LDS (to add the workers in order
// at FP32-routed positions) takes at most 64 KiB.
//
// Work is cut into chunks of G consecutive tiles of one bucket; a block
// takes one chunk and keeps the chunk's sign words in LDS until it ends.
// Above kOneLaunchChunks chunks (below), pass 1 runs as a sequence of
// launches of kEpochBlocks chunks each, so the bitmap stores of a launch
// reach memory together at its end rather than spread thinly through the
// gradient read stream.  Measured on MI355X:
// writes mixed into a streaming read cost far more than their own bytes (a
// 1/32 share of writes slows a plain 84 GB read by 35-45%); spread-out
// stores cost about 40% of the scan's time, launch-end bursts about 15-20%.
// One chunk per compute unit (256 on MI355X) per launch is the best epoch
// measured (128: -30%, 192 and 384: -7%, 512: -4%, 1024: -7%).
constexpr int kWaves = 16;
constexpr int kRowGroup = 64;     // worker rows per pass-1 group at most
constexpr int kWideWorkers = 32;  // above this: row groups, the decision's thread-per-worker reduction
constexpr int kThreads1 = kWaves * 64;
constexpr int kStageFloats = 16384;      // 64 KiB of LDS
#ifndef NF_BITS_WORDS
#define NF_BITS_WORDS 4096
#endif
#ifndef NF_EPOCH_BLOCKS
#define NF_EPOCH_BLOCKS 256
#endif
#ifndef NF_EPOCH_NOPACK
#define NF_EPOCH_NOPACK 1024
#endif
#ifndef NF_MAX_G
#define NF_MAX_G 32
#endif
constexpr int kBitsWords = NF_BITS_WORDS;      // LDS words for a chunk's sign words (32 KiB)
constexpr int kMaxSlots = 512;                 // partials the decision reduces per bucket at most
// ... above kWideWorkers workers (the decision then reads 64 * W partials
// per bucket: with 400 of 255 workers each, a 25 MiB bucket's decision
// took 0.28 ms)
constexpr int kMaxSlotsWide = 64;
constexpr int kEpochBlocks = NF_EPOCH_BLOCKS;  // chunks per pass-1 launch
// Without sign words (statistics and routed sums only) the writes are few and
// bigger launches lose less to tails: G-Ternary's first pass at GPT scale,
// 256 -> 13.7 ms, 1024 -> 12.8 ms, 4096 -> 12.8 ms, one launch -> 12.9 ms.
constexpr int64_t kEpochNoPack = NF_EPOCH_NOPACK;
constexpr int kMaxG = NF_MAX_G;                // tiles per chunk at most
static_assert(kMaxG <= 32, "pass 1 keeps a bit per tile of a chunk in 32 bits");
// Problems of at most 16 epochs of chunks (about 4 GiB of gradients) run as
// one launch: their stores cost less than the launch tails.  Measured: the
// 0.82 GB ResNet-50-scale workload's pass 1 0.28 -> 0.19 ms (up to 4
// epochs); up to 16 epochs, 30M elements at W = 32 (3,663 chunks) 0.946 ->
// 0.859 ms a step, 20M at W = 16 0.341 -> 0.317 ms, G-Ternary at W = 255
// 5.43 -> 5.29 ms.  ViT-B/16 scale (5,284 chunks) ran 2% slower as one
// launch, so larger problems keep launches of kEpochBlocks.
constexpr int64_t kOneLaunchChunks = 16 * kEpochBlocks;
// Chunks of a small problem: two rounds of two 16-wavefront blocks per
// compute unit.  One round and a part (ResNet-50 scale: 782 chunks of 32
// tiles) leaves most units idle in the second; 1,000 chunks of 25 tiles ran
// pass 1 0.185 -> 0.163 ms.
constexpr int64_t kFillChunks = 1024;
// ... and of a problem of at most kFillChunks tiles: one chunk per compute
// unit.  One block per unit with several tiles beat two or more blocks of
// one tile each at every size tried: the tiny bucket's step 0.057 -> 0.049
// ms, 2M elements at W = 4 0.074 -> 0.054 ms, 500K at W = 16 0.081 -> 0.055
// ms, 200K at W = 255 0.394 -> 0.315 ms (fewer slots also spare the
// decision its second level).
constexpr int64_t kSmallFillChunks = 256;
inline int64_t one_launch_epoch(int64_t total_chunks) {
  return total_chunks <= kOneLaunchChunks ? (total_chunks > 0 ? total_chunks : 1) : kEpochBlocks;
}

// Pass 2: a wavefront takes 64 consecutive bitmap words (4096 elements) per
// step, four wavefronts per block.
constexpr int kThreads2 = 256;
constexpr int kWordsPerWave2 = 64;
constexpr int kMaxBlocks2 = 1024;

// Words per worker and wavefront tile for WPW workers per wavefront: eight
// words for one worker and four for two keep pass 1 within 64 VGPRs (eight
// wavefronts per SIMD) without spills; more workers share 16 words.
constexpr NF_HD int pass1_words(int wpw) { return wpw == 1 ? 8 : wpw == 2 ? 4 : 16 / wpw; }
// Steps (64 elements) per wavefront of a whole chunk of kMaxG tiles of one
// element group, for NW words per worker and tile.
constexpr NF_HD int routed_steps(int nw) { return (kMaxG * nw + kWaves - 1) / kWaves; }

struct Geometry {
  int W, wg, eg, wpw, T, tile, G;
  int rows, ngroups;     // worker rows of the largest pass-1 group (<= 64), and groups
  int64_t n_total, bucket_n, nb;  // bucket_n: 0 for a bucket table
  bool table;            // buckets from a bucket table (sizes vary)
  int64_t chunks_full;   // chunks of a full bucket (of the largest, for a table)
  int64_t total_chunks;  // over all buckets
  int slots;             // partial-statistics slots per bucket (uniform): one per chunk
  int gs;                // slots per second-level group (0: no second level)
  int groups;            // second-level groups per full bucket (<= kMaxSlots)
  int bpb2;              // pass-2 blocks per bucket
};

// Bucket table: one row per bucket of a flat buffer whose buckets differ in
// size (DDP closes a bucket at a parameter boundary, §2.1).  Chunk q of
// pass 1 belongs to bucket cbucket[q] and owns partial slot q, so bucket b's
// slots are chunk0 .. chunk0 + (its chunks) - 1.
struct BucketRow {
  int64_t start;   // first element (a multiple of 64)
  int64_t len;     // elements (> 0)
  int64_t chunk0;  // first pass-1 chunk
  int64_t pad;
};

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Chunks per pass-1 launch (see kOneLaunchChunks), with or without sign words.
inline int64_t pass1_epoch(const Geometry& g) { return one_launch_epoch(g.total_chunks); }
inline int64_t pass1_launch_chunks(const Geometry& g, bool sign_words) {
  return sign_words || g.total_chunks <= kOneLaunchChunks ? pass1_epoch(g) : kEpochNoPack;
}

// Row group i of a geometry: its first worker and its rows (the first
// W % ngroups groups take one row more).
inline void row_group(const Geometry& g, int i, int* wbase, int* rows) {
  const int q = g.W / g.ngroups, r = g.W % g.ngroups;
  *wbase = i * q + (i < r ? i : r);
  *rows = q + (i < r ? 1 : 0);
}

// The worker-dependent part of the geometry (row groups, wavefront roles,
// tile, chunk length before the fill rule).
inline Geometry geometry_core(int W) {
  Geometry g;
  g.W = W;
  g.ngroups = W > kRowGroup ? (W + kRowGroup - 1) / kRowGroup : (W > kWideWorkers ? 2 : 1);
  g.rows = (W + g.ngroups - 1) / g.ngroups;
  const int R = g.rows;  // the pass-1 kernel's workers
  g.wg = R < kWaves ? R : kWaves;
  g.eg = kWaves / g.wg;
  // Workers per wavefront, rounded up to a power of two (a template
  // parameter of pass 1).
  int need = (R + g.wg - 1) / g.wg;
  g.wpw = 1;
  while (g.wpw < need) g.wpw *= 2;
  g.T = 64 * pass1_words(g.wpw);  // R * EG * T <= kStageFloats for every R <= 64
  g.tile = g.eg * g.T;
  // A chunk's sign words, R * G * EG * (T / 64), fit kBitsWords.
  int per_tile = R * g.eg * (g.T / 64);
  g.G = kBitsWords / per_tile;
  if (g.G > kMaxG) g.G = kMaxG;
  if (g.G < 1) g.G = 1;
  g.table = false;
  return g;
}

// A problem of fewer than kFillChunks chunks would leave compute units
// idle: it takes the smallest G that keeps it within kFillChunks chunks (so
// within one launch), or within kSmallFillChunks when it has at most
// kFillChunks tiles.  total_for(G): the problem's chunks at G tiles each.
template <typename F>
inline void fill_rule(Geometry& g, F total_for) {
  const int64_t target = total_for(1) <= kFillChunks ? kSmallFillChunks : kFillChunks;
  if (total_for(g.G) < target)
    for (int G = 1; G < g.G; ++G)
      if (total_for(G) <= target) {
        g.G = G;
        break;
      }
}

// Second-level groups and pass-2 blocks from the largest bucket's chunks
// and words.
inline void slot_groups(Geometry& g, int64_t max_len) {
  // Every chunk owns a slot, so no two chunks ever touch the same partial.
  // A bucket of more than kMaxSlots chunks (kMaxSlotsWide above kWideWorkers)
  // is first summed in groups of gs consecutive slots (at most that many
  // groups), which the decision reads.
  g.slots = (int)(g.chunks_full > 1 ? g.chunks_full : 1);
  const int cap = g.W > kWideWorkers ? kMaxSlotsWide : kMaxSlots;
  g.gs = g.chunks_full > cap ? (int)ceil_div(g.chunks_full, cap) : 0;
  g.groups = g.gs ? (int)ceil_div(g.chunks_full, g.gs) : 0;
  int64_t words = (max_len + 63) / 64;
  int64_t chunks2 = ceil_div(words, kWordsPerWave2 * 4);
  if (chunks2 < 1) chunks2 = 1;
  g.bpb2 = (int)(chunks2 < kMaxBlocks2 ? chunks2 : kMaxBlocks2);
}

// Equal buckets of bucket_n elements (the last one shorter).
inline Geometry make_geometry(int W, int64_t n_total, int64_t bucket_n) {
  Geometry g = geometry_core(W);
  g.n_total = n_total;
  g.bucket_n = bucket_n;
  g.nb = n_total <= 0 ? 1 : ceil_div(n_total, bucket_n);
  int64_t full = n_total < bucket_n ? n_total : bucket_n;
  if (full < 0) full = 0;
  int64_t last = n_total - (g.nb - 1) * bucket_n;
  if (last < 0) last = 0;
  const int64_t tiles_full = ceil_div(full, g.tile), tiles_last = ceil_div(last, g.tile);
  auto total_for = [&](int G) { return (g.nb - 1) * ceil_div(tiles_full, G) + ceil_div(tiles_last, G); };
  fill_rule(g, total_for);
  g.chunks_full = ceil_div(tiles_full, g.G);
  g.total_chunks = total_for(g.G);
  slot_groups(g, full);
  return g;
}

// Buckets [off[b], off[b+1]) of a bucket table (nb >= 1, off[0] = 0,
// off strictly increasing; validated by the caller).
inline Geometry make_geometry_table(int W, const int64_t* off, int64_t nb) {
  Geometry g = geometry_core(W);
  g.table = true;
  g.n_total = off[nb];
  g.bucket_n = 0;
  g.nb = nb;
  auto total_for = [&](int G) {
    int64_t t = 0;
    for (int64_t b = 0; b < nb; ++b) t += ceil_div(ceil_div(off[b + 1] - off[b], g.tile), G);
    return t;
  };
  fill_rule(g, total_for);
  int64_t max_len = 0;
  for (int64_t b = 0; b < nb; ++b)
    if (off[b + 1] - off[b] > max_len) max_len = off[b + 1] - off[b];
  g.chunks_full = ceil_div(ceil_div(max_len, g.tile), g.G);
  g.total_chunks = total_for(g.G);
  slot_groups(g, max_len);
  return g;
}

// Device bucket table of a table geometry: the rows, then the bucket of
// every chunk.
inline size_t table_rows_bytes(int64_t nb) { return (size_t)((nb * (int64_t)sizeof(BucketRow) + 255) & ~(int64_t)255); }
inline size_t table_bytes(const Geometry& g) {
  return table_rows_bytes(g.nb) + (size_t)((g.total_chunks * 4 + 255) & ~(int64_t)255);
}

// Per (bucket, slot, worker) partial statistics written by pass 1.  The |g|
// sum is carried as s + c with an error bound b (an XSum, nf_device.h): its
// exact value lies within b of sabs + sabs_c.  Pass 1 without sign words
// tracks every rounding error (exact mode); with sign words c and b start at
// 0 and only the reductions after pass 1 track theirs.
struct Partial {
  double sabs;
  double ssq;
  uint64_t nonfinite;
  double sabs_c;
  double sabs_b;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct WorkspaceLayout {
  size_t partials, ne, part2, ne2, total;
};

// [bucket][slot][W] partials, [bucket][slot] eligible counts, then the
// second-level [bucket][group][W] and [bucket][group] sums.
inline WorkspaceLayout workspace_layout(const Geometry& g) {
  WorkspaceLayout l;
  // one slot per chunk: chunk q's partials at slot q
  const size_t slots = g.table ? (size_t)(g.total_chunks > 0 ? g.total_chunks : 1) : (size_t)g.nb * (size_t)g.slots;
  const size_t groups = (size_t)g.nb * (size_t)g.groups;
  l.partials = 0;
  l.ne = align256(slots * (size_t)g.W * sizeof(Partial));
  l.part2 = l.ne + align256(slots * sizeof(uint64_t));
  l.ne2 = l.part2 + align256(groups * (size_t)g.W * sizeof(Partial));
  l.total = l.ne2 + align256(groups * sizeof(uint64_t));
  return l;
}

// ------------------------------------------------------- kernel arguments

enum SumMode { kSumsNone = 0, kSumsRouted = 1, kSumsAll = 2 };

struct Pass1Args {
  const float* g;  // the row group's first row
  int64_t wstride;
  const uint64_t* mask;
  uint64_t* bits;  // NULL: no sign payload; else the row group's first row
  int64_t bstride;
  float* out;      // FP32 sums (sum mode != none)
  Partial* part;
  uint64_t* part_ne;
  int64_t n_total, bucket_n, chunks_full, total_chunks;
  int32_t nb, W, wg, eg, T, G, slots, sums, mean;
  // Row groups: W is this group's rows; partials are [slot][wtot] with this
  // group's workers from wbase; racc: the routed FP32 sums continue from
  // out (not the first group); rfin: the last group (MEAN divides there).
  int32_t wtot, wbase, racc, rfin;
  const BucketRow* btab;   // NULL: equal buckets of bucket_n
  const int32_t* cbucket;  // bucket of every chunk (with btab)
};

struct DecideArgs {
  const Partial* part;
  const uint64_t* part_ne;
  // Exact mode (pass 1 without sign words): each worker's |g| sum is
  // rounded once from its exact value, re-summed from the gradients when
  // the carried error bound cannot certify the rounding.
  const float* g;
  int64_t wstride;
  const uint64_t* mask;
  int32_t exact;
  Partial* part2;          // second-level sums (gs > 0)
  uint64_t* part2_ne;
  nf_worker_stats* stats;
  nf_route_decision* dec;  // NULL: statistics only
  nf_route_policy pol;
  int64_t n_total, bucket_n;
  int32_t W, slots, tile, G, gs, groups;
  const BucketRow* btab;  // NULL: equal buckets of bucket_n
};

// kOpFallbackOnly: route-driven, FP32 sums of the buckets routed F only.
enum Pass2Op { kOpCountDecode = 0, kOpFp32 = 1, kOpFromDecision = 2, kOpFallbackOnly = 3 };

// G-Ternary pack and count/decode.  Route-driven (dec != NULL): only the
// buckets routed L, thresholds from stats and tau.  Standalone: one bucket,
// thresholds theta[W] and scale *scale.
struct TernArgs {
  const float* g;
  int64_t wstride;
  const uint64_t* mask;
  uint64_t* bits;  // 2W rows: positive planes 0..W-1, negative planes W..2W-1
  int64_t bstride;
  const nf_route_decision* dec;
  const nf_worker_stats* stats;  // [bucket][W]
  const float* theta;
  const float* scale;
  uint8_t* cpos;  // nullable
  uint8_t* cneg;  // nullable
  float* out;     // nullable
  float tau;
  int64_t n_total, bucket_n;
  int32_t W, decode_mode, bpb2;
  // pack geometry (filled by the pack launcher from the Geometry): the
  // launch's row group is workers wbase .. wbase + rows - 1
  int64_t chunks_full, total_chunks;
  int32_t nb, wg, eg, T, G, rows, wbase;
  const BucketRow* btab;   // NULL: equal buckets of bucket_n
  const int32_t* cbucket;  // bucket of every chunk (with btab)
};

struct Pass2Args {
  const uint64_t* bits;
  int64_t bstride;
  const float* g;
  int64_t wstride;
  const uint64_t* mask;
  const nf_route_decision* dec;  // kOpFromDecision: route and scale per bucket
  const float* scale;            // kOpCountDecode standalone
  uint8_t* counts;
  float* out;
  int64_t n_total, bucket_n;
  int32_t W, op, select, decode_mode, mean, bpb2;
  // grid z (0 or 1: one count): count z reads rows from z * z_rows and
  // writes counts + z * z_counts, out + z * z_out
  int32_t nz, z_rows;
  int64_t z_counts, z_out;
  const BucketRow* btab;  // NULL: equal buckets of bucket_n
};

// Partial-count reduction (inter-node sum of node-local counts + decode).
struct PsumArgs {
  const uint8_t* partial;  // G rows of n bytes, row g at partial + g * pstride
  int64_t pstride;
  const uint64_t* mask;    // required when out != NULL
  const float* scale;      // device, one float; required when out != NULL
  uint8_t* counts;         // nullable: n bytes
  float* out;              // nullable: written at mask = 1
  int64_t n;
  int32_t G, W, decode_mode;
};

// ------------------------------------------------------------ route rules
//
// Reasons and route of one bucket (§3.2 route states, §6.4 guard).  The
// caller supplies the lower median of the finite sums of squares (k finite
// values, median valid when k >= 2); host and device compute it by rank.

NF_HD inline float bucket_scale(const nf_worker_stats* st, int W, int64_t ne) {
  if (ne <= 0) return 0.0f;
  double acc = 0.0;
  for (int w = 0; w < W; ++w) acc += st[w].sum_abs_elig / (double)ne;
  return (float)(acc / (double)W);
}

NF_HD inline bool finite64(double x) { return x - x == 0.0; }

// Norm-spike threshold: kappa^2 times the lower median of the finite sums
// of squares; a worker spikes when its finite sum of squares exceeds it (with
// at least two finite sums).
NF_HD inline double spike_threshold(const nf_route_policy& p, double median) {
  return (p.kappa * p.kappa) * median;
}

// Route, reasons, scale and modeled bytes of a bucket from its per-worker
// findings: a non-finite value in some worker, a worker whose eligible |g|
// sum is 0, a norm spike.
NF_HD inline void decide_finish(int64_t n, int64_t ne, const nf_route_policy& p, bool nonf, bool zero,
                                bool spike, float scale, nf_route_decision* d) {
  uint32_t r = 0;
  if (!p.admitted) r |= NF_REASON_NOT_ADMITTED;
  if (ne == 0) r |= NF_REASON_NO_ELIGIBLE;
  if (p.veto) r |= NF_REASON_VETO;
  if (!p.guard_ok) r |= NF_REASON_GUARD;
  if (nonf) r |= NF_REASON_NONFINITE;
  if (zero && ne > 0) r |= NF_REASON_ZERO_WORKER;
  if (spike) r |= NF_REASON_NORM_SPIKE;
  int32_t route;
  if (r & (NF_REASON_NOT_ADMITTED | NF_REASON_NO_ELIGIBLE)) {
    route = NF_ROUTE_PLAIN;
  } else if (p.force_lowbit) {
    route = NF_ROUTE_LOWBIT;
    r |= NF_REASON_FORCED;
  } else if (r & (NF_REASON_VETO | NF_REASON_GUARD | NF_REASON_NONFINITE |
                  NF_REASON_ZERO_WORKER | NF_REASON_NORM_SPIKE)) {
    route = NF_ROUTE_FALLBACK;
  } else {
    route = NF_ROUTE_LOWBIT;
  }
  d->route = route;
  d->reasons = r;
  d->scale = scale;
  d->resummed = 0;
  d->n_eligible = ne;
  d->bytes_fp32 = 4.0 * (double)n;
  // one bit (binary) or two planes (ternary) per eligible element
  d->bytes_route = route == NF_ROUTE_LOWBIT
                       ? (p.format == NF_FORMAT_TERNARY ? 2.0 : 1.0) * (double)ne / 8.0 + 4.0 +
                             4.0 * (double)(n - ne)
                       : 4.0 * (double)n;
}

// The same from the statistics, one worker after another (the host's
// decision; the device kernel finds the per-worker facts in parallel).
NF_HD inline void decide_from(const nf_worker_stats* st, int W, int64_t n, int64_t ne,
                              const nf_route_policy& p, int kfinite, double median,
                              nf_route_decision* d) {
  uint64_t nonf = 0;
  bool zero = false, spike = false;
  const double thr = spike_threshold(p, median);
  for (int w = 0; w < W; ++w) {
    nonf += st[w].nonfinite;
    if (st[w].sum_abs_elig == 0.0) zero = true;
    if (kfinite >= 2 && finite64(st[w].sum_sq) && st[w].sum_sq > thr) spike = true;
  }
  decide_finish(n, ne, p, nonf != 0, zero, spike, bucket_scale(st, W, ne), d);
}

// G-Ternary write-side threshold: tau times the worker's mean |g| over
// eligible elements, the mean rounded to FP32 first; 0 without eligible
// elements.
NF_HD inline float ternary_threshold(const nf_worker_stats& st, int64_t ne, float tau) {
  if (ne <= 0) return 0.0f;
  const float mean_abs = (float)(st.sum_abs_elig / (double)ne);
  return tau * mean_abs;
}

// G-Ternary decode of the vote difference d = c+ - c- in [-W, W].
NF_HD inline float decode_qt(int d, int W, int mode) {
  if (mode == NF_DECODE_MAJORITY) return d > 0 ? 1.0f : (d < 0 ? -1.0f : 0.0f);
  return (float)d / (float)W;
}

// Rank of worker w among the finite sums of squares (ties by index).
NF_HD inline int ssq_rank(const nf_worker_stats* st, int W, int w) {
  double v = st[w].sum_sq;
  int rank = 0;
  for (int u = 0; u < W; ++u) {
    double x = st[u].sum_sq;
    if (!finite64(x)) continue;
    if (x < v || (x == v && u < w)) ++rank;
  }
  return rank;
}

// Decode value for count c: SOFT fl32((2c - W) / W), MAJORITY sign with tie 0.
NF_HD inline float decode_q(int c, int W, int mode) {
  int margin = 2 * c - W;
  if (mode == NF_DECODE_MAJORITY) return margin > 0 ? 1.0f : (margin < 0 ? -1.0f : 0.0f);
  return (float)margin / (float)W;
}

// Per-slice scales and the compacted payload (nf_sliced.hip).
constexpr int64_t kSliceSeg = 65536;  // elements per statistics segment of a slice

struct CompactArgs {
  const uint64_t* bits;     // positional rows
  int64_t bstride;
  const uint64_t* mask;
  const uint64_t* prefix;   // [nw + 1] eligible elements before word k
  const int64_t* start;     // [ceil(n_E / 64)] word holding rank 64 o
  uint64_t* cbits;          // compacted rows
  int64_t cstride;
  int64_t n, n_eligible;
  int32_t W;                // rows (filled by the launcher)
};

// Per-slice statistics from pass 1's chunk partials (one bucket of n
// elements, chunks of CH elements).
struct SliceChunkArgs {
  const float* g;
  int64_t wstride;
  const Partial* part;  // [chunk][W]: pass 1's partial slots
  const int64_t* off;   // [S]
  const int64_t* len;   // [S]
  double* sums;         // [S][W]
  float* scales;        // [S]
  int64_t S, CH;
  int32_t W;
};

struct SliceArgs {
  const float* g;
  int64_t wstride;
  const int64_t* off;       // [S]
  const int64_t* len;       // [S]
  const int64_t* segp;      // [S + 1] first segment of slice s
  double* part;             // [segments][W] workspace
  double* sums;             // [S][W]
  float* scales;            // [S]
  int64_t S;
  int32_t W;
};

struct ExpandArgs {
  const uint64_t* mask;
  const uint64_t* prefix;   // [nw + 1]
  const int32_t* wslice;    // [nw]
  const int64_t* rstart;    // [S + 1]
  const float* scales;      // [S]
  const uint8_t* counts_c;  // [n_E] counts in compacted order, 4-byte aligned
  float* out;
  int64_t n, S, n_eligible;
  int32_t W, decode_mode;
};

hipError_t launch_compact(const CompactArgs& a, int W, hipStream_t s);
hipError_t launch_slice_scales(const SliceArgs& a, int64_t segments, hipStream_t s);
hipError_t launch_slice_chunks(const SliceChunkArgs& a, hipStream_t s);
hipError_t launch_cexpand(const ExpandArgs& a, hipStream_t s);

// Sets the thread-local message of nf_last_error (nf_api.hip) and returns st.
nf_status set_error(nf_status st, const char* msg);

// Launchers (nf_pass1.hip, nf_pass2.hip, nf_ternary.hip, nf_sliced.hip).
hipError_t launch_pass1(const Geometry& geo, const Pass1Args& a, hipStream_t s);
hipError_t launch_decide(const Geometry& geo, const DecideArgs& a, hipStream_t s);
hipError_t launch_pass2(const Geometry& geo, const Pass2Args& a, hipStream_t s);
hipError_t launch_ternary_pack(const Geometry& geo, const TernArgs& a, hipStream_t s);
hipError_t launch_ternary_reduce(const Geometry& geo, const TernArgs& a, hipStream_t s);
hipError_t launch_psum(const PsumArgs& a, hipStream_t s);

}  // namespace nf
