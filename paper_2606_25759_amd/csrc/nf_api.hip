// nf_api.hip - the C ABI of include/nf.h: argument checks, workspace
// layout, and the launch sequence on the caller's stream.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>
#include <vector>

#include "nf_internal.h"

namespace {

// Device scratch of the allocation-free driver (nf_route_buckets_noalloc):
// the partial-statistics workspace of one call, in a file-scope array that
// every GPU running the library holds until the process ends.  In host code
// the array's name stands for a host-side shadow, never a device address:
// each device's address comes from hipGetSymbolAddress, taken once per
// device on the first call there, and only that address reaches a kernel.
constexpr size_t kStaticScratchBytes = (size_t)NF_STATIC_SCRATCH_BYTES;
constexpr int kMaxBuckets = NF_MAX_BUCKETS;
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

thread_local std::string g_err;
thread_local hipEvent_t g_phase_ev[4] = {nullptr, nullptr, nullptr, nullptr};

void record_phase(int i, hipStream_t s) {
  if (g_phase_ev[i]) (void)hipEventRecord(g_phase_ev[i], s);
}

nf_status fail(nf_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
nf_status fail(nf_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

nf_status ok() {
  g_err.clear();
  return NF_OK;
}

nf_status hip_fail(hipError_t e, const char* what) {
  return fail(NF_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// The current device's address of `scratch`, looked up on its first use.
nf_status scratch_address(void** p) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(NF_ERR_UNSUPPORTED, "device %d: the static scratch is tracked for devices 0..%d", dev,
                kMaxDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* a = nullptr;
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!a) return fail(NF_ERR_HIP, "hipGetSymbolAddress(scratch) gave a null address");
    g_scratch_dev[dev] = a;
  }
  *p = g_scratch_dev[dev];
  return NF_OK;
}

// Checks shared by every entry point that reads gradient rows.
nf_status check_grads(const float* g, int64_t stride, int32_t W, int64_t n) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (n < 0) return fail(NF_ERR_INVALID_ARG, "n=%lld < 0", (long long)n);
  if (stride < n) return fail(NF_ERR_INVALID_ARG, "worker_stride=%lld < n=%lld", (long long)stride, (long long)n);
  if (n > 0 && !g) return fail(NF_ERR_INVALID_ARG, "grads is NULL");
  if (!aligned(g, 16)) return fail(NF_ERR_ALIGNMENT, "grads not 16-byte aligned");
  if (stride % 4) return fail(NF_ERR_ALIGNMENT, "worker_stride=%lld not a multiple of 4", (long long)stride);
  return NF_OK;
}

nf_status check_mask(const uint64_t* mask, int64_t n) {
  if (n > 0 && !mask) return fail(NF_ERR_INVALID_ARG, "mask is NULL");
  if (!aligned(mask, 8)) return fail(NF_ERR_ALIGNMENT, "mask not 8-byte aligned");
  return NF_OK;
}

nf_status check_bits(const uint64_t* bits, int64_t bstride, int64_t n, int32_t W) {
  (void)W;
  if (n > 0 && !bits) return fail(NF_ERR_INVALID_ARG, "bits is NULL");
  if (!aligned(bits, 8)) return fail(NF_ERR_ALIGNMENT, "bits not 8-byte aligned");
  if (bstride < (n + 63) / 64)
    return fail(NF_ERR_INVALID_ARG, "bits_stride_words=%lld < ceil(n/64)=%lld", (long long)bstride,
                (long long)((n + 63) / 64));
  return NF_OK;
}

nf_status check_policy(const nf_route_policy* p) {
  if (!p) return fail(NF_ERR_INVALID_ARG, "policy is NULL");
  if (!(p->kappa > 0.0) || p->kappa != p->kappa || p->kappa - p->kappa != 0.0)
    return fail(NF_ERR_INVALID_ARG, "kappa must be finite and > 0");
  if (p->decode_mode != NF_DECODE_SOFT && p->decode_mode != NF_DECODE_MAJORITY)
    return fail(NF_ERR_INVALID_ARG, "decode_mode=%d", p->decode_mode);
  if (p->fp32_op != NF_FP32_SUM && p->fp32_op != NF_FP32_MEAN)
    return fail(NF_ERR_INVALID_ARG, "fp32_op=%d", p->fp32_op);
  if (p->format != NF_FORMAT_BINARY && p->format != NF_FORMAT_TERNARY)
    return fail(NF_ERR_INVALID_ARG, "format=%d", p->format);
  if (p->format == NF_FORMAT_TERNARY && !(p->tau >= 0.0f && p->tau - p->tau == 0.0f))
    return fail(NF_ERR_INVALID_ARG, "tau must be finite and >= 0");
  return NF_OK;
}

nf_status check_ws(const void* ws, size_t ws_bytes, size_t need) {
  if (ws_bytes < need)
    return fail(NF_ERR_WORKSPACE, "workspace of %zu bytes < %zu required", ws_bytes, need);
  if (need && !ws) return fail(NF_ERR_WORKSPACE, "workspace is NULL");
  if (!aligned(ws, 256)) return fail(NF_ERR_ALIGNMENT, "workspace not 256-byte aligned");
  return NF_OK;
}

void fill_pass1_geometry(const nf::Geometry& geo, nf::Pass1Args* a) {
  a->n_total = geo.n_total;
  a->bucket_n = geo.bucket_n;
  a->chunks_full = geo.chunks_full;
  a->total_chunks = geo.total_chunks;
  a->nb = (int32_t)geo.nb;
  a->W = geo.W;
  a->wg = geo.wg;
  a->eg = geo.eg;
  a->T = geo.T;
  a->G = geo.G;
  a->slots = geo.slots;
  a->btab = nullptr;
  a->cbucket = nullptr;
}

#define NF_TRY(x)                    \
  do {                               \
    nf_status st__ = (x);            \
    if (st__ != NF_OK) return st__;  \
  } while (0)

// Pass 1 + statistics (and optionally the decision) for buckets of one flat
// buffer.  Shared by the health, pack and route entry points.
nf_status run_pass1_decide(const nf::Geometry& geo, const float* g, int64_t stride,
                           const uint64_t* mask, uint64_t* bits, int64_t bstride, float* out,
                           int sums, int mean, nf_worker_stats* stats, nf_route_decision* dec,
                           const nf_route_policy* pol, void* ws, hipStream_t s,
                           bool phases = false, const nf::BucketRow* btab = nullptr,
                           const int32_t* cbucket = nullptr) {
  const nf::WorkspaceLayout lay = nf::workspace_layout(geo);
  char* w = static_cast<char*>(ws);
  nf::Pass1Args a;
  a.g = g;
  a.wstride = stride;
  a.mask = mask;
  a.bits = bits;
  a.bstride = bstride;
  a.out = out;
  a.part = reinterpret_cast<nf::Partial*>(w + lay.partials);
  a.part_ne = reinterpret_cast<uint64_t*>(w + lay.ne);
  fill_pass1_geometry(geo, &a);
  a.btab = btab;
  a.cbucket = cbucket;
  a.sums = sums;
  a.mean = mean;
  if (phases) record_phase(0, s);
  hipError_t e = nf::launch_pass1(geo, a, s);
  if (e != hipSuccess) return hip_fail(e, "pass-1 launch");
  if (phases) record_phase(1, s);
  nf::DecideArgs d;
  d.part = a.part;
  d.part_ne = a.part_ne;
  d.g = g;
  d.wstride = stride;
  d.mask = mask;
  d.exact = bits == nullptr;  // pass 1 without sign words tracks exact |g| sums
  d.stats = stats;
  d.dec = dec;
  if (pol) {
    d.pol = *pol;
  } else {
    memset(&d.pol, 0, sizeof d.pol);
    d.pol.kappa = 4.0;
  }
  d.n_total = geo.n_total;
  d.bucket_n = geo.bucket_n;
  d.part2 = reinterpret_cast<nf::Partial*>(w + lay.part2);
  d.part2_ne = reinterpret_cast<uint64_t*>(w + lay.ne2);
  d.W = geo.W;
  d.slots = geo.slots;
  d.tile = geo.tile;
  d.G = geo.G;
  d.gs = geo.gs;
  d.groups = geo.groups;
  d.btab = btab;
  e = nf::launch_decide(geo, d, s);
  if (e != hipSuccess) return hip_fail(e, "decide launch");
  if (phases) record_phase(2, s);
  return NF_OK;
}

// Pass-2 arguments for the buckets of a flat buffer.
nf::Pass2Args pass2_args(const nf::Geometry& geo) {
  nf::Pass2Args p;
  memset(&p, 0, sizeof p);
  p.n_total = geo.n_total;
  p.bucket_n = geo.bucket_n;
  p.W = geo.W;
  p.bpb2 = geo.bpb2;
  return p;
}

// Checks shared by the flat-buffer drivers (equal buckets or a table).
nf_status check_route_args(const float* g, int64_t stride, int32_t W, int64_t n_total, const uint64_t* mask,
                           const nf_route_policy* pol, float* out, nf_worker_stats* stats,
                           nf_route_decision* dec) {
  NF_TRY(check_grads(g, stride, W, n_total));
  NF_TRY(check_mask(mask, n_total));
  NF_TRY(check_policy(pol));
  if (n_total > 0 && !out) return fail(NF_ERR_INVALID_ARG, "out is NULL");
  if (!aligned(out, 4)) return fail(NF_ERR_ALIGNMENT, "out not 4-byte aligned");
  if (!stats || !dec) return fail(NF_ERR_INVALID_ARG, "stats and decision are required");
  if (!aligned(stats, 8) || !aligned(dec, 8)) return fail(NF_ERR_ALIGNMENT, "stats/decision not 8-byte aligned");
  return NF_OK;
}

// The route over every bucket of a geometry (checked arguments).
nf_status route_geo(const nf::Geometry& geo, const float* g, int64_t stride, int32_t W, const uint64_t* mask,
                    const nf_route_policy* pol, uint64_t* bits, int64_t bstride, uint8_t* counts, float* out,
                    nf_worker_stats* stats, nf_route_decision* dec, void* ws, size_t ws_bytes, void* stream,
                    const nf::BucketRow* btab, const int32_t* cbucket) {
  const int64_t n_total = geo.n_total;
  // pass 2 and the G-Ternary count run a grid row per bucket
  if (geo.nb > kMaxBuckets)
    return fail(NF_ERR_INVALID_ARG, "%lld buckets, at most %d per call", (long long)geo.nb, kMaxBuckets);
  NF_TRY(check_ws(ws, ws_bytes, nf::workspace_layout(geo).total));
  // The policy alone fixes the route when low-bit is not admitted, vetoed
  // or guard-rejected (and not forced): then no sign payload is built and
  // pass 1 writes the FP32 sums at every position.
  const bool predecided = !pol->admitted || (!pol->force_lowbit && (pol->veto || !pol->guard_ok));
  const bool ternary = pol->format == NF_FORMAT_TERNARY;
  if (!predecided) NF_TRY(check_bits(bits, bstride, n_total, W));
  hipStream_t s = static_cast<hipStream_t>(stream);
  // The G-Ternary payload needs each worker's threshold, known only once the
  // bucket has been read: pass 1 then builds no sign payload.
  NF_TRY(run_pass1_decide(geo, g, stride, mask, (predecided || ternary) ? nullptr : bits, bstride, out,
                          predecided ? nf::kSumsAll : nf::kSumsRouted, pol->fp32_op == NF_FP32_MEAN,
                          stats, dec, pol, ws, s, true, btab, cbucket));
  if (predecided || n_total == 0) {
    record_phase(3, s);
    return ok();
  }
  if (ternary) {
    nf::TernArgs t;
    memset(&t, 0, sizeof t);
    t.g = g;
    t.wstride = stride;
    t.mask = mask;
    t.bits = bits;
    t.bstride = bstride;
    t.dec = dec;
    t.stats = stats;
    t.cpos = counts;
    t.cneg = counts ? counts + n_total : nullptr;
    t.out = out;
    t.tau = pol->tau;
    t.n_total = n_total;
    t.bucket_n = geo.bucket_n;
    t.W = W;
    t.decode_mode = pol->decode_mode;
    t.bpb2 = geo.bpb2;
    t.btab = btab;
    t.cbucket = cbucket;
    hipError_t e = nf::launch_ternary_pack(geo, t, s);
    if (e != hipSuccess) return hip_fail(e, "ternary pack launch");
    e = nf::launch_ternary_reduce(geo, t, s);
    if (e != hipSuccess) return hip_fail(e, "ternary reduce launch");
  }
  nf::Pass2Args p = pass2_args(geo);
  p.bits = bits;
  p.bstride = bstride;
  p.g = g;
  p.wstride = stride;
  p.mask = mask;
  p.dec = dec;
  p.counts = counts;
  p.out = out;
  p.op = ternary ? nf::kOpFallbackOnly : nf::kOpFromDecision;
  p.decode_mode = pol->decode_mode;
  p.mean = pol->fp32_op == NF_FP32_MEAN;
  p.btab = btab;
  hipError_t e = nf::launch_pass2(geo, p, s);
  if (e != hipSuccess) return hip_fail(e, "pass-2 launch");
  record_phase(3, s);
  return ok();
}

nf_status route_flat(const float* g, int64_t stride, int32_t W, int64_t n_total, int64_t bucket_n,
                     const uint64_t* mask, const nf_route_policy* pol, uint64_t* bits,
                     int64_t bstride, uint8_t* counts, float* out, nf_worker_stats* stats,
                     nf_route_decision* dec, void* ws, size_t ws_bytes, void* stream) {
  NF_TRY(check_route_args(g, stride, W, n_total, mask, pol, out, stats, dec));
  const nf::Geometry geo = nf::make_geometry(W, n_total, bucket_n);
  return route_geo(geo, g, stride, W, mask, pol, bits, bstride, counts, out, stats, dec, ws, ws_bytes, stream,
                   nullptr, nullptr);
}

// A bucket table's offsets: nb >= 1, off[0] = 0, strictly increasing, every
// bucket start a multiple of 64 (its bitmap words start at off[b] / 64).
nf_status check_table_offsets(const int64_t* off, int32_t nb) {
  if (nb < 1) return fail(NF_ERR_INVALID_ARG, "nb=%d: a bucket table needs at least one bucket", nb);
  if (nb > kMaxBuckets) return fail(NF_ERR_INVALID_ARG, "nb=%d buckets, at most %d", nb, kMaxBuckets);
  if (!off) return fail(NF_ERR_INVALID_ARG, "bucket_offsets is NULL");
  if (off[0] != 0) return fail(NF_ERR_INVALID_ARG, "bucket_offsets[0]=%lld, must be 0", (long long)off[0]);
  for (int32_t b = 0; b < nb; ++b) {
    if (off[b + 1] <= off[b])
      return fail(NF_ERR_INVALID_ARG, "bucket %d is empty or negative: offsets %lld, %lld", b, (long long)off[b],
                  (long long)off[b + 1]);
    if (off[b] % 64) return fail(NF_ERR_INVALID_ARG, "bucket %d starts at %lld, not a multiple of 64", b,
                                 (long long)off[b]);
  }
  return NF_OK;
}

}  // namespace

namespace nf {
nf_status set_error(nf_status st, const char* msg) {
  g_err = msg;
  return st;
}
}  // namespace nf

extern "C" {

int nf_abi_version(void) { return NF_ABI_VERSION; }

nf_status nf_set_phase_events(void* before_pass1, void* after_pass1, void* after_decide,
                              void* after_pass2) {
  g_phase_ev[0] = static_cast<hipEvent_t>(before_pass1);
  g_phase_ev[1] = static_cast<hipEvent_t>(after_pass1);
  g_phase_ev[2] = static_cast<hipEvent_t>(after_decide);
  g_phase_ev[3] = static_cast<hipEvent_t>(after_pass2);
  return ok();
}

int64_t nf_pass1_launches(int32_t W, int64_t n_total, int64_t bucket_n, int32_t sign_words) {
  if (W < 1 || W > 255 || n_total <= 0 || bucket_n <= 0) return 0;
  const nf::Geometry geo = nf::make_geometry(W, n_total, bucket_n);
  return geo.ngroups * nf::ceil_div(geo.total_chunks, nf::pass1_launch_chunks(geo, sign_words != 0));
}

int64_t nf_pass1_chunk_elems(int32_t W, int64_t n_total, int64_t bucket_n, int64_t* chunks_per_bucket) {
  if (W < 1 || W > 255 || n_total <= 0 || bucket_n <= 0) return 0;
  const nf::Geometry geo = nf::make_geometry(W, n_total, bucket_n);
  if (chunks_per_bucket) *chunks_per_bucket = geo.chunks_full;
  return (int64_t)geo.tile * geo.G;
}

const char* nf_last_error(void) { return g_err.c_str(); }

nf_status nf_mask_from_segments(const int64_t* off_host, const int64_t* len_host,
                                const uint8_t* eligible_host, int64_t nseg, int64_t n,
                                uint64_t* mask_host) {
  if (n < 0 || nseg < 0) return fail(NF_ERR_INVALID_ARG, "negative n or nseg");
  if (nseg > 0 && (!off_host || !len_host || !eligible_host))
    return fail(NF_ERR_INVALID_ARG, "segment arrays are NULL");
  const int64_t nw = (n + 63) / 64;
  if (nw > 0 && !mask_host) return fail(NF_ERR_INVALID_ARG, "mask_host is NULL");
  for (int64_t s = 0; s < nseg; ++s)
    if (off_host[s] < 0 || len_host[s] < 0 || off_host[s] > n - len_host[s])
      return fail(NF_ERR_INVALID_ARG, "segment %lld [%lld, +%lld) outside [0, %lld)", (long long)s,
                  (long long)off_host[s], (long long)len_host[s], (long long)n);
  memset(mask_host, 0, (size_t)nw * sizeof(uint64_t));
  for (int64_t s = 0; s < nseg; ++s) {
    if (!eligible_host[s] || len_host[s] == 0) continue;
    int64_t lo = off_host[s], hi = off_host[s] + len_host[s];  // [lo, hi)
    int64_t wlo = lo >> 6, whi = (hi - 1) >> 6;
    for (int64_t k = wlo; k <= whi; ++k) {
      int64_t a = k == wlo ? (lo & 63) : 0;
      int64_t b = k == whi ? ((hi - 1) & 63) : 63;  // inclusive
      uint64_t m = (b == 63 ? ~0ull : ((1ull << (b + 1)) - 1ull)) & ~((1ull << a) - 1ull);
      mask_host[k] |= m;
    }
  }
  return ok();
}

size_t nf_workspace_bytes(int32_t W, int64_t n) {
  if (W < 1 || W > 255 || n < 0) return 0;
  return nf::workspace_layout(nf::make_geometry(W, n, n > 0 ? n : 1)).total;
}

size_t nf_workspace_bytes_buckets(int32_t W, int64_t n_total, int64_t bucket_n) {
  if (W < 1 || W > 255 || n_total < 0 || bucket_n <= 0) return 0;
  return nf::workspace_layout(nf::make_geometry(W, n_total, bucket_n)).total;
}

nf_status nf_bucket_health(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                           const uint64_t* mask, nf_worker_stats* stats, void* ws,
                           size_t ws_bytes, void* stream) {
  NF_TRY(check_grads(grads, worker_stride, W, n));
  NF_TRY(check_mask(mask, n));
  if (!stats) return fail(NF_ERR_INVALID_ARG, "stats is NULL");
  if (!aligned(stats, 8)) return fail(NF_ERR_ALIGNMENT, "stats not 8-byte aligned");
  const nf::Geometry geo = nf::make_geometry(W, n, n > 0 ? n : 1);
  NF_TRY(check_ws(ws, ws_bytes, nf::workspace_layout(geo).total));
  NF_TRY(run_pass1_decide(geo, grads, worker_stride, mask, nullptr, 0, nullptr, nf::kSumsNone, 0,
                          stats, nullptr, nullptr, ws, static_cast<hipStream_t>(stream)));
  return ok();
}

nf_status nf_pack_signs(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                        const uint64_t* mask, uint64_t* bits, int64_t bits_stride_words,
                        nf_worker_stats* stats, void* ws, size_t ws_bytes, void* stream) {
  NF_TRY(check_grads(grads, worker_stride, W, n));
  NF_TRY(check_mask(mask, n));
  NF_TRY(check_bits(bits, bits_stride_words, n, W));
  if (!aligned(stats, 8)) return fail(NF_ERR_ALIGNMENT, "stats not 8-byte aligned");
  const nf::Geometry geo = nf::make_geometry(W, n, n > 0 ? n : 1);
  NF_TRY(check_ws(ws, ws_bytes, nf::workspace_layout(geo).total));
  if (n == 0 && !stats) return ok();
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (stats) {
    NF_TRY(run_pass1_decide(geo, grads, worker_stride, mask, bits, bits_stride_words, nullptr,
                            nf::kSumsNone, 0, stats, nullptr, nullptr, ws, s));
  } else {
    const nf::WorkspaceLayout lay = nf::workspace_layout(geo);
    char* w = static_cast<char*>(ws);
    nf::Pass1Args a;
    a.g = grads;
    a.wstride = worker_stride;
    a.mask = mask;
    a.bits = bits;
    a.bstride = bits_stride_words;
    a.out = nullptr;
    a.part = reinterpret_cast<nf::Partial*>(w + lay.partials);
    a.part_ne = reinterpret_cast<uint64_t*>(w + lay.ne);
    fill_pass1_geometry(geo, &a);
    a.sums = nf::kSumsNone;
    a.mean = 0;
    hipError_t e = nf::launch_pass1(geo, a, s);
    if (e != hipSuccess) return hip_fail(e, "pass-1 launch");
  }
  return ok();
}

nf_status nf_fp32_reduce(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                         const uint64_t* mask, int32_t select, int32_t fp32_op, float* out,
                         void* stream) {
  NF_TRY(check_grads(grads, worker_stride, W, n));
  if (select != NF_SEL_ROUTED && select != NF_SEL_ELIGIBLE && select != NF_SEL_ALL)
    return fail(NF_ERR_INVALID_ARG, "select=%d", select);
  if (fp32_op != NF_FP32_SUM && fp32_op != NF_FP32_MEAN) return fail(NF_ERR_INVALID_ARG, "fp32_op=%d", fp32_op);
  if (select != NF_SEL_ALL) NF_TRY(check_mask(mask, n));
  if (n > 0 && !out) return fail(NF_ERR_INVALID_ARG, "out is NULL");
  if (!aligned(out, 4)) return fail(NF_ERR_ALIGNMENT, "out not 4-byte aligned");
  if (n == 0) return ok();
  const nf::Geometry geo = nf::make_geometry(W, n, n);
  nf::Pass2Args p = pass2_args(geo);
  p.g = grads;
  p.wstride = worker_stride;
  p.mask = select == NF_SEL_ALL ? nullptr : mask;
  p.out = out;
  p.op = nf::kOpFp32;
  p.select = select;
  p.mean = fp32_op == NF_FP32_MEAN;
  hipError_t e = nf::launch_pass2(geo, p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "fp32 launch");
  return ok();
}

nf_status nf_signcount_reduce(const uint64_t* bits, int64_t bits_stride_words, int32_t W, int64_t n,
                              const uint64_t* mask, const float* scale_dev, int32_t decode_mode,
                              uint8_t* counts, float* out, void* stream) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (n < 0) return fail(NF_ERR_INVALID_ARG, "n < 0");
  NF_TRY(check_bits(bits, bits_stride_words, n, W));
  if (decode_mode != NF_DECODE_SOFT && decode_mode != NF_DECODE_MAJORITY)
    return fail(NF_ERR_INVALID_ARG, "decode_mode=%d", decode_mode);
  if (out) {
    NF_TRY(check_mask(mask, n));
    if (!scale_dev) return fail(NF_ERR_INVALID_ARG, "scale_dev is NULL");
    if (!aligned(out, 4) || !aligned(scale_dev, 4)) return fail(NF_ERR_ALIGNMENT, "out/scale not 4-byte aligned");
  }
  if (n == 0 || (!out && !counts)) return ok();
  const nf::Geometry geo = nf::make_geometry(W, n, n);
  nf::Pass2Args p = pass2_args(geo);
  p.bits = bits;
  p.bstride = bits_stride_words;
  p.mask = mask;
  p.scale = scale_dev;
  p.counts = counts;
  p.out = out;
  p.op = nf::kOpCountDecode;
  p.decode_mode = decode_mode;
  hipError_t e = nf::launch_pass2(geo, p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "signcount launch");
  return ok();
}

nf_status nf_partial_counts(const uint64_t* bits, int64_t bits_stride_words, int32_t W, int32_t P,
                            int64_t n, uint8_t* partial, int64_t partial_stride, void* stream) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (P < 1 || P > W || W % P) return fail(NF_ERR_INVALID_ARG, "P=%d must divide W=%d", P, W);
  if (n < 0) return fail(NF_ERR_INVALID_ARG, "n < 0");
  NF_TRY(check_bits(bits, bits_stride_words, n, W));
  if (n > 0 && !partial) return fail(NF_ERR_INVALID_ARG, "partial is NULL");
  if (partial_stride < n) return fail(NF_ERR_INVALID_ARG, "partial_stride < n");
  if (n == 0) return ok();
  const nf::Geometry geo = nf::make_geometry(P, n, n);
  nf::Pass2Args p = pass2_args(geo);
  p.bits = bits;
  p.bstride = bits_stride_words;
  p.counts = partial;
  p.op = nf::kOpCountDecode;
  p.nz = W / P;
  p.z_rows = P;
  p.z_counts = partial_stride;
  hipError_t e = nf::launch_pass2(geo, p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "partial-count launch");
  return ok();
}

nf_status nf_partial_count_reduce(const uint8_t* partial, int64_t partial_stride, int32_t G, int32_t W,
                                  int64_t n, const uint64_t* mask, const float* scale_dev,
                                  int32_t decode_mode, uint8_t* counts, float* out, void* stream) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (G < 1 || G > W || W % G) return fail(NF_ERR_INVALID_ARG, "G=%d must divide W=%d", G, W);
  if (n < 0) return fail(NF_ERR_INVALID_ARG, "n < 0");
  if (n > 0 && !partial) return fail(NF_ERR_INVALID_ARG, "partial is NULL");
  if (partial_stride < n) return fail(NF_ERR_INVALID_ARG, "partial_stride < n");
  if (!aligned(partial, 16) || partial_stride % 16)
    return fail(NF_ERR_ALIGNMENT, "partial must be 16-byte aligned with a stride that is a multiple of 16");
  if (decode_mode != NF_DECODE_SOFT && decode_mode != NF_DECODE_MAJORITY)
    return fail(NF_ERR_INVALID_ARG, "decode_mode=%d", decode_mode);
  if (out) {
    NF_TRY(check_mask(mask, n));
    if (!scale_dev) return fail(NF_ERR_INVALID_ARG, "scale_dev is NULL");
    if (!aligned(out, 4) || !aligned(scale_dev, 4)) return fail(NF_ERR_ALIGNMENT, "out/scale not 4-byte aligned");
  }
  if (n == 0 || (!out && !counts)) return ok();
  nf::PsumArgs a;
  a.partial = partial;
  a.pstride = partial_stride;
  a.mask = mask;
  a.scale = scale_dev;
  a.counts = counts;
  a.out = out;
  a.n = n;
  a.G = G;
  a.W = W;
  a.decode_mode = decode_mode;
  hipError_t e = nf::launch_psum(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "partial-count reduce launch");
  return ok();
}

nf_status nf_stock_signcount(const uint64_t* bits, int64_t bits_stride_words, int32_t W, int64_t n,
                             const uint64_t* mask, const float* scale_dev, int32_t decode_mode,
                             int32_t replicas, uint8_t* counts, float* out, int64_t replica_stride,
                             void* stream) {
  if (replicas < 1 || replicas > 65535) return fail(NF_ERR_INVALID_ARG, "replicas=%d outside [1, 65535]", replicas);
  if (replica_stride < n) return fail(NF_ERR_INVALID_ARG, "replica_stride < n");
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (n < 0) return fail(NF_ERR_INVALID_ARG, "n < 0");
  NF_TRY(check_bits(bits, bits_stride_words, n, W));
  if (decode_mode != NF_DECODE_SOFT && decode_mode != NF_DECODE_MAJORITY)
    return fail(NF_ERR_INVALID_ARG, "decode_mode=%d", decode_mode);
  if (out) {
    NF_TRY(check_mask(mask, n));
    if (!scale_dev) return fail(NF_ERR_INVALID_ARG, "scale_dev is NULL");
    if (!aligned(out, 4) || !aligned(scale_dev, 4)) return fail(NF_ERR_ALIGNMENT, "out/scale not 4-byte aligned");
  }
  if (n == 0 || (!out && !counts)) return ok();
  const nf::Geometry geo = nf::make_geometry(W, n, n);
  nf::Pass2Args p = pass2_args(geo);
  p.bits = bits;
  p.bstride = bits_stride_words;
  p.mask = mask;
  p.scale = scale_dev;
  p.counts = counts;
  p.out = out;
  p.op = nf::kOpCountDecode;
  p.decode_mode = decode_mode;
  p.nz = replicas;
  p.z_rows = 0;
  p.z_counts = replica_stride;
  p.z_out = replica_stride;
  hipError_t e = nf::launch_pass2(geo, p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "stock signcount launch");
  return ok();
}

nf_status nf_sliced_layout_sizes(const int64_t* len_host, int64_t S, int64_t* n_eligible_host,
                                 int64_t* segments_host) {
  if (S < 0 || (S > 0 && !len_host) || !n_eligible_host || !segments_host)
    return fail(NF_ERR_INVALID_ARG, "S < 0 or NULL arrays");
  int64_t ne = 0, seg = 0;
  for (int64_t s = 0; s < S; ++s) {
    if (len_host[s] < 1) return fail(NF_ERR_INVALID_ARG, "slice %lld has length < 1", (long long)s);
    ne += len_host[s];
    seg += nf::ceil_div(len_host[s], nf::kSliceSeg);
  }
  *n_eligible_host = ne;
  *segments_host = seg;
  return ok();
}

nf_status nf_sliced_layout(const int64_t* off_host, const int64_t* len_host, int64_t S, int64_t n,
                           uint64_t* mask_host, uint64_t* prefix_host, int64_t* start_host,
                           int32_t* wslice_host, int64_t* rstart_host, int64_t* segp_host) {
  if (S < 0 || n < 0) return fail(NF_ERR_INVALID_ARG, "negative S or n");
  if (S > 0 && (!off_host || !len_host)) return fail(NF_ERR_INVALID_ARG, "slice arrays are NULL");
  if (S >= (int64_t)1 << 31) return fail(NF_ERR_INVALID_ARG, "too many slices");
  const int64_t nw = (n + 63) / 64;
  if (!prefix_host || !rstart_host || !segp_host || (nw > 0 && (!mask_host || !wslice_host)) ||
      (S > 0 && !start_host))
    return fail(NF_ERR_INVALID_ARG, "output arrays are NULL");
  int64_t end = 0;
  for (int64_t s = 0; s < S; ++s) {
    if (len_host[s] < 1 || off_host[s] < end || off_host[s] > n - len_host[s])
      return fail(NF_ERR_INVALID_ARG, "slice %lld [%lld, +%lld): slices must be sorted, disjoint, non-empty, inside [0, %lld)",
                  (long long)s, (long long)off_host[s], (long long)len_host[s], (long long)n);
    end = off_host[s] + len_host[s];
  }
  // mask: the union of the slices
  memset(mask_host, 0, (size_t)nw * sizeof(uint64_t));
  for (int64_t s = 0; s < S; ++s)
    for (int64_t i = off_host[s]; i < off_host[s] + len_host[s];) {
      const int64_t k = i / 64, b = i % 64;
      const int64_t take = (64 - b) < (off_host[s] + len_host[s] - i) ? (64 - b) : (off_host[s] + len_host[s] - i);
      mask_host[k] |= (take == 64 ? ~0ull : ((1ull << take) - 1ull)) << b;
      i += take;
    }
  // eligible elements before each word, and the word holding every 64th rank
  uint64_t acc = 0;
  int64_t o = 0;
  for (int64_t k = 0; k < nw; ++k) {
    prefix_host[k] = acc;
    const uint64_t next = acc + (uint64_t)__builtin_popcountll(mask_host[k]);
    for (; (uint64_t)(64 * o) < next; ++o) start_host[o] = k;
    acc = next;
  }
  prefix_host[nw] = acc;
  // slice of each word's first eligible element
  int64_t s = 0;
  for (int64_t k = 0; k < nw; ++k) {
    while (s < S && off_host[s] + len_host[s] <= 64 * k) ++s;
    wslice_host[k] = (int32_t)((s < S && off_host[s] < 64 * (k + 1)) ? s : S);
  }
  // compacted start of each slice and its first statistics segment
  rstart_host[0] = 0;
  segp_host[0] = 0;
  for (int64_t t = 0; t < S; ++t) {
    rstart_host[t + 1] = rstart_host[t] + len_host[t];
    segp_host[t + 1] = segp_host[t] + nf::ceil_div(len_host[t], nf::kSliceSeg);
  }
  return ok();
}

nf_status nf_compact_signs(const uint64_t* bits, int64_t bits_stride_words, int32_t W, int64_t n,
                           const uint64_t* mask, const uint64_t* prefix, const int64_t* start,
                           int64_t n_eligible, uint64_t* cbits, int64_t cbits_stride_words,
                           void* stream) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (n < 0 || n_eligible < 0 || n_eligible > n) return fail(NF_ERR_INVALID_ARG, "need 0 <= n_eligible <= n");
  NF_TRY(check_bits(bits, bits_stride_words, n, W));
  NF_TRY(check_mask(mask, n));
  if (n_eligible > 0 && (!prefix || !start || !cbits)) return fail(NF_ERR_INVALID_ARG, "NULL layout table or output");
  if (!aligned(cbits, 8) || !aligned(prefix, 8) || !aligned(start, 8)) return fail(NF_ERR_ALIGNMENT, "8-byte alignment");
  if (cbits_stride_words < (n_eligible + 63) / 64) return fail(NF_ERR_INVALID_ARG, "cbits_stride_words < ceil(n_E/64)");
  if (n_eligible == 0) return ok();
  nf::CompactArgs a;
  a.bits = bits;
  a.bstride = bits_stride_words;
  a.mask = mask;
  a.prefix = prefix;
  a.start = start;
  a.cbits = cbits;
  a.cstride = cbits_stride_words;
  a.n = n;
  a.n_eligible = n_eligible;
  hipError_t e = nf::launch_compact(a, W, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "compact launch");
  return ok();
}

size_t nf_slice_workspace_bytes(int32_t W, int64_t segments) {
  if (W < 1 || W > 255 || segments < 0) return 0;
  return nf::align256((size_t)segments * (size_t)W * sizeof(double));
}

nf_status nf_slice_scales(const float* grads, int64_t worker_stride, int32_t W, const int64_t* off,
                          const int64_t* len, const int64_t* segp, int64_t S, int64_t segments,
                          double* sums, float* scales, void* ws, size_t ws_bytes, void* stream) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (S < 0 || segments < S || segments > 0x7fffffff) return fail(NF_ERR_INVALID_ARG, "need 0 <= S <= segments < 2^31");
  if (S == 0) return ok();
  if (!grads || !off || !len || !segp || !sums || !scales) return fail(NF_ERR_INVALID_ARG, "NULL argument");
  if (!aligned(grads, 4) || !aligned(sums, 8) || !aligned(scales, 4) || !aligned(off, 8) || !aligned(len, 8) ||
      !aligned(segp, 8))
    return fail(NF_ERR_ALIGNMENT, "misaligned argument");
  NF_TRY(check_ws(ws, ws_bytes, nf_slice_workspace_bytes(W, segments)));
  nf::SliceArgs a;
  a.g = grads;
  a.wstride = worker_stride;
  a.off = off;
  a.len = len;
  a.segp = segp;
  a.part = static_cast<double*>(ws);
  a.sums = sums;
  a.scales = scales;
  a.S = S;
  a.W = W;
  hipError_t e = nf::launch_slice_scales(a, segments, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "slice scale launch");
  return ok();
}

nf_status nf_slice_scales_from_pass1(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                                     const int64_t* off, const int64_t* len, int64_t S, double* sums,
                                     float* scales, const void* ws, size_t ws_bytes, void* stream) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (n < 0 || S < 0 || S > n || S > 0x7fffffff) return fail(NF_ERR_INVALID_ARG, "need 0 <= S <= n, S < 2^31");
  if (worker_stride < n) return fail(NF_ERR_INVALID_ARG, "worker_stride %lld < n %lld", (long long)worker_stride,
                                     (long long)n);
  if (S == 0) return ok();
  if (!grads || !off || !len || !sums || !scales) return fail(NF_ERR_INVALID_ARG, "NULL argument");
  if (!aligned(grads, 4) || !aligned(sums, 8) || !aligned(scales, 4) || !aligned(off, 8) || !aligned(len, 8))
    return fail(NF_ERR_ALIGNMENT, "misaligned argument");
  const nf::Geometry geo = nf::make_geometry(W, n, n);
  const nf::WorkspaceLayout lay = nf::workspace_layout(geo);
  NF_TRY(check_ws(ws, ws_bytes, lay.total));
  nf::SliceChunkArgs a;
  a.g = grads;
  a.wstride = worker_stride;
  a.part = reinterpret_cast<const nf::Partial*>(static_cast<const char*>(ws) + lay.partials);
  a.off = off;
  a.len = len;
  a.sums = sums;
  a.scales = scales;
  a.S = S;
  a.CH = (int64_t)geo.G * geo.tile;
  a.W = W;
  hipError_t e = nf::launch_slice_chunks(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "slice statistics launch");
  return ok();
}

nf_status nf_compact_signcount_reduce(const uint64_t* cbits, int64_t cbits_stride_words, int32_t W,
                                      int64_t n, const uint64_t* mask, const uint64_t* prefix,
                                      const int32_t* wslice, const int64_t* rstart, int64_t S,
                                      int64_t n_eligible, const float* scales, int32_t decode_mode,
                                      uint8_t* counts_c, float* out, void* stream) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (n < 0 || n_eligible < 0 || n_eligible > n || S < 0) return fail(NF_ERR_INVALID_ARG, "need 0 <= n_eligible <= n, S >= 0");
  if (decode_mode != NF_DECODE_SOFT && decode_mode != NF_DECODE_MAJORITY)
    return fail(NF_ERR_INVALID_ARG, "decode_mode=%d", decode_mode);
  if (n_eligible == 0) return ok();
  NF_TRY(check_bits(cbits, cbits_stride_words, n_eligible, W));
  if (!counts_c) return fail(NF_ERR_INVALID_ARG, "counts_c is NULL");
  if (!aligned(counts_c, 4)) return fail(NF_ERR_ALIGNMENT, "counts_c not 4-byte aligned");
  if (out) {
    NF_TRY(check_mask(mask, n));
    if (S < 1 || !prefix || !wslice || !rstart || !scales) return fail(NF_ERR_INVALID_ARG, "NULL layout table or scales");
    if (!aligned(out, 4) || !aligned(prefix, 8) || !aligned(rstart, 8) || !aligned(wslice, 4) || !aligned(scales, 4))
      return fail(NF_ERR_ALIGNMENT, "misaligned argument");
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const nf::Geometry geo = nf::make_geometry(W, n_eligible, n_eligible);
  nf::Pass2Args p = pass2_args(geo);
  p.bits = cbits;
  p.bstride = cbits_stride_words;
  p.counts = counts_c;
  p.op = nf::kOpCountDecode;
  hipError_t e = nf::launch_pass2(geo, p, s);
  if (e != hipSuccess) return hip_fail(e, "compacted count launch");
  if (!out) return ok();
  nf::ExpandArgs x;
  x.mask = mask;
  x.prefix = prefix;
  x.wslice = wslice;
  x.rstart = rstart;
  x.scales = scales;
  x.counts_c = counts_c;
  x.out = out;
  x.n = n;
  x.S = S;
  x.n_eligible = n_eligible;
  x.W = W;
  x.decode_mode = decode_mode;
  e = nf::launch_cexpand(x, s);
  if (e != hipSuccess) return hip_fail(e, "sliced decode launch");
  return ok();
}

nf_status nf_ternary_threshold(const nf_worker_stats* stats_host, int32_t W, int64_t n_eligible,
                               float tau, float* theta_host) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (n_eligible < 0) return fail(NF_ERR_INVALID_ARG, "n_eligible < 0");
  if (!stats_host || !theta_host) return fail(NF_ERR_INVALID_ARG, "NULL stats or theta");
  if (!(tau >= 0.0f && tau - tau == 0.0f)) return fail(NF_ERR_INVALID_ARG, "tau must be finite and >= 0");
  for (int w = 0; w < W; ++w) theta_host[w] = nf::ternary_threshold(stats_host[w], n_eligible, tau);
  return ok();
}

nf_status nf_pack_ternary(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                          const uint64_t* mask, const float* theta_dev, uint64_t* bits,
                          int64_t bits_stride_words, void* stream) {
  NF_TRY(check_grads(grads, worker_stride, W, n));
  NF_TRY(check_mask(mask, n));
  NF_TRY(check_bits(bits, bits_stride_words, n, W));
  if (n > 0 && !theta_dev) return fail(NF_ERR_INVALID_ARG, "theta_dev is NULL");
  if (!aligned(theta_dev, 4)) return fail(NF_ERR_ALIGNMENT, "theta not 4-byte aligned");
  if (n == 0) return ok();
  const nf::Geometry geo = nf::make_geometry(W, n, n);
  nf::TernArgs t;
  memset(&t, 0, sizeof t);
  t.g = grads;
  t.wstride = worker_stride;
  t.mask = mask;
  t.bits = bits;
  t.bstride = bits_stride_words;
  t.theta = theta_dev;
  t.n_total = n;
  t.bucket_n = n;
  t.W = W;
  t.bpb2 = geo.bpb2;
  hipError_t e = nf::launch_ternary_pack(geo, t, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "ternary pack launch");
  return ok();
}

nf_status nf_ternary_reduce(const uint64_t* bits, int64_t bits_stride_words, int32_t W, int64_t n,
                            const uint64_t* mask, const float* scale_dev, int32_t decode_mode,
                            uint8_t* counts, float* out, void* stream) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (n < 0) return fail(NF_ERR_INVALID_ARG, "n < 0");
  NF_TRY(check_bits(bits, bits_stride_words, n, W));
  if (decode_mode != NF_DECODE_SOFT && decode_mode != NF_DECODE_MAJORITY)
    return fail(NF_ERR_INVALID_ARG, "decode_mode=%d", decode_mode);
  if (out) {
    NF_TRY(check_mask(mask, n));
    if (!scale_dev) return fail(NF_ERR_INVALID_ARG, "scale_dev is NULL");
    if (!aligned(out, 4) || !aligned(scale_dev, 4)) return fail(NF_ERR_ALIGNMENT, "out/scale not 4-byte aligned");
  }
  if (n == 0 || (!out && !counts)) return ok();
  const nf::Geometry geo = nf::make_geometry(W, n, n);
  nf::TernArgs t;
  memset(&t, 0, sizeof t);
  t.mask = mask;
  t.bits = const_cast<uint64_t*>(bits);
  t.bstride = bits_stride_words;
  t.scale = scale_dev;
  t.cpos = counts;
  t.cneg = counts ? counts + n : nullptr;
  t.out = out;
  t.n_total = n;
  t.bucket_n = n;
  t.W = W;
  t.decode_mode = decode_mode;
  t.bpb2 = geo.bpb2;
  hipError_t e = nf::launch_ternary_reduce(geo, t, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "ternary reduce launch");
  return ok();
}

nf_status nf_route_decide(const nf_worker_stats* stats_host, int32_t W, int64_t n, int64_t n_eligible,
                          const nf_route_policy* policy_host, nf_route_decision* decision_host) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (n < 0 || n_eligible < 0 || n_eligible > n) return fail(NF_ERR_INVALID_ARG, "need 0 <= n_eligible <= n");
  if (!stats_host || !decision_host) return fail(NF_ERR_INVALID_ARG, "NULL stats or decision");
  NF_TRY(check_policy(policy_host));
  int k = 0;
  for (int w = 0; w < W; ++w) k += nf::finite64(stats_host[w].sum_sq) ? 1 : 0;
  double med = 0.0;
  for (int w = 0; w < W; ++w)
    if (nf::finite64(stats_host[w].sum_sq) && nf::ssq_rank(stats_host, W, w) == (k - 1) / 2)
      med = stats_host[w].sum_sq;
  nf::decide_from(stats_host, W, n, n_eligible, *policy_host, k, med, decision_host);
  return ok();
}

nf_status nf_route_bucket(const float* grads, int64_t worker_stride, int32_t W, int64_t n,
                          const uint64_t* mask, const nf_route_policy* policy_host, uint64_t* bits,
                          int64_t bits_stride_words, uint8_t* counts, float* out,
                          nf_worker_stats* stats, nf_route_decision* decision, void* ws,
                          size_t ws_bytes, void* stream) {
  return route_flat(grads, worker_stride, W, n, n > 0 ? n : 1, mask, policy_host, bits,
                    bits_stride_words, counts, out, stats, decision, ws, ws_bytes, stream);
}

nf_status nf_route_buckets(const float* grads, int64_t worker_stride, int32_t W, int64_t n_total,
                           int64_t bucket_n, const uint64_t* mask, const nf_route_policy* policy_host,
                           uint64_t* bits, int64_t bits_stride_words, uint8_t* counts, float* out,
                           nf_worker_stats* stats, nf_route_decision* decisions, void* ws,
                           size_t ws_bytes, void* stream) {
  if (bucket_n <= 0) return fail(NF_ERR_INVALID_ARG, "bucket_n must be > 0");
  if (bucket_n < n_total && bucket_n % 64)
    return fail(NF_ERR_INVALID_ARG, "bucket_n=%lld must be a multiple of 64", (long long)bucket_n);
  return route_flat(grads, worker_stride, W, n_total, bucket_n, mask, policy_host, bits,
                    bits_stride_words, counts, out, stats, decisions, ws, ws_bytes, stream);
}

nf_status nf_route_buckets_noalloc(const float* grads, int64_t worker_stride, int32_t W,
                                   int64_t n_total, int64_t bucket_n, const uint64_t* mask,
                                   const nf_route_policy* policy_host, uint64_t* bits,
                                   int64_t bits_stride_words, uint8_t* counts, float* out,
                                   nf_worker_stats* stats, nf_route_decision* decisions,
                                   void* stream) {
  if (bucket_n <= 0) return fail(NF_ERR_INVALID_ARG, "bucket_n must be > 0");
  if (bucket_n < n_total && bucket_n % 64)
    return fail(NF_ERR_INVALID_ARG, "bucket_n=%lld must be a multiple of 64", (long long)bucket_n);
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  if (n_total < 0) return fail(NF_ERR_INVALID_ARG, "n_total < 0");
  const size_t need = nf::workspace_layout(nf::make_geometry(W, n_total, bucket_n)).total;
  if (need > kStaticScratchBytes)
    return fail(NF_ERR_WORKSPACE, "W=%d, n_total=%lld, bucket_n=%lld needs %zu bytes of scratch, above the "
                "static %zu", W, (long long)n_total, (long long)bucket_n, need, kStaticScratchBytes);
  void* ws = nullptr;
  NF_TRY(scratch_address(&ws));
  return route_flat(grads, worker_stride, W, n_total, bucket_n, mask, policy_host, bits,
                    bits_stride_words, counts, out, stats, decisions, ws, kStaticScratchBytes, stream);
}

size_t nf_bucket_table_bytes(int32_t W, const int64_t* bucket_offsets, int32_t nb) {
  if (W < 1 || W > 255 || check_table_offsets(bucket_offsets, nb) != NF_OK) return 0;
  return nf::table_bytes(nf::make_geometry_table(W, bucket_offsets, nb));
}

nf_status nf_bucket_table_init(int32_t W, const int64_t* bucket_offsets, int32_t nb, void* table,
                               size_t table_bytes, void* stream) {
  if (W < 1 || W > 255) return fail(NF_ERR_INVALID_ARG, "W=%d outside [1, 255]", W);
  NF_TRY(check_table_offsets(bucket_offsets, nb));
  const nf::Geometry geo = nf::make_geometry_table(W, bucket_offsets, nb);
  const size_t need = nf::table_bytes(geo);
  if (table_bytes < need) return fail(NF_ERR_WORKSPACE, "table of %zu bytes < %zu required", table_bytes, need);
  if (!table) return fail(NF_ERR_INVALID_ARG, "table is NULL");
  if (!aligned(table, 256)) return fail(NF_ERR_ALIGNMENT, "table not 256-byte aligned");
  // Rows and the bucket of every chunk, built here and copied once (no
  // exception crosses the C ABI: a failed host allocation is an error code).
  std::vector<unsigned char> host;
  try {
    host.assign(need, 0);
  } catch (...) {
    return fail(NF_ERR_WORKSPACE, "no host memory for a %zu-byte table", need);
  }
  nf::BucketRow* rows = reinterpret_cast<nf::BucketRow*>(host.data());
  int32_t* cb = reinterpret_cast<int32_t*>(host.data() + nf::table_rows_bytes(nb));
  int64_t q = 0;
  for (int32_t b = 0; b < nb; ++b) {
    const int64_t len = bucket_offsets[b + 1] - bucket_offsets[b];
    const int64_t chunks = nf::ceil_div(nf::ceil_div(len, geo.tile), geo.G);
    rows[b].start = bucket_offsets[b];
    rows[b].len = len;
    rows[b].chunk0 = q;
    rows[b].pad = 0;
    for (int64_t c = 0; c < chunks; ++c) cb[q + c] = b;
    q += chunks;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(table, host.data(), need, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "bucket table copy");
  return ok();
}

int64_t nf_pass1_launches_table(int32_t W, const int64_t* bucket_offsets, int32_t nb, int32_t sign_words) {
  if (W < 1 || W > 255 || check_table_offsets(bucket_offsets, nb) != NF_OK) return 0;
  const nf::Geometry geo = nf::make_geometry_table(W, bucket_offsets, nb);
  return geo.ngroups * nf::ceil_div(geo.total_chunks, nf::pass1_launch_chunks(geo, sign_words != 0));
}

size_t nf_workspace_bytes_table(int32_t W, const int64_t* bucket_offsets, int32_t nb) {
  if (W < 1 || W > 255 || check_table_offsets(bucket_offsets, nb) != NF_OK) return 0;
  return nf::workspace_layout(nf::make_geometry_table(W, bucket_offsets, nb)).total;
}

nf_status nf_route_bucket_table(const float* grads, int64_t worker_stride, int32_t W,
                                const int64_t* bucket_offsets, int32_t nb, const void* table,
                                const uint64_t* mask, const nf_route_policy* policy_host, uint64_t* bits,
                                int64_t bits_stride_words, uint8_t* counts, float* out,
                                nf_worker_stats* stats, nf_route_decision* decisions, void* ws,
                                size_t ws_bytes, void* stream) {
  NF_TRY(check_table_offsets(bucket_offsets, nb));
  const int64_t n_total = bucket_offsets[nb];
  NF_TRY(check_route_args(grads, worker_stride, W, n_total, mask, policy_host, out, stats, decisions));
  if (!table) return fail(NF_ERR_INVALID_ARG, "table is NULL");
  if (!aligned(table, 256)) return fail(NF_ERR_ALIGNMENT, "table not 256-byte aligned");
  const nf::Geometry geo = nf::make_geometry_table(W, bucket_offsets, nb);
  const unsigned char* t = static_cast<const unsigned char*>(table);
  return route_geo(geo, grads, worker_stride, W, mask, policy_host, bits, bits_stride_words, counts, out, stats,
                   decisions, ws, ws_bytes, stream, reinterpret_cast<const nf::BucketRow*>(t),
                   reinterpret_cast<const int32_t*>(t + nf::table_rows_bytes(nb)));
}

}  // extern "C"
