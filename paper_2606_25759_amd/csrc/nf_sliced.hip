// nf_sliced.hip - per-slice scales and the compacted eligible-only payload.
//
//   k_compact     positional sign rows -> compacted rows: bit r of a row is
//                 the r-th eligible element's bit (the payload's wire form)
//   k_slice_part  per (statistics segment, worker): FP64 sum of |g| over the
//                 segment, one fixed-order block reduction
//   k_slice_scale per slice: the segments' sums in order, then the slice's
//                 mean-absolute scale (the bucket scale's rule on one slice)
//   k_cexpand     counts in compacted order -> decoded values at the
//                 elements' own positions, each with its slice's scale
//
// The counts over the compacted rows come from pass 2's bit-sliced counter
// (k_pass2), run on the compacted rows as on any payload.
#include "nf_internal.h"

namespace nf {

namespace {

constexpr int kThreadsS = 256;

__device__ __forceinline__ uint64_t uniform64(uint64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t low_mask(int64_t r) {
  return r >= 64 ? ~0ull : (r <= 0 ? 0ull : ((1ull << r) - 1ull));
}

// The bits of x at the positions of the set bits of m, packed towards bit 0
// in their order ("compress", the generalized extract of Hacker's Delight,
// §7-4): six rounds, each moving the bits that have an odd number of
// cleared mask bits to their right (in the current round's unit) down by
// that unit, found with a parallel-suffix XOR.
__device__ __forceinline__ uint64_t compress64(uint64_t x, uint64_t m) {
  if (m == ~0ull) return x;
  x &= m;
  uint64_t mk = ~m << 1;  // counts the cleared mask bits to the right
#pragma unroll
  for (int i = 0; i < 6; ++i) {
    uint64_t mp = mk ^ (mk << 1);
    mp ^= mp << 2;
    mp ^= mp << 4;
    mp ^= mp << 8;
    mp ^= mp << 16;
    mp ^= mp << 32;
    const uint64_t mv = mp & m;  // mask bits that move in this round
    m = (m ^ mv) | (mv >> (1 << i));
    const uint64_t t = x & mv;
    x = (x ^ t) | (t >> (1 << i));
    mk &= ~mp;
  }
  return x;
}

// Compacted word o of row w = blockIdx.y gathers ranks 64o .. 64o + 63: it
// starts at the positional word holding rank 64o (start[o]), skips the
// ranks of that word below 64o, and appends the compressed words that
// follow until 64 ranks (or n_E) are covered.  A lane takes four compacted
// words, so that their table and payload loads are in flight together.
constexpr int kCompactPerLane = 4;

__global__ __launch_bounds__(kThreadsS) void k_compact(CompactArgs a) {
  const int w = blockIdx.y;
  const uint64_t* row = a.bits + (int64_t)w * a.bstride;
  uint64_t* crow = a.cbits + (int64_t)w * a.cstride;
  const int64_t nwc = (a.n_eligible + 63) / 64;
  const int64_t nw = (a.n + 63) / 64;
  // a wavefront takes 64 * kCompactPerLane consecutive compacted words; lane l
  // takes words l, l + 64, ... of them, so each batch of loads is contiguous
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * (kThreadsS / 64) + (threadIdx.x >> 6);
  const int64_t waves = (int64_t)gridDim.x * (kThreadsS / 64);
  for (int64_t t0 = wave * 64 * kCompactPerLane; t0 < nwc; t0 += waves * 64 * kCompactPerLane) {
    const int64_t o0 = t0 + lane;
    int64_t k[kCompactPerLane];
    uint64_t pk[kCompactPerLane], m0[kCompactPerLane], x0[kCompactPerLane];
#pragma unroll
    for (int j = 0; j < kCompactPerLane; ++j) k[j] = o0 + 64 * j < nwc ? a.start[o0 + 64 * j] : 0;
#pragma unroll
    for (int j = 0; j < kCompactPerLane; ++j) {
      pk[j] = a.prefix[k[j]];
      m0[j] = a.mask[k[j]];
      x0[j] = row[k[j]];
    }
#pragma unroll
    for (int j = 0; j < kCompactPerLane; ++j) {
      const int64_t o = o0 + 64 * j;
      if (o >= nwc) break;
      const int64_t r0 = o * 64;
      const int need = (int)((a.n_eligible - r0) < 64 ? (a.n_eligible - r0) : 64);
      int64_t kk = k[j];
      int skip = (int)(r0 - (int64_t)pk[j]);
      uint64_t m = m0[j], x = x0[j];
      uint64_t acc = 0;
      int got = 0;
      while (true) {
        if (kk == nw - 1) m &= low_mask(a.n - 64 * kk);
        const int cnt = __popcll(m) - skip;
        if (cnt > 0) {
          const uint64_t e = compress64(x, m) >> skip;
          acc |= got < 64 ? e << got : 0ull;
          got += cnt;
        }
        skip = 0;
        if (got >= need || ++kk >= nw) break;
        m = a.mask[kk];
        x = row[kk];
      }
      crow[o] = acc & low_mask(need);
    }
  }
}

// Block (segment, worker): FP64 sum of |g| over the segment.  Thread t takes
// elements t, t + 256, ...; the 256 partial sums are added by a fixed tree.
__global__ __launch_bounds__(kThreadsS) void k_slice_part(SliceArgs a) {
  __shared__ double red[kThreadsS];
  const int64_t seg = blockIdx.x;
  const int w = blockIdx.y;
  // slice of this segment: the last s with segp[s] <= seg (uniform search)
  int64_t lo = 0, hi = a.S - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) / 2;
    if (a.segp[mid] <= seg) lo = mid;
    else hi = mid - 1;
  }
  const int64_t s = lo;
  const int64_t j = seg - a.segp[s];
  const int64_t b0 = j * kSliceSeg;
  const int64_t len = a.len[s];
  const int64_t b1 = (b0 + kSliceSeg < len) ? b0 + kSliceSeg : len;
  const float* row = a.g + (int64_t)w * a.wstride + a.off[s];
  // thread t adds elements t, t + 256, ... in order; eight loads are in flight at a time
  double t = 0.0;
  int64_t i = b0 + threadIdx.x;
  for (; i + 7 * kThreadsS < b1; i += 8 * kThreadsS) {
    float x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = __builtin_nontemporal_load(row + i + u * kThreadsS);
#pragma unroll
    for (int u = 0; u < 8; ++u) t += __builtin_fabs((double)x[u]);
  }
  for (; i < b1; i += kThreadsS) t += __builtin_fabs((double)__builtin_nontemporal_load(row + i));
  red[threadIdx.x] = t;
  __syncthreads();
  for (int h = kThreadsS / 2; h > 0; h >>= 1) {
    if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) a.part[seg * a.W + w] = red[0];
}

// Block s: worker sums of slice s (its segments in order), then
// scale_s = fl32((sum over workers, in order, of sum_w / len_s) / W).
__global__ __launch_bounds__(kThreadsS) void k_slice_scale(SliceArgs a) {
  const int64_t s = blockIdx.x;
  for (int w = threadIdx.x; w < a.W; w += kThreadsS) {
    double t = 0.0;
    for (int64_t seg = a.segp[s]; seg < a.segp[s + 1]; ++seg) t += a.part[seg * a.W + w];
    a.sums[s * a.W + w] = t;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double acc = 0.0;
    for (int w = 0; w < a.W; ++w) acc += a.sums[s * a.W + w] / (double)a.len[s];
    a.scales[s] = (float)(acc / (double)a.W);
  }
}

// A wavefront takes 64 consecutive positional words per task.  Lane t loads
// mask word k0 + t; a scan of the popcounts gives each word's first rank
// (prefix[k0] + the eligible elements of the task's earlier words), so the
// task loads one prefix entry.  Then, word by word, lane j decodes element j:
// its rank is the word's first rank + the eligible bits below j, its count
// counts_c[rank], its slice the one whose compacted range holds the rank
// (walked forward per lane, ranks only grow).  Counts are loaded eight
// words at a time.  Slice starts and scales sit in LDS when the table has at
// most kExpandLdsSlices slices.
constexpr int kExpandBatch = 8;
constexpr int kExpandLdsSlices = 1024;

__device__ __forceinline__ int64_t slice_of_rank(const int64_t* rstart, int64_t S, int64_t r) {
  int64_t lo = 0, hi = S - 1;  // last s with rstart[s] <= r
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) / 2;
    if (rstart[mid] <= r) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

__global__ __launch_bounds__(kThreadsS) void k_cexpand(ExpandArgs a) {
  __shared__ float tab[256];
  __shared__ int64_t rs[kExpandLdsSlices + 1];
  __shared__ float sc[kExpandLdsSlices];
  const bool lds = a.S <= kExpandLdsSlices;
  for (int c = threadIdx.x; c <= a.W; c += kThreadsS) tab[c] = decode_q(c, a.W, a.decode_mode);
  if (lds) {
    for (int64_t t = threadIdx.x; t <= a.S; t += kThreadsS) rs[t] = a.rstart[t];
    for (int64_t t = threadIdx.x; t < a.S; t += kThreadsS) sc[t] = a.scales[t];
  }
  __syncthreads();
  const int64_t* rstart = lds ? rs : a.rstart;
  const float* scales = lds ? sc : a.scales;
  const int lane = threadIdx.x & 63;
  const int64_t nw = (a.n + 63) / 64;
  const int64_t wave = (int64_t)blockIdx.x * (kThreadsS / 64) + (threadIdx.x >> 6);
  const int64_t waves = (int64_t)gridDim.x * (kThreadsS / 64);
  for (int64_t k0 = wave * 64; k0 < nw; k0 += waves * 64) {
    const int nk = (int)((nw - k0) < 64 ? (nw - k0) : 64);
    uint64_t mw = lane < nk ? a.mask[k0 + lane] : 0ull;
    if (k0 + lane == nw - 1) mw &= low_mask(a.n - 64 * (nw - 1));
    // inclusive scan of the popcounts over the wavefront
    int incl = __popcll(mw);
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int v = __shfl_up(incl, d, 64);
      if (lane >= d) incl += v;
    }
    const int excl = incl - __popcll(mw);
    const int64_t base = (int64_t)a.prefix[k0];
    if (__shfl(incl, 63, 64) == 0) continue;  // no eligible element in the task
    int64_t s = slice_of_rank(rstart, a.S, base);  // every rank of the task is >= base
    for (int t0 = 0; t0 < nk; t0 += kExpandBatch) {
      uint8_t c[kExpandBatch];
      int64_t r[kExpandBatch];
      bool e[kExpandBatch];
#pragma unroll
      for (int u = 0; u < kExpandBatch; ++u) {
        const int t = t0 + u;
        const uint64_t m = uniform64(__shfl(mw, t < 64 ? t : 63, 64));
        const int ex = __shfl(excl, t < 64 ? t : 63, 64);
        e[u] = t < nk && ((m >> lane) & 1ull);
        r[u] = base + ex + __popcll(m & ((1ull << lane) - 1ull));
        c[u] = e[u] ? a.counts_c[r[u]] : 0;
      }
#pragma unroll
      for (int u = 0; u < kExpandBatch; ++u) {
        if (!e[u]) continue;
        while (s + 1 < a.S && r[u] >= rstart[s + 1]) ++s;
        a.out[64 * (k0 + t0 + u) + lane] = scales[s] * tab[c[u]];
      }
    }
  }
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, int W, hipStream_t s) {
  const int64_t nwc = (a.n_eligible + 63) / 64;
  int64_t blocks = (nwc + kThreadsS * kCompactPerLane - 1) / (kThreadsS * kCompactPerLane);
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_compact, dim3((unsigned)blocks, (unsigned)W), dim3(kThreadsS), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_slice_scales(const SliceArgs& a, int64_t segments, hipStream_t s) {
  hipLaunchKernelGGL(k_slice_part, dim3((unsigned)segments, (unsigned)a.W), dim3(kThreadsS), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_slice_scale, dim3((unsigned)a.S), dim3(kThreadsS), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_cexpand(const ExpandArgs& a, hipStream_t s) {
  const int64_t nw = (a.n + 63) / 64;
  int64_t blocks = (nw + 4 * 64 - 1) / (4 * 64);
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_cexpand, dim3((unsigned)blocks), dim3(kThreadsS), 0, s, a);
  return hipGetLastError();
}

}  // namespace nf
