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
#include "nf_device.h"

namespace nf {

namespace {

constexpr int kThreadsS = 256;

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

// Lane o (compacted word o, every row) gathers ranks 64o .. 64o + 63: it
// starts at the positional word holding rank 64o (start[o]), skips the ranks
// of that word below 64o, and appends the compressed words that follow until
// 64 ranks (or n_E) are covered.  The layout tables are read once per
// compacted word and serve all W rows.  When two positional words cover the
// 64 ranks (every word but those in sparse stretches of the mask), the rows
// go four at a time with both of their words in flight; otherwise each row
// walks the words one by one.
constexpr int kCompactRows = 4;

__global__ __launch_bounds__(kThreadsS) void k_compact(CompactArgs a) {
  const int64_t nwc = (a.n_eligible + 63) / 64;
  const int64_t nw = (a.n + 63) / 64;
  const int W = a.W;
  for (int64_t o = (int64_t)blockIdx.x * kThreadsS + threadIdx.x; o < nwc; o += (int64_t)gridDim.x * kThreadsS) {
    const int64_t r0 = o * 64;
    const int need = (int)((a.n_eligible - r0) < 64 ? (a.n_eligible - r0) : 64);
    const int64_t k = a.start[o];
    const int skip = (int)(r0 - (int64_t)a.prefix[k]);
    uint64_t m0 = a.mask[k];
    if (k == nw - 1) m0 &= low_bits(a.n - 64 * k);
    const int c0 = __popcll(m0) - skip;  // ranks of word k at or above 64o (>= 1)
    uint64_t m1 = 0;
    if (c0 < need && k + 1 < nw) {
      m1 = a.mask[k + 1];
      if (k + 1 == nw - 1) m1 &= low_bits(a.n - 64 * (k + 1));
    }
    const bool two = c0 >= need || c0 + __popcll(m1) >= need;
    const uint64_t keep = low_bits(need);
    if (two) {
      for (int w0 = 0; w0 < W; w0 += kCompactRows) {
        uint64_t x0[kCompactRows], x1[kCompactRows];
#pragma unroll
        for (int u = 0; u < kCompactRows; ++u) {
          const int w = w0 + u < W ? w0 + u : W - 1;
          x0[u] = a.bits[(int64_t)w * a.bstride + k];
          x1[u] = c0 < need ? a.bits[(int64_t)w * a.bstride + k + 1] : 0ull;
        }
#pragma unroll
        for (int u = 0; u < kCompactRows; ++u) {
          if (w0 + u >= W) break;
          uint64_t e = compress64(x0[u], m0) >> skip;
          if (c0 < need) e |= compress64(x1[u], m1) << c0;
          a.cbits[(int64_t)(w0 + u) * a.cstride + o] = e & keep;
        }
      }
      continue;
    }
    for (int w = 0; w < W; ++w) {
      const uint64_t* row = a.bits + (int64_t)w * a.bstride;
      int64_t kk = k;
      int sk = skip;
      uint64_t m = m0, acc = 0;
      int got = 0;
      while (true) {
        const int cnt = __popcll(m) - sk;
        if (cnt > 0) {
          const uint64_t e = compress64(row[kk], m) >> sk;
          acc |= got < 64 ? e << got : 0ull;
          got += cnt;
        }
        sk = 0;
        if (got >= need || ++kk >= nw) break;
        m = a.mask[kk];
        if (kk == nw - 1) m &= low_bits(a.n - 64 * kk);
      }
      a.cbits[(int64_t)w * a.cstride + o] = acc & keep;
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

// The same statistics without a second read of the gradients, from the
// partials pass 1 left in its workspace: block s takes slice s = [o, e), in
// chunks c0 = o / CH .. c1 = (e - 1) / CH.  A chunk that no other slice
// touches holds only slice s's eligible elements, so its pass-1 partial is
// slice s's share of it.  The first chunk is shared when the previous slice
// ends in it, the last when the next slice starts in it (slices are sorted
// and disjoint); a shared chunk's part of the slice is read and summed here.
// Thread t adds the owned chunks t, t + 256, ... in order, then its share of
// the shared parts' elements; a fixed tree adds the threads.
__global__ __launch_bounds__(kThreadsS) void k_slice_chunks(SliceChunkArgs a) {
  __shared__ double red[kThreadsS];
  const int64_t s = blockIdx.x;
  const int64_t o = a.off[s], e = o + a.len[s];
  const int64_t c0 = o / a.CH, c1 = (e - 1) / a.CH;
  const bool share0 = s > 0 && (a.off[s - 1] + a.len[s - 1] - 1) / a.CH == c0;
  const bool share1 = s + 1 < a.S && a.off[s + 1] / a.CH == c1;
  // parts of the slice read here: [r0, r0e) in chunk c0 and [r1, e) in c1
  int64_t r0 = o, r0e = o, r1 = e;
  if (c0 == c1) {
    if (share0 || share1) r0e = e;
  } else {
    if (share0) r0e = (c0 + 1) * a.CH;
    if (share1) r1 = c1 * a.CH;
  }
  const int64_t cb = r0e > r0 ? c0 + 1 : c0;  // owned chunks [cb, ce)
  const int64_t ce = (c0 == c1) ? (r0e > r0 ? c0 : c0 + 1) : (r1 < e ? c1 : c1 + 1);
  for (int w = 0; w < a.W; ++w) {
    double t = 0.0;
    for (int64_t c = cb + threadIdx.x; c < ce; c += kThreadsS) t += a.part[c * a.W + w].sabs;
    const float* row = a.g + (int64_t)w * a.wstride;
    for (int64_t i = r0 + threadIdx.x; i < r0e; i += kThreadsS) t += __builtin_fabs((double)row[i]);
    for (int64_t i = r1 + threadIdx.x; i < e; i += kThreadsS) t += __builtin_fabs((double)row[i]);
    red[threadIdx.x] = t;
    __syncthreads();
    for (int h = kThreadsS / 2; h > 0; h >>= 1) {
      if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
      __syncthreads();
    }
    if (threadIdx.x == 0) a.sums[s * a.W + w] = red[0];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    double acc = 0.0;
    for (int w = 0; w < a.W; ++w) acc += a.sums[s * a.W + w] / (double)a.len[s];
    a.scales[s] = (float)(acc / (double)a.W);
  }
}

// A wavefront takes 64 consecutive positional words per task.  Lane t loads
// mask word k0 + t; a scan of the popcounts gives each word's first rank
// (prefix[k0] + the eligible elements of the task's earlier words).  The
// task's counts, at most 4096 consecutive bytes of counts_c from rank
// prefix[k0] on, are brought into LDS with coalesced dword loads.  Then,
// word by word, lane j decodes element j: its count sits at (the word's
// first rank - prefix[k0] + the eligible bits below j) in LDS, its slice is
// the one whose compacted range holds its rank (walked forward per lane,
// ranks only grow).  The task's mask words and first ranks are read back
// from LDS as broadcasts, four words at a time.  A task inside one slice (the
// usual case) takes its scale once; others walk the slices per element.
// Slice starts and scales sit in LDS when the table has at most
// kExpandLdsSlices slices.
constexpr int kExpandLdsSlices = 1024;
constexpr int kExpandStageWords = 4096 / 4 + 2;  // dwords per wavefront: 4096 counts + alignment
constexpr int kExpandUnroll = 4;                 // words decoded together
constexpr int kExpandStageLoads = (kExpandStageWords + 63) / 64;  // dword loads per lane per task

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
  __shared__ uint32_t stage[kThreadsS / 64][kExpandStageWords];
  __shared__ uint64_t tmask[kThreadsS / 64][64];
  __shared__ int tex[kThreadsS / 64][64];
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
  uint32_t* st = stage[threadIdx.x >> 6];
  uint64_t* tw = tmask[threadIdx.x >> 6];
  int* te = tex[threadIdx.x >> 6];
  const uint8_t* stb = reinterpret_cast<const uint8_t*>(st);
  const int64_t nw = (a.n + 63) / 64;
  const int64_t ncw = a.n_eligible / 4;  // whole dwords of counts_c (the last 0-3 bytes go one by one)
  const uint32_t* cw = reinterpret_cast<const uint32_t*>(a.counts_c);
  const int64_t wave = (int64_t)blockIdx.x * (kThreadsS / 64) + (threadIdx.x >> 6);
  const int64_t waves = (int64_t)gridDim.x * (kThreadsS / 64);
  for (int64_t k0 = wave * 64; k0 < nw; k0 += waves * 64) {
    const int nk = (int)((nw - k0) < 64 ? (nw - k0) : 64);
    uint64_t mw = lane < nk ? a.mask[k0 + lane] : 0ull;
    if (k0 + lane == nw - 1) mw &= low_bits(a.n - 64 * (nw - 1));
    // inclusive scan of the popcounts over the wavefront
    int incl = __popcll(mw);
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int v = __shfl_up(incl, d, 64);
      if (lane >= d) incl += v;
    }
    const int excl = incl - __popcll(mw);
    const int total = __shfl(incl, 63, 64);
    if (total == 0) continue;  // no eligible element in the task
    const int64_t base = (int64_t)a.prefix[k0];
    // counts of ranks [base, base + total) into LDS, from the dword holding rank base
    const int64_t d0 = base / 4;
    const int off = (int)(base - 4 * d0);
    const int nd = (off + total + 3) / 4;
    // every load of the lane first, then the LDS stores (one round trip, not 17)
    uint32_t v[kExpandStageLoads];
#pragma unroll
    for (int j = 0; j < kExpandStageLoads; ++j) {
      const int i = lane + 64 * j;
      const int64_t d = d0 + i;
      v[j] = (i < nd && d < ncw) ? __builtin_nontemporal_load(cw + d) : 0u;
    }
#pragma unroll
    for (int j = 0; j < kExpandStageLoads; ++j) {
      const int i = lane + 64 * j;
      const int64_t d = d0 + i;
      if (i < nd && d >= ncw)  // the last 1-3 counts of counts_c, byte by byte
        for (int e = 0; e < 4 && 4 * d + e < a.n_eligible; ++e) v[j] |= (uint32_t)a.counts_c[4 * d + e] << (8 * e);
      if (i < nd) st[i] = v[j];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    tw[lane] = mw;    // the task's mask words and first ranks, read back as
    te[lane] = excl;  // wavefront-wide broadcasts
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    int64_t s = slice_of_rank(rstart, a.S, base);  // every rank of the task is >= base
    const uint64_t below = (1ull << lane) - 1ull;
    if (s + 1 >= a.S || rstart[s + 1] >= base + total) {
      // The whole task lies in slice s (the usual case: slices are far
      // longer than a task): one scale, no slice walk per element.
      const float scale = scales[s];
      float* orow = a.out + 64 * k0 + lane;
      for (int t = 0; t < nk; t += kExpandUnroll) {
        bool el[kExpandUnroll];
        uint8_t c[kExpandUnroll];
#pragma unroll
        for (int u = 0; u < kExpandUnroll; ++u) {
          const int tt = t + u < nk ? t + u : nk - 1;
          const uint64_t m = t + u < nk ? tw[tt] : 0ull;
          el[u] = (m >> lane) & 1ull;
          c[u] = el[u] ? stb[off + te[tt] + __popcll(m & below)] : 0;
        }
#pragma unroll
        for (int u = 0; u < kExpandUnroll; ++u)
          if (el[u]) orow[64 * (t + u)] = scale * tab[c[u]];
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      continue;
    }
    for (int t = 0; t < nk; t += kExpandUnroll) {
      bool el[kExpandUnroll];
      int rel[kExpandUnroll];
      uint8_t c[kExpandUnroll];
#pragma unroll
      for (int u = 0; u < kExpandUnroll; ++u) {
        const int tt = t + u < nk ? t + u : nk - 1;
        const uint64_t m = t + u < nk ? tw[tt] : 0ull;
        el[u] = (m >> lane) & 1ull;
        rel[u] = te[tt] + __popcll(m & below);  // rank - base
        c[u] = el[u] ? stb[off + rel[u]] : 0;
      }
#pragma unroll
      for (int u = 0; u < kExpandUnroll; ++u) {
        if (!el[u]) continue;
        const int64_t r = base + rel[u];
        while (s + 1 < a.S && r >= rstart[s + 1]) ++s;
        a.out[64 * (k0 + t + u) + lane] = scales[s] * tab[c[u]];
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a0, int W, hipStream_t s) {
  CompactArgs a = a0;
  a.W = W;
  const int64_t nwc = (a.n_eligible + 63) / 64;
  int64_t blocks = (nwc + kThreadsS - 1) / kThreadsS;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_compact, dim3((unsigned)blocks), dim3(kThreadsS), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_slice_scales(const SliceArgs& a, int64_t segments, hipStream_t s) {
  hipLaunchKernelGGL(k_slice_part, dim3((unsigned)segments, (unsigned)a.W), dim3(kThreadsS), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_slice_scale, dim3((unsigned)a.S), dim3(kThreadsS), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_slice_chunks(const SliceChunkArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_slice_chunks, dim3((unsigned)a.S), dim3(kThreadsS), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_cexpand(const ExpandArgs& a, hipStream_t s) {
  const int64_t nw = (a.n + 63) / 64;
  int64_t blocks = (nw + 4 * 64 - 1) / (4 * 64);
  // About one task per wavefront: a task's two dependent round trips are
  // better hidden by other queued wavefronts than by a grid-stride loop
  // (8,192 blocks: 2.54 ms at GPT scale; 2^20: 2.30 ms).
  if (blocks > (1 << 20)) blocks = 1 << 20;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_cexpand, dim3((unsigned)blocks), dim3(kThreadsS), 0, s, a);
  return hipGetLastError();
}

}  // namespace nf
