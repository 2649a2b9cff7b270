// nf_pass1.hip - write side and decision of the bucket reducer (gfx950).
//
//   k_pass1   write side (§3.3 step 5, §5.2): one read of the W gradient
//             rows; sign payload by wavefront ballot, per-worker health in
//             registers, FP32 sums at routed positions through an LDS stage.
//             Without sign words (PACK false) each lane's |g| sum is proven
//             exact tile by tile (or, past a failed proof, kept with its
//             rounding errors), so that the decision can round the exact sum
//             once.
//             A block takes a chunk of tiles by one of four loops: fast (all
//             eligible), mixed (all tiles full, some routed), routed
//             (nothing eligible, element-major) or general (ragged tails).
//   k_slotsum second level of the partials of buckets above kMaxSlots chunks
//   k_decide  one block per bucket: fixed-order reduction of the pass-1
//             partial statistics, then the route rules (§3.2, §6.4).  In
//             exact mode it certifies each |g| sum's rounding and re-sums
//             the worker exactly where it cannot.
//
// The path is bound by HBM bandwidth, so there is no MFMA: every step is a
// streaming scan with a handful of VALU operations per element and worker.
#include <hip/hip_ext.h>

#include "nf_device.h"

namespace nf {

// The wavefront's |g| sum of one worker as an XSum: in exact mode from the
// lanes' (s, c) pairs, otherwise the plain wavefront sum with no error kept.
template <bool EXACT>
__device__ __forceinline__ XSum lane_sum(double s, double c, uint32_t nz) {
  if constexpr (EXACT) return wave_xsum(xlane(s, c, nz));
  return XSum{wave_sum(s), 0.0, 0.0};
}

// p += q for partial statistics; in exact mode the |g| sums as XSums, else
// as plain FP64 sums (their error parts stay 0).
template <bool EXACT>
__device__ __forceinline__ void part_add(Partial& p, const Partial& q) {
  if constexpr (EXACT) {
    const XSum x = xcombine(XSum{p.sabs, p.sabs_c, p.sabs_b}, XSum{q.sabs, q.sabs_c, q.sabs_b});
    p.sabs = x.s;
    p.sabs_c = x.c;
    p.sabs_b = x.b;
  } else {
    p.sabs += q.sabs;
  }
  p.ssq += q.ssq;
  p.nonfinite += q.nonfinite;
}

// ------------------------------------------------------------------ pass 1
//
// WPW workers per wavefront and NW = pass1_words(WPW) words (64 elements
// each) per worker and tile.  Lane l of a wavefront loads element 64k + l of
// word k, so every load instruction reads 256 contiguous bytes and the ballot
// of "g > 0" over the wavefront is exactly bitmap word k.  A block takes one
// chunk (G tiles of one bucket); launch q0 takes chunks q0 .. q0 + grid - 1.
// Occupancy: eight wavefronts per SIMD (64 VGPRs) for one or two workers
// per wavefront with sign words; four without (the exact |g| sums need a few
// registers more, and at 64 they spilled: G-Ternary's first pass at GPT
// scale 23.2 ms against 13.6 ms at four) or with more workers.
template <int WPW, bool PACK>
__global__ __launch_bounds__(kThreads1) __attribute__((amdgpu_waves_per_eu(WPW <= 2 && PACK ? 8 : 4, WPW <= 2 && PACK ? 8 : 4))) void k_pass1(
    const float* __restrict__ g, const uint64_t* __restrict__ mask, uint64_t* __restrict__ bits,
    float* __restrict__ out, Partial* __restrict__ part, uint64_t* __restrict__ part_ne, Pass1Args a,
    int64_t q0) {
  constexpr int NW = pass1_words(WPW);
  extern __shared__ __align__(16) unsigned char smem[];
  const int64_t q = q0 + blockIdx.x;  // this block's chunk
  if (q >= a.total_chunks) return;     // whole block

  // chunk q -> bucket b, chunk c within it; the chunk's partials go to slot q
  int b;
  int64_t c, base, nbe, chunk0;
  chunk_home(q, a.btab, a.cbucket, a.nb, a.chunks_full, b, c);
  bucket_span(b, a.btab, a.n_total, a.bucket_n, a.slots, base, nbe, chunk0);
  const int v = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wavefront index, uniform
  const int lane = threadIdx.x & 63;
  const int wg = v % a.wg;
  const int eg = v / a.wg;
  const bool active = eg < a.eg;
  const int T = a.T;
  const int tile = a.eg * T;
  const int64_t ntiles = (nbe + tile - 1) / tile;
  const int64_t tb = c * a.G;
  const int64_t te = (tb + a.G < ntiles) ? tb + a.G : ntiles;
  const bool stage_on = a.sums != kSumsNone;
  // LDS: the chunk's sign words [W][G * EG * NW], then the FP32 stage [W][tile]
  const int cw = a.G * a.eg * NW;  // sign words per worker and chunk
  uint64_t* wbuf = reinterpret_cast<uint64_t*>(smem);
  const size_t stage_off = PACK ? (size_t)a.W * cw * sizeof(uint64_t) : 0;
  float* stage = reinterpret_cast<float*>(smem + stage_off);
  // then the chunk's mask words [G * EG * NW] (mixed chunks)
  uint64_t* mwords =
      reinterpret_cast<uint64_t*>(smem + stage_off + (stage_on ? (size_t)a.W * tile * sizeof(float) : 0));
  __shared__ uint32_t tflags;  // mixed chunks: bit i = tile tb + i has a routed element
  if (threadIdx.x == 0) tflags = 0;
  // FP32 sum at a position: an earlier row group's running sum comes first;
  // the mean divides by all workers after the last group.
  auto sum_first = [&](int64_t pos, float x0) { return a.racc ? out[pos] + x0 : x0; };
  auto sum_last = [&](float s) { return a.mean && a.rfin ? s / (float)a.wtot : s; };

  // Per-worker health of this lane.  Exact mode (no sign words): sabs[j] +
  // sabc[j] is the lane's exact |g| sum (TwoSum per term).
  constexpr bool EXACT = !PACK;
  double sabs[WPW], sabc[WPW], ssq[WPW];
  uint64_t nonf[WPW];
  uint32_t snz[WPW], um[WPW];  // exact mode: see tile_into_lane
  bool tw[WPW];
#pragma unroll
  for (int j = 0; j < WPW; ++j) {
    sabs[j] = 0.0;
    sabc[j] = 0.0;
    ssq[j] = 0.0;
    nonf[j] = 0;
    snz[j] = 0;
    um[j] = ~0u;
    tw[j] = false;
  }
  uint64_t ne = 0;

  // Fast chunks: every tile full and every element eligible, and no FP32
  // sums over all elements.  Then the loop needs no mask, bound or stage
  // work, and the next tile is in flight while one is examined (two
  // register buffers, tiles taken in pairs).  The per-tile instruction
  // count is what limits this loop: the ballots are the bitmap words as
  // they are, and addresses advance by constants.  Every issue makes the
  // same number of loads (past the chunk's end, in an idle wavefront or for
  // a missing worker it reads the bucket's first tile), so that the
  // compiler's wait counts leave the next tile in flight.
  constexpr int NX = WPW * NW;
  const bool all_full = te * tile <= nbe;
  float xa[NX], xb[NX];
  // Row pointers of this wavefront's workers at its element group, and the
  // bucket's first tile for loads that are not needed.
  const float* rp[WPW];
#pragma unroll
  for (int j = 0; j < WPW; ++j) {
    const int w = wg + j * a.wg;
    rp[j] = g + (int64_t)(w < a.W ? w : wg) * a.wstride + base + (int64_t)eg * T + lane;
  }
  const float* dp = g + (int64_t)wg * a.wstride + base + lane;
  auto issue_words = [&](int64_t tt, float (&X)[NX]) {
    const bool ok = active && tt < te;
    const int64_t o = tt * tile;
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
      const float* row = (ok && (j == 0 || wg + j * a.wg < a.W)) ? rp[j] + o : dp;
#pragma unroll
      for (int k = 0; k < NW; ++k) X[j * NW + k] = __builtin_nontemporal_load(row + 64 * k);
    }
  };
  // Loads whose values are not needed: waiting for them where they die
  // keeps the compiler from waiting for them later, with the next tile in
  // flight.
  auto consume = [&](const float (&X)[NX]) {
#pragma unroll
    for (int k = 0; k < NX; ++k) asm volatile("" ::"v"(X[k]));
  };
  // The mask load goes out first, unpredicated, so that only it is waited
  // for before the barrier.
  bool chunk_fast, chunk_routed, chunk_mixed;
  {
    const int64_t wbeg = (base + tb * tile) / 64;
    const int nwc = all_full ? (int)((te - tb) * (tile / 64)) : 0;
    uint64_t m0 = ~0ull;
    if (all_full) {
      m0 = mask[wbeg + ((int)threadIdx.x < nwc ? (int)threadIdx.x : nwc - 1)];
      issue_words(tb, xa);
    }
    const bool mine = (int)threadIdx.x < nwc;
    int some_not = !all_full || (mine && m0 != ~0ull);
    int some_set = !all_full || (mine && m0 != 0ull);
    for (int i = threadIdx.x + kThreads1; i < nwc; i += kThreads1) {
      const uint64_t m1 = mask[wbeg + i];
      some_not |= m1 != ~0ull;
      some_set |= m1 != 0ull;
    }
    chunk_fast = !__syncthreads_or(some_not) && a.sums != kSumsAll;
    // Every element routed to FP32 (all tiles full, no mask bit set).
    chunk_routed = stage_on && !__syncthreads_or(some_set) &&
                   (WPW == 1 || (te - tb) * (tile / 64) <= (int64_t)kWaves * routed_steps(NW));
    // Every tile full, some element routed (or FP32 sums over all
    // elements), one worker per wavefront: the chunk's mask words go to LDS,
    // with a bit per tile that has a routed element, and the first tile
    // stays in flight.  (With more workers per wavefront the registers of
    // this loop would spill; such chunks take the general loop.)
    chunk_mixed = WPW == 1 && all_full && !chunk_fast && !chunk_routed;
    if (chunk_mixed) {
      const int nwt = tile / 64;
      for (int i = threadIdx.x; i < nwc; i += kThreads1) {
        const uint64_t m1 = i < kThreads1 ? m0 : mask[wbeg + i];
        mwords[i] = m1;
        if (m1 != ~0ull) atomicOr(&tflags, 1u << (i / nwt));
      }
      __syncthreads();
    } else if (all_full && !chunk_fast) {
      consume(xa);
    }
  }

  // Chunks with every element routed to FP32, several workers per
  // wavefront: element-major like the one-worker case below, but the
  // workers go in groups of GW (their loads and FP64 sums of squares fit
  // the registers).  Lane l of wavefront v keeps the running FP32 sum of
  // element 64s + l for each of its steps s = v, v + 16, ... in a register
  // from one group to the next, so the workers are still added in order.
  // Each wavefront leaves its per-worker sums of squares in LDS; after the
  // last group, one barrier, and each worker's are added in wavefront order
  // (one barrier per group took 0.19 ms more on a 64-worker bucket).
  if constexpr (WPW > 1) {
    if (chunk_routed) {
      constexpr int GW = WPW <= 2 ? 8 : 16;  // workers per group
      constexpr int MS = routed_steps(NW);   // steps per wavefront at most
      const int64_t c0 = base + tb * tile;
      const int nsteps = (int)((te - tb) * (tile / 64));
      const int64_t slot = q;
      Partial* red = reinterpret_cast<Partial*>(smem);  // [kWaves][W]
      float run[MS];
#pragma unroll
      for (int i = 0; i < MS; ++i) run[i] = 0.0f;
      if (a.racc) {
#pragma unroll
        for (int i = 0; i < MS; ++i) {
          const int st = v + kWaves * i;
          if (st >= nsteps) break;
          run[i] = out[c0 + (int64_t)st * 64 + lane];
        }
      }
      for (int w0 = 0; w0 < a.W; w0 += GW) {
        double q2[GW];
        uint64_t nf2[GW];
#pragma unroll
        for (int w = 0; w < GW; ++w) {
          q2[w] = 0.0;
          nf2[w] = 0;
        }
#pragma unroll
        for (int i = 0; i < MS; ++i) {
          const int st = v + kWaves * i;
          if (st >= nsteps) break;  // wavefront-uniform
          const int64_t e = c0 + (int64_t)st * 64 + lane;
          float x[GW];
#pragma unroll
          for (int w = 0; w < GW; ++w)
            x[w] = w0 + w < a.W ? __builtin_nontemporal_load(g + (int64_t)(w0 + w) * a.wstride + e) : 0.0f;
          float sum = (w0 == 0 && !a.racc) ? x[0] : run[i] + x[0];
#pragma unroll
          for (int w = 1; w < GW; ++w)
            if (w0 + w < a.W) sum = sum + x[w];
          run[i] = sum;
#pragma unroll
          for (int w = 0; w < GW; ++w) {
            const double d = (double)x[w];
            q2[w] = __builtin_fma(d, d, q2[w]);
          }
          // A non-finite value makes the running sum non-finite from its
          // group on, so this finds every one.
          if (__ballot(!finite32(sum))) {
#pragma unroll
            for (int w = 0; w < GW; ++w) nf2[w] += __popcll(__ballot(!finite32(x[w])));
          }
        }
#pragma unroll
        for (int w = 0; w < GW; ++w) {
          const double s2 = wave_sum(q2[w]);
          if (lane == 0 && w0 + w < a.W) {
            Partial p;
            p.sabs = 0.0;
            p.sabs_c = 0.0;
            p.sabs_b = 0.0;
            p.ssq = s2;
            p.nonfinite = nf2[w];
            red[v * a.W + w0 + w] = p;
          }
        }
      }
      // one barrier for the chunk: each worker's wavefront partials in order
      __syncthreads();
      for (int w = threadIdx.x; w < a.W; w += kThreads1) {
        Partial p = red[w];
        for (int v2 = 1; v2 < kWaves; ++v2) {
          p.ssq += red[v2 * a.W + w].ssq;
          p.nonfinite += red[v2 * a.W + w].nonfinite;
        }
        part[slot * a.wtot + w] = p;
      }
#pragma unroll
      for (int i = 0; i < MS; ++i) {
        const int st = v + kWaves * i;
        if (st >= nsteps) break;
        out[c0 + (int64_t)st * 64 + lane] = sum_last(run[i]);
      }
      if (PACK) {
        const int64_t gw0 = c0 / 64;
        for (int i = threadIdx.x; i < a.W * nsteps; i += kThreads1) {
          const int w = i / nsteps;
          bits[(int64_t)w * a.bstride + gw0 + (i - w * nsteps)] = 0ull;
        }
      }
      if (threadIdx.x == 0) part_ne[slot] = 0;
      return;
    }
  }

  // Chunks with every element routed to FP32 (one worker per wavefront):
  // element-major, without the LDS stage or block barriers.  Lane l of
  // wavefront v takes element 64s + l for steps s = v, v + 16, ..., loads
  // that element of every worker (one 256-byte coalesced load per worker),
  // adds them in worker order in FP32 and keeps each worker's FP64 sum of
  // squares in its own register.  Nothing is eligible, so the sign words
  // are 0 and every |g| sum over eligible elements is 0.
  if (WPW == 1 && chunk_routed) {
    constexpr int WR = kWaves;  // workers at most on this path
    double q2[WR];
    uint64_t nf2[WR];
#pragma unroll
    for (int w = 0; w < WR; ++w) {
      q2[w] = 0.0;
      nf2[w] = 0;
    }
    const int64_t c0 = base + tb * tile;
    const int nsteps = (int)((te - tb) * (tile / 64));
    for (int st = v; st < nsteps; st += kWaves) {
      const int64_t e = c0 + (int64_t)st * 64 + lane;
      float x[WR];
#pragma unroll
      for (int w = 0; w < WR; ++w) x[w] = w < a.W ? __builtin_nontemporal_load(g + (int64_t)w * a.wstride + e) : 0.0f;
      float sum = sum_first(e, x[0]);
#pragma unroll
      for (int w = 1; w < WR; ++w)
        if (w < a.W) sum = sum + x[w];
      out[e] = sum_last(sum);
#pragma unroll
      for (int w = 0; w < WR; ++w) {
        const double d = (double)x[w];
        q2[w] = __builtin_fma(d, d, q2[w]);
      }
      // A non-finite value in any worker makes the sum non-finite.
      if (__ballot(!finite32(sum))) {
#pragma unroll
        for (int w = 0; w < WR; ++w) nf2[w] += __popcll(__ballot(!finite32(x[w])));
      }
    }
    // Zero sign words for the chunk, row by row.
    if (PACK) {
      const int64_t gw0 = c0 / 64;
      for (int i = threadIdx.x; i < a.W * nsteps; i += kThreads1) {
        const int w = i / nsteps;
        bits[(int64_t)w * a.bstride + gw0 + (i - w * nsteps)] = 0ull;
      }
    }
    // Block partials: wavefront sums, then wavefronts in order.
    Partial* red = reinterpret_cast<Partial*>(smem);
#pragma unroll
    for (int w = 0; w < WR; ++w) {
      const double s2 = wave_sum(q2[w]);
      if (lane == 0 && w < a.W) {
        Partial p;
        p.sabs = 0.0;
        p.sabs_c = 0.0;
        p.sabs_b = 0.0;
        p.ssq = s2;
        p.nonfinite = nf2[w];
        red[v * a.W + w] = p;
      }
    }
    __syncthreads();
    const int64_t slot = q;
    if ((int)threadIdx.x < a.W) {
      const int w = threadIdx.x;
      Partial p = red[w];
      for (int v2 = 1; v2 < kWaves; ++v2) {
        const Partial q3 = red[v2 * a.W + w];
        p.ssq += q3.ssq;
        p.nonfinite += q3.nonfinite;
      }
      part[slot * a.wtot + w] = p;
    }
    if (threadIdx.x == 0) part_ne[slot] = 0;
    return;
  }
  auto fast_body = [&](int64_t t, float (&X)[NX], float (&Xn)[NX]) {
    issue_words(t + 1, Xn);
    if (!active) {
      consume(X);
      return;
    }
    const int ti = (int)(t - tb);
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
      const int w = wg + j * a.wg;
      const float* x = &X[j * NW];
      if (j > 0 && w >= a.W) {
#pragma unroll
        for (int k = 0; k < NW; ++k) asm volatile("" ::"v"(x[k]));
        continue;
      }
      double s1 = 0.0, s2 = 0.0;
      uint32_t umt = ~0u;
      uint64_t bb[NW];
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        if (PACK) bb[k] = __ballot(x[k] > 0.0f);
        const double d = (double)x[k];
        s2 = __builtin_fma(d, d, s2);
        s1 += __builtin_fabs(d);
        if constexpr (EXACT) umt = term_umin(umt, x[k]);
      }
      if constexpr (EXACT) tile_into_lane<NW>(sabs[j], sabc[j], snz[j], um[j], tw[j], s1, umt, rp[j] + t * tile, ~0u);
      if (PACK) {
        uint32_t wlo, whi;
        lanes_from_ballots<NW>(bb, wlo, whi);
        if (lane < NW) wbuf[w * cw + (ti * a.eg + eg) * NW + lane] = ((uint64_t)whi << 32) | wlo;
      }
      if (__ballot(!finite64(s2))) {
#pragma unroll
        for (int k = 0; k < NW; ++k) nonf[j] += __popcll(__ballot(!finite32(x[k])));
      }
      if constexpr (!EXACT) sabs[j] += s1;
      ssq[j] += s2;
    }
  };
  if (chunk_fast) {
    if (active && wg == 0) ne = (uint64_t)(te - tb) * (uint64_t)T;
    // Pairs of tiles in a loop with a single exit, then the odd tile: the
    // loop head is reached only with xa in flight.
    int64_t t = tb;
    for (int64_t p = (te - tb) >> 1; p > 0; --p, t += 2) {
      fast_body(t, xa, xb);
      fast_body(t + 1, xb, xa);
    }
    if ((te - tb) & 1) {
      fast_body(t, xa, xb);
      consume(xb);
    } else {
      consume(xa);
    }
  }

  // Mixed chunks: the fast loop's structure (the next tile in flight while
  // one is examined), with each wavefront's mask words read from LDS, sign
  // and |g| contributions masked, and the tiles that hold a routed element
  // staged in LDS and added in worker order between two block barriers.
  if (WPW == 1 && chunk_mixed) {
    const int nwt = tile / 64;  // mask words per tile
    const uint32_t tfl = tflags;
    auto mixed_body = [&](int64_t t, float (&X)[NX], float (&Xn)[NX]) {
      issue_words(t + 1, Xn);
      const int ti = (int)(t - tb);
      const bool stage_tile = stage_on && (a.sums == kSumsAll || ((tfl >> ti) & 1u));  // block-uniform
      if (active) {
        uint64_t mw[NW];
        uint64_t mine = ~0ull;
#pragma unroll
        for (int k = 0; k < NW; ++k) {
          mw[k] = uniform64(mwords[ti * nwt + eg * NW + k]);
          mine &= mw[k];
        }
        if (wg == 0) {
          if (mine == ~0ull) {
            ne += (uint64_t)(64 * NW);
          } else {
#pragma unroll
            for (int k = 0; k < NW; ++k) ne += __popcll(mw[k]);
          }
        }
#pragma unroll
        for (int j = 0; j < WPW; ++j) {
          const int w = wg + j * a.wg;
          const float* x = &X[j * NW];
          if (j > 0 && w >= a.W) {
#pragma unroll
            for (int k = 0; k < NW; ++k) asm volatile("" ::"v"(x[k]));
            continue;
          }
          double s1 = 0.0, s2 = 0.0;
          uint32_t umt = ~0u;
          uint64_t bb[NW];
#pragma unroll
          for (int k = 0; k < NW; ++k) {
            if (PACK) bb[k] = __ballot(x[k] > 0.0f) & mw[k];
            const double d = (double)x[k];
            s2 = __builtin_fma(d, d, s2);
            const bool el = (mw[k] >> lane) & 1ull;
            s1 += el ? __builtin_fabs(d) : 0.0;
            if constexpr (EXACT) umt = term_umin(umt, el ? x[k] : 0.0f);
          }
          if constexpr (EXACT) {
            uint32_t el = 0;
#pragma unroll
            for (int k = 0; k < NW; ++k) el |= (uint32_t)((mw[k] >> lane) & 1ull) << k;
            tile_into_lane<NW>(sabs[j], sabc[j], snz[j], um[j], tw[j], s1, umt, rp[j] + t * tile, el);
          }
          if (PACK) {
            uint32_t wlo, whi;
            lanes_from_ballots<NW>(bb, wlo, whi);
            if (lane < NW) wbuf[w * cw + (ti * a.eg + eg) * NW + lane] = ((uint64_t)whi << 32) | wlo;
          }
          if (__ballot(!finite64(s2))) {
#pragma unroll
            for (int k = 0; k < NW; ++k) nonf[j] += __popcll(__ballot(!finite32(x[k])));
          }
          if constexpr (!EXACT) sabs[j] += s1;
          ssq[j] += s2;
          if (stage_tile) {
            float* st = stage + (int64_t)w * tile + eg * T + lane;
#pragma unroll
            for (int k = 0; k < NW; ++k) st[64 * k] = x[k];
          }
        }
      } else {
        consume(X);
      }
      if (stage_tile) {
        __syncthreads();
        const int64_t t0 = t * tile;
        for (int kw = v; kw < nwt; kw += kWaves) {
          const uint64_t pick = a.sums == kSumsAll ? ~0ull : ~mwords[ti * nwt + kw];
          const int e = kw * 64 + lane;
          if ((pick >> lane) & 1ull) {
            float s2 = sum_first(base + t0 + e, stage[e]);
            for (int w = 1; w < a.W; ++w) s2 = s2 + stage[w * tile + e];
            out[base + t0 + e] = sum_last(s2);
          }
        }
        __syncthreads();
      }
    };
    int64_t t = tb;
    for (int64_t p = (te - tb) >> 1; p > 0; --p, t += 2) {
      mixed_body(t, xa, xb);
      mixed_body(t + 1, xb, xa);
    }
    if ((te - tb) & 1) {
      mixed_body(t, xa, xb);
      consume(xb);
    } else {
      consume(xa);
    }
  }

  for (int64_t t = (chunk_fast || chunk_mixed) ? te : tb; t < te; ++t) {
    const int64_t t0 = t * tile;
    const bool full = t0 + tile <= nbe;  // block-uniform
    const int64_t e0 = t0 + (int64_t)eg * T;
    int64_t c64 = nbe - e0;
    const int cnt = active ? (int)(c64 < 0 ? 0 : (c64 > T ? T : c64)) : 0;
    const int64_t wrd0 = (base + e0) / 64;  // first word of my element group
    const uint64_t* tmask = mask + (base + t0) / 64;

    // Loads first, decisions after: the first worker's gradients, this
    // group's mask words and (several element groups) the tile's mask words
    // are all in flight before anything waits on them.
    float x0[NW];
    {
      const float* row = g + (int64_t)wg * a.wstride + base + e0 + lane;
      if (full) {
        if (active) {
#pragma unroll
          for (int k = 0; k < NW; ++k) x0[k] = __builtin_nontemporal_load(row + 64 * k);
        }
      } else {
#pragma unroll
        for (int k = 0; k < NW; ++k)
          x0[k] = (64 * k + lane < cnt) ? __builtin_nontemporal_load(row + 64 * k) : 0.0f;
      }
    }
    uint64_t mw[NW];
    uint64_t mine = ~0ull;
    if (full) {
      const uint64_t* mrow = active ? mask + wrd0 : tmask;  // in bounds for every wavefront
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        mw[k] = mrow[k];
        mine &= mw[k];
      }
    } else {
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        mw[k] = 64 * k < cnt ? (mask[wrd0 + k] & low_bits(cnt - 64 * k)) : 0ull;
        mine &= mw[k];
      }
    }
    // The tile needs the LDS stage (FP32 sums in worker order) unless every
    // element of it is eligible.  With one element group per block the
    // tile's words are every wavefront's own; otherwise every wavefront reads
    // them all, so the decision is block-uniform either way.
    bool tile_all = full && mine == ~0ull;
    if (a.eg > 1 && full) {
      uint64_t acc = ~0ull;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int k = lane + 64 * r;
        if (k < tile / 64) acc &= tmask[k];
      }
      tile_all = __all(acc == ~0ull);
    }
    const bool mine_all = full && mine == ~0ull;
    const bool stage_tile = stage_on && (a.sums == kSumsAll || !tile_all);
    if (active && wg == 0) {
      if (mine_all) {
        ne += (uint64_t)(64 * NW);
      } else {
#pragma unroll
        for (int k = 0; k < NW; ++k) ne += __popcll(mw[k]);
      }
    }

    if (active) {
      const int nwv = (cnt + 63) / 64;
#pragma unroll
      for (int j = 0; j < WPW; ++j) {
        const int w = wg + j * a.wg;
        if (j > 0 && w >= a.W) break;
        float x[NW];
        if (j == 0) {
#pragma unroll
          for (int k = 0; k < NW; ++k) x[k] = x0[k];
        } else {
          const float* row = g + (int64_t)w * a.wstride + base + e0 + lane;
          if (full) {
#pragma unroll
            for (int k = 0; k < NW; ++k) x[k] = __builtin_nontemporal_load(row + 64 * k);
          } else {
#pragma unroll
            for (int k = 0; k < NW; ++k)
              x[k] = (64 * k + lane < cnt) ? __builtin_nontemporal_load(row + 64 * k) : 0.0f;
          }
        }
        double s1 = 0.0, s2 = 0.0;
        uint32_t umt = ~0u;
        uint64_t bb[NW];
        if (mine_all) {
#pragma unroll
          for (int k = 0; k < NW; ++k) {
            if (PACK) bb[k] = __ballot(x[k] > 0.0f);
            const double d = (double)x[k];
            s2 = __builtin_fma(d, d, s2);
            s1 += __builtin_fabs(d);
            if constexpr (EXACT) umt = term_umin(umt, x[k]);
          }
        } else {
#pragma unroll
          for (int k = 0; k < NW; ++k) {
            if (PACK) bb[k] = __ballot(x[k] > 0.0f) & mw[k];
            const double d = (double)x[k];
            s2 = __builtin_fma(d, d, s2);
            const bool el = (mw[k] >> lane) & 1ull;
            s1 += el ? __builtin_fabs(d) : 0.0;
            if constexpr (EXACT) umt = term_umin(umt, el ? x[k] : 0.0f);
          }
        }
        if constexpr (EXACT) {
          uint32_t el = 0;
#pragma unroll
          for (int k = 0; k < NW; ++k) el |= (uint32_t)((mw[k] >> lane) & 1ull) << k;
          tile_into_lane<NW>(sabs[j], sabc[j], snz[j], um[j], tw[j], s1, umt,
                             g + (int64_t)w * a.wstride + base + e0 + lane, el);
        }
        if (PACK) {
          uint32_t wlo, whi;
          lanes_from_ballots<NW>(bb, wlo, whi);
          // word k of this group and tile -> chunk word ((t - tb) * EG + eg) * NW + k
          if (lane < nwv) wbuf[w * cw + ((t - tb) * a.eg + eg) * NW + lane] = ((uint64_t)whi << 32) | wlo;
        }
        if (__ballot(!finite64(s2))) {
#pragma unroll
          for (int k = 0; k < NW; ++k) nonf[j] += __popcll(__ballot(!finite32(x[k])));
        }
        if constexpr (!EXACT) sabs[j] += s1;
        ssq[j] += s2;
        if (stage_tile) {
          float* st = stage + (int64_t)w * tile + eg * T + lane;
#pragma unroll
          for (int k = 0; k < NW; ++k) st[64 * k] = x[k];
        }
      }
    }
    if (stage_tile) {
      __syncthreads();
      // Workers added in order w = 0..W-1 at each staged position; wavefront
      // v takes words v, v + 16, ... of the tile.
      const int lim = (int)((nbe - t0) < tile ? (nbe - t0) : tile);
      const int nwt = (lim + 63) / 64;
      for (int kw = v; kw < nwt; kw += kWaves) {
        const int e = kw * 64 + lane;
        const uint64_t pick = (a.sums == kSumsAll ? ~0ull : ~tmask[kw]) & low_bits(lim - kw * 64);
        if ((pick >> lane) & 1ull) {
          float s = sum_first(base + t0 + e, stage[e]);
          for (int w = 1; w < a.W; ++w) s = s + stage[w * tile + e];
          out[base + t0 + e] = sum_last(s);
        }
      }
      __syncthreads();
    }
  }

  const int64_t slot = q;  // the chunk's own partial slot
  if (a.eg == 1) {
    // One element group: each worker lives in exactly one wavefront, which
    // stores its own rows of sign words and its own partials, so the block
    // ends without a barrier.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int64_t e_beg = tb * tile;
    const int64_t e_end = (te * tile < nbe) ? te * tile : nbe;
    const int valid = te > tb ? (int)((e_end - e_beg + 63) / 64) : 0;
    const int64_t gw0 = (base + e_beg) / 64;
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
      const int w = wg + j * a.wg;
      if (w >= a.W) break;
      if (PACK)
        for (int o = lane; o < valid; o += 64) bits[(int64_t)w * a.bstride + gw0 + o] = wbuf[w * cw + o];
      const XSum x1 = lane_sum<EXACT>(sabs[j], sabc[j], snz[j]);
      const double s2 = wave_sum(ssq[j]);
      if (lane == 0) {
        Partial p;
        p.sabs = x1.s;
        p.sabs_c = x1.c;
        p.sabs_b = x1.b;
        p.ssq = s2;
        p.nonfinite = nonf[j];
        part[slot * a.wtot + w] = p;
      }
    }
    if (wg == 0 && lane == 0) part_ne[slot] = ne;
    return;
  }

  __syncthreads();
  // The chunk's sign words, row by row, as coalesced stores.
  if (PACK && te > tb) {
    const int64_t e_beg = tb * tile;
    const int64_t e_end = (te * tile < nbe) ? te * tile : nbe;
    const int valid = (int)((e_end - e_beg + 63) / 64);
    const int64_t gw0 = (base + e_beg) / 64;
    for (int i = threadIdx.x; i < a.W * valid; i += kThreads1) {
      const int w = i / valid;
      const int o = i - w * valid;
      bits[(int64_t)w * a.bstride + gw0 + o] = wbuf[w * cw + o];
    }
    __syncthreads();
  }

  // Block partials: wavefront sums, then element groups in order, to the
  // chunk's own slot.
  Partial* red = reinterpret_cast<Partial*>(smem);
  uint64_t* red_ne = reinterpret_cast<uint64_t*>(red + a.eg * a.W);
  if (active) {
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
      const int w = wg + j * a.wg;
      if (w >= a.W) break;
      const XSum x1 = lane_sum<EXACT>(sabs[j], sabc[j], snz[j]);
      const double s2 = wave_sum(ssq[j]);
      if (lane == 0) {
        Partial p;
        p.sabs = x1.s;
        p.sabs_c = x1.c;
        p.sabs_b = x1.b;
        p.ssq = s2;
        p.nonfinite = nonf[j];
        red[eg * a.W + w] = p;
      }
    }
    if (wg == 0 && lane == 0) red_ne[eg] = ne;
  }
  __syncthreads();
  for (int w = threadIdx.x; w < a.W; w += kThreads1) {
    Partial p = red[w];
    for (int e = 1; e < a.eg; ++e) part_add<EXACT>(p, red[e * a.W + w]);
    part[slot * a.wtot + w] = p;
  }
  if (threadIdx.x == 0) {
    uint64_t s = 0;
    for (int e = 0; e < a.eg; ++e) s += red_ne[e];
    part_ne[slot] = s;
  }
}

// ------------------------------------------------------------------ decide
// Second level for buckets of more than kMaxSlots chunks: block x sums
// group x % groups (gs consecutive slots) of bucket x / groups.  Thread
// t < parts * W takes worker t % W and every parts-th slot from t / W on;
// the parts are then added in order, so the result does not depend on
// timing.
template <bool EXACT>
__global__ __launch_bounds__(256) void k_slotsum(DecideArgs a) {
  __shared__ Partial red[256];
  const int b = (int)(blockIdx.x / (unsigned)a.groups);
  const int grp = (int)(blockIdx.x - (unsigned)b * (unsigned)a.groups);
  int64_t base, nbe, chunk0;
  bucket_span(b, a.btab, a.n_total, a.bucket_n, a.slots, base, nbe, chunk0);
  const int64_t chunks = ((nbe + a.tile - 1) / a.tile + a.G - 1) / a.G;
  const int64_t s0 = (int64_t)grp * a.gs;
  if (s0 >= chunks) return;  // whole block: this bucket has fewer groups
  const int cnt = (int)(chunks - s0 < a.gs ? chunks - s0 : a.gs);
  const int parts = 256 / a.W;
  const int t = threadIdx.x;
  const Partial* P = a.part + (chunk0 + s0) * a.W;
  if (t < parts * a.W) {
    const int w = t % a.W;
    Partial r;
    r.sabs = r.sabs_c = r.sabs_b = r.ssq = 0.0;
    r.nonfinite = 0;
#pragma unroll 8
    for (int k = t / a.W; k < cnt; k += parts) part_add<EXACT>(r, P[(int64_t)k * a.W + w]);
    red[t] = r;
  }
  __syncthreads();
  if (t < a.W) {
    Partial r = red[t];
    for (int p = 1; p < parts; ++p) part_add<EXACT>(r, red[p * a.W + t]);
    a.part2[((int64_t)b * a.groups + grp) * a.W + t] = r;
  }
  if (t < 64) {
    const uint64_t* N = a.part_ne + chunk0 + s0;
    uint64_t ne = 0;
    for (int k = t; k < cnt; k += 64) ne += N[k];
    ne = wave_sum_u64(ne);
    if (t == 0) a.part2_ne[(int64_t)b * a.groups + grp] = ne;
  }
}

// 1024 threads: up to 32 workers, sixteen wavefronts take the workers in
// turn (at W = 32, two each), the lanes of one splitting its slots, so
// that fewer slot sums wait on each other.  Above 32 workers (a wavefront
// would take up to sixteen in turn: 0.28 ms at W = 255; at W = 64 this
// way halves the stress bucket's decision, 88 -> 38 us) thread t takes
// worker t % W and every P-th slot from t / W, P the largest power of two
// with P * W <= 1024; the P parts of a worker are then added in order.
constexpr int kDecideThreads = 1024;

template <bool EXACT>
__global__ __launch_bounds__(kDecideThreads) void k_decide(DecideArgs a) {
  __shared__ nf_worker_stats st[256];
  __shared__ uint8_t redo[256];            // exact mode: re-sum this worker
  __shared__ unsigned long long hist[256];  // exponent bins of the re-summation
  __shared__ uint64_t ne_s;
  __shared__ double med_s;
  __shared__ double qterm[256];  // |g| sum / n_E per worker (the scale's terms)
  __shared__ Partial wide[kDecideThreads];  // W > kWideWorkers: [part][W]
  const int b = blockIdx.x;
  const int v = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wavefront index, uniform
  const int lane = threadIdx.x & 63;
  // One slot per chunk of this bucket, or its second-level group sums.
  int64_t base, nbe, chunk0;
  bucket_span(b, a.btab, a.n_total, a.bucket_n, a.slots, base, nbe, chunk0);
  const int64_t chunks = ((nbe + a.tile - 1) / a.tile + a.G - 1) / a.G;
  const bool two = a.gs > 0;
  const Partial* P = two ? a.part2 + (int64_t)b * a.groups * a.W : a.part + chunk0 * a.W;
  const uint64_t* PN = two ? a.part2_ne + (int64_t)b * a.groups : a.part_ne + chunk0;
  const int used = (int)(two ? (chunks + a.gs - 1) / a.gs : chunks);
  // The slot loops are unrolled so that their loads are in flight together;
  // the adds keep their order.
  if (a.W > kWideWorkers) {
    int parts = 1;
    while (2 * parts * a.W <= kDecideThreads) parts *= 2;
    const int t = threadIdx.x;
    if (t < parts * a.W) {
      const int w = t % a.W;
      Partial r;
      r.sabs = r.sabs_c = r.sabs_b = r.ssq = 0.0;
      r.nonfinite = 0;
#pragma unroll 8
      for (int k = t / a.W; k < used; k += parts) part_add<EXACT>(r, P[(int64_t)k * a.W + w]);
      wide[t] = r;
    }
    __syncthreads();
    if (t < a.W) {
      Partial r = wide[t];
      for (int p = 1; p < parts; ++p) part_add<EXACT>(r, wide[p * a.W + t]);
      double s1;
      const bool certified = xround(XSum{r.sabs, r.sabs_c, r.sabs_b}, s1);
      st[t].nonfinite = r.nonfinite;
      st[t].sum_abs_elig = s1;
      st[t].sum_sq = r.ssq;
      redo[t] = EXACT && !certified;
    }
  } else {
    for (int w = v; w < a.W; w += kDecideThreads / 64) {
      Partial r;
      r.sabs = r.sabs_c = r.sabs_b = r.ssq = 0.0;
      r.nonfinite = 0;
#pragma unroll 8
      for (int k = lane; k < used; k += 64) part_add<EXACT>(r, P[(int64_t)k * a.W + w]);
      const XSum x1 = EXACT ? wave_xsum(XSum{r.sabs, r.sabs_c, r.sabs_b}) : XSum{wave_sum(r.sabs), 0.0, 0.0};
      const double s2 = wave_sum(r.ssq);
      const uint64_t nf = wave_sum_u64(r.nonfinite);
      if (lane == 0) {
        double s1;
        const bool certified = xround(x1, s1);
        st[w].nonfinite = nf;
        st[w].sum_abs_elig = s1;
        st[w].sum_sq = s2;
        redo[w] = EXACT && !certified;
      }
    }
  }
  if (v == 0) {
    uint64_t s = 0;
#pragma unroll 8
    for (int k = lane; k < used; k += 64) s += PN[k];
    s = wave_sum_u64(s);
    if (lane == 0) ne_s = s;
  }
  __syncthreads();
  // Exact mode: a worker whose rounding the bound could not certify is
  // summed again from its gradients, exactly (rare: it takes a total within
  // the bound of a rounding midpoint).
  uint32_t resummed = 0;
  if (EXACT) {
    for (int w = 0; w < a.W; ++w) {
      if (!redo[w]) continue;  // block-uniform
      const double e = exact_abs_sum(a.g + (int64_t)w * a.wstride, a.mask, base, nbe, hist);
      if (threadIdx.x == 0) st[w].sum_abs_elig = e;
      ++resummed;
    }
    __syncthreads();
  }
  for (int w = threadIdx.x; w < a.W; w += kDecideThreads) a.stats[(int64_t)b * a.W + w] = st[w];
  if (!a.dec) return;
  // The per-worker facts of the route rules, thread t for worker t (W <=
  // 255): finite sums of squares counted by a block vote, the lower median
  // by rank, the scale's terms |g| sum / n_E divided in parallel and added
  // in worker order by one thread (as the host's decision adds them), and
  // the reason flags by block votes.  (With one thread scanning the workers
  // the decision of two 255-worker buckets took 88 us; this way, 49 us.)
  const int t = threadIdx.x;
  const bool mine = t < a.W;
  const double ssq = mine ? st[t].sum_sq : 0.0;
  const double sab = mine ? st[t].sum_abs_elig : 0.0;
  const bool fin = mine && finite64(ssq);
  if (t == 0) med_s = 0.0;
  const int kfin = __syncthreads_count(fin);
  if (fin && ssq_rank(st, a.W, t) == (kfin - 1) / 2) med_s = ssq;
  const int64_t ne = (int64_t)ne_s;
  if (mine) qterm[t] = ne > 0 ? sab / (double)ne : 0.0;
  const int nonf = __syncthreads_or(mine && st[t].nonfinite != 0);
  const int zero = __syncthreads_or(mine && sab == 0.0);
  const int spike = __syncthreads_or(kfin >= 2 && fin && ssq > spike_threshold(a.pol, med_s));
  if (t == 0) {
    float scale = 0.0f;
    if (ne > 0) {
      double acc = 0.0;
      for (int w = 0; w < a.W; ++w) acc += qterm[w];
      scale = (float)(acc / (double)a.W);
    }
    nf_route_decision d;
    decide_finish(nbe, ne, a.pol, nonf != 0, zero != 0, spike != 0, scale, &d);
    d.resummed = resummed;
    a.dec[b] = d;
  }
}

// --------------------------------------------------------------- launchers

template <bool PACK>
static hipError_t pass1_dispatch(const Geometry& geo, const Pass1Args& a0, hipStream_t s) {
  const dim3 block(kThreads1);
  const int R = geo.rows;  // workers of the largest row group
  const int cw = geo.G * geo.eg * pass1_words(geo.wpw);
  size_t smem = PACK ? (size_t)R * cw * sizeof(uint64_t) : 0;
  if (a0.sums != kSumsNone) smem += (size_t)R * geo.tile * sizeof(float);
  smem += (size_t)geo.G * geo.eg * pass1_words(geo.wpw) * sizeof(uint64_t);  // mask words of a mixed chunk
  size_t red = (size_t)geo.eg * R * sizeof(Partial) + (size_t)geo.eg * sizeof(uint64_t);
  // routed chunks with several workers per wavefront: [kWaves][W] partials
  if (geo.wpw > 1 && a0.sums != kSumsNone && red < (size_t)kWaves * R * sizeof(Partial))
    red = (size_t)kWaves * R * sizeof(Partial);
  if (smem < red) smem = red;
  if (smem > 65536) {
    // Above 64 KiB of dynamic LDS the kernel must opt in (gfx950 has 160 KiB per CU).
    hipError_t e = hipSuccess;
    switch (geo.wpw) {
      case 1: e = hipFuncSetAttribute((const void*)k_pass1<1, PACK>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
      case 2: e = hipFuncSetAttribute((const void*)k_pass1<2, PACK>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
      case 4: e = hipFuncSetAttribute((const void*)k_pass1<4, PACK>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
      default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
  }
  // One launch per epoch of chunks (see the geometry notes) and row group.
  // The first launch is ordered after earlier work on the stream; later ones
  // may start while the one before drains: every chunk writes only its own
  // partial slots and sign words.  A later row group's first launch is
  // ordered too when it continues the FP32 sums in the output.  The next
  // ordered launch (the decision) waits for all.
  const uint32_t overlap = hipExtAnyOrderLaunch;
  const int64_t epoch = pass1_launch_chunks(geo, PACK);
  for (int grp = 0; grp < geo.ngroups; ++grp) {
    Pass1Args a = a0;
    int wb, rows;
    row_group(geo, grp, &wb, &rows);
    // every wavefront's first worker (wg < geo.wg) must be a row of the group
    if (rows < geo.wg || rows > R) return hipErrorInvalidValue;
    a.W = rows;
    a.wtot = geo.W;
    a.wbase = wb;
    a.racc = grp > 0;
    a.rfin = grp == geo.ngroups - 1;
    a.g = a0.g + (int64_t)wb * a0.wstride;
    if (a0.bits) a.bits = a0.bits + (int64_t)wb * a0.bstride;
    a.part = a0.part + wb;
    const bool chained = grp > 0 && a0.sums != kSumsNone;
    for (int64_t q0 = 0; q0 < geo.total_chunks; q0 += epoch) {
      const int64_t left = geo.total_chunks - q0;
      const dim3 grid((unsigned)(left < epoch ? left : epoch));
      const uint32_t fl = (q0 == 0 && (grp == 0 || chained)) ? 0u : overlap;
      switch (geo.wpw) {
        case 1: hipExtLaunchKernelGGL((k_pass1<1, PACK>), grid, block, smem, s, nullptr, nullptr, fl, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a, q0); break;
        case 2: hipExtLaunchKernelGGL((k_pass1<2, PACK>), grid, block, smem, s, nullptr, nullptr, fl, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a, q0); break;
        case 4: hipExtLaunchKernelGGL((k_pass1<4, PACK>), grid, block, smem, s, nullptr, nullptr, fl, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a, q0); break;
        default: return hipErrorInvalidValue;
      }
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

hipError_t launch_pass1(const Geometry& geo, const Pass1Args& a, hipStream_t s) {
  return a.bits ? pass1_dispatch<true>(geo, a, s) : pass1_dispatch<false>(geo, a, s);
}

hipError_t launch_decide(const Geometry& geo, const DecideArgs& a, hipStream_t s) {
  if (geo.gs > 0) {
    if (a.exact)
      hipLaunchKernelGGL(k_slotsum<true>, dim3((unsigned)(geo.nb * geo.groups)), dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL(k_slotsum<false>, dim3((unsigned)(geo.nb * geo.groups)), dim3(256), 0, s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (a.exact)
    hipLaunchKernelGGL(k_decide<true>, dim3((unsigned)geo.nb), dim3(kDecideThreads), 0, s, a);
  else
    hipLaunchKernelGGL(k_decide<false>, dim3((unsigned)geo.nb), dim3(kDecideThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace nf
