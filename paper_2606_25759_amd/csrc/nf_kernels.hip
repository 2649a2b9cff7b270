// nf_kernels.hip - gfx950 kernels of the bucket reducer.
//
//   k_pass1   write side (§3.3 step 5, §5.2): one read of the W gradient
//             rows; sign payload by wavefront ballot, per-worker health in
//             registers, FP32 sums at routed positions through an LDS stage.
//             A block takes a chunk of tiles by one of four loops: fast (all
//             eligible), mixed (all tiles full, some routed), routed
//             (nothing eligible, element-major) or general (ragged tails).
//   k_slotsum second level of the partials of buckets above kMaxSlots chunks
//   k_decide  one block per bucket: fixed-order reduction of the pass-1
//             partial statistics, then the route rules (§3.2, §6.4).
//   k_pass2   read side (§3.3 step 7, §6.1): per-coordinate sign counts over
//             the W bitmaps and the scaled decode; or the FP32 sum of the
//             eligible positions when the bucket falls back.
//
// The path is bound by HBM bandwidth, so there is no MFMA: every step is a
// streaming scan with a handful of VALU operations per element and worker.
#include <hip/hip_ext.h>

#include "nf_internal.h"

namespace nf {

// Four floats / four dwords as one 16-byte vector (for vector nontemporal
// loads and stores).
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bool finite32(float x) {
  return (__float_as_uint(x) & 0x7f800000u) != 0x7f800000u;
}

// Sum over the wavefront by an xor butterfly.  Lane 0 always adds in the
// same order, so its result is deterministic; callers use lane 0.
__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// Sign words k = 0..NW-1 of one worker tile, already held as wavefront
// ballots (scalar register pairs), moved into lanes k of two VGPRs so that
// lanes 0..NW-1 can store them with one instruction.  v_writelane_b32 reads
// its data operand early: a scalar register written by a VALU compare just
// before is not yet visible to it, and the compiler does not model that
// dependence through inline assembly, so the block waits first (s_nop 4).
template <int NW>
__device__ __forceinline__ void lanes_from_ballots(const uint64_t (&bb)[NW], uint32_t& lo,
                                                   uint32_t& hi) {
  uint32_t l[8], h[8];
#pragma unroll
  for (int k = 0; k < NW; ++k) {
    l[k] = (uint32_t)bb[k];
    h[k] = (uint32_t)(bb[k] >> 32);
  }
  if constexpr (NW == 8) {
    // two blocks of four words keep at most eight scalar inputs live
    asm volatile(
        "s_nop 4\n"
        "v_writelane_b32 %0, %2, 0\n v_writelane_b32 %1, %3, 0\n"
        "v_writelane_b32 %0, %4, 1\n v_writelane_b32 %1, %5, 1\n"
        "v_writelane_b32 %0, %6, 2\n v_writelane_b32 %1, %7, 2\n"
        "v_writelane_b32 %0, %8, 3\n v_writelane_b32 %1, %9, 3\n"
        : "=v"(lo), "=v"(hi)
        : "s"(l[0]), "s"(h[0]), "s"(l[1]), "s"(h[1]), "s"(l[2]), "s"(h[2]), "s"(l[3]), "s"(h[3]));
    asm volatile(
        "s_nop 4\n"
        "v_writelane_b32 %0, %2, 4\n v_writelane_b32 %1, %3, 4\n"
        "v_writelane_b32 %0, %4, 5\n v_writelane_b32 %1, %5, 5\n"
        "v_writelane_b32 %0, %6, 6\n v_writelane_b32 %1, %7, 6\n"
        "v_writelane_b32 %0, %8, 7\n v_writelane_b32 %1, %9, 7\n"
        : "+v"(lo), "+v"(hi)
        : "s"(l[4]), "s"(h[4]), "s"(l[5]), "s"(h[5]), "s"(l[6]), "s"(h[6]), "s"(l[7]), "s"(h[7]));
  } else if constexpr (NW == 4) {
    asm volatile(
        "s_nop 4\n"
        "v_writelane_b32 %0, %2, 0\n v_writelane_b32 %1, %3, 0\n"
        "v_writelane_b32 %0, %4, 1\n v_writelane_b32 %1, %5, 1\n"
        "v_writelane_b32 %0, %6, 2\n v_writelane_b32 %1, %7, 2\n"
        "v_writelane_b32 %0, %8, 3\n v_writelane_b32 %1, %9, 3\n"
        : "=v"(lo), "=v"(hi)
        : "s"(l[0]), "s"(h[0]), "s"(l[1]), "s"(h[1]), "s"(l[2]), "s"(h[2]), "s"(l[3]), "s"(h[3]));
  } else if constexpr (NW == 2) {
    asm volatile(
        "s_nop 4\n"
        "v_writelane_b32 %0, %2, 0\n v_writelane_b32 %1, %3, 0\n"
        "v_writelane_b32 %0, %4, 1\n v_writelane_b32 %1, %5, 1\n"
        : "=v"(lo), "=v"(hi)
        : "s"(l[0]), "s"(h[0]), "s"(l[1]), "s"(h[1]));
  } else {
    static_assert(NW == 1, "tile words");
    asm volatile(
        "s_nop 4\n"
        "v_writelane_b32 %0, %2, 0\n v_writelane_b32 %1, %3, 0\n"
        : "=v"(lo), "=v"(hi)
        : "s"(l[0]), "s"(h[0]));
  }
}

// A wavefront-uniform 64-bit value held in a vector register, as a scalar.
__device__ __forceinline__ uint64_t uniform64(uint64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// c + bit `lane` of the wavefront-uniform word (the word read as a lane mask).
__device__ __forceinline__ uint32_t add_lane_bit(uint32_t c, uint64_t word) {
  return c + (uint32_t)__builtin_amdgcn_inverse_ballot_w64(word);
}

__device__ __forceinline__ uint64_t low_bits(int64_t r) {
  return r >= 64 ? ~0ull : (r <= 0 ? 0ull : ((1ull << r) - 1ull));
}

__device__ __forceinline__ int64_t bucket_len(int64_t n_total, int64_t bucket_n, int b) {
  int64_t base = (int64_t)b * bucket_n;
  int64_t r = n_total - base;
  return r < 0 ? 0 : (r < bucket_n ? r : bucket_n);
}

// ------------------------------------------------------------------ pass 1
//
// WPW workers per wavefront and NW = pass1_words(WPW) words (64 elements
// each) per worker and tile.  Lane l of a wavefront loads element 64k + l of
// word k, so every load instruction reads 256 contiguous bytes and the ballot
// of "g > 0" over the wavefront is exactly bitmap word k.  A block takes one
// chunk (G tiles of one bucket); launch q0 takes chunks q0 .. q0 + grid - 1.
template <int WPW, bool PACK>
__global__ __launch_bounds__(kThreads1) __attribute__((amdgpu_waves_per_eu(WPW <= 2 ? 8 : 4, WPW <= 2 ? 8 : 4))) void k_pass1(
    const float* __restrict__ g, const uint64_t* __restrict__ mask, uint64_t* __restrict__ bits,
    float* __restrict__ out, Partial* __restrict__ part, uint64_t* __restrict__ part_ne, Pass1Args a,
    int64_t q0) {
  constexpr int NW = pass1_words(WPW);
  extern __shared__ __align__(16) unsigned char smem[];
  const int64_t q = q0 + blockIdx.x;  // this block's chunk
  if (q >= a.total_chunks) return;     // whole block

  // chunk q -> bucket b, chunk c within it (all buckets but the last are full)
  int b;
  int64_t c;
  if (q < (int64_t)(a.nb - 1) * a.chunks_full) {
    b = (int)(q / a.chunks_full);
    c = q - (int64_t)b * a.chunks_full;
  } else {
    b = a.nb - 1;
    c = q - (int64_t)b * a.chunks_full;
  }
  const int64_t base = (int64_t)b * a.bucket_n;
  const int64_t nbe = bucket_len(a.n_total, a.bucket_n, b);
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

  double sabs[WPW], ssq[WPW];
  uint64_t nonf[WPW];
#pragma unroll
  for (int j = 0; j < WPW; ++j) {
    sabs[j] = 0.0;
    ssq[j] = 0.0;
    nonf[j] = 0;
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
  // After each group the wavefronts' sums of squares are added in wavefront
  // order, through LDS, into the group's partials.
  if constexpr (WPW > 1) {
    if (chunk_routed) {
      constexpr int GW = WPW <= 2 ? 8 : 16;  // workers per group
      constexpr int MS = routed_steps(NW);   // steps per wavefront at most
      const int64_t c0 = base + tb * tile;
      const int nsteps = (int)((te - tb) * (tile / 64));
      const int64_t slot = (int64_t)b * a.slots + c;
      Partial* red = reinterpret_cast<Partial*>(smem);  // [kWaves][GW]
      float run[MS];
#pragma unroll
      for (int i = 0; i < MS; ++i) run[i] = 0.0f;
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
          float sum = w0 == 0 ? x[0] : run[i] + x[0];
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
          if (lane == 0) {
            Partial p;
            p.sabs = 0.0;
            p.ssq = s2;
            p.nonfinite = nf2[w];
            red[v * GW + w] = p;
          }
        }
        __syncthreads();
        if ((int)threadIdx.x < GW && w0 + (int)threadIdx.x < a.W) {
          const int w = threadIdx.x;
          Partial p = red[w];
          for (int v2 = 1; v2 < kWaves; ++v2) {
            p.ssq += red[v2 * GW + w].ssq;
            p.nonfinite += red[v2 * GW + w].nonfinite;
          }
          part[slot * a.W + w0 + w] = p;
        }
        __syncthreads();  // red is reused by the next group
      }
#pragma unroll
      for (int i = 0; i < MS; ++i) {
        const int st = v + kWaves * i;
        if (st >= nsteps) break;
        out[c0 + (int64_t)st * 64 + lane] = a.mean ? run[i] / (float)a.W : run[i];
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
      float sum = x[0];
#pragma unroll
      for (int w = 1; w < WR; ++w)
        if (w < a.W) sum = sum + x[w];
      out[e] = a.mean ? sum / (float)a.W : sum;
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
        p.ssq = s2;
        p.nonfinite = nf2[w];
        red[v * a.W + w] = p;
      }
    }
    __syncthreads();
    const int64_t slot = (int64_t)b * a.slots + c;
    if ((int)threadIdx.x < a.W) {
      const int w = threadIdx.x;
      Partial p = red[w];
      for (int v2 = 1; v2 < kWaves; ++v2) {
        const Partial q3 = red[v2 * a.W + w];
        p.ssq += q3.ssq;
        p.nonfinite += q3.nonfinite;
      }
      part[slot * a.W + w] = p;
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
      uint64_t bb[NW];
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        if (PACK) bb[k] = __ballot(x[k] > 0.0f);
        const double d = (double)x[k];
        s2 = __builtin_fma(d, d, s2);
        s1 += __builtin_fabs(d);
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
      sabs[j] += s1;
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
          uint64_t bb[NW];
#pragma unroll
          for (int k = 0; k < NW; ++k) {
            if (PACK) bb[k] = __ballot(x[k] > 0.0f) & mw[k];
            const double d = (double)x[k];
            s2 = __builtin_fma(d, d, s2);
            s1 += ((mw[k] >> lane) & 1ull) ? __builtin_fabs(d) : 0.0;
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
          sabs[j] += s1;
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
            float s2 = stage[e];
            for (int w = 1; w < a.W; ++w) s2 = s2 + stage[w * tile + e];
            if (a.mean) s2 = s2 / (float)a.W;
            out[base + t0 + e] = s2;
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
        uint64_t bb[NW];
        if (mine_all) {
#pragma unroll
          for (int k = 0; k < NW; ++k) {
            if (PACK) bb[k] = __ballot(x[k] > 0.0f);
            const double d = (double)x[k];
            s2 = __builtin_fma(d, d, s2);
            s1 += __builtin_fabs(d);
          }
        } else {
#pragma unroll
          for (int k = 0; k < NW; ++k) {
            if (PACK) bb[k] = __ballot(x[k] > 0.0f) & mw[k];
            const double d = (double)x[k];
            s2 = __builtin_fma(d, d, s2);
            s1 += ((mw[k] >> lane) & 1ull) ? __builtin_fabs(d) : 0.0;
          }
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
        sabs[j] += s1;
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
          float s = stage[e];
          for (int w = 1; w < a.W; ++w) s = s + stage[w * tile + e];
          if (a.mean) s = s / (float)a.W;
          out[base + t0 + e] = s;
        }
      }
      __syncthreads();
    }
  }

  const int64_t slot = (int64_t)b * a.slots + c;  // the chunk's own partial slot
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
      const double s1 = wave_sum(sabs[j]);
      const double s2 = wave_sum(ssq[j]);
      if (lane == 0) {
        Partial p;
        p.sabs = s1;
        p.ssq = s2;
        p.nonfinite = nonf[j];
        part[slot * a.W + w] = p;
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
      const double s1 = wave_sum(sabs[j]);
      const double s2 = wave_sum(ssq[j]);
      if (lane == 0) {
        Partial p;
        p.sabs = s1;
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
    for (int e = 1; e < a.eg; ++e) {
      const Partial q2 = red[e * a.W + w];
      p.sabs += q2.sabs;
      p.ssq += q2.ssq;
      p.nonfinite += q2.nonfinite;
    }
    part[slot * a.W + w] = p;
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
__global__ __launch_bounds__(256) void k_slotsum(DecideArgs a) {
  __shared__ Partial red[256];
  const int b = (int)(blockIdx.x / (unsigned)a.groups);
  const int grp = (int)(blockIdx.x - (unsigned)b * (unsigned)a.groups);
  const int64_t nbe = bucket_len(a.n_total, a.bucket_n, b);
  const int64_t chunks = ((nbe + a.tile - 1) / a.tile + a.G - 1) / a.G;
  const int64_t s0 = (int64_t)grp * a.gs;
  if (s0 >= chunks) return;  // whole block: this bucket has fewer groups
  const int cnt = (int)(chunks - s0 < a.gs ? chunks - s0 : a.gs);
  const int parts = 256 / a.W;
  const int t = threadIdx.x;
  const Partial* P = a.part + ((int64_t)b * a.slots + s0) * a.W;
  if (t < parts * a.W) {
    const int w = t % a.W;
    double s1 = 0.0, s2 = 0.0;
    uint64_t nf = 0;
#pragma unroll 8
    for (int k = t / a.W; k < cnt; k += parts) {
      const Partial q = P[(int64_t)k * a.W + w];
      s1 += q.sabs;
      s2 += q.ssq;
      nf += q.nonfinite;
    }
    red[t].sabs = s1;
    red[t].ssq = s2;
    red[t].nonfinite = nf;
  }
  __syncthreads();
  if (t < a.W) {
    Partial r = red[t];
    for (int p = 1; p < parts; ++p) {
      r.sabs += red[p * a.W + t].sabs;
      r.ssq += red[p * a.W + t].ssq;
      r.nonfinite += red[p * a.W + t].nonfinite;
    }
    a.part2[((int64_t)b * a.groups + grp) * a.W + t] = r;
  }
  if (t < 64) {
    const uint64_t* N = a.part_ne + (int64_t)b * a.slots + s0;
    uint64_t ne = 0;
    for (int k = t; k < cnt; k += 64) ne += N[k];
    ne = wave_sum_u64(ne);
    if (t == 0) a.part2_ne[(int64_t)b * a.groups + grp] = ne;
  }
}

__global__ __launch_bounds__(256) void k_decide(DecideArgs a) {
  __shared__ nf_worker_stats st[256];
  __shared__ uint64_t ne_s;
  __shared__ int kfin_s;
  __shared__ double med_s;
  const int b = blockIdx.x;
  const int v = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wavefront index, uniform
  const int lane = threadIdx.x & 63;
  // One slot per chunk of this bucket, or its second-level group sums.
  const int64_t nbe = bucket_len(a.n_total, a.bucket_n, b);
  const int64_t chunks = ((nbe + a.tile - 1) / a.tile + a.G - 1) / a.G;
  const bool two = a.gs > 0;
  const Partial* P = two ? a.part2 + (int64_t)b * a.groups * a.W : a.part + (int64_t)b * a.slots * a.W;
  const uint64_t* PN = two ? a.part2_ne + (int64_t)b * a.groups : a.part_ne + (int64_t)b * a.slots;
  const int used = (int)(two ? (chunks + a.gs - 1) / a.gs : chunks);
  // The slot loops are unrolled so that their loads are in flight together;
  // the adds keep their order.
  for (int w = v; w < a.W; w += 4) {
    double s1 = 0.0, s2 = 0.0;
    uint64_t nf = 0;
#pragma unroll 8
    for (int k = lane; k < used; k += 64) {
      const Partial p = P[(int64_t)k * a.W + w];
      s1 += p.sabs;
      s2 += p.ssq;
      nf += p.nonfinite;
    }
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    nf = wave_sum_u64(nf);
    if (lane == 0) {
      st[w].nonfinite = nf;
      st[w].sum_abs_elig = s1;
      st[w].sum_sq = s2;
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
  for (int w = threadIdx.x; w < a.W; w += 256) a.stats[(int64_t)b * a.W + w] = st[w];
  if (!a.dec) return;
  if (threadIdx.x == 0) {
    int k = 0;
    for (int w = 0; w < a.W; ++w) k += finite64(st[w].sum_sq) ? 1 : 0;
    kfin_s = k;
    med_s = 0.0;
  }
  __syncthreads();
  const int kfin = kfin_s;
  for (int w = threadIdx.x; w < a.W; w += 256)
    if (finite64(st[w].sum_sq) && ssq_rank(st, a.W, w) == (kfin - 1) / 2) med_s = st[w].sum_sq;
  __syncthreads();
  if (threadIdx.x == 0) {
    nf_route_decision d;
    decide_from(st, a.W, nbe, (int64_t)ne_s, a.pol, kfin, med_s, &d);
    a.dec[b] = d;
  }
}

// ------------------------------------------------------------------ pass 2
//
// A wavefront takes 64 consecutive bitmap words (4096 elements) per step.
// Counting (route L): lane l loads word k0 + l of every worker row (one
// 512-byte coalesced load per worker) and adds the W words into a
// bit-sliced counter, planes P[0..B) with bit j of P[b] = bit b of the count
// of element 64(k0+l) + j.  Eight words at a time go through a carry-save
// tree of full adders (Harley-Seal), the rest ripple in.  The planes are then
// transposed through LDS so that lane j decodes element j of each word: its
// count selects fl32(scale * q[c]) from an LDS table, and every store is a
// coalesced 64- or 256-byte row, nontemporal (they are not read again here;
// measured 4% faster than cached stores).  Fallback (route F) and the
// standalone FP32 reduction add the workers in order at the selected
// positions instead.
constexpr int kRec = 12;  // dwords per (word, half) record: 8 planes, mask half, pad
constexpr int kFp32Rows = 8;  // worker rows in flight in the FP32 sums

struct FullAdd {
  uint64_t sum, carry;
};

__device__ __forceinline__ FullAdd full_add(uint64_t a, uint64_t b, uint64_t c) {
  const uint64_t t = a ^ b;
  return FullAdd{t ^ c, (a & b) | (c & t)};
}

// Bit-sliced count of one bitmap word position over W rows (row w at
// col[w * bstride]): P[b] holds bit b of each element's count, for the
// nplanes planes that counts 0..W need.  Eight words at a time go through a
// carry-save tree of full adders (Harley-Seal), the rest ripple in.
__device__ __forceinline__ void count_column(const uint64_t* col, int64_t bstride, int W, bool valid,
                                             int nplanes, uint64_t (&P)[8]) {
#pragma unroll
  for (int q = 0; q < 8; ++q) P[q] = 0;
  int w = 0;
  for (; w + 8 <= W; w += 8) {
    uint64_t x[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = valid ? col[(int64_t)(w + i) * bstride] : 0ull;
    FullAdd f0 = full_add(P[0], x[0], x[1]);
    FullAdd f1 = full_add(f0.sum, x[2], x[3]);
    FullAdd f2 = full_add(P[1], f0.carry, f1.carry);
    FullAdd f3 = full_add(f1.sum, x[4], x[5]);
    FullAdd f4 = full_add(f3.sum, x[6], x[7]);
    FullAdd f5 = full_add(f2.sum, f3.carry, f4.carry);
    FullAdd f6 = full_add(P[2], f2.carry, f5.carry);
    P[0] = f4.sum;
    P[1] = f5.sum;
    P[2] = f6.sum;
    uint64_t c = f6.carry;  // weight 8
#pragma unroll
    for (int q = 3; q < 8; ++q) {
      if (q < nplanes) {
        const uint64_t t = P[q] & c;
        P[q] ^= c;
        c = t;
      }
    }
  }
  for (; w < W; ++w) {
    uint64_t c = valid ? col[(int64_t)w * bstride] : 0ull;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if (q < nplanes) {
        const uint64_t t = P[q] & c;
        P[q] ^= c;
        c = t;
      }
    }
  }
}

__global__ __launch_bounds__(kThreads2) void k_pass2(
    const uint64_t* __restrict__ bits0, const float* __restrict__ g, const uint64_t* __restrict__ mask,
    const nf_route_decision* __restrict__ dec, const float* __restrict__ scale_p,
    uint8_t* __restrict__ counts0, float* __restrict__ out0, Pass2Args a) {
  __shared__ float tab[256];
  __shared__ __align__(16) uint32_t rec[4][64 * 2 * kRec];
  // Grid z: independent counts over rows z * z_rows .. z * z_rows + W - 1,
  // written z * z_counts / z * z_out further on (node-local partial counts,
  // replicated stock counting); z = 0 for every other call.
  const int z = blockIdx.z;
  const uint64_t* bits = bits0 ? bits0 + (int64_t)z * a.z_rows * a.bstride : nullptr;
  uint8_t* counts = counts0 ? counts0 + (int64_t)z * a.z_counts : nullptr;
  float* out = out0 ? out0 + (int64_t)z * a.z_out : nullptr;
  const int b = blockIdx.y;
  const int64_t base = (int64_t)b * a.bucket_n;
  const int64_t nbe = bucket_len(a.n_total, a.bucket_n, b);
  int op = a.op;
  int sel = a.select;
  float scale = 0.0f;
  if (op == kOpFallbackOnly) {
    if (dec[b].route != NF_ROUTE_FALLBACK) return;  // whole block
    op = kOpFp32;
    sel = NF_SEL_ELIGIBLE;
  } else if (op == kOpFromDecision) {
    const int route = dec[b].route;
    if (route == NF_ROUTE_PLAIN) return;  // whole block: pass 1 wrote every position
    if (route == NF_ROUTE_LOWBIT) {
      op = kOpCountDecode;
      scale = dec[b].scale;
    } else {
      op = kOpFp32;
      sel = NF_SEL_ELIGIBLE;
    }
  } else if (op == kOpCountDecode && out) {
    scale = *scale_p;
  }
  if (op == kOpCountDecode) {
    for (int c = threadIdx.x; c <= a.W; c += kThreads2) tab[c] = scale * decode_q(c, a.W, a.decode_mode);
    __syncthreads();
  }
  const int64_t nwords = (nbe + 63) / 64;
  const int64_t wbase = base / 64;
  const int v = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wavefront index, uniform
  const int lane = threadIdx.x & 63;
  int nplanes = 1;
  while ((1 << nplanes) <= a.W) ++nplanes;  // counts 0..W need nplanes bits
  uint32_t* my = rec[v];

  for (int64_t ch = (int64_t)blockIdx.x * 4 + v; ch * 64 < nwords; ch += (int64_t)a.bpb2 * 4) {
    const int64_t k0 = ch * 64;
    const int nk = (int)((nwords - k0) < 64 ? (nwords - k0) : 64);
    if (op == kOpCountDecode) {
      // ---- bit-sliced counts, lane = word k0 + lane
      const bool valid = lane < nk;
      uint64_t P[8];
      count_column(bits + wbase + k0 + lane, a.bstride, a.W, valid, nplanes, P);
      const uint64_t mw = (valid && mask) ? mask[wbase + k0 + lane] : 0ull;
      // ---- transpose through LDS: record (word, half) holds the planes' and
      // the mask's 32-bit halves
      uint4* r0 = reinterpret_cast<uint4*>(my + (lane * 2) * kRec);
      uint4* r1 = reinterpret_cast<uint4*>(my + (lane * 2 + 1) * kRec);
      r0[0] = make_uint4((uint32_t)P[0], (uint32_t)P[1], (uint32_t)P[2], (uint32_t)P[3]);
      r0[1] = make_uint4((uint32_t)P[4], (uint32_t)P[5], (uint32_t)P[6], (uint32_t)P[7]);
      r0[2] = make_uint4((uint32_t)mw, 0u, 0u, 0u);
      r1[0] = make_uint4((uint32_t)(P[0] >> 32), (uint32_t)(P[1] >> 32), (uint32_t)(P[2] >> 32),
                         (uint32_t)(P[3] >> 32));
      r1[1] = make_uint4((uint32_t)(P[4] >> 32), (uint32_t)(P[5] >> 32), (uint32_t)(P[6] >> 32),
                         (uint32_t)(P[7] >> 32));
      r1[2] = make_uint4((uint32_t)(mw >> 32), 0u, 0u, 0u);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // ---- decode: per 256 elements (four words), lane l takes elements
      // 4l .. 4l + 3, i.e. nibble l % 16 of word l / 16.  A nibble of each
      // plane spreads into the low bits of four bytes by one multiply
      // (copies of the nibble at bits 0, 7, 14, 21 put its bit i at bit 8i),
      // so the four counts form one 32-bit word: one dword store of counts
      // and, where all four elements are eligible, one 16-byte store of
      // decoded values.
      const bool c4 = counts && ((reinterpret_cast<uintptr_t>(counts + base) & 3) == 0);
      const bool o16 = out && ((reinterpret_cast<uintptr_t>(out + base) & 15) == 0);
      for (int grp = 0; grp * 4 < nk; ++grp) {
        const int kk = grp * 4 + (lane >> 4);
        const int shn = 4 * (lane & 7);
        const uint4* r = reinterpret_cast<const uint4*>(my + (kk * 2 + ((lane >> 3) & 1)) * kRec);
        const uint4 p03 = r[0];
        const uint4 p47 = r[1];
        const uint32_t mnib = (r[2].x >> shn) & 15u;
        auto spread = [&](uint32_t plane) { return (((plane >> shn) & 15u) * 0x00204081u) & 0x01010101u; };
        uint32_t cw4 = spread(p03.x) | (spread(p03.y) << 1) | (spread(p03.z) << 2) | (spread(p03.w) << 3);
        if (nplanes > 4)
          cw4 |= (spread(p47.x) << 4) | (spread(p47.y) << 5) | (spread(p47.z) << 6) | (spread(p47.w) << 7);
        const int64_t i0 = (k0 + grp * 4) * 64 + 4 * lane;  // first of my four elements in the bucket
        if (kk >= nk || i0 >= nbe) continue;
        if (i0 + 3 < nbe) {
          if (c4) {
            __builtin_nontemporal_store(cw4, reinterpret_cast<uint32_t*>(counts + base + i0));
          } else if (counts) {
#pragma unroll
            for (int e = 0; e < 4; ++e) counts[base + i0 + e] = (uint8_t)(cw4 >> (8 * e));
          }
          if (out) {
            if (o16 && mnib == 15u) {
              const f32x4 y = {tab[cw4 & 255u], tab[(cw4 >> 8) & 255u], tab[(cw4 >> 16) & 255u],
                               tab[cw4 >> 24]};
              __builtin_nontemporal_store(y, reinterpret_cast<f32x4*>(out + base + i0));
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if ((mnib >> e) & 1u) out[base + i0 + e] = tab[(cw4 >> (8 * e)) & 255u];
            }
          }
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (i0 + e < nbe) {
              if (counts) counts[base + i0 + e] = (uint8_t)(cw4 >> (8 * e));
              if (out && ((mnib >> e) & 1u)) out[base + i0 + e] = tab[(cw4 >> (8 * e)) & 255u];
            }
          }
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    } else {
      // ---- FP32 sums: 256 elements (four words) per step; lane l takes
      // elements 4l .. 4l + 3 with one 16-byte load per worker row, eight
      // rows in flight at a time, and loads nothing when none of its four
      // elements is selected.  Rows are 16-byte aligned and buckets start on
      // 64-element boundaries, so every full group of four is aligned.
      const bool o16 = (reinterpret_cast<uintptr_t>(out + base) & 15) == 0;
      for (int grp = 0; grp * 4 < nk; ++grp) {
        const int64_t e = (k0 + grp * 4) * 64 + 4 * lane;  // my first element in the bucket
        const int64_t left = nbe - e;
        const int cnt = left <= 0 ? 0 : (left >= 4 ? 4 : (int)left);
        uint32_t pick = cnt ? (1u << cnt) - 1u : 0u;
        if (sel != NF_SEL_ALL && cnt) {
          const uint32_t nib = (uint32_t)(mask[wbase + e / 64] >> (e & 63)) & 15u;
          pick &= sel == NF_SEL_ELIGIBLE ? nib : ~nib;
        }
        if (!pick) continue;
        const float* p = g + base + e;
        if (cnt == 4) {
          f32x4 acc = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
          int w = 1;
          for (; w + kFp32Rows <= a.W; w += kFp32Rows) {
            f32x4 x[kFp32Rows];
#pragma unroll
            for (int u = 0; u < kFp32Rows; ++u)
              x[u] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + (int64_t)(w + u) * a.wstride));
#pragma unroll
            for (int u = 0; u < kFp32Rows; ++u) acc = acc + x[u];
          }
          for (; w < a.W; ++w)
            acc = acc + __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + (int64_t)w * a.wstride));
          if (a.mean) acc = acc / (float)a.W;
          if (pick == 15u && o16) {
            __builtin_nontemporal_store(acc, reinterpret_cast<f32x4*>(out + base + e));
          } else {
#pragma unroll
            for (int c = 0; c < 4; ++c)
              if ((pick >> c) & 1u) out[base + e + c] = acc[c];
          }
        } else {
          // the bucket's last, partial group of four
          for (int c = 0; c < cnt; ++c) {
            if (!((pick >> c) & 1u)) continue;
            float y = p[c];
            for (int w = 1; w < a.W; ++w) y = y + p[(int64_t)w * a.wstride + c];
            if (a.mean) y = y / (float)a.W;
            out[base + e + c] = y;
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------- G-Ternary
//
// Pack (write side), laid out as pass 1: a block takes one chunk (G tiles of
// one bucket) and wavefront v serves worker group v % WG and element group
// v / WG; lane l loads element 64k + l of word k, so the ballots of
// "eligible, not gated, g > 0" and "eligible, not gated, g < 0" are the
// two planes' words.  The next tile's loads (and mask words) are in flight
// while one tile is examined.  The chunk's words of both planes stay in LDS
// and leave at its end as coalesced rows; launches of pass 1's epochs
// bring the plane stores of a launch together, as in pass 1.
template <int WPW>
__global__ __launch_bounds__(kThreads1) __attribute__((amdgpu_waves_per_eu(WPW <= 2 ? 8 : 4, WPW <= 2 ? 8 : 4))) void k_tpack(
    TernArgs a, int64_t q0) {
  constexpr int NW = pass1_words(WPW);
  constexpr int NX = WPW * NW;
  extern __shared__ __align__(16) unsigned char smem[];
  const int64_t q = q0 + blockIdx.x;  // this block's chunk
  if (q >= a.total_chunks) return;     // whole block
  int b;
  int64_t c;
  if (q < (int64_t)(a.nb - 1) * a.chunks_full) {
    b = (int)(q / a.chunks_full);
    c = q - (int64_t)b * a.chunks_full;
  } else {
    b = a.nb - 1;
    c = q - (int64_t)b * a.chunks_full;
  }
  if (a.dec && a.dec[b].route != NF_ROUTE_LOWBIT) return;  // whole block: no planes
  const int64_t base = (int64_t)b * a.bucket_n;
  const int64_t nbe = bucket_len(a.n_total, a.bucket_n, b);
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
  const int64_t te_full = (te * tile <= nbe) ? te : te - 1;  // tiles [tb, te_full) are full
  const int cw = a.G * a.eg * NW;                             // words per worker row and chunk
  uint64_t* ppos = reinterpret_cast<uint64_t*>(smem);
  uint64_t* pneg = ppos + (size_t)a.W * cw;

  float th[WPW];
  const float* rp[WPW];
#pragma unroll
  for (int j = 0; j < WPW; ++j) {
    const int w = wg + j * a.wg;
    const int wl = w < a.W ? w : wg;
    th[j] = a.dec ? ternary_threshold(a.stats[(int64_t)b * a.W + wl], a.dec[b].n_eligible, a.tau)
                  : a.theta[wl];
    rp[j] = a.g + (int64_t)wl * a.wstride + base + (int64_t)eg * T + lane;
  }
  const uint64_t* mbase = a.mask + base / 64 + (int64_t)eg * (T / 64);
  // The first NW words of the bucket's first tile (full whenever any tile of
  // this chunk is): read by loads whose values are not needed.
  const float* dp = a.g + (int64_t)wg * a.wstride + base + lane;
  const uint64_t* dm = a.mask + base / 64;

  // Loads of a full tile (or, for an idle wavefront or a tile past the full
  // ones, of the bucket's first words).
  auto issue = [&](int64_t tt, float (&X)[NX], uint64_t (&M)[NW]) {
    const bool ok = active && tt < te_full;
    const int64_t o = tt * tile;
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
      const float* row = ok ? rp[j] + o : dp;
#pragma unroll
      for (int k = 0; k < NW; ++k) X[j * NW + k] = __builtin_nontemporal_load(row + 64 * k);
    }
    const uint64_t* mrow = ok ? mbase + o / 64 : dm;
#pragma unroll
    for (int k = 0; k < NW; ++k) M[k] = uniform64(mrow[k]);
  };
  auto body = [&](int64_t t, const float (&X)[NX], const uint64_t (&M)[NW]) {
    const int ti = (int)(t - tb);
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
      const int w = wg + j * a.wg;
      if (j > 0 && w >= a.W) continue;
      uint64_t pb[NW], nb[NW];
#pragma unroll
      for (int k = 0; k < NW; ++k) {
        const float x = X[j * NW + k];
        const bool keep = !(__builtin_fabsf(x) < th[j]);  // gated to 0 below the threshold
        pb[k] = __ballot(keep && x > 0.0f) & M[k];
        nb[k] = __ballot(keep && x < 0.0f) & M[k];
      }
      uint32_t lo, hi;
      const int at = w * cw + (ti * a.eg + eg) * NW + lane;
      lanes_from_ballots<NW>(pb, lo, hi);
      if (lane < NW) ppos[at] = ((uint64_t)hi << 32) | lo;
      lanes_from_ballots<NW>(nb, lo, hi);
      if (lane < NW) pneg[at] = ((uint64_t)hi << 32) | lo;
    }
  };
  auto consume = [&](const float (&X)[NX]) {
#pragma unroll
    for (int k = 0; k < NX; ++k) asm volatile("" ::"v"(X[k]));
  };

  float xa[NX], xb[NX];
  uint64_t ma[NW], mb[NW];
  int64_t t = tb;
  if (te_full > tb) {
    issue(tb, xa, ma);
    // Pairs of full tiles with the next one in flight, then the odd one.
    for (int64_t p = (te_full - tb) >> 1; p > 0; --p, t += 2) {
      issue(t + 1, xb, mb);
      if (active) body(t, xa, ma);
      issue(t + 2, xa, ma);
      if (active) body(t + 1, xb, mb);
    }
    if ((te_full - tb) & 1) {
      if (active) body(t, xa, ma);
      ++t;
    } else {
      consume(xa);
    }
  }
  if (t < te && active) {
    // The bucket's last, partial tile: loads and mask bits stop at its end.
    const int64_t e0 = t * tile + (int64_t)eg * T;
    const int64_t c64 = nbe - e0;
    const int cnt = (int)(c64 < 0 ? 0 : (c64 > T ? T : c64));
#pragma unroll
    for (int j = 0; j < WPW; ++j)
#pragma unroll
      for (int k = 0; k < NW; ++k)
        xb[j * NW + k] = (64 * k + lane < cnt) ? __builtin_nontemporal_load(rp[j] + t * tile + 64 * k) : 0.0f;
#pragma unroll
    for (int k = 0; k < NW; ++k)
      mb[k] = 64 * k < cnt ? uniform64(mbase[t * (tile / 64) + k] & low_bits(cnt - 64 * k)) : 0ull;
    body(t, xb, mb);
  }

  // The chunk's words of both planes, row by row.
  const int64_t e_beg = tb * tile;
  const int64_t e_end = (te * tile < nbe) ? te * tile : nbe;
  const int valid = te > tb ? (int)((e_end - e_beg + 63) / 64) : 0;
  const int64_t gw0 = (base + e_beg) / 64;
  if (a.eg == 1) {
    // each worker's words were written by its own wavefront only
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
      const int w = wg + j * a.wg;
      if (w >= a.W) break;
      for (int o = lane; o < valid; o += 64) {
        a.bits[(int64_t)w * a.bstride + gw0 + o] = ppos[w * cw + o];
        a.bits[(int64_t)(a.W + w) * a.bstride + gw0 + o] = pneg[w * cw + o];
      }
    }
    return;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < a.W * valid; i += kThreads1) {
    const int w = i / valid;
    const int o = i - w * valid;
    a.bits[(int64_t)w * a.bstride + gw0 + o] = ppos[w * cw + o];
    a.bits[(int64_t)(a.W + w) * a.bstride + gw0 + o] = pneg[w * cw + o];
  }
}

// Count and decode (read side), as pass 2 with two counters: lane l counts
// word k0 + l of the positive rows and of the negative rows; the planes of
// both go through LDS so that each lane decodes four consecutive elements
// (one nibble per plane, spread into four count bytes by a multiply) from
// the difference of the two counts, d = c+ - c-, through a table of
// fl32(scale * q[d]).
constexpr int kRecT = 20;  // dwords per (word, half): 8 + 8 plane halves, mask half, pad

__global__ __launch_bounds__(kThreads2) void k_tpass2(TernArgs a) {
  __shared__ float tab[2 * 255 + 1];
  __shared__ __align__(16) uint32_t rec[4][64 * 2 * kRecT];
  const int b = blockIdx.y;
  float scale = 0.0f;
  if (a.dec) {
    if (a.dec[b].route != NF_ROUTE_LOWBIT) return;  // whole block
    scale = a.dec[b].scale;
  } else if (a.out) {
    scale = *a.scale;
  }
  if (a.out) {
    for (int d = threadIdx.x; d <= 2 * a.W; d += kThreads2) tab[d] = scale * decode_qt(d - a.W, a.W, a.decode_mode);
    __syncthreads();
  }
  const int64_t base = (int64_t)b * a.bucket_n;
  const int64_t nbe = bucket_len(a.n_total, a.bucket_n, b);
  const int64_t nwords = (nbe + 63) / 64;
  const int64_t wbase = base / 64;
  const int v = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wavefront index, uniform
  const int lane = threadIdx.x & 63;
  int nplanes = 1;
  while ((1 << nplanes) <= a.W) ++nplanes;  // counts 0..W need nplanes bits
  uint32_t* my = rec[v];
  const bool c4 = a.cpos && a.cneg && ((reinterpret_cast<uintptr_t>(a.cpos + base) & 3) == 0) &&
                  ((reinterpret_cast<uintptr_t>(a.cneg + base) & 3) == 0);
  const bool o16 = a.out && ((reinterpret_cast<uintptr_t>(a.out + base) & 15) == 0);

  for (int64_t ch = (int64_t)blockIdx.x * 4 + v; ch * 64 < nwords; ch += (int64_t)a.bpb2 * 4) {
    const int64_t k0 = ch * 64;
    const int nk = (int)((nwords - k0) < 64 ? (nwords - k0) : 64);
    const bool valid = lane < nk;
    uint64_t P[8], N[8];
    count_column(a.bits + wbase + k0 + lane, a.bstride, a.W, valid, nplanes, P);
    count_column(a.bits + (int64_t)a.W * a.bstride + wbase + k0 + lane, a.bstride, a.W, valid, nplanes, N);
    const uint64_t mw = (valid && a.mask) ? a.mask[wbase + k0 + lane] : 0ull;
    uint4* r0 = reinterpret_cast<uint4*>(my + (lane * 2) * kRecT);
    uint4* r1 = reinterpret_cast<uint4*>(my + (lane * 2 + 1) * kRecT);
    r0[0] = make_uint4((uint32_t)P[0], (uint32_t)P[1], (uint32_t)P[2], (uint32_t)P[3]);
    r0[1] = make_uint4((uint32_t)P[4], (uint32_t)P[5], (uint32_t)P[6], (uint32_t)P[7]);
    r0[2] = make_uint4((uint32_t)N[0], (uint32_t)N[1], (uint32_t)N[2], (uint32_t)N[3]);
    r0[3] = make_uint4((uint32_t)N[4], (uint32_t)N[5], (uint32_t)N[6], (uint32_t)N[7]);
    r0[4] = make_uint4((uint32_t)mw, 0u, 0u, 0u);
    r1[0] = make_uint4((uint32_t)(P[0] >> 32), (uint32_t)(P[1] >> 32), (uint32_t)(P[2] >> 32), (uint32_t)(P[3] >> 32));
    r1[1] = make_uint4((uint32_t)(P[4] >> 32), (uint32_t)(P[5] >> 32), (uint32_t)(P[6] >> 32), (uint32_t)(P[7] >> 32));
    r1[2] = make_uint4((uint32_t)(N[0] >> 32), (uint32_t)(N[1] >> 32), (uint32_t)(N[2] >> 32), (uint32_t)(N[3] >> 32));
    r1[3] = make_uint4((uint32_t)(N[4] >> 32), (uint32_t)(N[5] >> 32), (uint32_t)(N[6] >> 32), (uint32_t)(N[7] >> 32));
    r1[4] = make_uint4((uint32_t)(mw >> 32), 0u, 0u, 0u);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int grp = 0; grp * 4 < nk; ++grp) {
      const int kk = grp * 4 + (lane >> 4);
      const int shn = 4 * (lane & 7);
      const uint4* r = reinterpret_cast<const uint4*>(my + (kk * 2 + ((lane >> 3) & 1)) * kRecT);
      const uint4 p03 = r[0];
      const uint4 p47 = r[1];
      const uint4 n03 = r[2];
      const uint4 n47 = r[3];
      const uint32_t mnib = (r[4].x >> shn) & 15u;
      auto spread = [&](uint32_t plane) { return (((plane >> shn) & 15u) * 0x00204081u) & 0x01010101u; };
      uint32_t cp4 = spread(p03.x) | (spread(p03.y) << 1) | (spread(p03.z) << 2) | (spread(p03.w) << 3);
      uint32_t cn4 = spread(n03.x) | (spread(n03.y) << 1) | (spread(n03.z) << 2) | (spread(n03.w) << 3);
      if (nplanes > 4) {
        cp4 |= (spread(p47.x) << 4) | (spread(p47.y) << 5) | (spread(p47.z) << 6) | (spread(p47.w) << 7);
        cn4 |= (spread(n47.x) << 4) | (spread(n47.y) << 5) | (spread(n47.z) << 6) | (spread(n47.w) << 7);
      }
      const int64_t i0 = (k0 + grp * 4) * 64 + 4 * lane;  // first of my four elements in the bucket
      if (kk >= nk || i0 >= nbe) continue;
      auto value = [&](int e) {
        return tab[(int)((cp4 >> (8 * e)) & 255u) - (int)((cn4 >> (8 * e)) & 255u) + a.W];
      };
      if (i0 + 3 < nbe) {
        if (c4) {
          __builtin_nontemporal_store(cp4, reinterpret_cast<uint32_t*>(a.cpos + base + i0));
          __builtin_nontemporal_store(cn4, reinterpret_cast<uint32_t*>(a.cneg + base + i0));
        } else if (a.cpos && a.cneg) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            a.cpos[base + i0 + e] = (uint8_t)(cp4 >> (8 * e));
            a.cneg[base + i0 + e] = (uint8_t)(cn4 >> (8 * e));
          }
        }
        if (a.out) {
          if (o16 && mnib == 15u) {
            const f32x4 y = {value(0), value(1), value(2), value(3)};
            __builtin_nontemporal_store(y, reinterpret_cast<f32x4*>(a.out + base + i0));
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if ((mnib >> e) & 1u) a.out[base + i0 + e] = value(e);
          }
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (i0 + e < nbe) {
            if (a.cpos && a.cneg) {
              a.cpos[base + i0 + e] = (uint8_t)(cp4 >> (8 * e));
              a.cneg[base + i0 + e] = (uint8_t)(cn4 >> (8 * e));
            }
            if (a.out && ((mnib >> e) & 1u)) a.out[base + i0 + e] = value(e);
          }
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// --------------------------------------------------------------- launchers

template <bool PACK>
static hipError_t pass1_dispatch(const Geometry& geo, const Pass1Args& a, hipStream_t s) {
  const dim3 block(kThreads1);
  const int cw = geo.G * geo.eg * pass1_words(geo.wpw);
  size_t smem = PACK ? (size_t)geo.W * cw * sizeof(uint64_t) : 0;
  if (a.sums != kSumsNone) smem += (size_t)geo.W * geo.tile * sizeof(float);
  smem += (size_t)geo.G * geo.eg * pass1_words(geo.wpw) * sizeof(uint64_t);  // mask words of a mixed chunk
  const size_t red = (size_t)geo.eg * geo.W * sizeof(Partial) + (size_t)geo.eg * sizeof(uint64_t);
  if (smem < red) smem = red;
  if (smem > 65536) {
    // Above 64 KiB of dynamic LDS the kernel must opt in (gfx950 has 160 KiB per CU).
    hipError_t e = hipSuccess;
    switch (geo.wpw) {
      case 1: e = hipFuncSetAttribute((const void*)k_pass1<1, PACK>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
      case 2: e = hipFuncSetAttribute((const void*)k_pass1<2, PACK>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
      case 4: e = hipFuncSetAttribute((const void*)k_pass1<4, PACK>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
      case 8: e = hipFuncSetAttribute((const void*)k_pass1<8, PACK>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
      case 16: e = hipFuncSetAttribute((const void*)k_pass1<16, PACK>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
      default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
  }
  // One launch per epoch of chunks (see the geometry notes).  The first
  // launch is ordered after earlier work on the stream; later ones may
  // start while the one before drains: every chunk writes only its own
  // partial slot and sign words.  The next ordered launch (the decision)
  // waits for all.
  const uint32_t overlap = hipExtAnyOrderLaunch;
  const int64_t epoch = pass1_launch_chunks(geo, PACK);
  for (int64_t q0 = 0; q0 < geo.total_chunks; q0 += epoch) {
    const int64_t left = geo.total_chunks - q0;
    const dim3 grid((unsigned)(left < epoch ? left : epoch));
    const uint32_t fl = q0 > 0 ? overlap : 0u;
    switch (geo.wpw) {
      case 1: hipExtLaunchKernelGGL((k_pass1<1, PACK>), grid, block, smem, s, nullptr, nullptr, fl, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a, q0); break;
      case 2: hipExtLaunchKernelGGL((k_pass1<2, PACK>), grid, block, smem, s, nullptr, nullptr, fl, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a, q0); break;
      case 4: hipExtLaunchKernelGGL((k_pass1<4, PACK>), grid, block, smem, s, nullptr, nullptr, fl, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a, q0); break;
      case 8: hipExtLaunchKernelGGL((k_pass1<8, PACK>), grid, block, smem, s, nullptr, nullptr, fl, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a, q0); break;
      case 16: hipExtLaunchKernelGGL((k_pass1<16, PACK>), grid, block, smem, s, nullptr, nullptr, fl, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a, q0); break;
      default: return hipErrorInvalidValue;
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_pass1(const Geometry& geo, const Pass1Args& a, hipStream_t s) {
  return a.bits ? pass1_dispatch<true>(geo, a, s) : pass1_dispatch<false>(geo, a, s);
}

hipError_t launch_decide(const Geometry& geo, const DecideArgs& a, hipStream_t s) {
  if (geo.gs > 0) {
    hipLaunchKernelGGL(k_slotsum, dim3((unsigned)(geo.nb * geo.groups)), dim3(256), 0, s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_decide, dim3((unsigned)geo.nb), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_ternary_pack(const Geometry& geo, const TernArgs& a0, hipStream_t s) {
  TernArgs a = a0;
  a.chunks_full = geo.chunks_full;
  a.total_chunks = geo.total_chunks;
  a.nb = (int32_t)geo.nb;
  a.wg = geo.wg;
  a.eg = geo.eg;
  a.T = geo.T;
  a.G = geo.G;
  // Both planes of a chunk: 2 * W * G * EG * (T / 64) words, at most 64 KiB.
  const size_t smem = 2 * (size_t)geo.W * geo.G * geo.eg * pass1_words(geo.wpw) * sizeof(uint64_t);
  if (smem > 65536) return hipErrorInvalidValue;
  // No chunk shares state with another, so every launch after the first may
  // start while the one before drains.
  const int64_t epoch = one_launch_epoch(geo.total_chunks);  // chunks share no state here
  for (int64_t q0 = 0; q0 < geo.total_chunks; q0 += epoch) {
    const int64_t left = geo.total_chunks - q0;
    const dim3 grid((unsigned)(left < epoch ? left : epoch));
    const uint32_t fl = q0 > 0 ? hipExtAnyOrderLaunch : 0u;
    switch (geo.wpw) {
      case 1: hipExtLaunchKernelGGL((k_tpack<1>), grid, dim3(kThreads1), smem, s, nullptr, nullptr, fl, a, q0); break;
      case 2: hipExtLaunchKernelGGL((k_tpack<2>), grid, dim3(kThreads1), smem, s, nullptr, nullptr, fl, a, q0); break;
      case 4: hipExtLaunchKernelGGL((k_tpack<4>), grid, dim3(kThreads1), smem, s, nullptr, nullptr, fl, a, q0); break;
      case 8: hipExtLaunchKernelGGL((k_tpack<8>), grid, dim3(kThreads1), smem, s, nullptr, nullptr, fl, a, q0); break;
      case 16: hipExtLaunchKernelGGL((k_tpack<16>), grid, dim3(kThreads1), smem, s, nullptr, nullptr, fl, a, q0); break;
      default: return hipErrorInvalidValue;
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_ternary_reduce(const Geometry& geo, const TernArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_tpass2, dim3((unsigned)geo.bpb2, (unsigned)geo.nb), dim3(kThreads2), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_pass2(const Geometry& geo, const Pass2Args& a, hipStream_t s) {
  const unsigned nz = a.nz > 0 ? (unsigned)a.nz : 1u;
  hipLaunchKernelGGL(k_pass2, dim3((unsigned)geo.bpb2, (unsigned)geo.nb, nz), dim3(kThreads2), 0, s,
                     a.bits, a.g, a.mask, a.dec, a.scale, a.counts, a.out, a);
  return hipGetLastError();
}

// ------------------------------------------------- partial-count reduction
//
// Inter-node step of the hierarchical reducer: c_i = sum over the G rows of
// uint8 partial counts, then the aggregate return (decode) as in pass 2.  A
// thread takes 16 consecutive elements: one 16-byte load per partial row,
// summed as packed bytes in 32-bit adds (every byte's sum is at most W <=
// 255, so no carry crosses a byte), one 16-byte store of counts, and the
// 16 decoded values through an LDS table of fl32(scale * q[c]).
__global__ __launch_bounds__(kThreads2) void k_psum(PsumArgs a) {
  __shared__ float tab[256];
  if (a.out) {
    const float scale = *a.scale;
    for (int c = threadIdx.x; c <= a.W; c += kThreads2) tab[c] = scale * decode_q(c, a.W, a.decode_mode);
    __syncthreads();
  }
  const int64_t ngroups = (a.n + 15) / 16;
  const bool c16 = a.counts && ((reinterpret_cast<uintptr_t>(a.counts) & 15) == 0);
  const bool o16 = a.out && ((reinterpret_cast<uintptr_t>(a.out) & 15) == 0);
  for (int64_t t = (int64_t)blockIdx.x * kThreads2 + threadIdx.x; t < ngroups; t += (int64_t)gridDim.x * kThreads2) {
    const int64_t i0 = t * 16;
    const int cnt = (a.n - i0) < 16 ? (int)(a.n - i0) : 16;
    uint32_t c[4] = {0u, 0u, 0u, 0u};
    if (cnt == 16) {
      for (int gr = 0; gr < a.G; ++gr) {
        const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(a.partial + (int64_t)gr * a.pstride + i0));
        c[0] += v[0];
        c[1] += v[1];
        c[2] += v[2];
        c[3] += v[3];
      }
    } else {
      for (int gr = 0; gr < a.G; ++gr)
        for (int e = 0; e < cnt; ++e) c[e / 4] += (uint32_t)a.partial[(int64_t)gr * a.pstride + i0 + e] << (8 * (e % 4));
    }
    if (a.counts) {
      if (cnt == 16 && c16) {
        const u32x4 cv = {c[0], c[1], c[2], c[3]};
        __builtin_nontemporal_store(cv, reinterpret_cast<u32x4*>(a.counts + i0));
      } else {
        for (int e = 0; e < cnt; ++e) a.counts[i0 + e] = (uint8_t)(c[e / 4] >> (8 * (e % 4)));
      }
    }
    if (a.out) {
      const uint32_t m16 = (uint32_t)(a.mask[i0 / 64] >> (i0 & 63)) & 0xffffu;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t cw = c[q];
        const uint32_t mq = (m16 >> (4 * q)) & 15u;
        const int64_t j = i0 + 4 * q;
        if (cnt == 16 && o16 && mq == 15u) {
          const f32x4 y = {tab[cw & 255u], tab[(cw >> 8) & 255u], tab[(cw >> 16) & 255u], tab[cw >> 24]};
          __builtin_nontemporal_store(y, reinterpret_cast<f32x4*>(a.out + j));
        } else {
          for (int e = 0; e < 4; ++e)
            if (4 * q + e < cnt && ((mq >> e) & 1u)) a.out[j + e] = tab[(cw >> (8 * e)) & 255u];
        }
      }
    }
  }
}

hipError_t launch_psum(const PsumArgs& a, hipStream_t s) {
  const int64_t ngroups = (a.n + 15) / 16;
  int64_t blocks = (ngroups + kThreads2 - 1) / kThreads2;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_psum, dim3((unsigned)blocks), dim3(kThreads2), 0, s, a);
  return hipGetLastError();
}

}  // namespace nf
