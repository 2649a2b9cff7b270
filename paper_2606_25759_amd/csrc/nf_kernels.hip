// nf_kernels.hip - gfx950 kernels of the bucket reducer.
//
//   k_pass1   write side (§3.3 step 5, §5.2): one read of the W gradient
//             rows; sign payload by wavefront ballot, per-worker health in
//             registers, FP32 sums at routed positions through an LDS stage.
//   k_decide  one block per bucket: fixed-order reduction of the pass-1
//             partial statistics, then the route rules (§3.2, §6.4).
//   k_pass2   read side (§3.3 step 7, §6.1): per-coordinate sign counts over
//             the W bitmaps and the scaled decode; or the FP32 sum of the
//             eligible positions when the bucket falls back.
//
// The path is bound by HBM bandwidth, so there is no MFMA: every step is a
// streaming scan with a handful of VALU operations per element and worker.
#include "nf_internal.h"

namespace nf {

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
    asm volatile(
        "s_nop 4\n"
        "v_writelane_b32 %0, %2, 0\n v_writelane_b32 %1, %3, 0\n"
        "v_writelane_b32 %0, %4, 1\n v_writelane_b32 %1, %5, 1\n"
        "v_writelane_b32 %0, %6, 2\n v_writelane_b32 %1, %7, 2\n"
        "v_writelane_b32 %0, %8, 3\n v_writelane_b32 %1, %9, 3\n"
        "v_writelane_b32 %0, %10, 4\n v_writelane_b32 %1, %11, 4\n"
        "v_writelane_b32 %0, %12, 5\n v_writelane_b32 %1, %13, 5\n"
        "v_writelane_b32 %0, %14, 6\n v_writelane_b32 %1, %15, 6\n"
        "v_writelane_b32 %0, %16, 7\n v_writelane_b32 %1, %17, 7\n"
        : "=v"(lo), "=v"(hi)
        : "s"(l[0]), "s"(h[0]), "s"(l[1]), "s"(h[1]), "s"(l[2]), "s"(h[2]), "s"(l[3]), "s"(h[3]),
          "s"(l[4]), "s"(h[4]), "s"(l[5]), "s"(h[5]), "s"(l[6]), "s"(h[6]), "s"(l[7]), "s"(h[7]));
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
// each) per worker and tile.  Lane l of a wavefront loads element 64k + l of word k, so
// every load instruction reads 256 contiguous bytes and the ballot of
// "g > 0" over the wavefront is exactly bitmap word k.
template <int WPW, bool PACK>
__global__ __launch_bounds__(kThreads1) __attribute__((amdgpu_waves_per_eu(WPW <= 2 ? 8 : 4))) void k_pass1(const float* __restrict__ g,
                                                     const uint64_t* __restrict__ mask,
                                                     uint64_t* __restrict__ bits,
                                                     float* __restrict__ out,
                                                     Partial* __restrict__ part,
                                                     uint64_t* __restrict__ part_ne, Pass1Args a) {
  constexpr int NW = pass1_words(WPW);
  extern __shared__ __align__(16) unsigned char smem[];
  float* stage = reinterpret_cast<float*>(smem);

  const int b = blockIdx.y;
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
  const bool stage_on = a.sums != kSumsNone;

  double sabs[WPW], ssq[WPW];
  uint64_t nonf[WPW];
#pragma unroll
  for (int j = 0; j < WPW; ++j) {
    sabs[j] = 0.0;
    ssq[j] = 0.0;
    nonf[j] = 0;
  }
  uint64_t ne = 0;

  for (int64_t t = blockIdx.x; t < ntiles; t += a.bpb) {
    const int64_t t0 = t * tile;
    // Tile class, identical in every wavefront: full and eligible everywhere
    // (no FP32 sums needed) or general (partial, mixed or routed).
    bool fast = (t0 + tile <= nbe) && a.sums != kSumsAll;
    if (fast) {
      const uint64_t* mt = mask + (base + t0) / 64;
      bool ok = true;
      for (int k = lane; k < tile / 64; k += 64) ok = ok && (mt[k] == ~0ull);
      fast = __all(ok);
    }
    const int64_t e0 = t0 + (int64_t)eg * T;
    int64_t c64 = nbe - e0;
    const int cnt = active ? (int)(c64 < 0 ? 0 : (c64 > T ? T : c64)) : 0;
    const int64_t wrd0 = (base + e0) / 64;  // first word of my element group

    if (fast) {
      if (active) {
#pragma unroll
        for (int j = 0; j < WPW; ++j) {
          const int w = wg + j * a.wg;
          if (j > 0 && w >= a.W) break;
          const float* row = g + (int64_t)w * a.wstride + base + e0 + lane;
          float x[NW];
#pragma unroll
          for (int k = 0; k < NW; ++k) x[k] = __builtin_nontemporal_load(row + 64 * k);
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
            if (lane < NW) bits[(int64_t)w * a.bstride + wrd0 + lane] = ((uint64_t)whi << 32) | wlo;
          }
          if (__ballot(!finite64(s2))) {
#pragma unroll
            for (int k = 0; k < NW; ++k) nonf[j] += __popcll(__ballot(!finite32(x[k])));
          }
          sabs[j] += s1;
          ssq[j] += s2;
        }
        if (wg == 0) ne += (uint64_t)T;
      }
    } else {
      if (active) {
        const uint64_t* mrow = mask + wrd0;
        uint64_t mw[NW];
#pragma unroll
        for (int k = 0; k < NW; ++k) mw[k] = 64 * k < cnt ? (mrow[k] & low_bits(cnt - 64 * k)) : 0ull;
        const int nwv = (cnt + 63) / 64;
#pragma unroll
        for (int j = 0; j < WPW; ++j) {
          const int w = wg + j * a.wg;
          if (j > 0 && w >= a.W) break;
          const float* row = g + (int64_t)w * a.wstride + base + e0 + lane;
          float x[NW];
#pragma unroll
          for (int k = 0; k < NW; ++k) x[k] = (64 * k + lane < cnt) ? __builtin_nontemporal_load(row + 64 * k) : 0.0f;
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
            if (lane < nwv) bits[(int64_t)w * a.bstride + wrd0 + lane] = ((uint64_t)whi << 32) | wlo;
          }
          if (__ballot(!finite64(s2))) {
#pragma unroll
            for (int k = 0; k < NW; ++k) nonf[j] += __popcll(__ballot(!finite32(x[k])));
          }
          sabs[j] += s1;
          ssq[j] += s2;
          if (stage_on) {
            float* st = stage + (int64_t)w * tile + eg * T + lane;
#pragma unroll
            for (int k = 0; k < NW; ++k) st[64 * k] = x[k];
          }
        }
        if (wg == 0) {
#pragma unroll
          for (int k = 0; k < NW; ++k) ne += __popcll(mw[k]);
        }
      }
      if (stage_on) {
        __syncthreads();
        // Workers added in order w = 0..W-1 at each staged position.
        const int lim = (int)((nbe - t0) < tile ? (nbe - t0) : tile);
        for (int e = threadIdx.x; e < lim; e += kThreads1) {
          const int64_t i = base + t0 + e;
          const bool routed = !((mask[i >> 6] >> (i & 63)) & 1ull);
          if (a.sums == kSumsAll || routed) {
            float s = stage[e];
            for (int w = 1; w < a.W; ++w) s = s + stage[w * tile + e];
            if (a.mean) s = s / (float)a.W;
            out[i] = s;
          }
        }
        __syncthreads();
      }
    }
  }

  // Block partials: wavefront sums, then element groups in order.
  __syncthreads();
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
  const int64_t slot = (int64_t)b * a.bpb + blockIdx.x;
  for (int w = threadIdx.x; w < a.W; w += kThreads1) {
    Partial p = red[w];
    for (int e = 1; e < a.eg; ++e) {
      const Partial q = red[e * a.W + w];
      p.sabs += q.sabs;
      p.ssq += q.ssq;
      p.nonfinite += q.nonfinite;
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
__global__ __launch_bounds__(256) void k_decide(DecideArgs a) {
  __shared__ nf_worker_stats st[256];
  __shared__ uint64_t ne_s;
  __shared__ int kfin_s;
  __shared__ double med_s;
  const int b = blockIdx.x;
  const int v = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wavefront index, uniform
  const int lane = threadIdx.x & 63;
  const Partial* P = a.part + (int64_t)b * a.bpb * a.W;
  for (int w = v; w < a.W; w += 4) {
    double s1 = 0.0, s2 = 0.0;
    uint64_t nf = 0;
    for (int k = lane; k < a.bpb; k += 64) {
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
    for (int k = lane; k < a.bpb; k += 64) s += a.part_ne[(int64_t)b * a.bpb + k];
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
    const int64_t n = bucket_len(a.n_total, a.bucket_n, b);
    decide_from(st, a.W, n, (int64_t)ne_s, a.pol, kfin, med_s, &d);
    a.dec[b] = d;
  }
}

// ------------------------------------------------------------------ pass 2
__global__ __launch_bounds__(kThreads2) void k_pass2(
    const uint64_t* __restrict__ bits, const float* __restrict__ g, const uint64_t* __restrict__ mask,
    const nf_route_decision* __restrict__ dec, const float* __restrict__ scale_p,
    uint8_t* __restrict__ counts, float* __restrict__ out, Pass2Args a) {
  __shared__ float tab[256];
  const int b = blockIdx.y;
  const int64_t base = (int64_t)b * a.bucket_n;
  const int64_t nbe = bucket_len(a.n_total, a.bucket_n, b);
  int op = a.op;
  int sel = a.select;
  float scale = 0.0f;
  if (op == kOpFromDecision) {
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
  constexpr int K = kWordsPerWave2;
  for (int64_t ch = (int64_t)blockIdx.x * 4 + v; ch * K < nwords; ch += (int64_t)a.bpb2 * 4) {
    const int64_t k0 = ch * K;
    const int nk = (int)((nwords - k0) < K ? (nwords - k0) : K);
    if (op == kOpCountDecode) {
      uint32_t c[K];
#pragma unroll
      for (int k = 0; k < K; ++k) c[k] = 0;
      for (int w = 0; w < a.W; ++w) {
        const uint64_t* brow = bits + (int64_t)w * a.bstride + wbase + k0;
        if (nk == K) {
#pragma unroll
          for (int k = 0; k < K; ++k) c[k] = add_lane_bit(c[k], brow[k]);
        } else {
#pragma unroll
          for (int k = 0; k < K; ++k)
            if (k < nk) c[k] = add_lane_bit(c[k], brow[k]);
        }
      }
#pragma unroll
      for (int k = 0; k < K; ++k) {
        if (k >= nk) break;
        const int64_t i = (k0 + k) * 64 + lane;
        if (i < nbe) {
          if (counts) counts[base + i] = (uint8_t)c[k];
          if (out && ((mask[wbase + k0 + k] >> lane) & 1ull)) out[base + i] = tab[c[k]];
        }
      }
    } else {
      float s[K];
      uint64_t selw[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        uint64_t m = 0;
        if (k < nk) {
          const uint64_t mw = mask ? mask[wbase + k0 + k] : ~0ull;
          m = sel == NF_SEL_ALL ? ~0ull : (sel == NF_SEL_ELIGIBLE ? mw : ~mw);
          m &= low_bits(nbe - (k0 + k) * 64);
        }
        selw[k] = m;
        s[k] = 0.0f;
      }
      for (int w = 0; w < a.W; ++w) {
        const float* row = g + (int64_t)w * a.wstride + base + k0 * 64 + lane;
#pragma unroll
        for (int k = 0; k < K; ++k) {
          if ((selw[k] >> lane) & 1ull) {
            const float x = __builtin_nontemporal_load(row + 64 * k);
            s[k] = w == 0 ? x : s[k] + x;
          }
        }
      }
#pragma unroll
      for (int k = 0; k < K; ++k) {
        if ((selw[k] >> lane) & 1ull) {
          float y = s[k];
          if (a.mean) y = y / (float)a.W;
          out[base + (k0 + k) * 64 + lane] = y;
        }
      }
    }
  }
}

// --------------------------------------------------------------- launchers

template <bool PACK>
static hipError_t pass1_dispatch(const Geometry& geo, const Pass1Args& a, hipStream_t s) {
  const dim3 grid((unsigned)geo.bpb, (unsigned)geo.nb);
  const dim3 block(kThreads1);
  size_t red = (size_t)geo.eg * geo.W * sizeof(Partial) + (size_t)geo.eg * sizeof(uint64_t);
  size_t smem = a.sums != kSumsNone ? (size_t)geo.W * geo.tile * sizeof(float) : 0;
  if (smem < red) smem = red;
  switch (geo.wpw) {
    case 1: hipLaunchKernelGGL((k_pass1<1, PACK>), grid, block, smem, s, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a); break;
    case 2: hipLaunchKernelGGL((k_pass1<2, PACK>), grid, block, smem, s, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a); break;
    case 4: hipLaunchKernelGGL((k_pass1<4, PACK>), grid, block, smem, s, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a); break;
    case 8: hipLaunchKernelGGL((k_pass1<8, PACK>), grid, block, smem, s, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a); break;
    case 16: hipLaunchKernelGGL((k_pass1<16, PACK>), grid, block, smem, s, a.g, a.mask, a.bits, a.out, a.part, a.part_ne, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_pass1(const Geometry& geo, const Pass1Args& a, hipStream_t s) {
  return a.bits ? pass1_dispatch<true>(geo, a, s) : pass1_dispatch<false>(geo, a, s);
}

hipError_t launch_decide(const Geometry& geo, const DecideArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_decide, dim3((unsigned)geo.nb), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_pass2(const Geometry& geo, const Pass2Args& a, hipStream_t s) {
  hipLaunchKernelGGL(k_pass2, dim3((unsigned)geo.bpb2, (unsigned)geo.nb), dim3(kThreads2), 0, s,
                     a.bits, a.g, a.mask, a.dec, a.scale, a.counts, a.out, a);
  return hipGetLastError();
}

}  // namespace nf
