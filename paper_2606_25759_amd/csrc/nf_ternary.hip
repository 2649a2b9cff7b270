// nf_ternary.hip - G-Ternary write side and count/decode (§2.2; gfx950).
//
//   k_tpack   both planes per worker, laid out as pass 1's chunks
//   k_tpass2  pass 2's bit-sliced counter over the positive and the negative
//             planes, decoded from their difference
#include <hip/hip_ext.h>

#include "nf_device.h"

namespace nf {

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
  int64_t c, base, nbe, chunk0;
  chunk_home(q, a.btab, a.cbucket, a.nb, a.chunks_full, b, c);
  if (a.dec && a.dec[b].route != NF_ROUTE_LOWBIT) return;  // whole block: no planes
  bucket_span(b, a.btab, a.n_total, a.bucket_n, 0, base, nbe, chunk0);
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
  // This launch's rows: workers wbase .. wbase + R - 1; w below is a row of
  // the group, and the planes of the group's rows start at pbits (positive)
  // and nbits (negative).
  const int R = a.rows;
  const float* g = a.g + (int64_t)a.wbase * a.wstride;
  uint64_t* pbits = a.bits + (int64_t)a.wbase * a.bstride;
  uint64_t* nbits = a.bits + (int64_t)(a.W + a.wbase) * a.bstride;
  uint64_t* ppos = reinterpret_cast<uint64_t*>(smem);
  uint64_t* pneg = ppos + (size_t)R * cw;

  float th[WPW];
  const float* rp[WPW];
#pragma unroll
  for (int j = 0; j < WPW; ++j) {
    const int w = wg + j * a.wg;
    const int wl = w < R ? w : wg;
    th[j] = a.dec ? ternary_threshold(a.stats[(int64_t)b * a.W + a.wbase + wl], a.dec[b].n_eligible, a.tau)
                  : a.theta[a.wbase + wl];
    rp[j] = g + (int64_t)wl * a.wstride + base + (int64_t)eg * T + lane;
  }
  const uint64_t* mbase = a.mask + base / 64 + (int64_t)eg * (T / 64);
  // The first NW words of the bucket's first tile (full whenever any tile of
  // this chunk is): read by loads whose values are not needed.
  const float* dp = g + (int64_t)wg * a.wstride + base + lane;
  const uint64_t* dm = a.mask + base / 64;

  bool chunk_all = false, chunk_any = true;  // set below, after the first tile's loads are out

  // Loads of a full tile (or, for an idle wavefront or a tile past the full
  // ones, of the bucket's first words).
  auto issue_data = [&](int64_t tt, float (&X)[NX]) {
    const bool ok = active && tt < te_full;
    const int64_t o = tt * tile;
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
      const float* row = ok ? rp[j] + o : dp;
#pragma unroll
      for (int k = 0; k < NW; ++k) X[j * NW + k] = __builtin_nontemporal_load(row + 64 * k);
    }
  };
  auto issue_mask = [&](int64_t tt, uint64_t (&M)[NW]) {
    const bool ok = active && tt < te_full;
    const int64_t o = tt * tile;
    if (chunk_all) {
      // every element of the chunk eligible: no mask words to load
#pragma unroll
      for (int k = 0; k < NW; ++k) M[k] = ~0ull;
      return;
    }
    const uint64_t* mrow = ok ? mbase + o / 64 : dm;
#pragma unroll
    for (int k = 0; k < NW; ++k) M[k] = uniform64(mrow[k]);
  };
  auto issue = [&](int64_t tt, float (&X)[NX], uint64_t (&M)[NW]) {
    issue_data(tt, X);
    issue_mask(tt, M);
  };
  auto body = [&](int64_t t, const float (&X)[NX], const uint64_t (&M)[NW]) {
    const int ti = (int)(t - tb);
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
      const int w = wg + j * a.wg;
      if (j > 0 && w >= R) continue;
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
  if (te_full > tb) issue_data(tb, xa);
  // Whether every element of the chunk is eligible (then the tiles need no
  // mask words), and whether any is: a chunk with none is not read.
  {
    const int64_t cn = ((te * tile < nbe) ? te * tile : nbe) - tb * tile;  // elements of the chunk
    const int nwc = cn > 0 ? (int)((cn + 63) / 64) : 0;
    const uint64_t* cm = a.mask + (base + tb * tile) / 64;
    int any = 0, notall = cn % 64 != 0;  // a ragged chunk keeps its mask loads
    for (int i = threadIdx.x; i < nwc; i += kThreads1) {
      const uint64_t m = cm[i] & (i == nwc - 1 ? low_bits(cn - 64 * (int64_t)i) : ~0ull);
      any |= m != 0ull;
      notall |= m != ~0ull;
    }
    chunk_any = __syncthreads_or(any);
    chunk_all = !__syncthreads_or(notall);
  }

  // A chunk with no eligible element: both planes are zero and nothing more
  // is read (mask bits past the bucket's end do not count).
  if (!chunk_any) {
    if (te_full > tb) consume(xa);
    {
      const int64_t cn = ((te * tile < nbe) ? te * tile : nbe) - tb * tile;
      const int nwc = cn > 0 ? (int)((cn + 63) / 64) : 0;
      const int64_t gz = (base + tb * tile) / 64;
      for (int i = threadIdx.x; i < R * nwc; i += kThreads1) {
        const int w = i / nwc;
        const int o = i - w * nwc;
        pbits[(int64_t)w * a.bstride + gz + o] = 0ull;
        nbits[(int64_t)w * a.bstride + gz + o] = 0ull;
      }
      return;
    }
  }
  if (te_full > tb) issue_mask(tb, ma);
  int64_t t = tb;
  if (te_full > tb) {
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
      if (w >= R) break;
      for (int o = lane; o < valid; o += 64) {
        pbits[(int64_t)w * a.bstride + gw0 + o] = ppos[w * cw + o];
        nbits[(int64_t)w * a.bstride + gw0 + o] = pneg[w * cw + o];
      }
    }
    return;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < R * valid; i += kThreads1) {
    const int w = i / valid;
    const int o = i - w * valid;
    pbits[(int64_t)w * a.bstride + gw0 + o] = ppos[w * cw + o];
    nbits[(int64_t)w * a.bstride + gw0 + o] = pneg[w * cw + o];
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
  int64_t base, nbe, chunk0;
  bucket_span(b, a.btab, a.n_total, a.bucket_n, 0, base, nbe, chunk0);
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

hipError_t launch_ternary_pack(const Geometry& geo, const TernArgs& a0, hipStream_t s) {
  TernArgs a = a0;
  a.chunks_full = geo.chunks_full;
  a.total_chunks = geo.total_chunks;
  a.nb = (int32_t)geo.nb;
  a.wg = geo.wg;
  a.eg = geo.eg;
  a.T = geo.T;
  a.G = geo.G;
  // Both planes of a chunk: 2 * R * G * EG * (T / 64) words, at most 64 KiB.
  const size_t smem = 2 * (size_t)geo.rows * geo.G * geo.eg * pass1_words(geo.wpw) * sizeof(uint64_t);
  if (smem > 65536) return hipErrorInvalidValue;
  // No chunk or row group shares state with another, so every launch after
  // the first may start while the one before drains.
  const int64_t epoch = one_launch_epoch(geo.total_chunks);  // chunks share no state here
  for (int grp = 0; grp < geo.ngroups; ++grp) {
    row_group(geo, grp, &a.wbase, &a.rows);
    // every wavefront's first worker (wg < geo.wg) must be a row of the group
    if (a.rows < geo.wg || a.rows > geo.rows) return hipErrorInvalidValue;
    for (int64_t q0 = 0; q0 < geo.total_chunks; q0 += epoch) {
      const int64_t left = geo.total_chunks - q0;
      const dim3 grid((unsigned)(left < epoch ? left : epoch));
      const uint32_t fl = (q0 > 0 || grp > 0) ? hipExtAnyOrderLaunch : 0u;
      switch (geo.wpw) {
        case 1: hipExtLaunchKernelGGL((k_tpack<1>), grid, dim3(kThreads1), smem, s, nullptr, nullptr, fl, a, q0); break;
        case 2: hipExtLaunchKernelGGL((k_tpack<2>), grid, dim3(kThreads1), smem, s, nullptr, nullptr, fl, a, q0); break;
        case 4: hipExtLaunchKernelGGL((k_tpack<4>), grid, dim3(kThreads1), smem, s, nullptr, nullptr, fl, a, q0); break;
        default: return hipErrorInvalidValue;
      }
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

hipError_t launch_ternary_reduce(const Geometry& geo, const TernArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_tpass2, dim3((unsigned)geo.bpb2, (unsigned)geo.nb), dim3(kThreads2), 0, s, a);
  return hipGetLastError();
}

}  // namespace nf
