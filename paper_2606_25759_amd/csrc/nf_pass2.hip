// nf_pass2.hip - read side of the bucket reducer (gfx950).
//
//   k_pass2   read side (§3.3 step 7, §6.1): per-coordinate sign counts over
//             the W bitmaps and the scaled decode; or the FP32 sum of the
//             eligible positions when the bucket falls back.
//   k_psum    inter-node step of the hierarchical reducer (§6.1): the sum of
//             uint8 partial counts and the aggregate return.
#include <hip/hip_ext.h>

#include "nf_device.h"

namespace nf {

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
  int64_t base, nbe, chunk0;
  bucket_span(b, a.btab, a.n_total, a.bucket_n, 0, base, nbe, chunk0);
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
      // unrolled so that the partial rows' loads are in flight together
#pragma unroll 8
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
          // A cached store: the four stores of a thread are 64 bytes apart
          // across the lanes, and L2 merges them into whole lines (as
          // nontemporal stores the exchange took 38 us instead of 16 us at
          // 6,553,600 elements).
          *reinterpret_cast<f32x4*>(a.out + j) = y;
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
