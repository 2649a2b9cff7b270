// nf_device.h - device helpers shared by the reducer's kernels: vector
// types, finiteness tests, wavefront sums, ballots moved into lanes, and the
// bit-sliced (carry-save) counter of sign words over worker rows.
#pragma once

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

// ------------------------------------------------- exactly rounded sums
//
// A sum of non-negative FP64 terms carried as XSum {s, c, b}: s is the
// running FP64 sum, c gathers the exact rounding error of every addition
// into s (Knuth's TwoSum), and b bounds how far c, itself summed in FP64, is
// from the sum of those errors.  So the exact total lies within b of s + c,
// and with b = 0 it is s + c exactly, whose one FP64 rounding fl(s + c) is
// then the exact total rounded to nearest even.  b stays 0 while every
// addition into c is exact, which holds whenever the terms' exponents span
// less than about 100 binades.  A non-finite s (a NaN or infinite term) is
// the IEEE sum itself.
struct XSum {
  double s, c, b;
};

// t + e == a + x exactly, t = fl(a + x) (finite a, x; no reassociation).
__device__ __forceinline__ void two_sum(double a, double x, double& t, double& e) {
  t = a + x;
  const double z = t - a;
  e = (a - (t - z)) + (x - z);
}

// One term into a lane's running (s, c); nz counts the nonzero errors added
// to c (c is exact while at most one has been: 0 + e is exact).
__device__ __forceinline__ void xadd(double& s, double& c, uint32_t& nz, double x) {
  double t, e;
  two_sum(s, x, t, e);
  s = t;
  c += e;
  nz += e != 0.0 ? 1u : 0u;
}

// Exact mode.  A plain FP64 sum of non-negative FP32 terms (in any order of
// additions) is exact when its result p < 2^53 q, q the quantum of the
// smallest nonzero term: every exact partial sum is a multiple of q, and
// multiples of q up to 2^53 q are representable, so a first inexact step
// would need an exact partial above 2^53 q, after which every computed
// partial stays >= 2^53 q (rounding is monotonic and the terms are >= 0).
// um tracks the minimum of (bits(x) << 1) - 1 over the terms (zeros wrap to
// the top, and the shift drops the sign), so (um + 1) >> 24 is the smallest
// nonzero term's exponent field e, whose quantum is 2^(max(e, 1) - 150).
__device__ __forceinline__ uint32_t term_umin(uint32_t um, float x) {
  const uint32_t v = (__float_as_uint(x) << 1) - 1u;
  return v < um ? v : um;  // unsigned: a zero's wrapped value stays the largest
}

__device__ __forceinline__ bool sum_is_exact(double p, uint32_t um) {
  const uint32_t e = (um + 1u) >> 24;
  const uint32_t eb = (e > 1u ? e : 1u) + 926u;  // biased FP64 exponent of 2^53 q
  return p < __longlong_as_double((long long)((uint64_t)eb << 52));
}

// One tile of a lane's |g| terms into its running sum.  p is the tile's
// plain sum and umt its terms' um.  While the lane's plain sum s stays
// proven exact (s + p checked against every term so far, uml), the tile
// enters by one plain addition.  The first tile that breaks the proof (a
// term below about 2^-29 of the lane's sum, or a non-finite one; rare)
// switches the lane to TwoSum for the rest of its terms (tw): a tile then
// enters (s, c) by TwoSum as one term p when p alone is proven exact, else
// term by term (rarer still: a term below about 2^-29 of its tile's sum),
// reading the tile's NW values again from tp[64 k] (the bits k of el are
// its eligible ones), so that no register is held for this path.
template <int NW>
__device__ __forceinline__ void tile_into_lane(double& s, double& c, uint32_t& nz, uint32_t& uml, bool& tw,
                                               double p, uint32_t umt, const float* tp, uint32_t el) {
  const double sp = s + p;
  const uint32_t un = umt < uml ? umt : uml;
  uml = un;
  if (!tw && sum_is_exact(sp, un)) {
    s = sp;
  } else {
    tw = true;
    if (sum_is_exact(p, umt)) {
      xadd(s, c, nz, p);
    } else {
#pragma unroll 1
      for (int k = 0; k < NW; ++k)
        if ((el >> k) & 1u) xadd(s, c, nz, __builtin_fabs((double)tp[64 * k]));
    }
  }
}

// A lane's (s, c) after m <= 2^13 terms, nz of whose errors were nonzero,
// as an XSum (a plain sum proven exact enters as (s, 0) with nz = 0).  With nz <= 1, c is exact (b = 0).  Otherwise: each TwoSum error
// is at most 2^-53 of the running sum (<= s: terms are non-negative) and
// each of the m roundings of c at most 2^-53 of |c| <= m 2^-53 s, so c is off
// by at most m^2 2^-106 s (1 + 2^-40) < 2^-80 s.
__device__ __forceinline__ XSum xlane(double s, double c, uint32_t nz) {
  return XSum{s, c, nz <= 1u ? 0.0 : s * 0x1p-80};
}

// x + y: the two sums added by TwoSum, the error parts by TwoSum as well, so
// the bound grows by exactly the magnitudes of their two rounding errors
// (0 when both additions are exact); (1 + 2^-50) covers the rounding of the
// bound's own sum.
__device__ __forceinline__ XSum xcombine(const XSum& x, const XSum& y) {
  XSum r;
  double e, c12, f1, f2;
  two_sum(x.s, y.s, r.s, e);
  two_sum(x.c, y.c, c12, f1);
  two_sum(c12, e, r.c, f2);
  r.b = (x.b + y.b + (__builtin_fabs(f1) + __builtin_fabs(f2))) * (1.0 + 0x1p-50);
  return r;
}

__device__ __forceinline__ XSum wave_xsum(XSum x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    XSum y;
    y.s = __shfl_xor(x.s, m, 64);
    y.c = __shfl_xor(x.c, m, 64);
    y.b = __shfl_xor(x.b, m, 64);
    x = xcombine(x, y);
  }
  return x;
}

// The FP64 value nearest to the exact total (ties to even) when it is
// proven: r = fl(s + c).  With b = 0 the total is s + c and r its correct
// rounding.  Otherwise rho = s + c - r exactly, the total lies within b of
// r + rho, and it rounds to r when it stays strictly inside r's rounding
// interval, whose half-widths are ulp(r)/2 above and ulp(r)/2 below
// (ulp(r)/4 when r is a power of two); fl(rho + b) < h implies rho + b < h
// for a power of two h, so the test is exact.  Returns false when the
// rounding is not proven.
__device__ __forceinline__ bool xround(const XSum& x, double& out) {
  if (!(x.s - x.s == 0.0)) {  // NaN or infinite term
    out = x.s;
    return true;
  }
  double r, rho;
  two_sum(x.s, x.c, r, rho);
  out = r;
  if (x.b == 0.0) return true;
  if (r == 0.0) return false;
  const uint64_t bits = (uint64_t)__double_as_longlong(r);
  const int64_t be = (int64_t)((bits >> 52) & 0x7ff);  // r >= 2^-149: normal
  const double half_up = __longlong_as_double((long long)((uint64_t)(be - 53) << 52));
  const double half_dn = (bits & 0xfffffffffffffull) ? half_up : 0.5 * half_up;
  return r > 0.0 && rho + x.b < half_up && x.b - rho < half_dn;
}

// The exact sum of |g| over the eligible elements [base, base + len) of one
// worker row, rounded once to FP64 (ties to even), by the whole block.  Used
// only where xround cannot certify the fast sum, so it favours plainness
// over speed: each eligible finite |g| = m 2^(e-150) adds its 24-bit
// significand m to an LDS bin of its exponent e (integer adds, exact), and
// one thread then adds the bins into base-2^32 digits of units 2^-149 and
// rounds.  hist: 256 LDS words; every thread must call.
__device__ double exact_abs_sum(const float* row, const uint64_t* mask, int64_t base, int64_t len,
                                unsigned long long* hist) {
  for (int i = threadIdx.x; i < 256; i += blockDim.x) hist[i] = 0;
  __syncthreads();
  for (int64_t i = threadIdx.x; i < len; i += blockDim.x) {
    const int64_t e = base + i;
    if (!((mask[e >> 6] >> (e & 63)) & 1ull)) continue;
    const uint32_t u = __float_as_uint(row[e]) & 0x7fffffffu;
    const uint32_t ex = u >> 23;
    const unsigned long long m = (u & 0x7fffffu) | (ex ? 0x800000u : 0u);
    if (ex < 255 && m) atomicAdd(&hist[ex ? ex : 1], m);
  }
  __syncthreads();
  double res = 0.0;
  if (threadIdx.x == 0) {
    // bin e holds sum m with weight 2^(e-1) units; bins e <= 254 and sums
    // below 2^64 fit 12 digits (384 bits)
    uint64_t d[12];
    for (int i = 0; i < 12; ++i) d[i] = 0;
    for (int ex = 1; ex < 255; ++ex) {
      const uint64_t v = hist[ex];
      if (!v) continue;
      const int p = ex - 1, k = p >> 5, r = p & 31;
      const uint64_t lo = (v & 0xffffffffu) << r, hi = (v >> 32) << r;  // each < 2^63
      d[k] += lo & 0xffffffffu;
      d[k + 1] += (lo >> 32) + (hi & 0xffffffffu);
      d[k + 2] += hi >> 32;
    }
    for (int i = 0; i < 11; ++i) {
      d[i + 1] += d[i] >> 32;
      d[i] &= 0xffffffffu;
    }
    int top = -1;
    for (int i = 11; i >= 0 && top < 0; --i)
      if (d[i]) top = 32 * i + 63 - __builtin_clzll(d[i]);
    if (top >= 0) {
      auto bit = [&](int i) { return (int)((d[i >> 5] >> (i & 31)) & 1u); };
      const int low = top > 52 ? top - 52 : 0;
      uint64_t m = 0;
      for (int i = top; i >= low; --i) m = (m << 1) | (uint64_t)bit(i);
      if (low > 0 && bit(low - 1)) {
        int rest = 0;
        for (int i = low - 2; i >= 0 && !rest; --i) rest = bit(i);
        if (rest || (m & 1u)) m += 1;
      }
      res = ldexp((double)m, low - 149);
    }
  }
  __syncthreads();
  return res;  // thread 0's value
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

// The bucket b of pass-1 chunk q and the chunk's index c in it: equal
// buckets of chunks_full chunks (btab NULL; the last may have fewer), or a
// bucket table.
__device__ __forceinline__ void chunk_home(int64_t q, const BucketRow* btab, const int32_t* cbucket, int nb,
                                           int64_t chunks_full, int& b, int64_t& c) {
  if (btab) {
    b = cbucket[q];
    c = q - btab[b].chunk0;
  } else if (q < (int64_t)(nb - 1) * chunks_full) {
    b = (int)(q / chunks_full);
    c = q - (int64_t)b * chunks_full;
  } else {
    b = nb - 1;
    c = q - (int64_t)b * chunks_full;
  }
}

// First element, length and first chunk (partial slot) of bucket b.
__device__ __forceinline__ void bucket_span(int b, const BucketRow* btab, int64_t n_total, int64_t bucket_n,
                                            int64_t slots, int64_t& base, int64_t& len, int64_t& chunk0) {
  if (btab) {
    base = btab[b].start;
    len = btab[b].len;
    chunk0 = btab[b].chunk0;
  } else {
    base = (int64_t)b * bucket_n;
    len = bucket_len(n_total, bucket_n, b);
    chunk0 = (int64_t)b * slots;
  }
}

// ------------------------------------------------------ bit-sliced counts

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

}  // namespace nf
