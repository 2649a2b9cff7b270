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
