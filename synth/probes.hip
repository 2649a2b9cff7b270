// probes.hip - reference kernels for measurement, not part of the reducer.
//
//   nfs_read_probe  streams n floats once with 128-bit loads (the
//                   "achievable" HBM read rate the reducer is compared to)
//   nfs_copy        copies n floats with 128-bit loads and stores (a kernel
//                   of known traffic, 4n bytes each way, used to scale the
//                   hardware byte counters)
//   nfs_pattern_probe  reads 16 rows in the reducer's first-pass schedule
//                   (chunks of 16 x 16,384 elements, a row per wavefront,
//                   512-element tiles with the next one in flight, launches
//                   of 256 chunks that may overlap) and, if asked, writes 1/32
//                   (or 2/32: two rows of words per row, as two bit planes)
//                   of the bytes read as 2 KiB rows at each chunk's end: the
//                   read pattern alone and with the writes mixed in, without
//                   the reducer's arithmetic (each word is a ballot of a data
//                   bit)
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(1024) void k_read(const f4* __restrict__ src, int64_t nq, float* __restrict__ sink) {
  float acc = 0.0f;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nq; i += (int64_t)gridDim.x * blockDim.x) {
    const f4 y = __builtin_nontemporal_load(src + i);
    acc += (y.x + y.y) + (y.z + y.w);
  }
  // Never true for finite data of the probe's size; keeps the loads live.
  if (acc == -1.0f) sink[threadIdx.x] = acc;
}

__global__ __launch_bounds__(1024) void k_copy(const f4* __restrict__ src, f4* __restrict__ dst, int64_t nq) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nq; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = __builtin_nontemporal_load(src + i);
}

constexpr int kPatRows = 16;       // rows: one per wavefront
constexpr int kPatChunk = 16384;   // elements per row and chunk
constexpr int kPatEpoch = 256;     // chunks per launch

// Block = chunk c of every row; wavefront v = row v.  Lane l loads element
// 64k + l of each 512-element tile's eight words; the word of 64 elements
// is the ballot of their lowest mantissa bit.
template <int NSTORE>
__global__ __launch_bounds__(1024) void k_pattern(const float* __restrict__ src, int64_t stride,
                                                  uint64_t* __restrict__ dst, int64_t dstride, int64_t q0,
                                                  int64_t nchunks) {
  __shared__ uint64_t words[kPatRows * (kPatChunk / 64)];
  const int64_t c = q0 + blockIdx.x;
  if (c >= nchunks) return;
  const int v = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float* row = src + (int64_t)v * stride + c * kPatChunk + lane;
  float xa[8], xb[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) xa[k] = __builtin_nontemporal_load(row + 64 * k);
  for (int t = 0; t < kPatChunk / 512; t += 2) {
#pragma unroll
    for (int k = 0; k < 8; ++k) xb[k] = __builtin_nontemporal_load(row + (t + 1) * 512 + 64 * k);
    uint64_t my = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const uint64_t b = __ballot((__float_as_uint(xa[k]) & 1u) != 0u);
      if (lane == k) my = b;
    }
    if (lane < 8) words[v * (kPatChunk / 64) + t * 8 + lane] = my;
    const int tn = t + 2 < kPatChunk / 512 ? t + 2 : 0;  // the last issue re-reads the chunk's first tile
#pragma unroll
    for (int k = 0; k < 8; ++k) xa[k] = __builtin_nontemporal_load(row + tn * 512 + 64 * k);
    my = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const uint64_t b = __ballot((__float_as_uint(xb[k]) & 1u) != 0u);
      if (lane == k) my = b;
    }
    if (lane < 8) words[v * (kPatChunk / 64) + (t + 1) * 8 + lane] = my;
  }
  uint32_t keep = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) keep ^= __float_as_uint(xa[k]);
  __syncthreads();
  if (NSTORE > 0) {
    // row r of words to dst row r (and to row 16 + r, inverted, for the second plane)
    for (int i = threadIdx.x; i < kPatRows * (kPatChunk / 64); i += 1024) {
      const int r = i / (kPatChunk / 64), o = i - r * (kPatChunk / 64);
      dst[(int64_t)r * dstride + c * (kPatChunk / 64) + o] = words[i];
      if (NSTORE > 1) dst[(int64_t)(kPatRows + r) * dstride + c * (kPatChunk / 64) + o] = ~words[i];
    }
  } else if (keep == 0x9e3779b9u && lane == 0) {
    dst[0] = words[threadIdx.x];  // keeps the words live; practically never taken
  }
}

bool bad(const void* p, int64_t n) { return ((uintptr_t)p & 15) != 0 || n < 0 || (n & 3) != 0; }

}  // namespace

// n: floats, a multiple of 4; src 16-byte aligned; sink holds 1024 floats.
extern "C" int nfs_read_probe(const float* src, int64_t n, float* sink, void* stream) {
  if (bad(src, n)) return 1;
  if (n == 0) return 0;
  hipLaunchKernelGGL(k_read, dim3(4096), dim3(1024), 0, (hipStream_t)stream, reinterpret_cast<const f4*>(src),
                     n / 4, sink);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

// 16 rows of n floats at src + r * stride (n a multiple of 16,384; stride a
// multiple of 4 and >= n); dst: 16 * store rows (16 for store = 0) of
// dstride >= n / 64 words.  store (0, 1 or 2): rows of words written per row
// read; with 0 nothing is written (dst is touched only by a branch the data
// practically never takes).  Returns the number of launches, or -1.
extern "C" int nfs_pattern_probe(const float* src, int64_t stride, int64_t n, uint64_t* dst, int64_t dstride,
                                 int store, void* stream) {
  if (((uintptr_t)src & 15) || (stride & 3) || stride < n || n <= 0 || n % kPatChunk || dstride < n / 64 ||
      ((uintptr_t)dst & 7) || store < 0 || store > 2)
    return -1;
  const int64_t nchunks = n / kPatChunk;
  int launches = 0;
  for (int64_t q0 = 0; q0 < nchunks; q0 += kPatEpoch, ++launches) {
    const int64_t left = nchunks - q0;
    const dim3 grid((unsigned)(left < kPatEpoch ? left : kPatEpoch));
    const uint32_t fl = q0 > 0 ? hipExtAnyOrderLaunch : 0u;
    if (store == 2)
      hipExtLaunchKernelGGL(k_pattern<2>, grid, dim3(1024), 0, (hipStream_t)stream, nullptr, nullptr, fl, src,
                            stride, dst, dstride, q0, nchunks);
    else if (store == 1)
      hipExtLaunchKernelGGL(k_pattern<1>, grid, dim3(1024), 0, (hipStream_t)stream, nullptr, nullptr, fl, src,
                            stride, dst, dstride, q0, nchunks);
    else
      hipExtLaunchKernelGGL(k_pattern<0>, grid, dim3(1024), 0, (hipStream_t)stream, nullptr, nullptr, fl, src,
                            stride, dst, dstride, q0, nchunks);
    if (hipGetLastError() != hipSuccess) return -1;
  }
  return launches;
}

// n: floats, a multiple of 4; src and dst 16-byte aligned, not overlapping.
extern "C" int nfs_copy(const float* src, float* dst, int64_t n, void* stream) {
  if (bad(src, n) || bad(dst, n)) return 1;
  if (n == 0) return 0;
  hipLaunchKernelGGL(k_copy, dim3(4096), dim3(1024), 0, (hipStream_t)stream, reinterpret_cast<const f4*>(src),
                     reinterpret_cast<f4*>(dst), n / 4);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
