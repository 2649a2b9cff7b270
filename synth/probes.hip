// probes.hip - reference kernels for measurement, not part of the reducer.
//
//   nfs_read_probe  streams n floats once with 128-bit loads (the
//                   "achievable" HBM read rate the reducer is compared to)
//   nfs_copy        copies n floats with 128-bit loads and stores (a kernel
//                   of known traffic, 4n bytes each way, used to scale the
//                   hardware byte counters)
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

// n: floats, a multiple of 4; src and dst 16-byte aligned, not overlapping.
extern "C" int nfs_copy(const float* src, float* dst, int64_t n, void* stream) {
  if (bad(src, n) || bad(dst, n)) return 1;
  if (n == 0) return 0;
  hipLaunchKernelGGL(k_copy, dim3(4096), dim3(1024), 0, (hipStream_t)stream, reinterpret_cast<const f4*>(src),
                     reinterpret_cast<f4*>(dst), n / 4);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
