// gen.hip - seeded synthetic gradient buckets generated on the device.
//
// Input generation only: nothing here computes any step of the reducer.
// Random numbers come from Philox4x32-10 (Salmon, Moraes, Dror, Shaw,
// "Parallel random numbers: as easy as 1, 2, 3", SC 2011), written from that
// definition, keyed by (seed, worker) with the element index as counter;
// Box-Muller turns pairs of uniforms into normals.  Element i of worker w is
//   g = scale_w * sigma_s * Z                        (normal segments)
//   g = scale_w * sigma_s / sqrt(3) * Z / sqrt(V/3)  (Student-t, 3 dof)
// where s is the segment holding i, Z and V's three terms are independent
// standard normals.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {


__device__ inline void philox10(uint32_t ctr[4], uint32_t k0, uint32_t k1) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)M0 * ctr[0];
    const uint64_t p1 = (uint64_t)M1 * ctr[2];
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t n0 = hi1 ^ ctr[1] ^ k0;
    const uint32_t n2 = hi0 ^ ctr[3] ^ k1;
    ctr[0] = n0;
    ctr[1] = lo1;
    ctr[2] = n2;
    ctr[3] = lo0;
    k0 += W0;
    k1 += W1;
  }
}

// Four standard normals from one Philox block.
__device__ inline void normals4(uint64_t seed, uint32_t w, uint64_t group, uint32_t stream, float z[4]) {
  uint32_t c[4] = {(uint32_t)group, (uint32_t)(group >> 32), w, stream};
  philox10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
  const float inv = 2.3283064365386963e-10f;  // 2^-32
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const float u1 = ((float)c[2 * p] + 1.0f) * inv;  // (0, 1]
    const float u2 = (float)c[2 * p + 1] * inv;       // [0, 1)
    const float r = sqrtf(-2.0f * logf(u1));
    float sn, cs;
    sincosf(6.283185307179586f * u2, &sn, &cs);
    z[2 * p] = r * cs;
    z[2 * p + 1] = r * sn;
  }
}

__global__ void k_generate(float* __restrict__ g, int64_t stride, int32_t W, int64_t n,
                           const int64_t* __restrict__ seg_start, const float* __restrict__ seg_sigma,
                           const int32_t* __restrict__ seg_dist, int32_t nseg,
                           const float* __restrict__ wscale, uint64_t seed) {
  const int w = blockIdx.y;
  const int64_t group = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // 4 elements
  const int64_t i0 = group * 4;
  if (i0 >= n) return;
  float z[4];
  normals4(seed, (uint32_t)w, (uint64_t)group, 0u, z);
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  bool need_t = false;
  int sidx[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int64_t i = i0 + e;
    int lo = 0, hi = nseg - 1;  // last segment with start <= i
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (seg_start[mid] <= i) lo = mid; else hi = mid - 1;
    }
    sidx[e] = lo;
    need_t |= seg_dist[lo] == 1;
  }
  if (need_t) {
    float a[4], b[4], c[4];
    normals4(seed, (uint32_t)w, (uint64_t)group, 1u, a);
    normals4(seed, (uint32_t)w, (uint64_t)group, 2u, b);
    normals4(seed, (uint32_t)w, (uint64_t)group, 3u, c);
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = (a[e] * a[e] + b[e] * b[e] + c[e] * c[e]) / 3.0f;
  }
  const float ws = wscale[w];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int64_t i = i0 + e;
    if (i >= n) break;
    const int s = sidx[e];
    float x = z[e];
    if (seg_dist[s] == 1) x = x / sqrtf(v[e]) * 0.5773502691896258f;  // t3 with unit variance
    g[(int64_t)w * stride + i] = ws * (seg_sigma[s] * x);
  }
}

__global__ void k_inject(float* __restrict__ g, int64_t stride, const int32_t* __restrict__ w,
                         const int64_t* __restrict__ idx, const float* __restrict__ val, int64_t m) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j < m) g[(int64_t)w[j] * stride + idx[j]] = val[j];
}

}  // namespace

extern "C" int nfs_generate(float* g, int64_t stride, int32_t W, int64_t n, const int64_t* seg_start,
                            const float* seg_sigma, const int32_t* seg_dist, int32_t nseg,
                            const float* wscale, uint64_t seed, void* stream) {
  if (W < 1 || n < 0 || stride < n || nseg < 1) return 1;
  if (n == 0) return 0;
  const int64_t groups = (n + 3) / 4;
  const int threads = 256;
  dim3 grid((unsigned)((groups + threads - 1) / threads), (unsigned)W);
  hipLaunchKernelGGL(k_generate, grid, dim3(threads), 0, (hipStream_t)stream, g, stride, W, n,
                     seg_start, seg_sigma, seg_dist, nseg, wscale, seed);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

extern "C" int nfs_inject(float* g, int64_t stride, const int32_t* w, const int64_t* idx,
                          const float* val, int64_t m, void* stream) {
  if (m <= 0) return 0;
  hipLaunchKernelGGL(k_inject, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, (hipStream_t)stream,
                     g, stride, w, idx, val, m);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
