// Measured ceilings for the roofline fractions the benchmark reports beside
// the published peaks: a plain streaming copy (what HBM delivers to a simple
// kernel, and the reference reading of the memory-traffic counters) and a
// register-only loop of fp32 matrix-core products (what the matrix cores
// deliver at the clock they hold under sustained load).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "scn_internal.h"

namespace scn {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int COPY_THREADS = 256;

// float4 copy, one vector per lane (the loop runs once unless the grid is
// capped): a wave moves 1 KB of consecutive addresses.  One vector per lane
// over a grid as large as the data measured 6.26 TB/s on a 1 GiB copy; a
// grid-stride loop over 2048 work-groups, 4.76 TB/s, and four or eight
// vectors per lane, 5.76 and 4.34 TB/s.
__global__ void __launch_bounds__(COPY_THREADS) copy_kernel(const float4* __restrict__ src,
                                                            float4* __restrict__ dst, int64_t n4) {
  const int64_t stride = (int64_t)gridDim.x * COPY_THREADS;
  for (int64_t i = (int64_t)blockIdx.x * COPY_THREADS + threadIdx.x; i < n4; i += stride)
    dst[i] = src[i];
}

constexpr int MFMA_CHAINS = 8;  // independent accumulators per wave

// Each wave issues iters * MFMA_CHAINS products of 16x16x4 (2048 flops
// each) on operands held in registers; the chains are independent, so the
// matrix core never waits for a result.
__global__ void __launch_bounds__(256) mfma_loop_kernel(float* __restrict__ out, int iters) {
  const int lane = threadIdx.x & 63;
  float a = 1.0f + 1e-3f * lane, b = 1.0f - 1e-3f * lane;
  v4f acc[MFMA_CHAINS];
#pragma unroll
  for (int c = 0; c < MFMA_CHAINS; ++c) acc[c] = v4f{0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < MFMA_CHAINS; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < MFMA_CHAINS; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  if (lane == 0) out[(int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)] = s;
}

}  // namespace
}  // namespace scn

using namespace scn;

extern "C" {

scn_status scn_ceiling_copy(const void* src, void* dst, size_t bytes, hipStream_t st) {
  clear_error();
  if (!src || !dst || (bytes & 15) != 0 ||
      ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15) != 0) {
    set_error("scn_ceiling_copy: invalid argument");
    return SCN_ERR_INVALID;
  }
  const int64_t n4 = (int64_t)(bytes / 16);
  if (n4 == 0) return SCN_OK;
  const int64_t blocks = std::min<int64_t>(ceil_div(n4, COPY_THREADS), int64_t(1) << 30);
  hipLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(COPY_THREADS), 0, st,
                     static_cast<const float4*>(src), static_cast<float4*>(dst), n4);
  SCN_LAUNCH_CHECK();
  return SCN_OK;
}

scn_status scn_ceiling_mfma_f32(float* out, int64_t workgroups, int32_t iters, double* flops,
                                hipStream_t st) {
  clear_error();
  if (!out || !flops || workgroups < 1 || workgroups > INT32_MAX || iters < 1) {
    set_error("scn_ceiling_mfma_f32: invalid argument");
    return SCN_ERR_INVALID;
  }
  hipLaunchKernelGGL(mfma_loop_kernel, dim3((unsigned)workgroups), dim3(256), 0, st, out, iters);
  SCN_LAUNCH_CHECK();
  *flops = (double)workgroups * 4 * iters * MFMA_CHAINS * 2048.0;
  return SCN_OK;
}

}  // extern "C"
