// Sparse max-pooling (end of section 1.3: pooling works like the convolution,
// over the same active-site rules and ground state) and its gradient, for
// non-overlapping windows (filter == stride).  Max-pooling only moves data, so
// the kernels are organised for coalesced HBM traffic: one thread per
// (site, channel) with channels innermost, window rows from the rulebook's
// per-output neighbour table, no atomics.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "scn_internal.h"

namespace scn {
namespace {

// y[o][c] = max over the window (inactive positions hold g_in[c]); first
// strict maximum in ascending k wins.
__global__ void __launch_bounds__(256) maxpool_fwd_kernel(const float* __restrict__ x,
                                                          const float* __restrict__ g_in,
                                                          const int32_t* __restrict__ nbr,
                                                          int64_t a_out, int C, int K,
                                                          float* __restrict__ y,
                                                          uint8_t* __restrict__ argmax) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a_out * C) return;
  const int64_t o = i / C;
  const int c = (int)(i - o * C);
  const float g = g_in[c];
  const int32_t* nb = nbr + o * K;
  float best = 0.f;
  int bk = -1;
  for (int k = 0; k < K; ++k) {
    const int32_t r = nb[k];
    const float v = r >= 0 ? x[(int64_t)r * C + c] : g;
    if (bk < 0 || v > best) {
      best = v;
      bk = k;
    }
  }
  y[i] = best;
  argmax[i] = (uint8_t)bk;
}

__global__ void copy_vec_kernel(const float* __restrict__ a, float* __restrict__ b, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) b[i] = a[i];
}

// dx[r][c] = dy[o][c] if input r sits at the winning offset of (o, c), else 0.
// Every input row lies in at most one window (filter == stride).
__global__ void __launch_bounds__(256) maxpool_bwd_dx_kernel(const int32_t* __restrict__ inv,
                                                             const uint8_t* __restrict__ argmax,
                                                             const float* __restrict__ dy,
                                                             int64_t a_in, int C, int K,
                                                             float* __restrict__ dx) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a_in * C) return;
  const int64_t r = i / C;
  const int c = (int)(i - r * C);
  const int32_t t = inv[r];
  float v = 0.f;
  if (t >= 0) {
    const int64_t o = t / K;
    const int k = (int)(t - o * K);
    const int64_t j = o * C + c;
    if (argmax[j] == k) v = dy[j];
  }
  dx[i] = v;
}

constexpr int PB_ROWS = 1024;

// partial[blk][c] = sum over the block's outputs of dy[o][c] where the winner is inactive
__global__ void __launch_bounds__(256) maxpool_bwd_ground_kernel(const int32_t* __restrict__ nbr,
                                                                 const uint8_t* __restrict__ argmax,
                                                                 const float* __restrict__ dy,
                                                                 int64_t a_out, int C, int K,
                                                                 float* __restrict__ part) {
  __shared__ float red[256];
  const int64_t o0 = (int64_t)blockIdx.x * PB_ROWS;
  const int64_t o1 = min<int64_t>(o0 + PB_ROWS, a_out);
  const int rg = threadIdx.x >> 6, cl = threadIdx.x & 63;
  for (int cb = 0; cb < C; cb += 64) {
    const int c = cb + cl;
    float s = 0.f;
    if (c < C)
      for (int64_t o = o0 + rg; o < o1; o += 4) {
        const int64_t j = o * C + c;
        if (nbr[o * K + argmax[j]] < 0) s += dy[j];
      }
    red[threadIdx.x] = s;
    __syncthreads();
    if (rg == 0 && c < C)
      part[(int64_t)blockIdx.x * C + c] = ((red[cl] + red[64 + cl]) + red[128 + cl]) + red[192 + cl];
    __syncthreads();
  }
}

__global__ void maxpool_bwd_ground_finish(const float* __restrict__ part, int64_t nblk, int C,
                                          const float* __restrict__ dg_out,
                                          float* __restrict__ dg_in) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= C) return;
  float s = dg_out ? dg_out[c] : 0.f;
  for (int64_t b = 0; b < nblk; ++b) s += part[b * C + c];
  dg_in[c] = s;
}

inline unsigned nblocks(int64_t n, int t) { return (unsigned)std::max<int64_t>(1, ceil_div(n, t)); }

}  // namespace
}  // namespace scn

using namespace scn;

extern "C" {

scn_status scn_maxpool_fwd(const scn_rulebook* rb, const float* x, const float* g_in, int32_t C,
                           float* y, float* g_out, uint8_t* argmax, hipStream_t st) {
  clear_error();
  if (!rb || !g_in || !g_out || C < 1 || (rb->a_in > 0 && !x) ||
      (rb->a_out > 0 && (!y || !argmax))) {
    set_error("scn_maxpool_fwd: invalid argument");
    return SCN_ERR_INVALID;
  }
  if (rb->f != rb->s || !rb->nbr) {
    set_error("scn_maxpool_fwd: only non-overlapping windows (filter == stride) are supported");
    return SCN_ERR_UNSUPPORTED;
  }
  if (rb->a_out > 0) {
    hipLaunchKernelGGL(maxpool_fwd_kernel, dim3(nblocks(rb->a_out * C, 256)), dim3(256), 0, st, x,
                       g_in, rb->nbr, rb->a_out, C, rb->K, y, argmax);
    SCN_LAUNCH_CHECK();
  }
  hipLaunchKernelGGL(copy_vec_kernel, dim3(nblocks(C, 256)), dim3(256), 0, st, g_in, g_out, C);
  SCN_LAUNCH_CHECK();
  return SCN_OK;
}

size_t scn_maxpool_bwd_workspace_bytes(const scn_rulebook* rb, int32_t C) {
  if (!rb || C < 1) return 0;
  return (size_t)std::max<int64_t>(1, ceil_div(rb->a_out, PB_ROWS)) * C * sizeof(float);
}

scn_status scn_maxpool_bwd(const scn_rulebook* rb, const uint8_t* argmax, const float* dy,
                           const float* dg_out, int32_t C, float* dx, float* dg_in, void* ws,
                           size_t ws_bytes, hipStream_t st) {
  clear_error();
  if (!rb || C < 1 || (rb->a_out > 0 && (!argmax || !dy)) || (rb->a_in > 0 && !dx)) {
    set_error("scn_maxpool_bwd: invalid argument");
    return SCN_ERR_INVALID;
  }
  if (rb->f != rb->s || !rb->nbr) {
    set_error("scn_maxpool_bwd: only non-overlapping windows (filter == stride) are supported");
    return SCN_ERR_UNSUPPORTED;
  }
  const size_t need = scn_maxpool_bwd_workspace_bytes(rb, C);
  if (dg_in && (!ws || ws_bytes < need)) {
    set_error("scn_maxpool_bwd: workspace of %zu bytes needed, %zu given", need, ws_bytes);
    return SCN_ERR_WORKSPACE;
  }
  if (rb->a_in > 0) {
    hipLaunchKernelGGL(maxpool_bwd_dx_kernel, dim3(nblocks(rb->a_in * C, 256)), dim3(256), 0, st,
                       rb->inv, argmax, dy, rb->a_in, C, rb->K, dx);
    SCN_LAUNCH_CHECK();
  }
  if (dg_in) {
    const int64_t nblk = std::max<int64_t>(1, ceil_div(rb->a_out, PB_ROWS));
    float* part = static_cast<float*>(ws);
    if (rb->a_out > 0) {
      hipLaunchKernelGGL(maxpool_bwd_ground_kernel, dim3((unsigned)nblk), dim3(256), 0, st,
                         rb->nbr, argmax, dy, rb->a_out, C, rb->K, part);
      SCN_LAUNCH_CHECK();
    }
    hipLaunchKernelGGL(maxpool_bwd_ground_finish, dim3(nblocks(C, 64)), dim3(64), 0, st, part,
                       rb->a_out > 0 ? nblk : 0, C, dg_out, dg_in);
    SCN_LAUNCH_CHECK();
  }
  return SCN_OK;
}

}  // extern "C"
