// Device-wide exclusive prefix sum (reduce, scan of block totals, downsweep;
// one work-group for short inputs).
// Deterministic: integer sums, fixed partition.  Used by the rulebook builder
// to number active sites (popcounts of occupancy words) and to place pair
// lists (per-tile pair counts).
//
// Each thread owns 16 consecutive elements.  Whole chunks move as 16-byte
// vectors (four per thread for 32-bit elements, eight for 64-bit ones), so a
// wave touches each cache line with as few instructions as the data needs;
// only the last, partial chunk goes element by element.
#pragma once

#include "scn_internal.h"

namespace scn {

constexpr int SCAN_THREADS = 256;
constexpr int SCAN_ITEMS = 16;  // consecutive elements per thread
constexpr int SCAN_BLOCK = SCAN_THREADS * SCAN_ITEMS;

template <typename T>
__device__ inline T block_exclusive_scan(T v, T* total) {
  // 256 threads = 4 waves of 64
  __shared__ T wsum[SCAN_THREADS / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  T inc = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    T t = __shfl_up(inc, d, 64);
    if (lane >= d) inc += t;
  }
  if (lane == 63) wsum[w] = inc;
  __syncthreads();
  T before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < SCAN_THREADS / 64; ++i) {
    if (i < w) before += wsum[i];
    all += wsum[i];
  }
  __syncthreads();
  *total = all;
  return before + inc - v;
}

// Load functor: T operator()(int64_t i) const, valid for i < n, and
// void chunk(int64_t i, T (&v)[SCAN_ITEMS]) const for a whole chunk starting at
// a multiple of SCAN_ITEMS with i + SCAN_ITEMS <= n.
template <typename T, class Load>
__device__ inline void load_items(const Load& ld, int64_t base, int64_t n, T (&v)[SCAN_ITEMS]) {
  if (base + SCAN_ITEMS <= n) {
    ld.chunk(base, v);
  } else {
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j) v[j] = base + j < n ? ld(base + j) : T(0);
  }
}

// 16 consecutive elements at p (16-byte aligned) as 16-byte vectors
template <typename T>
__device__ inline void load16(const T* p, T (&v)[SCAN_ITEMS]) {
  constexpr int PER = 16 / sizeof(T);
  const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
  for (int u = 0; u < SCAN_ITEMS / PER; ++u) {
    const uint4 x = q[u];
    const T* e = reinterpret_cast<const T*>(&x);
#pragma unroll
    for (int j = 0; j < PER; ++j) v[u * PER + j] = e[j];
  }
}

template <typename T>
__device__ inline void store16(T* p, const T (&v)[SCAN_ITEMS]) {
  constexpr int PER = 16 / sizeof(T);
  uint4* q = reinterpret_cast<uint4*>(p);
#pragma unroll
  for (int u = 0; u < SCAN_ITEMS / PER; ++u) {
    uint4 x;
    T* e = reinterpret_cast<T*>(&x);
#pragma unroll
    for (int j = 0; j < PER; ++j) e[j] = v[u * PER + j];
    q[u] = x;
  }
}

// loader of a plain array
template <typename T>
struct PlainLoad {
  const T* v;
  __device__ T operator()(int64_t i) const { return v[i]; }
  __device__ void chunk(int64_t i, T (&x)[SCAN_ITEMS]) const { load16<T>(v + i, x); }
};

template <typename T, class Load>
__global__ void __launch_bounds__(SCAN_THREADS) scan_reduce_kernel(Load ld, int64_t n,
                                                                   T* block_sums) {
  const int64_t base = (int64_t)blockIdx.x * SCAN_BLOCK + (int64_t)threadIdx.x * SCAN_ITEMS;
  T v[SCAN_ITEMS];
  load_items<T>(ld, base, n, v);
  T s = 0;
#pragma unroll
  for (int j = 0; j < SCAN_ITEMS; ++j) s += v[j];
  T tot;
  block_exclusive_scan<T>(s, &tot);
  if (threadIdx.x == 0) block_sums[blockIdx.x] = tot;
}

// One block: exclusive scan of nb block totals in place; grand total to *total.
template <typename T>
__global__ void __launch_bounds__(SCAN_THREADS) scan_top_kernel(T* sums, int64_t nb, T* total) {
  T carry = 0;
  for (int64_t c = 0; c < nb; c += SCAN_THREADS) {
    const int64_t i = c + threadIdx.x;
    T v = i < nb ? sums[i] : T(0);
    T tot;
    T ex = block_exclusive_scan<T>(v, &tot);
    if (i < nb) sums[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) *total = carry;
}

template <typename T, class Load>
__global__ void __launch_bounds__(SCAN_THREADS) scan_down_kernel(Load ld, int64_t n,
                                                                 const T* block_off, T* out) {
  const int64_t base = (int64_t)blockIdx.x * SCAN_BLOCK + (int64_t)threadIdx.x * SCAN_ITEMS;
  T v[SCAN_ITEMS];
  load_items<T>(ld, base, n, v);
  T s = 0;
#pragma unroll
  for (int j = 0; j < SCAN_ITEMS; ++j) s += v[j];
  T tot;
  T ex = block_exclusive_scan<T>(s, &tot) + block_off[blockIdx.x];
  T o[SCAN_ITEMS];
#pragma unroll
  for (int j = 0; j < SCAN_ITEMS; ++j) {
    o[j] = ex;
    ex += v[j];
  }
  if (base + SCAN_ITEMS <= n) {
    store16<T>(out + base, o);
  } else {
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j)
      if (base + j < n) out[base + j] = o[j];
  }
}

// The whole scan in one work-group, chunk by chunk with a running carry: for
// inputs of a few chunks one launch costs less than the three above.
template <typename T, class Load>
__global__ void __launch_bounds__(SCAN_THREADS) scan_single_kernel(Load ld, int64_t n, T* out,
                                                                   T* total) {
  T carry = 0;
  for (int64_t c = 0; c < n; c += SCAN_BLOCK) {
    const int64_t base = c + (int64_t)threadIdx.x * SCAN_ITEMS;
    T v[SCAN_ITEMS];
    load_items<T>(ld, base, n, v);
    T s = 0;
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j) s += v[j];
    T tot;
    T ex = block_exclusive_scan<T>(s, &tot) + carry;
    T o[SCAN_ITEMS];
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j) {
      o[j] = ex;
      ex += v[j];
    }
    if (base + SCAN_ITEMS <= n) {
      store16<T>(out + base, o);
    } else {
#pragma unroll
      for (int j = 0; j < SCAN_ITEMS; ++j)
        if (base + j < n) out[base + j] = o[j];
    }
    carry += tot;
  }
  if (threadIdx.x == 0) *total = carry;
}

// inputs of at most this many chunks take scan_single_kernel
constexpr int64_t SCAN_SINGLE_MAX_BLOCKS = 4;

inline int64_t scan_blocks(int64_t n) { return n > 0 ? ceil_div(n, SCAN_BLOCK) : 1; }

// out[i] = sum_{j<i} ld(j) for i < n; *total = sum of all (device).  tmp holds
// scan_blocks(n) elements of T (unused for inputs of a few chunks).  out (and
// the loader's array) must be 16-byte aligned.
template <typename T, class Load>
scn_status exclusive_scan(Load ld, int64_t n, T* out, T* total, T* tmp, hipStream_t s) {
  const int64_t nb = scan_blocks(n);
  if (nb <= SCAN_SINGLE_MAX_BLOCKS) {
    hipLaunchKernelGGL((scan_single_kernel<T, Load>), dim3(1), dim3(SCAN_THREADS), 0, s, ld, n,
                       out, total);
    SCN_LAUNCH_CHECK();
    return SCN_OK;
  }
  if (n > 0) {
    hipLaunchKernelGGL((scan_reduce_kernel<T, Load>), dim3((unsigned)nb), dim3(SCAN_THREADS), 0,
                       s, ld, n, tmp);
    SCN_LAUNCH_CHECK();
  }
  hipLaunchKernelGGL((scan_top_kernel<T>), dim3(1), dim3(SCAN_THREADS), 0, s, tmp,
                     n > 0 ? nb : 0, total);
  SCN_LAUNCH_CHECK();
  if (n > 0) {
    hipLaunchKernelGGL((scan_down_kernel<T, Load>), dim3((unsigned)nb), dim3(SCAN_THREADS), 0,
                       s, ld, n, (const T*)tmp, out);
    SCN_LAUNCH_CHECK();
  }
  return SCN_OK;
}

}  // namespace scn
