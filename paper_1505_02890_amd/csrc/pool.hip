// Sparse max-pooling (end of section 1.3: pooling works like the convolution,
// over the same active-site rules and ground state) and its gradient, for
// windows that tile the grid (filter == stride), leave gaps (filter < stride)
// or overlap (filter > stride, the MP3/2 of the paper's networks), on the
// cubic lattice (K = f^3 positions per window), the tetrahedral one
// (K = C(f+2, 3)) or the 2D square and triangular ones (K = f^2, C(f+1, 2)).  Max-pooling only moves data, so the kernels are organised
// for coalesced HBM traffic: threads over (site, channel) with channels
// innermost, window rows from the rulebook's per-output neighbour table, no
// atomics.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <initializer_list>
#include <type_traits>

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

// ---- four channels per thread (C % 4 == 0, aligned rows) ------------------
// A block holds `per` sites with nc4 = C/4 threads each; argmax bytes of four
// channels travel as one 32-bit word (byte e = channel 4*c4 + e).

// The block's window-table rows are contiguous in nbr: the block loads them
// into LDS with a few coalesced loads, instead of every lane of an output
// loading each entry (for 64 channels, 16 lanes per output asked for the same
// word, one load instruction per window position).
template <int K>
__device__ inline const int32_t* stage_rows(const int32_t* __restrict__ nbr, int64_t o_first,
                                            int64_t a_out, int rows, int32_t* sh) {
  const int64_t n = (o_first + rows < a_out ? (int64_t)rows : a_out - o_first) * K;
  const int32_t* src = nbr + o_first * K;
  for (int i = threadIdx.x; i < n; i += blockDim.x) sh[i] = src[i];
  __syncthreads();
  return sh;
}

typedef float pool_v4f __attribute__((ext_vector_type(4)));


// A streaming store, for rows nothing reads again soon (dx): 5-10% faster
// than a plain store in the backward kernels.
__device__ inline void store_stream(float4* p, float4 v) {
  __builtin_nontemporal_store(pool_v4f{v.x, v.y, v.z, v.w}, reinterpret_cast<pool_v4f*>(p));
}

template <int K>
__global__ void __launch_bounds__(256) maxpool_fwd_vec_kernel(const float4* __restrict__ x,
                                                              const float4* __restrict__ g_in,
                                                              const int32_t* __restrict__ nbr,
                                                              int64_t a_out, int nc4, int per,
                                                              float4* __restrict__ y,
                                                              uint32_t* __restrict__ argmax,
                                                              int chunk) {
  extern __shared__ int32_t nsh[];  // per * K entries
  const int ol = threadIdx.x / nc4, c4 = threadIdx.x - ol * nc4;
  // overlapping windows share inputs with the windows of nearby blocks
  const int64_t blk = xcd_block(blockIdx.x, chunk);
  if (blk * per >= a_out) return;  // the whole block: a launch rounded up to whole runs
  const int64_t ob = blk * per, o = ob + ol;
  stage_rows<K>(nbr, ob, a_out, per, nsh);
  if (ol >= per || o >= a_out) return;
  const float4 g = g_in[c4];
  const int32_t* nb = nsh + ol * K;
  // first strict maximum in ascending k, per channel
  // (the 27 positions of a 3-wide cube window a plane of 9 at a time;
  // smaller windows all at once)
  constexpr int PL = K == 27 ? 9 : K, NPL = K / PL;
  float4 best = make_float4(0.f, 0.f, 0.f, 0.f);
  uint32_t b0 = 0, b1 = 0, b2 = 0, b3 = 0;
#pragma unroll 1
  for (int kz = 0; kz < NPL; ++kz) {
    // an inactive position takes g and loads nothing (its lanes are masked
    // off); a plane's loads are all in flight together
    float4 v[PL];
#pragma unroll
    for (int i = 0; i < PL; ++i) {
      const int32_t r = nb[kz * PL + i];
      v[i] = g;
      if (r >= 0) v[i] = x[(int64_t)r * nc4 + c4];
    }
#pragma unroll
    for (int i = 0; i < PL; ++i) {
      const uint32_t k = kz * PL + i;
      if (k == 0) {
        best = v[i];
        continue;
      }
      if (v[i].x > best.x) { best.x = v[i].x; b0 = k; }
      if (v[i].y > best.y) { best.y = v[i].y; b1 = k; }
      if (v[i].z > best.z) { best.z = v[i].z; b2 = k; }
      if (v[i].w > best.w) { best.w = v[i].w; b3 = k; }
    }
  }
  // streaming stores: the outputs are not read again here, and the input
  // rows that nearby windows re-read keep the cache (2x2x2 forward on 4.4M
  // rows 0.251 -> 0.241 ms)
  store_stream(y + o * nc4 + c4, best);
  __builtin_nontemporal_store(b0 | (b1 << 8) | (b2 << 16) | (b3 << 24), argmax + o * nc4 + c4);
}

// outputs per block of the four-channel backward: 2x2x2 windows on 4.4M rows
// 0.273 ms at 64 (four per lane group at 64 channels), 0.258 at 32, 0.245 at
// 16 (one per lane group), 0.264 at 8
constexpr int PBV_ROWS = 16;
constexpr int CELL_ROWS = 32;  // windows per block of the MP3/2 cell backward (0.347 -> 0.341 ms
                                // against 64; 16: 0.385)

// Output-major backward: an input lies in at most one window, so each window
// writes its inputs' dx rows (dy where the input won, else 0) and dx is
// written once per element with no atomics (rows in no window are zeroed by
// zero_uncovered_kernel).  A winner at an inactive
// position sends dy to the ground state: part[blk][c] sums those, over the
// block's outputs in a fixed order (part may be null).
template <int K>
__global__ void __launch_bounds__(256) maxpool_bwd_vec_kernel(const int32_t* __restrict__ nbr,
                                                              const uint32_t* __restrict__ argmax,
                                                              const float4* __restrict__ dy,
                                                              int64_t a_out, int nc4,
                                                              float4* __restrict__ dx,
                                                              float4* __restrict__ part) {
  __shared__ float4 red[256];
  __shared__ int32_t nsh[PBV_ROWS * K];
  const int rows = 256 / nc4;  // outputs in flight per block
  const int rl = threadIdx.x / nc4, c4 = threadIdx.x - rl * nc4;
  const int64_t o0 = (int64_t)blockIdx.x * PBV_ROWS;
  const int64_t o1 = min<int64_t>(o0 + PBV_ROWS, a_out);
  stage_rows<K>(nbr, o0, a_out, PBV_ROWS, nsh);
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  if (rl < rows)
    for (int64_t o = o0 + rl; o < o1; o += rows) {
      const int64_t j = o * nc4 + c4;
      const uint32_t am = argmax[j];
      const float4 d = dy[j];
      const uint32_t k0 = am & 255u, k1 = (am >> 8) & 255u, k2 = (am >> 16) & 255u, k3 = am >> 24;
      const int32_t* nb = nsh + (o - o0) * K;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int32_t r = nb[k];
        const float4 v = make_float4(k0 == (uint32_t)k ? d.x : 0.f, k1 == (uint32_t)k ? d.y : 0.f,
                                     k2 == (uint32_t)k ? d.z : 0.f, k3 == (uint32_t)k ? d.w : 0.f);
        if (r >= 0) {
          if (dx) store_stream(dx + (int64_t)r * nc4 + c4, v);
        } else {
          s.x += v.x;
          s.y += v.y;
          s.z += v.z;
          s.w += v.w;
        }
      }
    }
  if (!part) return;
  red[threadIdx.x] = s;
  __syncthreads();
  if (rl == 0) {
    for (int i = 1; i < rows; ++i) {
      const float4 t = red[i * nc4 + c4];
      s.x += t.x;
      s.y += t.y;
      s.z += t.z;
      s.w += t.w;
    }
    part[(int64_t)blockIdx.x * nc4 + c4] = s;
  }
}

// dx[r] of one input over its (up to 8) windows: win8 = its slots (o*K + k
// or -1), summed in slot order, a fixed order; nc4 lanes, channels 4*c4 ..
template <int K>
__device__ inline float4 input_grad(const int32_t (&t)[8], const uint32_t* __restrict__ argmax,
                                    const float4* __restrict__ dy, int nc4, int c4) {
  uint32_t am[8];
  float4 d[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    am[j] = 0u;
    d[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (t[j] >= 0) {  // an empty slot loads nothing: its lanes are masked off
      const int64_t jj = (int64_t)((uint32_t)t[j] / K) * nc4 + c4;
      am[j] = argmax[jj];
      d[j] = dy[jj];
    }
  }
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    // 255: an empty slot, which no argmax byte holds
    const uint32_t k = t[j] >= 0 ? (uint32_t)t[j] % K : 255u;
    v.x += (am[j] & 255u) == k ? d[j].x : 0.f;
    v.y += ((am[j] >> 8) & 255u) == k ? d[j].y : 0.f;
    v.z += ((am[j] >> 16) & 255u) == k ? d[j].z : 0.f;
    v.w += (am[j] >> 24) == k ? d[j].w : 0.f;
  }
  return v;
}

// Overlapping windows (filter > stride), input-major: an input lies in up to 8
// windows, win[r*8 + j] = o*K + k or -1.  dx[r][c] = sum over its windows
// (slot order) of dy[o][c] where the input won channel c of window o.  nc4
// lanes per input.  (3-wide windows of stride 2 on the cubic lattice take the
// cell-major kernel below instead, with about a third of the gathers.)
template <int K>
__global__ void __launch_bounds__(256) maxpool_bwd_overlap_vec_kernel(
    const int32_t* __restrict__ win, const uint32_t* __restrict__ argmax,
    const float4* __restrict__ dy, int64_t a_in, int nc4, int per, float4* __restrict__ dx) {
  const int rl = threadIdx.x / nc4, c4 = threadIdx.x - rl * nc4;
  const int64_t r = (int64_t)blockIdx.x * per + rl;
  if (rl >= per || r >= a_in) return;
  const int4 w0 = reinterpret_cast<const int4*>(win)[2 * r];
  const int4 w1 = reinterpret_cast<const int4*>(win)[2 * r + 1];
  const int32_t t[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
  store_stream(dx + r * nc4 + c4, input_grad<K>(t, argmax, dy, nc4, c4));
}

// Inputs without a home window (3-wide windows of stride 2, cubic lattice):
// the listed inputs, input-major as above (all slots empty: dx = 0).  A
// grid-stride loop up to the count the rulebook build left on the device.
__global__ void __launch_bounds__(256) maxpool_bwd_homeless_vec_kernel(
    const int32_t* __restrict__ list, const int32_t* __restrict__ count,
    const int32_t* __restrict__ win, const uint32_t* __restrict__ argmax,
    const float4* __restrict__ dy, int nc4, int per, float4* __restrict__ dx) {
  const int rl = threadIdx.x / nc4, c4 = threadIdx.x - rl * nc4;
  if (rl >= per) return;
  const int64_t n = *count;
  for (int64_t i = (int64_t)blockIdx.x * per + rl; i < n; i += (int64_t)gridDim.x * per) {
    const int64_t r = list[i];
    const int4 w0 = reinterpret_cast<const int4*>(win)[2 * r];
    const int4 w1 = reinterpret_cast<const int4*>(win)[2 * r + 1];
    const int32_t t[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
    dx[r * nc4 + c4] = input_grad<27>(t, argmax, dy, nc4, c4);
  }
}

// 3-wide windows of stride 2 on the cubic lattice, cell-major.  Window h's
// home cell holds the inputs at its offsets w = (wx, wy, wz) in {0,1}^3
// (position wx + 3wy + 9wz); such an input also lies in window h - b for each
// b in {0,1}^3 with no bit where w has a 1 (low[h*8 + b]), at position
// (wx + 2bx) + 3(wy + 2by) + 9(wz + 2bz), b being its slot there.  Each lane
// group (nc4 lanes) takes a window, gathers dy and argmax of the windows h - b
// its active home inputs need (avg about 5 for surfaces), and writes each
// home input's dx row: the sum over its slots in slot order, the same sum
// the input-major kernel forms.  Every input with a home window is written
// exactly once (the others are listed as homeless).  The gathers per input
// drop from 3.4 rows to about 1.2.  The window's own dy and argmax also give
// the ground-state sums (dy where the winner is inactive), so no separate
// pass reads them: part[blk][c] sums the block's windows in a fixed order
// (part may be null).  CELL_ROWS windows per block: their home entries and
// lower windows are staged in LDS once.  Five waves per SIMD (96 VGPRs; the
// compiler's own choice, 98, allowed four): 0.373 -> 0.366 ms on 4.4M inputs.
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(5))) maxpool_bwd_cells_kernel(
    const int32_t* __restrict__ nbr, const int32_t* __restrict__ low,
    const uint32_t* __restrict__ pmask, const uint32_t* __restrict__ argmax,
    const float4* __restrict__ dy, int64_t a_out, int nc4, float4* __restrict__ dx,
    float4* __restrict__ part, int chunk) {
  __shared__ int32_t home[CELL_ROWS * 8];
  __shared__ int4 lows[CELL_ROWS * 2];
  __shared__ float4 red[256];
  const int64_t blk = xcd_block(blockIdx.x, chunk);
  const int64_t h0 = blk * CELL_ROWS;
  if (h0 >= a_out) return;  // the whole block: a launch rounded up to whole runs
  const int nh = (int)min<int64_t>(CELL_ROWS, a_out - h0);
  if ((int)threadIdx.x < nh) {
    const int t = threadIdx.x;
    const int32_t* row = nbr + (h0 + t) * 27;
#pragma unroll
    for (int w = 0; w < 8; ++w) home[t * 8 + w] = row[(w & 1) + 3 * ((w >> 1) & 1) + 9 * (w >> 2)];
  }
  for (int i = threadIdx.x; i < 2 * nh; i += 256)
    lows[i] = reinterpret_cast<const int4*>(low + h0 * 8)[i];
  __syncthreads();
  const int rows = 256 / nc4;
  const int rl = threadIdx.x / nc4, c4 = threadIdx.x - rl * nc4;
  float4 g = make_float4(0.f, 0.f, 0.f, 0.f);
  if (rl < rows)
    for (int i = rl; i < nh; i += rows) {
      const int32_t* hm = home + i * 8;
      const int4 la = lows[2 * i], lb = lows[2 * i + 1];
      const int32_t lw[8] = {la.x, la.y, la.z, la.w, lb.x, lb.y, lb.z, lb.w};
      uint32_t act = 0u;
#pragma unroll
      for (int w = 0; w < 8; ++w) act |= (hm[w] >= 0 ? 1u : 0u) << w;
      uint32_t am[8];
      float4 d[8];
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        // home offsets with no 1 along b's axes: these lie in window h - b
        constexpr uint32_t ZX = 0x55u, ZY = 0x33u, ZZ = 0x0Fu;
        const uint32_t zm = ((b & 1) ? ZX : 0xFFu) & ((b & 2) ? ZY : 0xFFu) & ((b & 4) ? ZZ : 0xFFu);
        am[b] = 0u;
        d[b] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (b == 0 || (lw[b] >= 0 && (act & zm))) {
          const int64_t jj = (int64_t)lw[b] * nc4 + c4;
          am[b] = argmax[jj];
          d[b] = dy[jj];
        }
      }
      // ground state: channels of window h whose winner is an inactive position
      const uint32_t m = pmask[h0 + i];
      if (!((m >> (am[0] & 255u)) & 1u)) g.x += d[0].x;
      if (!((m >> ((am[0] >> 8) & 255u)) & 1u)) g.y += d[0].y;
      if (!((m >> ((am[0] >> 16) & 255u)) & 1u)) g.z += d[0].z;
      if (!((m >> (am[0] >> 24)) & 1u)) g.w += d[0].w;
#pragma unroll
      for (int w = 0; w < 8; ++w) {
        if (hm[w] < 0) continue;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          if (b & w) continue;  // not a window of this input
          if (b != 0 && lw[b] < 0) continue;
          const uint32_t k = ((w & 1) + 2 * (b & 1)) + 3 * (((w >> 1) & 1) + 2 * ((b >> 1) & 1)) +
                             9 * ((w >> 2) + 2 * (b >> 2));
          v.x += (am[b] & 255u) == k ? d[b].x : 0.f;
          v.y += ((am[b] >> 8) & 255u) == k ? d[b].y : 0.f;
          v.z += ((am[b] >> 16) & 255u) == k ? d[b].z : 0.f;
          v.w += (am[b] >> 24) == k ? d[b].w : 0.f;
        }
        store_stream(dx + (int64_t)hm[w] * nc4 + c4, v);
      }
    }
  if (!part) return;
  red[threadIdx.x] = g;
  __syncthreads();
  if (rl == 0) {
    for (int i = 1; i < rows; ++i) {
      const float4 t = red[i * nc4 + c4];
      g.x += t.x;
      g.y += t.y;
      g.z += t.z;
      g.w += t.w;
    }
    part[blk * nc4 + c4] = g;
  }
}

__global__ void __launch_bounds__(256) maxpool_bwd_overlap_kernel(const int32_t* __restrict__ win,
                                                                  const uint8_t* __restrict__ argmax,
                                                                  const float* __restrict__ dy,
                                                                  int64_t a_in, int C, int K,
                                                                  float* __restrict__ dx) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a_in * C) return;
  const int64_t r = i / C;
  const int c = (int)(i - r * C);
  float v = 0.f;
  for (int j = 0; j < 8; ++j) {
    const int32_t t = win[r * 8 + j];
    if (t < 0) continue;
    const int32_t o = t / K;
    const int k = t - o * K;
    const int64_t jj = (int64_t)o * C + c;
    if (argmax[jj] == k) v += dy[jj];
  }
  dx[i] = v;
}

// Ground-state partial sums alone (the overlapping case computes dx input-
// major): part[blk][c] sums, over the block's outputs in a fixed order, dy[o][c]
// where the winner of (o, c) is an inactive position (bit am of pmask[o]
// clear).  A stream over argmax and dy.
__global__ void __launch_bounds__(256) maxpool_ground_vec_kernel(const uint32_t* __restrict__ pmask,
                                                                 const uint32_t* __restrict__ argmax,
                                                                 const float4* __restrict__ dy,
                                                                 int64_t a_out, int nc4,
                                                                 float4* __restrict__ part) {
  __shared__ float4 red[256];
  const int rows = 256 / nc4;
  const int rl = threadIdx.x / nc4, c4 = threadIdx.x - rl * nc4;
  const int64_t o0 = (int64_t)blockIdx.x * PBV_ROWS;
  const int64_t o1 = min<int64_t>(o0 + PBV_ROWS, a_out);
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  if (rl < rows)
#pragma unroll 4
    for (int64_t o = o0 + rl; o < o1; o += rows) {
      const int64_t j = o * nc4 + c4;
      const uint32_t am = argmax[j], m = pmask[o];
      const float4 d = dy[j];
      if (!((m >> (am & 255u)) & 1u)) s.x += d.x;
      if (!((m >> ((am >> 8) & 255u)) & 1u)) s.y += d.y;
      if (!((m >> ((am >> 16) & 255u)) & 1u)) s.z += d.z;
      if (!((m >> (am >> 24)) & 1u)) s.w += d.w;
    }
  red[threadIdx.x] = s;
  __syncthreads();
  if (rl == 0) {
    for (int i = 1; i < rows; ++i) {
      const float4 t = red[i * nc4 + c4];
      s.x += t.x;
      s.y += t.y;
      s.z += t.z;
      s.w += t.w;
    }
    part[(int64_t)blockIdx.x * nc4 + c4] = s;
  }
}

// dx rows of inputs that lie in no window (a grid edge the windows do not
// reach) are zero; one thread per input row
__global__ void __launch_bounds__(256) zero_uncovered_kernel(const int32_t* __restrict__ inv,
                                                             int64_t a_in, int nc4,
                                                             float4* __restrict__ dx) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= a_in || inv[r] >= 0) return;
  for (int c4 = 0; c4 < nc4; ++c4) dx[r * nc4 + c4] = make_float4(0.f, 0.f, 0.f, 0.f);
}

constexpr int PB_ROWS = 1024;  // outputs per block of the one-channel ground gradient

// ---- any channel count (one channel per thread) -----------------------------

// partial[blk][c] = sum over the block's outputs of dy[o][c] where the winner is inactive
__global__ void __launch_bounds__(256) maxpool_bwd_ground_kernel(const uint32_t* __restrict__ pmask,
                                                                 const uint8_t* __restrict__ argmax,
                                                                 const float* __restrict__ dy,
                                                                 int64_t a_out, int C,
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
        if (!((pmask[o] >> argmax[j]) & 1u)) s += dy[j];
      }
    red[threadIdx.x] = s;
    __syncthreads();
    if (rg == 0 && c < C)
      part[(int64_t)blockIdx.x * C + c] = ((red[cl] + red[64 + cl]) + red[128 + cl]) + red[192 + cl];
    __syncthreads();
  }
}

// The ground-state sums dg_in[c] = dg_out[c] + sum_b part[b][c], in two
// passes of fixed shape.  First GF_BLOCKS work-groups each add a contiguous
// range of part's rows: rg = 256 / C row groups of C lanes, so a wave reads
// whole rows (one work-group per channel took 22 us for 15k rows of 64
// channels: every load touched 64 lines); the row groups' sums are added in
// order.  Then each work-group of the second pass takes 64 channels: four
// row groups of 64 lanes add every fourth of the GF_BLOCKS partial rows, and
// their sums are added in order.
constexpr int GF_BLOCKS = 256;
__global__ void __launch_bounds__(256) maxpool_ground_rows_kernel(const float* __restrict__ part,
                                                                  int64_t nblk, int C,
                                                                  float* __restrict__ part2) {
  __shared__ float red[256];
  const int64_t per = (nblk + GF_BLOCKS - 1) / GF_BLOCKS;
  const int64_t b0 = (int64_t)blockIdx.x * per, b1 = min<int64_t>(nblk, b0 + per);
  if (C <= 256) {
    const int rg_n = 256 / C, rg = threadIdx.x / C, c = threadIdx.x - rg * C;
    float s = 0.f;
    if (rg < rg_n) {
#pragma unroll 4
      for (int64_t b = b0 + rg; b < b1; b += rg_n) s += part[b * C + c];
    }
    red[threadIdx.x] = s;
    __syncthreads();
    if (rg == 0) {
      for (int g = 1; g < rg_n; ++g) s += red[g * C + c];
      part2[(int64_t)blockIdx.x * C + c] = s;
    }
  } else {
    for (int c = threadIdx.x; c < C; c += 256) {
      float s = 0.f;
      for (int64_t b = b0; b < b1; ++b) s += part[b * C + c];
      part2[(int64_t)blockIdx.x * C + c] = s;
    }
  }
}

__global__ void __launch_bounds__(256) maxpool_bwd_ground_finish(const float* __restrict__ part2,
                                                                 int C,
                                                                 const float* __restrict__ dg_out,
                                                                 float* __restrict__ dg_in) {
  __shared__ float red[256];
  const int rg = threadIdx.x >> 6, c = blockIdx.x * 64 + (threadIdx.x & 63);
  float s = 0.f;
  if (c < C) {
#pragma unroll 8
    for (int g = rg; g < GF_BLOCKS; g += 4) s += part2[(int64_t)g * C + c];
  }
  red[threadIdx.x] = s;
  __syncthreads();
  if (rg == 0 && c < C)
    dg_in[c] = (dg_out ? dg_out[c] : 0.f) + (((s + red[64 + threadIdx.x]) + red[128 + threadIdx.x]) +
                                             red[192 + threadIdx.x]);
}

inline unsigned nblocks(int64_t n, int t) { return (unsigned)std::max<int64_t>(1, ceil_div(n, t)); }

// calls fn(std::integral_constant<int, K>{}) for the window sizes of the
// lattices: 1, 8, 27 (cube), 4, 10 (tetrahedron), 4, 9 (square), 3, 6
// (triangle), 2, 3 (line) and 16 (the 4D hypercube of 2); false for others
template <typename Fn>
bool with_window(int K, Fn fn) {
  switch (K) {
    case 1: fn(std::integral_constant<int, 1>{}); return true;
    case 2: fn(std::integral_constant<int, 2>{}); return true;
    case 3: fn(std::integral_constant<int, 3>{}); return true;
    case 4: fn(std::integral_constant<int, 4>{}); return true;
    case 6: fn(std::integral_constant<int, 6>{}); return true;
    case 8: fn(std::integral_constant<int, 8>{}); return true;
    case 9: fn(std::integral_constant<int, 9>{}); return true;
    case 10: fn(std::integral_constant<int, 10>{}); return true;
    case 16: fn(std::integral_constant<int, 16>{}); return true;
    case 27: fn(std::integral_constant<int, 27>{}); return true;
    default: return false;
  }
}

inline bool window_size_ok(int K) {
  return with_window(K, [](auto) {});
}

// four-channel path: C % 4 == 0, C <= 1024, float rows 16-byte aligned, argmax
// words 4-byte aligned
inline bool pool_vec_ok(int C, std::initializer_list<const void*> rows, const void* argmax) {
  if (C % 4 != 0 || C > 1024 || (reinterpret_cast<uintptr_t>(argmax) & 3) != 0) return false;
  for (const void* p : rows)
    if (reinterpret_cast<uintptr_t>(p) & 15) return false;
  return true;
}



// floats of the per-block ground-state partial sums, rounded to 16 bytes;
// enough for every path (the four-channel paths use blocks of PBV_ROWS or
// CELL_ROWS outputs)
inline size_t part_floats(const scn_rulebook* rb, int C) {
  const int64_t rows = C % 4 == 0 ? (PBV_ROWS < CELL_ROWS ? PBV_ROWS : CELL_ROWS) : PB_ROWS;
  return ((size_t)std::max<int64_t>(1, ceil_div(rb->a_out, rows)) * C + 3) & ~size_t(3);
}

}  // namespace
}  // namespace scn

using namespace scn;

extern "C" {

scn_status scn_maxpool_fwd(const scn_rulebook* rb, const float* x, const float* g_in, int32_t C,
                           float* y, float* g_out, uint8_t* argmax, hipStream_t st) {
  clear_error();
  if (scn_status rc0 = after_build(rb, st)) return rc0;
  if (!rb || !g_in || !g_out || C < 1 || (rb->a_in > 0 && !x) ||
      (rb->a_out > 0 && (!y || !argmax))) {
    set_error("scn_maxpool_fwd: invalid argument");
    return SCN_ERR_INVALID;
  }
  if (!rb->nbr) {
    set_error("scn_maxpool_fwd: the rulebook has no pooling tables (stride 1, or windows wider "
              "than their stride on sites of other than 3 coordinates)");
    return SCN_ERR_UNSUPPORTED;
  }
  if (!window_size_ok(rb->K)) {
    set_error("scn_maxpool_fwd: windows of %d sites are not supported", rb->K);
    return SCN_ERR_UNSUPPORTED;
  }
  if (rb->a_out > 0) {
    if (pool_vec_ok(C, {x, g_in, y}, argmax)) {
      const int nc4 = C / 4, per = 256 / nc4;
      const int64_t nb = nblocks(rb->a_out, per);
      // runs of 16 blocks per XCD: MP3/2 forward on 4.4M rows 0.363 -> 0.337 ms;
      // of 128 for the 2x2x2 forward: 0.257 -> 0.251 ms
      const int chunk = xcd_chunk(nb, rb->K == 27 ? 16 : (rb->K == 8 ? 128 : 1));
      const dim3 grid(xcd_grid(nb, chunk));
      const auto* x4 = reinterpret_cast<const float4*>(x);
      const auto* g4 = reinterpret_cast<const float4*>(g_in);
      auto* y4 = reinterpret_cast<float4*>(y);
      auto* am4 = reinterpret_cast<uint32_t*>(argmax);
      with_window(rb->K, [&](auto k) {
        constexpr int K = decltype(k)::value;
        hipLaunchKernelGGL(maxpool_fwd_vec_kernel<K>, grid, dim3(256), per * K * sizeof(int32_t),
                           st, x4, g4, rb->nbr, rb->a_out, nc4, per, y4, am4, chunk);
      });
    } else {
      hipLaunchKernelGGL(maxpool_fwd_kernel, dim3(nblocks(rb->a_out * C, 256)), dim3(256), 0, st,
                         x, g_in, rb->nbr, rb->a_out, C, rb->K, y, argmax);
    }
    SCN_LAUNCH_CHECK();
  }
  hipLaunchKernelGGL(copy_vec_kernel, dim3(nblocks(C, 256)), dim3(256), 0, st, g_in, g_out, C);
  SCN_LAUNCH_CHECK();
  return SCN_OK;
}

size_t scn_maxpool_bwd_workspace_bytes(const scn_rulebook* rb, int32_t C) {
  if (!rb || C < 1) return 0;
  // the per-block partial sums, then the GF_BLOCKS partial rows
  return (part_floats(rb, C) + (size_t)GF_BLOCKS * C) * sizeof(float);
}

scn_status scn_maxpool_bwd(const scn_rulebook* rb, const uint8_t* argmax, const float* dy,
                           const float* dg_out, int32_t C, float* dx, float* dg_in, void* ws,
                           size_t ws_bytes, hipStream_t st) {
  clear_error();
  if (scn_status rc0 = after_build(rb, st)) return rc0;
  if (!rb || C < 1 || (rb->a_out > 0 && (!argmax || !dy)) || (rb->a_in > 0 && !dx)) {
    set_error("scn_maxpool_bwd: invalid argument");
    return SCN_ERR_INVALID;
  }
  if (!rb->nbr) {
    set_error("scn_maxpool_bwd: the rulebook has no pooling tables (stride 1, or windows wider "
              "than their stride on sites of other than 3 coordinates)");
    return SCN_ERR_UNSUPPORTED;
  }
  if (!window_size_ok(rb->K)) {
    set_error("scn_maxpool_bwd: windows of %d sites are not supported", rb->K);
    return SCN_ERR_UNSUPPORTED;
  }
  const size_t need = scn_maxpool_bwd_workspace_bytes(rb, C);
  if (dg_in && (!ws || ws_bytes < need)) {
    set_error("scn_maxpool_bwd: workspace of %zu bytes needed, %zu given", need, ws_bytes);
    return SCN_ERR_WORKSPACE;
  }
  float* part = dg_in ? static_cast<float*>(ws) : nullptr;
  const bool vec = pool_vec_ok(C, {dy, dx, part}, argmax);
  const bool overlap = rb->inv_slots == 8;
  int64_t nblk = 0;
  if (overlap && vec && rb->lowwin) {
    // cell-major (3-wide windows of stride 2, cubic lattice): the inputs
    // without a home window, then every window's home cell and ground sums
    const int nc4 = C / 4, per = 256 / nc4;
    const auto* am4 = reinterpret_cast<const uint32_t*>(argmax);
    const auto* dy4 = reinterpret_cast<const float4*>(dy);
    auto* dx4 = reinterpret_cast<float4*>(dx);
    if (rb->a_in > 0) {
      hipLaunchKernelGGL(maxpool_bwd_homeless_vec_kernel,
                         dim3(std::min<unsigned>(nblocks(rb->a_in, per), 1024)), dim3(256), 0, st,
                         rb->homeless, rb->n_homeless, rb->inv, am4, dy4, nc4, per, dx4);
      SCN_LAUNCH_CHECK();
    }
    nblk = std::max<int64_t>(1, ceil_div(rb->a_out, CELL_ROWS));
    if (rb->a_out > 0) {
      const int chunk = xcd_chunk(nblk, 32);  // runs of 1024 windows per XCD
      hipLaunchKernelGGL(maxpool_bwd_cells_kernel, dim3(xcd_grid(nblk, chunk)), dim3(256), 0, st,
                         rb->nbr, rb->lowwin, rb->pmask, am4, dy4, rb->a_out, nc4, dx4,
                         reinterpret_cast<float4*>(part), chunk);
      SCN_LAUNCH_CHECK();
    }
  } else if (overlap) {
    // dx per input over its (up to 8) windows, then the ground-state sums
    // output-major
    if (rb->a_in > 0) {
      if (vec) {
        const int nc4 = C / 4;
        const auto* am4 = reinterpret_cast<const uint32_t*>(argmax);
        const auto* dy4 = reinterpret_cast<const float4*>(dy);
        auto* dx4 = reinterpret_cast<float4*>(dx);
        const int per = 256 / nc4;
        with_window(rb->K, [&](auto k) {
          hipLaunchKernelGGL(maxpool_bwd_overlap_vec_kernel<decltype(k)::value>,
                             dim3(nblocks(rb->a_in, per)), dim3(256), 0, st, rb->inv,
                             am4, dy4, rb->a_in, nc4, per, dx4);
        });
      } else {
        hipLaunchKernelGGL(maxpool_bwd_overlap_kernel, dim3(nblocks(rb->a_in * C, 256)), dim3(256),
                           0, st, rb->inv, argmax, dy, rb->a_in, C, rb->K, dx);
      }
      SCN_LAUNCH_CHECK();
    }
    if (dg_in) {
      nblk = std::max<int64_t>(1, ceil_div(rb->a_out, vec ? PBV_ROWS : PB_ROWS));
      if (rb->a_out > 0) {
        if (vec) {
          hipLaunchKernelGGL(maxpool_ground_vec_kernel, dim3((unsigned)nblk), dim3(256), 0, st,
                             rb->pmask, reinterpret_cast<const uint32_t*>(argmax),
                             reinterpret_cast<const float4*>(dy), rb->a_out, C / 4,
                             reinterpret_cast<float4*>(part));
        } else {
          hipLaunchKernelGGL(maxpool_bwd_ground_kernel, dim3((unsigned)nblk), dim3(256), 0, st,
                             rb->pmask, argmax, dy, rb->a_out, C, part);
        }
        SCN_LAUNCH_CHECK();
      }
    }
  } else if (vec) {
    // one pass: dx of the inputs in windows and the ground-state partial sums
    nblk = std::max<int64_t>(1, ceil_div(rb->a_out, PBV_ROWS));
    if (rb->a_in > 0) {
      hipLaunchKernelGGL(zero_uncovered_kernel, dim3(nblocks(rb->a_in, 256)), dim3(256), 0, st,
                         rb->inv, rb->a_in, C / 4, reinterpret_cast<float4*>(dx));
      SCN_LAUNCH_CHECK();
    }
    if (rb->a_out > 0) {
      const dim3 grid((unsigned)nblk);
      const auto* am4 = reinterpret_cast<const uint32_t*>(argmax);
      const auto* dy4 = reinterpret_cast<const float4*>(dy);
      auto* dx4 = reinterpret_cast<float4*>(dx);
      auto* p4 = reinterpret_cast<float4*>(part);
      with_window(rb->K, [&](auto k) {
        hipLaunchKernelGGL(maxpool_bwd_vec_kernel<decltype(k)::value>, grid, dim3(256), 0, st,
                           rb->nbr, am4, dy4, rb->a_out, C / 4, dx4, p4);
      });
      SCN_LAUNCH_CHECK();
    }
  } else {
    if (rb->a_in > 0) {
      hipLaunchKernelGGL(maxpool_bwd_dx_kernel, dim3(nblocks(rb->a_in * C, 256)), dim3(256), 0,
                         st, rb->inv, argmax, dy, rb->a_in, C, rb->K, dx);
      SCN_LAUNCH_CHECK();
    }
    nblk = std::max<int64_t>(1, ceil_div(rb->a_out, PB_ROWS));
    if (dg_in && rb->a_out > 0) {
      hipLaunchKernelGGL(maxpool_bwd_ground_kernel, dim3((unsigned)nblk), dim3(256), 0, st,
                         rb->pmask, argmax, dy, rb->a_out, C, part);
      SCN_LAUNCH_CHECK();
    }
  }
  if (dg_in) {
    float* part2 = part + part_floats(rb, C);
    hipLaunchKernelGGL(maxpool_ground_rows_kernel, dim3(GF_BLOCKS), dim3(256), 0, st, part,
                       rb->a_out > 0 ? nblk : 0, C, part2);
    SCN_LAUNCH_CHECK();
    hipLaunchKernelGGL(maxpool_bwd_ground_finish, dim3(nblocks(C, 64)), dim3(256), 0, st, part2,
                       C, dg_out, dg_in);
    SCN_LAUNCH_CHECK();
  }
  return SCN_OK;
}

}  // extern "C"
