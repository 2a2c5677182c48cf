// Sparse convolution, steps 2 and 3 of section 1.3 (gather the rows of Q, then
// Q W + B) and the gradients, on fp32 matrix cores (v_mfma_f32_16x16x4f32).
//
// Q is never formed.  Its row for output o holds, per offset k, either an
// input row or the ground state g_in.  Writing v_k(o) = g_in + (x[r] - g_in)
// when site s*o+k is active,
//     Q W + B = g_pre + sum_{pairs (r, o) of offset k} (x[r] - g_in) W_k,
//     g_pre   = B + sum_k g_in W_k,
// so only the active blocks are gathered and multiplied.
//
// Gather kernel (forward and input gradient).  A work-group owns a tile of
// accumulator rows (output rows for the forward, input ranks for the input
// gradient) and 64 columns; the accumulators live in LDS.  For each offset k
// the tile's pairs form one contiguous range of list k (lists ascend by output
// row and by input key), so the work-group stages up to 64 gathered rows in
// LDS, each wave multiplies them by its 16 columns of W_k with MFMA and adds
// the 16x16 results into the accumulator rows named by the pairs.  A wave is
// the only writer of its columns and pair rows are distinct within an offset,
// so the scatter needs no atomics and the summation order is fixed.
//
// Weight gradient.  dW_k = X_k^T dY_k over the P_k pairs of offset k is a
// contraction along the pair axis: split into fixed chunks, each chunk's
// partial product goes to the workspace, and a reduction sums the chunks in
// index order (deterministic).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "scn_internal.h"

namespace scn {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int NT = 256;     // threads per work-group (4 waves)
constexpr int CB = 64;      // columns per work-group
constexpr int CH = 64;      // gathered rows per stage
constexpr int ACC_LD = CB + 16;

__device__ inline v4f mfma4(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Ground state of the convolution output: g_pre = B + sum_k g_in W_k
// ---------------------------------------------------------------------------
__global__ void ground_pre_kernel(const float* __restrict__ g_in, const float* __restrict__ W,
                                  const float* __restrict__ bias, int K, int Cin, int Cout,
                                  float* __restrict__ g_pre) {
  const int co = blockIdx.x * blockDim.x + threadIdx.x;
  if (co >= Cout) return;
  float acc = bias ? bias[co] : 0.f;
  for (int k = 0; k < K; ++k)
    for (int ci = 0; ci < Cin; ++ci) acc = fmaf(g_in[ci], W[((int64_t)k * Cin + ci) * Cout + co], acc);
  g_pre[co] = acc;
}

__global__ void relu_vec_kernel(float* __restrict__ v, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) v[i] = v[i] > 0.f ? v[i] : 0.f;
}

// ---------------------------------------------------------------------------
// Gather -> MFMA -> LDS scatter
// ---------------------------------------------------------------------------
struct GatherArgs {
  const float* src;      // gathered rows [*][Rk]
  const int32_t* gidx;   // per pair: row of src
  const int32_t* aidx;   // per pair: accumulator row
  const int64_t* tpos;   // [K*ntile + 1] pair ranges per tile of TILE accumulator rows
  int64_t ntile;
  const float* W;        // B(j, n) = W[k*ks + j*sj + n*sn]
  int64_t ks, sj, sn;
  int Rk;                // reduction length (channels of src)
  int RkP;               // Rk rounded up to 16
  int Nc;                // output columns
  const float* sub;      // [Rk] subtracted from gathered rows, or null
  const float* add;      // [Nc] added to every accumulator row, or null
  int relu;
  float* dst;            // [nrows][Nc]
  const int32_t* wmap;   // dst row of accumulator row r (null = identity)
  int64_t nrows;
  int K;
  int TM;                // tiles of TILE rows per work-group
  int vec_ok;            // rows of src are 16-byte aligned (float4 gathers)
};

__global__ void __launch_bounds__(NT) gather_mfma_kernel(GatherArgs a) {
  extern __shared__ float smem[];
  const int T = a.TM * TILE;
  const int XS_LD = a.RkP + 4;
  float* acc = smem;                                  // [T][ACC_LD]
  float* xs = acc + (size_t)T * ACC_LD;               // [CH][XS_LD]
  int* ids = reinterpret_cast<int*>(xs + (size_t)CH * XS_LD);  // [CH]

  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int n16 = lane & 15, q = lane >> 4;
  const int64_t t0 = (int64_t)blockIdx.x * a.TM;
  const int64_t t1 = min(t0 + a.TM, a.ntile);
  const int64_t row0 = t0 * TILE;
  const int c0 = blockIdx.y * CB;
  const int col = c0 + 16 * w + n16;     // this lane's output column in MFMA results
  const bool wave_live = c0 + 16 * w < a.Nc;
  const int nkt = a.RkP >> 4;            // 16-wide reduction steps

  for (int i = tid; i < T * ACC_LD; i += NT) acc[i] = 0.f;

  const int vec_ok = a.vec_ok;
  for (int k = 0; k < a.K; ++k) {
    const int64_t p_begin = a.tpos[(int64_t)k * a.ntile + t0];
    const int64_t p_end = a.tpos[(int64_t)k * a.ntile + t1];
    if (p_begin >= p_end) continue;   // uniform across the work-group
    // B fragments of W_k for this wave's 16 columns: b[t][e] = B(16t + 4q + e, col)
    float b[64];
#pragma unroll
    for (int t = 0; t < 16; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = 16 * t + 4 * q + e;
        float v = 0.f;
        if (t < nkt && j < a.Rk && col < a.Nc) v = a.W[(int64_t)k * a.ks + j * a.sj + col * a.sn];
        b[4 * t + e] = v;
      }
    for (int64_t p0 = p_begin; p0 < p_end; p0 += CH) {
      const int n = (int)min<int64_t>(CH, p_end - p0);
      __syncthreads();  // previous stage fully consumed
      if (tid < CH) ids[tid] = tid < n ? (int)(a.aidx[p0 + tid] - row0) : 0;
      // gather n rows (zero rows up to the next multiple of 16 and zero padding columns)
      const int nr = (n + 15) & ~15;
      const int q4 = a.RkP >> 2;  // float4 per staged row
      for (int i = tid; i < nr * q4; i += NT) {
        const int r = i / q4, c4 = (i - r * q4) * 4;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (r < n) {
          const int64_t srow = a.gidx[p0 + r];
          const float* sp = a.src + srow * a.Rk;
          if (vec_ok && c4 + 3 < a.Rk) {
            v = *reinterpret_cast<const float4*>(sp + c4);
          } else {
            if (c4 + 0 < a.Rk) v.x = sp[c4 + 0];
            if (c4 + 1 < a.Rk) v.y = sp[c4 + 1];
            if (c4 + 2 < a.Rk) v.z = sp[c4 + 2];
            if (c4 + 3 < a.Rk) v.w = sp[c4 + 3];
          }
          if (a.sub) {
            if (c4 + 0 < a.Rk) v.x -= a.sub[c4 + 0];
            if (c4 + 1 < a.Rk) v.y -= a.sub[c4 + 1];
            if (c4 + 2 < a.Rk) v.z -= a.sub[c4 + 2];
            if (c4 + 3 < a.Rk) v.w -= a.sub[c4 + 3];
          }
        }
        *reinterpret_cast<float4*>(xs + r * XS_LD + c4) = v;
      }
      __syncthreads();
      if (!wave_live) continue;
      for (int rb = 0; rb < nr; rb += 16) {
        v4f c = {0.f, 0.f, 0.f, 0.f};
        const float* arow = xs + (rb + n16) * XS_LD + 4 * q;
#pragma unroll
        for (int t = 0; t < 16; ++t) {
          if (t < nkt) {
            const float4 av = *reinterpret_cast<const float4*>(arow + 16 * t);
            c = mfma4(av.x, b[4 * t + 0], c);
            c = mfma4(av.y, b[4 * t + 1], c);
            c = mfma4(av.z, b[4 * t + 2], c);
            c = mfma4(av.w, b[4 * t + 3], c);
          }
        }
        // lane holds rows rb + 4q + v, column col
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int r = rb + 4 * q + v;
          if (r < n) {
            float* ap = acc + ids[r] * ACC_LD + 16 * w + n16;
            *ap += c[v];
          }
        }
      }
    }
  }
  __syncthreads();
  // epilogue: dst[row] = act(acc + add)
  const int ncols = min(CB, a.Nc - c0);
  for (int i = tid; i < T * CB; i += NT) {
    const int r = i / CB, cc = i - r * CB;
    const int64_t grow = row0 + r;
    if (cc >= ncols || grow >= a.nrows) continue;
    float v = acc[r * ACC_LD + cc];
    if (a.add) v += a.add[c0 + cc];
    if (a.relu) v = v > 0.f ? v : 0.f;
    const int64_t drow = a.wmap ? (int64_t)a.wmap[grow] : grow;
    a.dst[drow * a.Nc + c0 + cc] = v;
  }
}

size_t gather_smem_bytes(int TM, int RkP) {
  return ((size_t)TM * TILE * ACC_LD + (size_t)CH * (RkP + 4)) * sizeof(float) + CH * sizeof(int);
}

scn_status launch_gather(GatherArgs a, hipStream_t st) {
  if (a.nrows <= 0) return SCN_OK;
  a.vec_ok = ((a.Rk & 3) == 0) && ((reinterpret_cast<uintptr_t>(a.src) & 15) == 0);
  const int64_t nwg = ceil_div(a.ntile, a.TM);
  const unsigned ncb = (unsigned)ceil_div(a.Nc, CB);
  const size_t smem = gather_smem_bytes(a.TM, a.RkP);
  static bool attr_set = false;
  if (!attr_set) {
    SCN_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(gather_mfma_kernel),
                                hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024));
    attr_set = true;
  }
  hipLaunchKernelGGL(gather_mfma_kernel, dim3((unsigned)nwg, ncb), dim3(NT), smem, st, a);
  SCN_LAUNCH_CHECK();
  return SCN_OK;
}

// ---------------------------------------------------------------------------
// Backward helpers
// ---------------------------------------------------------------------------
constexpr int RB_ROWS = 1024;  // rows per column-sum block

// dyb = relu ? dy * (y > 0) : dy (written only under relu);  partS[blk][c] = sum of dyb rows
__global__ void __launch_bounds__(NT) colsum_kernel(const float* __restrict__ dy,
                                                    const float* __restrict__ y, int relu,
                                                    int64_t rows, int C, float* __restrict__ dyb,
                                                    float* __restrict__ partS) {
  __shared__ float red[NT];
  const int64_t r0 = (int64_t)blockIdx.x * RB_ROWS;
  const int64_t r1 = min<int64_t>(r0 + RB_ROWS, rows);
  const int rg = threadIdx.x >> 6, cl = threadIdx.x & 63;
  for (int cbase = 0; cbase < C; cbase += 64) {
    const int c = cbase + cl;
    float s = 0.f;
    if (c < C) {
      for (int64_t r = r0 + rg; r < r1; r += 4) {
        float v = dy[r * C + c];
        if (relu) {
          v = y[r * C + c] > 0.f ? v : 0.f;
          dyb[r * C + c] = v;
        }
        s += v;
      }
    }
    red[threadIdx.x] = s;
    __syncthreads();
    if (rg == 0 && c < C)
      partS[(int64_t)blockIdx.x * C + c] = ((red[cl] + red[64 + cl]) + red[128 + cl]) + red[192 + cl];
    __syncthreads();
  }
}

// S, dḡ, dbias; u0 = S + dḡ
__global__ void finish_vec_kernel(const float* __restrict__ partS, int64_t nblk, int C,
                                  const float* __restrict__ g_out, const float* __restrict__ dg_out,
                                  int relu, float* __restrict__ S, float* __restrict__ u0,
                                  float* __restrict__ dbias) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= C) return;
  float s = 0.f;
  for (int64_t b = 0; b < nblk; ++b) s += partS[b * C + c];
  float dg = dg_out ? dg_out[c] : 0.f;
  if (relu && dg_out) dg = g_out[c] > 0.f ? dg : 0.f;
  S[c] = s;
  u0[c] = s + dg;
  if (dbias) dbias[c] = s + dg;
}

// Weight gradient partials.  grid (chunk, k, cin-block * n_co_blocks + co-block)
constexpr int DW_SC = 64;          // pairs per stage
constexpr int DW_LD = DW_SC + 4;

struct DwArgs {
  const float* x;        // [a_in][Cin]
  const float* dyb;      // [a_out][Cout]
  const float* g_in;     // [Cin]
  const int32_t* in_rows;
  const int32_t* out_rows;
  const int64_t* off;    // [K+1]
  int Cin, Cout;
  int64_t chp;           // pairs per chunk
  int64_t maxc;          // chunks per offset (slot count)
  float* part;           // [K][maxc][Cin][Cout]
  float* partT;          // [K][maxc][Cout]
};

__global__ void __launch_bounds__(NT) dw_partial_kernel(DwArgs a) {
  __shared__ float xsT[64 * DW_LD];  // [ci][pair]
  __shared__ float dsT[64 * DW_LD];  // [co][pair]
  const int k = blockIdx.y;
  const int64_t c = blockIdx.x;
  const int64_t lb = a.off[k], le = a.off[k + 1];
  const int64_t p_begin = lb + c * a.chp;
  if (p_begin >= le) return;
  const int64_t p_end = min(le, p_begin + a.chp);
  const int nco = (a.Cout + 63) / 64;
  const int ci0 = (blockIdx.z / nco) * 64, co0 = (blockIdx.z % nco) * 64;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n16 = lane & 15, q = lane >> 4;

  v4f acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = (v4f){0.f, 0.f, 0.f, 0.f};
  float tsum = 0.f;  // column sum of dyb over this lane's quarter of every stage
  const int tcol = 16 * w + n16;

  // gather mapping: lane -> (pair = i16 + 16*rep, channel quad)
  for (int64_t p0 = p_begin; p0 < p_end; p0 += DW_SC) {
    const int n = (int)min<int64_t>(DW_SC, p_end - p0);
    __syncthreads();
    // 64 pairs x 16 quads = 1024 items, 4 per thread; consecutive lanes = consecutive pairs
    for (int it = tid; it < DW_SC * 16; it += NT) {
      const int pr = it & 63, c4 = (it >> 6) * 4;
      float4 xv = make_float4(0.f, 0.f, 0.f, 0.f), dv = xv;
      if (pr < n) {
        const int64_t ri = a.in_rows[p0 + pr], ro = a.out_rows[p0 + pr];
        const float* xp = a.x + ri * a.Cin + ci0;
        const float* dp = a.dyb + ro * a.Cout + co0;
        float xe[4], de[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int ci = ci0 + c4 + e, co = co0 + c4 + e;
          xe[e] = ci < a.Cin ? xp[c4 + e] - a.g_in[ci] : 0.f;
          de[e] = co < a.Cout ? dp[c4 + e] : 0.f;
        }
        xv = make_float4(xe[0], xe[1], xe[2], xe[3]);
        dv = make_float4(de[0], de[1], de[2], de[3]);
      }
      xsT[(c4 + 0) * DW_LD + pr] = xv.x;
      xsT[(c4 + 1) * DW_LD + pr] = xv.y;
      xsT[(c4 + 2) * DW_LD + pr] = xv.z;
      xsT[(c4 + 3) * DW_LD + pr] = xv.w;
      dsT[(c4 + 0) * DW_LD + pr] = dv.x;
      dsT[(c4 + 1) * DW_LD + pr] = dv.y;
      dsT[(c4 + 2) * DW_LD + pr] = dv.z;
      dsT[(c4 + 3) * DW_LD + pr] = dv.w;
    }
    __syncthreads();
    // A(m = ci, kk = pair) = xsT[16w + m][pair];  B(kk = pair, n = co) = dsT[16j + n][pair]
    const float* ar = xsT + (16 * w + n16) * DW_LD + 4 * q;
#pragma unroll
    for (int t = 0; t < DW_SC / 16; ++t) {
      const float4 av = *reinterpret_cast<const float4*>(ar + 16 * t);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 bv = *reinterpret_cast<const float4*>(dsT + (16 * j + n16) * DW_LD + 4 * q + 16 * t);
        acc[j] = mfma4(av.x, bv.x, acc[j]);
        acc[j] = mfma4(av.y, bv.y, acc[j]);
        acc[j] = mfma4(av.z, bv.z, acc[j]);
        acc[j] = mfma4(av.w, bv.w, acc[j]);
      }
    }
    if (ci0 == 0) {
      // this lane sums column tcol over pairs [16q, 16q + 16) of the stage
      const float* tr = dsT + tcol * DW_LD + 16 * q;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 v = *reinterpret_cast<const float4*>(tr + 4 * i);
        tsum += ((v.x + v.y) + v.z) + v.w;
      }
    }
  }
  // write partial dW: lane holds rows 4q + v (ci), column n16 of tile j (co)
  float* out = a.part + ((int64_t)k * a.maxc + c) * a.Cin * a.Cout;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int ci = ci0 + 16 * w + 4 * q + v, co = co0 + 16 * j + n16;
      if (ci < a.Cin && co < a.Cout) out[(int64_t)ci * a.Cout + co] = acc[j][v];
    }
  if (ci0 == 0) {
    // combine the four quarters in a fixed order
    const float t1 = __shfl_xor(tsum, 16, 64);
    const float s01 = q & 1 ? t1 + tsum : tsum + t1;
    const float t2 = __shfl_xor(s01, 32, 64);
    const float s = q & 2 ? t2 + s01 : s01 + t2;
    const int co = co0 + tcol;
    if (q == 0 && co < a.Cout) a.partT[((int64_t)k * a.maxc + c) * a.Cout + co] = s;
  }
}

// dW[k][ci][co] = sum_c part + g_in[ci] * u0[co];  T[k][co] = sum_c partT
__global__ void dw_reduce_kernel(const float* __restrict__ part, const float* __restrict__ partT,
                                 const int64_t* __restrict__ off, int K, int Cin, int Cout,
                                 int64_t chp, int64_t maxc, const float* __restrict__ g_in,
                                 const float* __restrict__ u0, float* __restrict__ dW,
                                 float* __restrict__ T) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t per = (int64_t)Cin * Cout;
  if (i < (int64_t)K * per) {
    const int k = (int)(i / per);
    const int64_t e = i - k * per;
    const int ci = (int)(e / Cout), co = (int)(e - (int64_t)ci * Cout);
    const int64_t nch = ceil_div(off[k + 1] - off[k], chp);
    const float* p = part + (int64_t)k * maxc * per + e;
    float s = 0.f;
    for (int64_t c = 0; c < nch; ++c) s += p[c * per];
    if (dW) dW[i] = s + g_in[ci] * u0[co];
  }
  if (i < (int64_t)K * Cout) {
    const int k = (int)(i / Cout), co = (int)(i % Cout);
    const int64_t nch = ceil_div(off[k + 1] - off[k], chp);
    float s = 0.f;
    for (int64_t c = 0; c < nch; ++c) s += partT[((int64_t)k * maxc + c) * Cout + co];
    T[i] = s;
  }
}

// dg_in[ci] = sum_k sum_co W[k][ci][co] * (u0[co] - T[k][co])
__global__ void dgin_kernel(const float* __restrict__ W, const float* __restrict__ u0,
                            const float* __restrict__ T, int K, int Cin, int Cout,
                            float* __restrict__ dg_in) {
  const int ci = blockIdx.x * blockDim.x + threadIdx.x;
  if (ci >= Cin) return;
  float s = 0.f;
  for (int k = 0; k < K; ++k)
    for (int co = 0; co < Cout; ++co)
      s = fmaf(W[((int64_t)k * Cin + ci) * Cout + co], u0[co] - T[(int64_t)k * Cout + co], s);
  dg_in[ci] = s;
}

inline int64_t dw_chunk(int64_t P) {
  const int64_t want = ceil_div(std::max<int64_t>(P, 1), 2048);
  return std::max<int64_t>(1024, ceil_div(want, 256) * 256);
}

struct BwdLayout {
  int64_t chp, maxc, nblk;
  size_t o_dyb, o_part, o_partT, o_partS, o_S, o_u0, o_T, total;
};

BwdLayout bwd_layout(const scn_rulebook* rb, int Cin, int Cout, uint32_t flags) {
  BwdLayout L{};
  int64_t pmax = 0;
  for (int k = 0; k < rb->K; ++k) pmax = std::max(pmax, rb->off_host[k + 1] - rb->off_host[k]);
  L.chp = dw_chunk(rb->n_pairs);
  L.maxc = std::max<int64_t>(1, ceil_div(pmax, L.chp));
  L.nblk = std::max<int64_t>(1, ceil_div(rb->a_out, RB_ROWS));
  auto al = [](size_t b) { return (b + 255) & ~size_t(255); };
  size_t cur = 0;
  L.o_dyb = cur;
  cur += (flags & SCN_RELU) ? al((size_t)rb->a_out * Cout * 4) : 0;
  L.o_part = cur;
  cur += al((size_t)rb->K * L.maxc * Cin * Cout * 4);
  L.o_partT = cur;
  cur += al((size_t)rb->K * L.maxc * Cout * 4);
  L.o_partS = cur;
  cur += al((size_t)L.nblk * Cout * 4);
  L.o_S = cur;
  cur += al((size_t)Cout * 4);
  L.o_u0 = cur;
  cur += al((size_t)Cout * 4);
  L.o_T = cur;
  cur += al((size_t)rb->K * Cout * 4);
  L.total = cur;
  return L;
}

constexpr int pick_tm() { return 2; }

}  // namespace
}  // namespace scn

using namespace scn;

extern "C" {

scn_status scn_conv_fwd(const scn_rulebook* rb, const float* x, const float* g_in,
                        const float* W, const float* bias, int32_t Cin, int32_t Cout,
                        uint32_t flags, float* y, float* g_out, hipStream_t st) {
  clear_error();
  if (!rb || !g_in || !W || !g_out || Cin < 1 || Cout < 1 || (rb->a_in > 0 && !x) ||
      (rb->a_out > 0 && !y)) {
    set_error("scn_conv_fwd: invalid argument");
    return SCN_ERR_INVALID;
  }
  if (Cin > 256) {
    set_error("scn_conv_fwd: Cin %d > 256 is not supported", Cin);
    return SCN_ERR_UNSUPPORTED;
  }
  const int relu = (flags & SCN_RELU) ? 1 : 0;
  hipLaunchKernelGGL(ground_pre_kernel, dim3((unsigned)ceil_div(Cout, 64)), dim3(64), 0, st, g_in,
                     W, bias, rb->K, Cin, Cout, g_out);
  SCN_LAUNCH_CHECK();
  GatherArgs a{};
  a.src = x;
  a.gidx = rb->in_rows;
  a.aidx = rb->out_rows;
  a.tpos = rb->otile;
  a.ntile = rb->n_otiles;
  a.W = W;
  a.ks = (int64_t)Cin * Cout;
  a.sj = Cout;
  a.sn = 1;
  a.Rk = Cin;
  a.RkP = (int)ceil_div(Cin, 16) * 16;
  a.Nc = Cout;
  a.sub = g_in;
  a.add = g_out;  // holds g_pre until the ReLU below
  a.relu = relu;
  a.dst = y;
  a.wmap = nullptr;
  a.nrows = rb->a_out;
  a.K = rb->K;
  a.TM = pick_tm();
  scn_status rc = launch_gather(a, st);
  if (rc) return rc;
  if (relu) {
    hipLaunchKernelGGL(relu_vec_kernel, dim3((unsigned)ceil_div(Cout, 256)), dim3(256), 0, st,
                       g_out, Cout);
    SCN_LAUNCH_CHECK();
  }
  return SCN_OK;
}

size_t scn_conv_bwd_workspace_bytes(const scn_rulebook* rb, int32_t Cin, int32_t Cout,
                                    uint32_t flags) {
  if (!rb || Cin < 1 || Cout < 1) return 0;
  return bwd_layout(rb, Cin, Cout, flags).total;
}

scn_status scn_conv_bwd(const scn_rulebook* rb, const float* x, const float* g_in,
                        const float* W, const float* y, const float* g_out, const float* dy,
                        const float* dg_out, int32_t Cin, int32_t Cout, uint32_t flags,
                        float* dx, float* dg_in, float* dW, float* dbias, void* ws,
                        size_t ws_bytes, hipStream_t st) {
  clear_error();
  const int relu = (flags & SCN_RELU) ? 1 : 0;
  if (!rb || !g_in || !W || Cin < 1 || Cout < 1 || (rb->a_out > 0 && !dy) ||
      (rb->a_in > 0 && !x) || (relu && rb->a_out > 0 && !y) || (relu && dg_out && !g_out)) {
    set_error("scn_conv_bwd: invalid argument");
    return SCN_ERR_INVALID;
  }
  if (Cin > 256 || Cout > 256) {
    set_error("scn_conv_bwd: channels > 256 are not supported");
    return SCN_ERR_UNSUPPORTED;
  }
  const BwdLayout L = bwd_layout(rb, Cin, Cout, flags);
  if (!ws || ws_bytes < L.total) {
    set_error("scn_conv_bwd: workspace of %zu bytes needed, %zu given", L.total, ws_bytes);
    return SCN_ERR_WORKSPACE;
  }
  char* base = static_cast<char*>(ws);
  float* dyb = relu ? reinterpret_cast<float*>(base + L.o_dyb) : const_cast<float*>(dy);
  float* part = reinterpret_cast<float*>(base + L.o_part);
  float* partT = reinterpret_cast<float*>(base + L.o_partT);
  float* partS = reinterpret_cast<float*>(base + L.o_partS);
  float* S = reinterpret_cast<float*>(base + L.o_S);
  float* u0 = reinterpret_cast<float*>(base + L.o_u0);
  float* T = reinterpret_cast<float*>(base + L.o_T);
  const int K = rb->K;

  // dȳ and S (column sums over active outputs)
  if (rb->a_out > 0) {
    hipLaunchKernelGGL(colsum_kernel, dim3((unsigned)L.nblk), dim3(NT), 0, st, dy, y, relu,
                       rb->a_out, Cout, dyb, partS);
    SCN_LAUNCH_CHECK();
  }
  hipLaunchKernelGGL(finish_vec_kernel, dim3((unsigned)ceil_div(Cout, 64)), dim3(64), 0, st,
                     partS, rb->a_out > 0 ? L.nblk : 0, Cout, g_out, dg_out, relu, S, u0, dbias);
  SCN_LAUNCH_CHECK();

  // input gradient: accumulate over input ranks with W_k^T
  if (dx && rb->a_in > 0) {
    GatherArgs a{};
    a.src = dyb;
    a.gidx = rb->out_rows;
    a.aidx = rb->in_rank;
    a.tpos = rb->itile;
    a.ntile = rb->n_itiles;
    a.W = W;
    a.ks = (int64_t)Cin * Cout;
    a.sj = 1;      // reduction index j = output channel
    a.sn = Cout;   // result column n = input channel
    a.Rk = Cout;
    a.RkP = (int)ceil_div(Cout, 16) * 16;
    a.Nc = Cin;
    a.sub = nullptr;
    a.add = nullptr;
    a.relu = 0;
    a.dst = dx;
    a.wmap = rb->input_sorted ? nullptr : rb->perm;
    a.nrows = rb->a_in;
    a.K = K;
    a.TM = pick_tm();
    scn_status rc = launch_gather(a, st);
    if (rc) return rc;
  }

  // weight gradient partials (also the per-offset column sums T_k)
  if (dW || dg_in) {
    DwArgs d{};
    d.x = x;
    d.dyb = dyb;
    d.g_in = g_in;
    d.in_rows = rb->in_rows;
    d.out_rows = rb->out_rows;
    d.off = rb->off_dev;
    d.Cin = Cin;
    d.Cout = Cout;
    d.chp = L.chp;
    d.maxc = L.maxc;
    d.part = part;
    d.partT = partT;
    if (rb->n_pairs > 0) {
      const unsigned nz = (unsigned)(ceil_div(Cin, 64) * ceil_div(Cout, 64));
      hipLaunchKernelGGL(dw_partial_kernel, dim3((unsigned)L.maxc, (unsigned)K, nz), dim3(NT), 0,
                         st, d);
      SCN_LAUNCH_CHECK();
    }
    const int64_t nred = std::max<int64_t>((int64_t)K * Cin * Cout, (int64_t)K * Cout);
    hipLaunchKernelGGL(dw_reduce_kernel, dim3((unsigned)ceil_div(nred, 256)), dim3(256), 0, st,
                       part, partT, rb->off_dev, K, Cin, Cout, L.chp, L.maxc, g_in, u0, dW, T);
    SCN_LAUNCH_CHECK();
    if (dg_in) {
      hipLaunchKernelGGL(dgin_kernel, dim3((unsigned)ceil_div(Cin, 64)), dim3(64), 0, st, W, u0,
                         T, K, Cin, Cout, dg_in);
      SCN_LAUNCH_CHECK();
    }
  }
  return SCN_OK;
}

}  // extern "C"
