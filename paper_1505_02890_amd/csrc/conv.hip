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
// Gather kernel (forward and input gradient).  A work-group of four waves owns
// a tile of accumulator rows (output rows for the forward, input ranks for the
// input gradient) and 64 columns; the accumulators live in LDS and each wave
// owns 16 of the columns.  For each offset k the tile's pairs form one
// contiguous range of list k (lists ascend by output row and by input key).
// The tile's ranges are read once into lanes; the work-group walks them in
// stages of 32 pairs of one offset.  Per stage it gathers the 32 rows into an
// LDS buffer (one gather per row, shared by the four waves), each wave
// multiplies them by its slice of W_k on the matrix cores and adds the
// products into the LDS rows named by the pairs.  Rows, row indices and
// weights are fetched two stages ahead, and a stage's products are added one
// stage later, so no wave waits for memory or for its own matrix-core
// results in steady state.  A wave is the only writer of its columns and pair
// rows are distinct within an offset, so the scatter needs no atomics and the
// summation order is fixed.
//
// Weight gradient.  dW_k = X_k^T dY_k over the P_k pairs of offset k is a
// contraction along the pair axis: split into fixed chunks, each chunk's
// partial product goes to the workspace, and a reduction sums the chunks in
// index order (deterministic).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "scn_internal.h"

namespace scn {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int NT = 256;     // threads per work-group (4 waves)
constexpr int CB = 64;      // columns per work-group
constexpr int ACC_LD = CB + 4;

__device__ inline v4f mfma4(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Work-groups are dispatched round-robin over the 8 XCDs; give each XCD a
// contiguous range of work items so neighbouring tiles share its L2.
__device__ inline int64_t xcd_remap(int64_t b, int64_t n) {
  const int64_t x = b & 7, j = b >> 3, base = n >> 3, rem = n & 7;
  return x * base + min(x, rem) + j;
}

// ---------------------------------------------------------------------------
// Ground-state terms of the convolution.
//   gw[k][co]  = sum_ci g_in[ci] W[k][ci][co]       (what an inactive site at
//                offset k contributes; subtracted per pair in the residual form)
//   g_pre[co]  = B[co] + sum_k gw[k][co]
// ---------------------------------------------------------------------------
// One block per (k, 64 columns): thread (group g, column c) sums the input
// channels ci = g (mod GW_GROUPS) in ascending order, then the group sums are
// added in group order (fixed order, so the result is deterministic).
constexpr int GW_GROUPS = 4;
__global__ void __launch_bounds__(256) ground_w_kernel(const float* __restrict__ g_in,
                                                       const float* __restrict__ W, int K, int Cin,
                                                       int Cout, int ld, float* __restrict__ gw) {
  __shared__ float part[GW_GROUPS][64];
  const int nb = ld / 64;  // column blocks (ld is a multiple of 64)
  const int k = blockIdx.x / nb, c0 = (blockIdx.x - k * nb) * 64;
  const int c = threadIdx.x & 63, grp = threadIdx.x >> 6;
  const int co = c0 + c;
  float s = 0.f;
  if (co < Cout) {
    const float* wp = W + (int64_t)k * Cin * Cout + co;
#pragma unroll 4
    for (int ci = grp; ci < Cin; ci += GW_GROUPS) s = fmaf(g_in[ci], wp[(int64_t)ci * Cout], s);
  }
  part[grp][c] = s;
  __syncthreads();
  if (grp == 0) {
    float t = part[0][c];
#pragma unroll
    for (int g = 1; g < GW_GROUPS; ++g) t += part[g][c];
    gw[(int64_t)k * ld + co] = t;
  }
}

// g_pre (kept for the contraction's epilogue) and g_out = act(g_pre)
__global__ void ground_pre_kernel(const float* __restrict__ gw, int ld,
                                  const float* __restrict__ bias, int K, int Cout, int relu,
                                  float* __restrict__ g_pre, float* __restrict__ g_out) {
  const int co = blockIdx.x * blockDim.x + threadIdx.x;
  if (co >= Cout) return;
  float s = bias ? bias[co] : 0.f;
  for (int k = 0; k < K; ++k) s += gw[(int64_t)k * ld + co];
  g_pre[co] = s;
  g_out[co] = relu && !(s > 0.f) ? 0.f : s;
}

__global__ void zero_kernel(float* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.f;
}

// Packed weights for the gather kernel, in MFMA fragment order:
//   Wp[k][cb][w][t][lane][e] = W_k(j = 16t + 4q + e, n = 64cb + 16w + n16),
//   lane = n16 + 16q, zero outside j < Rk, n < Nc;  RkP = 16*NKT, NcP = 64*NCB.
//   forward:        W_k(j = ci, n = co) = W[k][ci][co]
//   input gradient: W_k(j = co, n = ci) = W[k][ci][co]
__global__ void __launch_bounds__(256) pack_w_kernel(const float* __restrict__ W, int K, int Cin,
                                                     int Cout, int transpose, int RkP, int NcP,
                                                     float* __restrict__ Wp) {
  const int Nc = transpose ? Cout : Cin, Rk = transpose ? Cin : Cout;
  const int nkt = RkP / 16, ncb = NcP / 64;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)K * NcP * RkP) return;
  const int e = (int)(i & 3), ln = (int)((i >> 2) & 63);
  const int64_t f = i >> 8;  // ((k*ncb + cb)*4 + w)*nkt + t
  const int t = (int)(f % nkt);
  const int64_t g = f / nkt;
  const int wv = (int)(g & 3);
  const int64_t h = g >> 2;
  const int cbk = (int)(h % ncb);
  const int64_t k = h / ncb;
  const int j = 16 * t + 4 * (ln >> 4) + e;
  const int n = 64 * cbk + 16 * wv + (ln & 15);
  float v = 0.f;
  if (j < Rk && n < Nc) {
    const int ci = transpose ? j : n, co = transpose ? n : j;
    v = W[(k * Cin + ci) * Cout + co];
  }
  Wp[i] = v;
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
  const float* Wp;       // W_k(j, n) = Wp[(k*NcP + n)*RkP + j], zero-padded (RkP = 16*ceil(Rk/16))
  const float* gwp;      // [K][NcP] subtracted from every pair's product (zeros if none)
  int NcP;               // Nc rounded up to 64
  int Rk;                // reduction length (channels of src)
  int Nc;                // output columns
  const float* add;      // [Nc] added to every accumulator row, or null
  int relu;
  float* dst;            // [nrows][Nc]
  const int32_t* wmap;   // dst row of accumulator row r (null = identity)
  int64_t nrows;
  int K;
  int vec_ok;            // rows of src are 16-byte aligned and Rk % 4 == 0
  int dvec_ok;           // rows of dst are 16-byte aligned and Nc % 4 == 0
};

// One pipeline stage covers up to 32 consecutive pairs of one offset (two
// 16-pair blocks).  The work-group gathers the stage's rows once into an LDS
// buffer (8 threads per row, float4 loads); each wave then reads MFMA
// fragments from LDS: lane (n16, q) takes channels 16t + 4q .. +3 of pair n16
// of each block, which is the B-operand layout of v_mfma_f32_16x16x4f32 when
// the contraction is computed transposed (R^T = W_k^T X^T).  The result holds
// pair n16, output columns 4q .. 4q+3 of the wave's 16 in one lane, so the
// lane adds one contiguous float4 into its pair's accumulator row.  The
// pair's accumulator row travels with its gathered row, in the padding word
// of the LDS row.
constexpr int SROWS = 32;  // pairs per stage

template <int NKT>
struct WFrag {
  float4 w[NKT];  // W_k(j = 16t + 4q + 0..3, column 16w + n16)
  float4 g;       // gw[k][16w + 4q .. +3]
};

// Weights in fragment order: Wp[k][cb][w][t][lane][e] = W_k(j = 16t + 4q + e,
// n = 64cb + 16w + n16) with lane = n16 + 16q, zero-padded to 16*NKT rows and
// NcP = 64*ceil(Nc/64) columns, so a wave's fragment is NKT contiguous 1 KB
// blocks.  gw is [K][NcP].
template <int NKT>
__device__ inline WFrag<NKT> load_w(const GatherArgs& a, int k, int cb, int w, int lane, int gcol) {
  WFrag<NKT> f;
  const float* wp =
      a.Wp + (((int64_t)k * (a.NcP >> 6) + cb) * 4 + w) * (int64_t)(NKT * 256) + lane * 4;
#pragma unroll
  for (int t = 0; t < NKT; ++t) f.w[t] = *reinterpret_cast<const float4*>(wp + 256 * t);
  f.g = *reinterpret_cast<const float4*>(a.gwp + (int64_t)k * a.NcP + gcol);
  return f;
}

// Per-thread share of one stage's gather: row tid/8, channel quads
// (tid%8) + 8u, and the row's accumulator index.  Positions past the stage's
// pairs are clamped to its last pair (loads stay in bounds; those rows are
// never scattered).  Reduction slots j >= Rk read some channel of the row;
// the matching W entries are zero.
template <int NKT>
struct StageRegs {
  static constexpr int NQ = (4 * NKT + 7) / 8;  // float4 per thread
  v4f v[NQ];  // (arrays of HIP's float4 struct were left in scratch memory)
  int acc_row;
};

template <int NKT, bool VEC>
__device__ inline StageRegs<NKT> load_stage(const GatherArgs& a, int gi, int ai, int tid) {
  StageRegs<NKT> R;
  const float* rp = a.src + (int64_t)gi * a.Rk;
  const int part = tid & 7;
#pragma unroll
  for (int u = 0; u < StageRegs<NKT>::NQ; ++u) {
    const int c = 4 * (part + 8 * u);
    if (VEC) {
      const int cc = c < a.Rk ? c : 0;
      R.v[u] = *reinterpret_cast<const v4f*>(rp + cc);
    } else {
#pragma unroll
      for (int z = 0; z < 4; ++z) R.v[u][z] = rp[c + z < a.Rk ? c + z : 0];
    }
  }
  R.acc_row = ai;
  return R;
}

template <int NKT>
__device__ inline void store_stage(float* xs, int tid, const StageRegs<NKT>& R) {
  constexpr int XLD = 16 * NKT + 4;
  const int row = tid >> 3, part = tid & 7;
#pragma unroll
  for (int u = 0; u < StageRegs<NKT>::NQ; ++u) {
    const int quad = part + 8 * u;
    if (quad < 4 * NKT) *reinterpret_cast<v4f*>(xs + row * XLD + 4 * quad) = R.v[u];
  }
  reinterpret_cast<int*>(xs)[row * XLD + 16 * NKT] = R.acc_row;  // same value from all 8
}

// Products of one stage held by a lane: pair n16 of each 16-pair block,
// output columns cq .. cq+3, already offset by -gw (the accumulator starts at
// -gw), and the accumulator rows they go to.
struct StageOut {
  v4f c0, c1;
  int i0, i1;
};

// Multiply one stage (cnt live pairs, possibly none) by the wave's W_k slice.
// Lanes past the live pairs target the spare row `spare` (never read), so
// the code has no branch.
template <int NKT>
__device__ inline StageOut stage_mfma(const float* xs, const WFrag<NKT>& B, int cnt, int spare,
                                      int n16, int q) {
  constexpr int XLD = 16 * NKT + 4;
  const float* r0 = xs + n16 * XLD + 4 * q;
  const float* r1 = xs + (16 + n16) * XLD + 4 * q;
  const int* ai = reinterpret_cast<const int*>(xs) + 16 * NKT;
  StageOut o;
  const int a0 = ai[n16 * XLD], a1 = ai[(16 + n16) * XLD];
  o.i0 = n16 < cnt ? a0 : spare;
  o.i1 = 16 + n16 < cnt ? a1 : spare;
  v4f c0v = {-B.g.x, -B.g.y, -B.g.z, -B.g.w}, c1v = c0v;
#pragma unroll
  for (int t = 0; t < NKT; ++t) {
    const float4 x0 = *reinterpret_cast<const float4*>(r0 + 16 * t);
    const float4 x1 = *reinterpret_cast<const float4*>(r1 + 16 * t);
    c0v = mfma4(B.w[t].x, x0.x, c0v);
    c1v = mfma4(B.w[t].x, x1.x, c1v);
    c0v = mfma4(B.w[t].y, x0.y, c0v);
    c1v = mfma4(B.w[t].y, x1.y, c1v);
    c0v = mfma4(B.w[t].z, x0.z, c0v);
    c1v = mfma4(B.w[t].z, x1.z, c1v);
    c0v = mfma4(B.w[t].w, x0.w, c0v);
    c1v = mfma4(B.w[t].w, x1.w, c1v);
  }
  o.c0 = c0v;
  o.c1 = c1v;
  return o;
}

// Add a stage's products into its accumulator rows (columns cq .. cq+3).
__device__ inline void stage_scatter(const StageOut& o, float* acc, int cq) {
  float4* r = reinterpret_cast<float4*>(&acc[o.i0 * ACC_LD + cq]);
  float4 v = *r;
  v.x += o.c0[0];
  v.y += o.c0[1];
  v.z += o.c0[2];
  v.w += o.c0[3];
  *r = v;
  r = reinterpret_cast<float4*>(&acc[o.i1 * ACC_LD + cq]);
  v = *r;
  v.x += o.c1[0];
  v.y += o.c1[1];
  v.z += o.c1[2];
  v.w += o.c1[3];
  *r = v;
}

// Stage schedule of one tile.  Lane k (< K) of every wave holds the tile's
// pair range of list k: start P and length N (at most TM*64: one pair per
// accumulator row and offset); `live` has bit k set when N > 0.  Stages are
// stepped with readlane, so the main loop makes no memory access to find its
// next stage.
struct Sched {
  int64_t P;
  int N;
  uint64_t live;
  int K;
};

__device__ inline int64_t lane64(int64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(uint64_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// A stage position: offset k, pairs [p, p + min(n, 32)) of list k; k == K
// (n == 0) past the tile's last stage.
struct Pos {
  int k, n;
  int64_t p;
};

__device__ inline Pos jump(const Sched& s, uint64_t m) {
  Pos x;
  if (!m) {
    x.k = s.K;
    x.n = 0;
    x.p = 0;
    return x;
  }
  x.k = __builtin_ctzll(m);
  x.p = lane64(s.P, x.k);
  x.n = __builtin_amdgcn_readlane(s.N, x.k);
  return x;
}

__device__ inline Pos next_stage(const Sched& s, Pos x) {
  if (x.k >= s.K) return x;
  x.p += SROWS;
  x.n -= SROWS;
  if (x.n > 0) return x;
  return jump(s, s.live & ~((2ull << x.k) - 1ull));
}

// Main loop, unrolled by two so that the register sets of the software
// pipeline keep fixed names (X = iteration parity); a tile with an odd number
// of stages ends with one empty stage.  Iteration i computes
// stage s_i; in flight meanwhile: the rows of s_{i+1} (landed, stored to LDS
// at the top of the iteration), the rows of s_{i+2} and s_{i+3}, the row
// indices of s_{i+4} and s_{i+5}, and the weights of s_{i+1} and s_{i+2}.
// The row and index loads of an iteration are unconditional; the weights are
// loaded only when the offset changes.
template <int NKT, bool VEC, int TM, int MINB>
__global__ void __launch_bounds__(NT, MINB) gather_mfma_kernel(GatherArgs a) {
  extern __shared__ float smem[];
  constexpr int T = TM * TILE;
  constexpr int XLD = 16 * NKT + 4;
  float* acc = smem;                      // [T + 1][ACC_LD], row T is the spare row
  float* xsb = smem + (T + 1) * ACC_LD;   // [2][SROWS][XLD]
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int n16 = lane & 15, q = lane >> 4;
  const int64_t tile = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t t0 = tile * TM;
  const int64_t t1 = min(t0 + TM, a.ntile);
  const int64_t row0 = t0 * TILE;
  const int cb = blockIdx.y;
  const int c0 = cb * CB;
  const int cq = 16 * w + 4 * q;      // tile-local columns this lane accumulates
  const int lrow = tid >> 3;          // stage row this thread gathers

  for (int i = tid; i < T * ACC_LD / 4; i += NT)
    reinterpret_cast<float4*>(acc)[i] = make_float4(0.f, 0.f, 0.f, 0.f);

  Sched sc;
  sc.K = a.K;
  {
    const int k = lane < a.K ? lane : 0;
    sc.P = a.tpos[(int64_t)k * a.ntile + t0];
    sc.N = lane < a.K ? (int)(a.tpos[(int64_t)k * a.ntile + t1] - sc.P) : 0;
    sc.live = __ballot(sc.N > 0);
  }
  Pos s0 = jump(sc, sc.live);
  if (s0.k < a.K) {
    const Pos first = s0;
    // loads for a position past the last stage use the first stage (in
    // bounds, never scattered)
    auto real = [&](const Pos x) -> Pos { return x.k < a.K ? x : first; };
    auto gidx_of = [&](const Pos x) -> int {
      const Pos r = real(x);
      return a.gidx[r.p + min(lrow, r.n - 1)];
    };
    auto aidx_of = [&](const Pos x) -> int {
      const Pos r = real(x);
      return (int)(a.aidx[r.p + min(lrow, r.n - 1)] - row0);
    };
    auto wk = [&](const Pos x) { return load_w<NKT>(a, real(x).k, cb, w, lane, c0 + cq); };
    Pos s1 = next_stage(sc, s0), s2 = next_stage(sc, s1), s3 = next_stage(sc, s2);
    Pos s4 = next_stage(sc, s3), s5 = next_stage(sc, s4);

    store_stage<NKT>(xsb, tid, load_stage<NKT, VEC>(a, gidx_of(s0), aidx_of(s0), tid));
    StageRegs<NKT> R0 = load_stage<NKT, VEC>(a, gidx_of(s1), aidx_of(s1), tid);
    StageRegs<NKT> R1 = load_stage<NKT, VEC>(a, gidx_of(s2), aidx_of(s2), tid);
    int G0 = gidx_of(s3), G1 = gidx_of(s4);
    WFrag<NKT> B0 = wk(s0), B1 = wk(s1);
    // drain the prologue's loads once per tile, so that the wait counts in
    // the loop follow from the loop's own loads
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    // one iteration: parity X selects the register sets.  The products of
    // s_i are added to the accumulators one iteration later, so the wave
    // never waits for its own matrix-core results.
    auto step = [&](StageRegs<NKT>& R, int& G, WFrag<NKT>& B, StageOut& Onew, const StageOut& Oprev,
                    float* xs_cur, float* xs_nxt) {
      // s_i is past the last stage (no live pairs) only in the second half
      // of the final pair
      Onew = stage_mfma<NKT>(xs_cur, B, min(s0.n, SROWS), T, n16, q);
      stage_scatter(Oprev, acc, cq);
      // rows of s_{i+1} -> the other buffer
      store_stage<NKT>(xs_nxt, tid, R);
      // rows of s_{i+3} (index loaded two iterations ago), index of s_{i+5}
      R = load_stage<NKT, VEC>(a, G, aidx_of(s3), tid);
      G = gidx_of(s5);
      // weights of s_{i+2} into the set just used, unless that set already
      // holds them (s_{i+2} continues s_i's offset: a full 128-row tile has
      // four stages per offset).  The branch tightens the compiler's wait
      // counts; fewer weight loads still win (input gradient 2.35 -> 2.26 ms)
      if (s2.k != s0.k) B = wk(s2);
    };
    auto shift = [&]() {
      s0 = s1;
      s1 = s2;
      s2 = s3;
      s3 = s4;
      s4 = s5;
      s5 = next_stage(sc, s5);
    };
    float* const xa = xsb;
    float* const xb = xsb + SROWS * XLD;
    // stages in pairs; the only exit is after the second of a pair, behind
    // its barrier (every path through the loop issues the same loads)
    StageOut O0, O1;
    O1.c0 = v4f{0.f, 0.f, 0.f, 0.f};
    O1.c1 = O1.c0;
    O1.i0 = O1.i1 = T;
    while (true) {
      step(R0, G0, B0, O0, O1, xa, xb);
      __syncthreads();
      shift();
      step(R1, G1, B1, O1, O0, xb, xa);
      __syncthreads();
      shift();
      if (s0.k >= a.K) break;
    }
    stage_scatter(O1, acc, cq);
  }
  __syncthreads();
  // epilogue: dst[row] = act(acc + add)
  const int ncols = min(CB, a.Nc - c0);
  for (int i = tid; i < T * (CB / 4); i += NT) {
    const int r = i / (CB / 4), cc = (i - r * (CB / 4)) * 4;
    const int64_t grow = row0 + r;
    if (cc >= ncols || grow >= a.nrows) continue;
    float4 v = *reinterpret_cast<const float4*>(&acc[r * ACC_LD + cc]);
    float e[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (a.add && cc + u < ncols) e[u] += a.add[c0 + cc + u];
      if (a.relu) e[u] = e[u] > 0.f ? e[u] : 0.f;
    }
    const int64_t drow = a.wmap ? (int64_t)a.wmap[grow] : grow;
    float* dp = a.dst + drow * a.Nc + c0 + cc;
    if (a.dvec_ok && cc + 3 < ncols) {
      *reinterpret_cast<float4*>(dp) = make_float4(e[0], e[1], e[2], e[3]);
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (cc + u < ncols) dp[u] = e[u];
    }
  }
}

typedef void (*GatherFn)(GatherArgs);

// Tile rows (TM * 64) and work-groups per CU: the accumulators and the two
// stage buffers must fit the 160 KB of LDS.  Reductions over up to 160
// channels use 128-row tiles, three work-groups per CU up to 64 channels and
// two past that (several work-groups per CU hide the gather latency); longer
// reductions use 256-row tiles, one work-group per CU.
template <int NKT>
constexpr int gather_tm() {
  return NKT > 10 ? 4 : 2;
}

template <int NKT>
GatherFn pick_gather(bool vec) {
  constexpr int TM = gather_tm<NKT>(), MINB = NKT > 10 ? 1 : (NKT > 4 ? 2 : 3);
  return vec ? gather_mfma_kernel<NKT, true, TM, MINB> : gather_mfma_kernel<NKT, false, TM, MINB>;
}

GatherFn gather_fn(int nkt, bool vec) {
  switch (nkt) {
    case 1: return pick_gather<1>(vec);
    case 2: return pick_gather<2>(vec);
    case 3: return pick_gather<3>(vec);
    case 4: return pick_gather<4>(vec);
    case 5: return pick_gather<5>(vec);
    case 6: return pick_gather<6>(vec);
    case 7: return pick_gather<7>(vec);
    case 8: return pick_gather<8>(vec);
    case 9: return pick_gather<9>(vec);
    case 10: return pick_gather<10>(vec);
    case 11: return pick_gather<11>(vec);
    case 12: return pick_gather<12>(vec);
    case 13: return pick_gather<13>(vec);
    case 14: return pick_gather<14>(vec);
    case 15: return pick_gather<15>(vec);
    default: return pick_gather<16>(vec);
  }
}

scn_status launch_gather(GatherArgs a, hipStream_t st) {
  if (a.nrows <= 0) return SCN_OK;
  a.vec_ok = ((a.Rk & 3) == 0) && ((reinterpret_cast<uintptr_t>(a.src) & 15) == 0);

  a.dvec_ok = ((a.Nc & 3) == 0) && ((reinterpret_cast<uintptr_t>(a.dst) & 15) == 0);
  const int nkt = (int)ceil_div(a.Rk, 16);
  const int TM = nkt > 10 ? gather_tm<11>() : gather_tm<1>();
  const int64_t nwg = ceil_div(a.ntile, TM);
  const unsigned ncb = (unsigned)ceil_div(a.Nc, CB);
  const size_t smem =
      ((size_t)(TM * TILE + 1) * ACC_LD + 2 * (size_t)SROWS * (16 * nkt + 4)) * sizeof(float);
  const bool vec = a.vec_ok;
  GatherFn fn = gather_fn(nkt, vec);
  static bool attr_done[2][17] = {};
  bool& done = attr_done[vec][nkt];
  if (!done) {
    SCN_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem));
    done = true;
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)nwg, ncb), dim3(NT), smem, st, a);
  SCN_LAUNCH_CHECK();
  return SCN_OK;
}

// ---------------------------------------------------------------------------
// Dense-block forward (stride-1 rulebooks)
// ---------------------------------------------------------------------------
// The rulebook sorts the output rows by neighbour mask; cut into blocks of 32
// (DENSE_ROWS) the rows of a block mostly share one mask.  One wave owns a
// block and 64 output columns, with its 32 x 64 accumulators in registers:
// for each offset k of the union of the block's masks it gathers the block's
// 32 input rows (a row without offset k contributes zero) and multiplies them
// by W_k, 64 input channels at a time.  Lane (n16, q) gathers block rows n16
// and 16 + n16; a row's input at offset k is entry popcount(mask & (2^k - 1))
// of its output-major neighbour list.  There is no scatter: the rows of a
// block are distinct outputs, and the epilogue writes each once.  Rows hold
// x - g_in, so y = g_pre + sum over active offsets of (x - g_in) W_k.  The
// next (offset, channel chunk)'s rows are loaded while the current one is
// multiplied.
struct DenseArgs {
  const float* x;          // [a_in][Cin]
  const float* g_in;       // [Cin]
  const float* Wp;         // packed like GatherArgs::Wp (fragment order, transposed W)
  const float* add;        // [Cout] g_pre
  const int32_t* nb;       // rulebook fnb
  const uint32_t* nb_off;  // rulebook fnb_off
  const int32_t* fperm;    // rulebook fperm
  const uint32_t* fmask;   // rulebook fmask
  float* y;                // [a_out][Cout]
  int64_t a_out, nblk;
  int K, Cin, Cout, NcP, relu, dvec_ok;
};

// One block row as the lane sees it: its mask and the start of its list.
struct DRow {
  uint32_t m, off;
};

// The rows of one (offset, 64-channel chunk) item: lane (n16, q) holds
// channels 64ch + 16t + 4q .. +3 of block rows n16 and 16 + n16.
template <int TC>
struct DRows {
  float4 v[2][TC];
  int r0, r1;
};

__device__ inline int dense_src(const DenseArgs& a, const DRow& w, int k) {
  // the list entry is read unconditionally (the list has a spare entry)
  const int r = a.nb[w.off + __popc(w.m & ((1u << k) - 1u))];
  return (w.m >> k) & 1u ? r : -1;
}

template <int NKT, bool VEC>
__device__ inline DRows<(NKT < 4 ? NKT : 4)> dense_rows(const DenseArgs& a, const DRow& w0,
                                                        const DRow& w1, int k, int ch, int q) {
  constexpr int TC = NKT < 4 ? NKT : 4;
  DRows<TC> R;
  R.r0 = dense_src(a, w0, k);
  R.r1 = dense_src(a, w1, k);
  const float* p0 = a.x + (int64_t)(R.r0 >= 0 ? R.r0 : 0) * a.Cin;
  const float* p1 = a.x + (int64_t)(R.r1 >= 0 ? R.r1 : 0) * a.Cin;
#pragma unroll
  for (int t = 0; t < TC; ++t) {
    const int c = 64 * ch + 16 * t + 4 * q;
    if (VEC) {
      // channels past Cin read channel 0; their weights are zero
      const int cc = c < a.Cin ? c : 0;
      R.v[0][t] = *reinterpret_cast<const float4*>(p0 + cc);
      R.v[1][t] = *reinterpret_cast<const float4*>(p1 + cc);
    } else {
      float e0[4], e1[4];
#pragma unroll
      for (int z = 0; z < 4; ++z) {
        const int cz = c + z < a.Cin ? c + z : 0;
        e0[z] = p0[cz];
        e1[z] = p1[cz];
      }
      R.v[0][t] = make_float4(e0[0], e0[1], e0[2], e0[3]);
      R.v[1][t] = make_float4(e1[0], e1[1], e1[2], e1[3]);
    }
  }
  return R;
}

// rows of an item whose input rows are already known
template <int NKT, bool VEC>
__device__ inline DRows<(NKT < 4 ? NKT : 4)> dense_rows_i(const DenseArgs& a, int r0, int r1,
                                                          int ch, int q) {
  constexpr int TC = NKT < 4 ? NKT : 4;
  DRows<TC> R;
  R.r0 = r0;
  R.r1 = r1;
  const float* p0 = a.x + (int64_t)(r0 >= 0 ? r0 : 0) * a.Cin;
  const float* p1 = a.x + (int64_t)(r1 >= 0 ? r1 : 0) * a.Cin;
#pragma unroll
  for (int t = 0; t < TC; ++t) {
    const int c = 64 * ch + 16 * t + 4 * q;
    if (VEC) {
      const int cc = c < a.Cin ? c : 0;
      R.v[0][t] = *reinterpret_cast<const float4*>(p0 + cc);
      R.v[1][t] = *reinterpret_cast<const float4*>(p1 + cc);
    } else {
      float e0[4], e1[4];
#pragma unroll
      for (int z = 0; z < 4; ++z) {
        const int cz = c + z < a.Cin ? c + z : 0;
        e0[z] = p0[cz];
        e1[z] = p1[cz];
      }
      R.v[0][t] = make_float4(e0[0], e0[1], e0[2], e0[3]);
      R.v[1][t] = make_float4(e1[0], e1[1], e1[2], e1[3]);
    }
  }
  return R;
}

template <int NKT, bool VEC>
__global__ void __launch_bounds__(NT) dense_fwd_kernel(DenseArgs a) {
  constexpr int TC = NKT < 4 ? NKT : 4;        // 16-channel steps per chunk
  constexpr int NCH = (NKT + 3) / 4;           // 64-channel chunks
  __shared__ float gsh[16 * NKT];  // g_in, zero past Cin (those weights are zero)
  for (int c = threadIdx.x; c < 16 * NKT; c += NT) gsh[c] = c < a.Cin ? a.g_in[c] : 0.f;
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int64_t b = (int64_t)blockIdx.x * (NT / 64) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (b >= a.nblk) return;
  const int cb = blockIdx.y;
  // Two lane layouts.  MFMA layout: lane (n16, q) = n16 + 16q holds row n16
  // (and 16 + n16), channels 4q .. 4q + 3 of each 16; the operand fixes it.
  // Load layout: lane (rl, cq) = 4rl + cq loads row rl (and 16 + rl),
  // channels 4cq .. 4cq + 3, so four adjacent lanes read one row's 64
  // contiguous bytes (in the MFMA layout four adjacent lanes read four
  // rows, and the L1 serves each 16-byte piece on its own).  The rows are
  // gathered in the load layout and moved to the MFMA layout by ds_bpermute.
  const int n16 = lane & 15, q = lane >> 4;
  const int rl = lane >> 2, cq = lane & 3;
  const int from = (n16 * 4 + q) * 4;  // bpermute address: MFMA lane <- load lane 4 n16 + q
  const int ncb = a.NcP >> 6;
  const int64_t pos0 = b * DENSE_ROWS + n16, pos1 = pos0 + 16;      // MFMA layout
  const int64_t lpos0 = b * DENSE_ROWS + rl, lpos1 = lpos0 + 16;    // load layout
  const int o0 = pos0 < a.a_out ? a.fperm[pos0] : 0, o1 = pos1 < a.a_out ? a.fperm[pos1] : 0;
  const int lo0 = lpos0 < a.a_out ? a.fperm[lpos0] : 0, lo1 = lpos1 < a.a_out ? a.fperm[lpos1] : 0;
  DRow w0, w1;
  w0.m = lpos0 < a.a_out ? a.fmask[lpos0] : 0u;
  w1.m = lpos1 < a.a_out ? a.fmask[lpos1] : 0u;
  w0.off = a.nb_off[lo0];
  w1.off = a.nb_off[lo1];
  uint32_t u = w0.m | w1.m;
#pragma unroll
  for (int d = 4; d < 64; d <<= 1) u |= (uint32_t)__shfl_xor((int)u, d, 64);
  const uint32_t U = (uint32_t)__builtin_amdgcn_readfirstlane((int)u);
  v4f acc[2][4];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int g = 0; g < 4; ++g) acc[r][g] = v4f{0.f, 0.f, 0.f, 0.f};
  if (U) {
    // item = (offset k, channel chunk ch), in order; `rest` holds the offsets
    // after k; past the last item an item stays where it is (its loads are in
    // bounds and unused)
    struct Item {
      int k, ch;
      uint32_t rest;
    };
    auto advance = [&](Item& t) {
      if (t.ch + 1 < NCH) {
        ++t.ch;
      } else if (t.rest) {
        t.k = __builtin_ctz(t.rest);
        t.rest &= t.rest - 1;
        t.ch = 0;
      }
    };
    Item c{__builtin_ctz(U), 0, U & (U - 1)};
    Item n = c;
    advance(n);
    Item nn = n;
    advance(nn);
    const int nit = __builtin_popcount(U) * NCH;
    int n0 = dense_src(a, w0, n.k), n1 = dense_src(a, w1, n.k);
    DRows<TC> cur = dense_rows_i<NKT, VEC>(a, dense_src(a, w0, c.k), dense_src(a, w1, c.k), 0, cq);
    DRows<TC> nxt;
    int nn0 = 0, nn1 = 0;
    for (int it = 0; it < nit; ++it) {
      const int ch = c.ch;
      const float* wp = a.Wp + (((int64_t)c.k * ncb + cb) * 4) * (NKT * 256) + lane * 4;
      auto wload = [&](int t, float4 (&A)[4]) {
        const int tg = 4 * ch + t < NKT ? 4 * ch + t : NKT - 1;  // past NKT: never used
#pragma unroll
        for (int g = 0; g < 4; ++g)
          A[g] = *reinterpret_cast<const float4*>(wp + (int64_t)g * (NKT * 256) + tg * 256);
      };
      // the next item's rows and the indices after it: issued after this
      // item's last weight load, so the waits for the weights leave them in
      // flight
      auto prefetch = [&]() {
        nxt = dense_rows_i<NKT, VEC>(a, n0, n1, n.ch, cq);
        nn0 = dense_src(a, w0, nn.k);
        nn1 = dense_src(a, w1, nn.k);
      };
      auto mult = [&](int t, const float4 (&A)[4]) {
        const int tg = 4 * ch + t;
        // x - g_in, zero for an absent row, in the load layout; then to the
        // MFMA layout
        const float4 gq = *reinterpret_cast<const float4*>(&gsh[16 * tg + 4 * cq]);
        const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
        float4 d0 = cur.v[0][t], d1 = cur.v[1][t];
        d0.x -= gq.x; d0.y -= gq.y; d0.z -= gq.z; d0.w -= gq.w;
        d1.x -= gq.x; d1.y -= gq.y; d1.z -= gq.z; d1.w -= gq.w;
        const float4 L0 = cur.r0 >= 0 ? d0 : z, L1 = cur.r1 >= 0 ? d1 : z;
        auto perm = [&](float v) {
          return __int_as_float(__builtin_amdgcn_ds_bpermute(from, __float_as_int(v)));
        };
        const float4 B0 = make_float4(perm(L0.x), perm(L0.y), perm(L0.z), perm(L0.w));
        const float4 B1 = make_float4(perm(L1.x), perm(L1.y), perm(L1.z), perm(L1.w));
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          acc[0][g] = mfma4(A[g].x, B0.x, acc[0][g]);
          acc[1][g] = mfma4(A[g].x, B1.x, acc[1][g]);
          acc[0][g] = mfma4(A[g].y, B0.y, acc[0][g]);
          acc[1][g] = mfma4(A[g].y, B1.y, acc[1][g]);
          acc[0][g] = mfma4(A[g].z, B0.z, acc[0][g]);
          acc[1][g] = mfma4(A[g].z, B1.z, acc[1][g]);
          acc[0][g] = mfma4(A[g].w, B0.w, acc[0][g]);
          acc[1][g] = mfma4(A[g].w, B1.w, acc[1][g]);
        }
      };
      // weights two 16-channel steps ahead of their products (two register
      // sets, alternating)
      float4 A0[4], A1[4];
      wload(0, A0);
      if (TC > 1) wload(1, A1);
      if (TC <= 2) prefetch();
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int t = 0; t < TC; ++t) {
        if (NCH > 1 && 4 * ch + t >= NKT) {
          // a last chunk shorter than the step that issues the prefetch
          // (t = TC - 3) issues it here, so the next item's rows are loaded
          if (t <= TC - 3) prefetch();
          break;
        }
        // step t's products, then step t + 2's weights into the set just read
        if (t & 1) mult(t, A1); else mult(t, A0);
        if (t + 2 < TC) {
          if (t & 1) wload(t + 2, A1); else wload(t + 2, A0);
          if (t + 2 == TC - 1) prefetch();
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      c = n;
      n = nn;
      advance(nn);
      n0 = nn0;
      n1 = nn1;
      cur = nxt;
    }
  }
  // epilogue: rows n16 and 16 + n16 of the block, columns 64cb + 16g + 4q .. +3
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int64_t pos = r ? pos1 : pos0;
    if (pos >= a.a_out) continue;
    float* dp = a.y + (int64_t)(r ? o1 : o0) * a.Cout;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int col = 64 * cb + 16 * g + 4 * q;
      if (col >= a.Cout) continue;
      float e[4] = {acc[r][g][0], acc[r][g][1], acc[r][g][2], acc[r][g][3]};
#pragma unroll
      for (int u2 = 0; u2 < 4; ++u2) {
        if (col + u2 < a.Cout) e[u2] += a.add[col + u2];
        if (a.relu) e[u2] = e[u2] > 0.f ? e[u2] : 0.f;
      }
      if (a.dvec_ok && col + 3 < a.Cout) {
        // a streaming store: y is read only by later calls (kernel 2.669 ->
        // 2.653 ms on the 1M-site layer)
        __builtin_nontemporal_store(v4f{e[0], e[1], e[2], e[3]}, reinterpret_cast<v4f*>(dp + col));
      } else {
#pragma unroll
        for (int u2 = 0; u2 < 4; ++u2)
          if (col + u2 < a.Cout) dp[col + u2] = e[u2];
      }
    }
  }
}

typedef void (*DenseFn)(DenseArgs);

template <int NKT>
DenseFn pick_dense(bool vec) {
  return vec ? dense_fwd_kernel<NKT, true> : dense_fwd_kernel<NKT, false>;
}

DenseFn dense_fn(int nkt, bool vec) {
  switch (nkt) {
    case 1: return pick_dense<1>(vec);
    case 2: return pick_dense<2>(vec);
    case 3: return pick_dense<3>(vec);
    case 4: return pick_dense<4>(vec);
    case 5: return pick_dense<5>(vec);
    case 6: return pick_dense<6>(vec);
    case 7: return pick_dense<7>(vec);
    case 8: return pick_dense<8>(vec);
    case 9: return pick_dense<9>(vec);
    case 10: return pick_dense<10>(vec);
    case 11: return pick_dense<11>(vec);
    case 12: return pick_dense<12>(vec);
    case 13: return pick_dense<13>(vec);
    case 14: return pick_dense<14>(vec);
    case 15: return pick_dense<15>(vec);
    default: return pick_dense<16>(vec);
  }
}

scn_status launch_dense(DenseArgs a, hipStream_t st) {
  if (a.a_out <= 0 || a.nblk <= 0) return SCN_OK;
  const bool vec = ((a.Cin & 3) == 0) && ((reinterpret_cast<uintptr_t>(a.x) & 15) == 0) &&
                   ((reinterpret_cast<uintptr_t>(a.g_in) & 15) == 0);
  a.dvec_ok = ((a.Cout & 3) == 0) && ((reinterpret_cast<uintptr_t>(a.y) & 15) == 0);
  const int nkt = (int)ceil_div(a.Cin, 16);
  const int64_t nwg = ceil_div(a.nblk, NT / 64);
  hipLaunchKernelGGL(dense_fn(nkt, vec), dim3((unsigned)nwg, (unsigned)(a.NcP / 64)), dim3(NT), 0,
                     st, a);
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

// Four channels per thread (C % 4 == 0, 16-byte aligned rows): a block reads
// RB_ROWS rows as float4, `per` rows at a time, and combines the rows in a
// fixed order.
__global__ void __launch_bounds__(NT) colsum_vec_kernel(const float4* __restrict__ dy,
                                                        const float4* __restrict__ y, int relu,
                                                        int64_t rows, int nc4,
                                                        float4* __restrict__ dyb,
                                                        float4* __restrict__ partS) {
  __shared__ float4 red[NT];
  const int per = NT / nc4;
  const int rl = threadIdx.x / nc4, c4 = threadIdx.x - rl * nc4;
  const int64_t r0 = (int64_t)blockIdx.x * RB_ROWS;
  const int64_t r1 = min<int64_t>(r0 + RB_ROWS, rows);
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  if (rl < per) {
    int64_t r = r0 + rl;
    // four rows in flight per thread
    for (; r + 3 * per < r1; r += 4 * per) {
      float4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = dy[(r + u * per) * nc4 + c4];
      if (relu) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float4 m = y[(r + u * per) * nc4 + c4];
          v[u].x = m.x > 0.f ? v[u].x : 0.f;
          v[u].y = m.y > 0.f ? v[u].y : 0.f;
          v[u].z = m.z > 0.f ? v[u].z : 0.f;
          v[u].w = m.w > 0.f ? v[u].w : 0.f;
          dyb[(r + u * per) * nc4 + c4] = v[u];
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        s.x += v[u].x;
        s.y += v[u].y;
        s.z += v[u].z;
        s.w += v[u].w;
      }
    }
    for (; r < r1; r += per) {
      float4 v = dy[r * nc4 + c4];
      if (relu) {
        const float4 m = y[r * nc4 + c4];
        v.x = m.x > 0.f ? v.x : 0.f;
        v.y = m.y > 0.f ? v.y : 0.f;
        v.z = m.z > 0.f ? v.z : 0.f;
        v.w = m.w > 0.f ? v.w : 0.f;
        dyb[r * nc4 + c4] = v;
      }
      s.x += v.x;
      s.y += v.y;
      s.z += v.z;
      s.w += v.w;
    }
  }
  red[threadIdx.x] = s;
  __syncthreads();
  if (rl == 0) {
    for (int i = 1; i < per; ++i) {
      const float4 t = red[i * nc4 + c4];
      s.x += t.x;
      s.y += t.y;
      s.z += t.z;
      s.w += t.w;
    }
    partS[(int64_t)blockIdx.x * nc4 + c4] = s;
  }
}

// S, dḡ, dbias; u0 = S + dḡ.  One block per column: each thread sums a
// strided share of the partials, then a fixed-shape tree.
__global__ void __launch_bounds__(NT) finish_vec_kernel(const float* __restrict__ partS,
                                                        int64_t nblk, int C,
                                                        const float* __restrict__ g_out,
                                                        const float* __restrict__ dg_out, int relu,
                                                        float* __restrict__ S,
                                                        float* __restrict__ u0,
                                                        float* __restrict__ dbias) {
  __shared__ float red[NT];
  const int c = blockIdx.x;
  float s = 0.f;
  for (int64_t b = threadIdx.x; b < nblk; b += NT) s += partS[b * C + c];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int h = NT / 2; h > 0; h >>= 1) {
    if (threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float t = red[0];
    float dg = dg_out ? dg_out[c] : 0.f;
    if (relu && dg_out) dg = g_out[c] > 0.f ? dg : 0.f;
    S[c] = t;
    u0[c] = t + dg;
    if (dbias) dbias[c] = t + dg;
  }
}

// Weight gradient partials.  A work-group accumulates one 64x64 block of
// dW_k = sum_pairs (x[r] - g_in)^T dy[o] over a fixed chunk of list k, 64 pairs
// per stage.  The stage is stored transposed in LDS ([channel][pair]) so that
// MFMA fragments along the pair axis are single ds_read_b128s.  Thread
// (channel c = tid % 64, pair quad group w = tid / 64) loads channel c of 16
// pairs: every wave-wide load reads 64 consecutive channels of one row (two
// cache lines), and each 4 pairs of one channel leave as one ds_write_b128.
// Pair indices are staged through LDS two stages ahead, rows one stage ahead.
constexpr int DW_SC = 64;          // pairs per stage
constexpr int DW_LD = DW_SC + 4;   // pitch of a channel row (floats)
// Pair quad p of channel row r sits at quad p ^ (r / 16) of the row: with the
// 17-quad pitch this keeps every 16-lane group of both the transposed stores
// and the fragment reads on 16 distinct bank groups.

struct DwArgs {
  const float* x;        // [a_in][Cin]
  const float* dyb;      // [a_out][Cout]
  const float* g_in;     // [Cin]
  const int32_t* in_rows;
  const int32_t* out_rows;
  const int64_t* off;    // [K+1]
  int K;
  int Cin, Cout;
  int nco;               // 64-column blocks of Cout
  int nblk;              // (Cin blocks) * nco
  int64_t chp;           // pairs per chunk
  int64_t maxc;          // chunks per offset (slot count)
  float* part;           // [K][maxc][Cin][Cout]
  float* partT;          // [K][maxc][Cout]
};

// channel c of pairs 4*(w + 4v) + u, v < 4, u < 4 of a stage
struct DwRows {
  float x[16], d[16];
};

__device__ inline void dw_rows(const DwArgs& a, const int* ix, const int* io, int cx, int cd,
                               int w, DwRows& R) {
#pragma unroll
  for (int v = 0; v < 4; ++v)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int pr = 4 * (w + 4 * v) + u;
      R.x[4 * v + u] = a.x[(int64_t)ix[pr] * a.Cin + cx];
      R.d[4 * v + u] = a.dyb[(int64_t)io[pr] * a.Cout + cd];
    }
}

// V4 (Cin and Cout multiples of 4, 16-byte aligned rows): thread (pair quad
// pq = tid / 16, channel quad cq = tid % 16) loads channels 4cq .. 4cq+3 of
// pairs 4pq .. 4pq+3 of each operand as float4 (a wave reads four whole
// 256-byte row segments per load) and transposes the 4x4 blocks in registers.
struct DwRows4 {
  float4 x[4], d[4];
};

__device__ inline void dw_rows4(const DwArgs& a, const int* ix, const int* io, int cx4, int cd4,
                                int pq, DwRows4& R) {
  const float4* x4 = reinterpret_cast<const float4*>(a.x);
  const float4* d4 = reinterpret_cast<const float4*>(a.dyb);
  const int nx4 = a.Cin >> 2, nd4 = a.Cout >> 2;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    R.x[u] = x4[(int64_t)ix[4 * pq + u] * nx4 + cx4];
    R.d[u] = d4[(int64_t)io[4 * pq + u] * nd4 + cd4];
  }
}

template <bool V4>
__global__ void __launch_bounds__(NT) dw_partial_kernel(DwArgs a) {
  __shared__ float xsT[64 * DW_LD];  // [ci][pair], x - g_in
  __shared__ float dsT[64 * DW_LD];  // [co][pair]
  __shared__ int idx[2][2][DW_SC];   // [buffer][input row, output row][pair]
  // flattened (chunk, offset, block) work item, blocks then offsets fastest,
  // contiguous per XCD
  const int64_t item = xcd_remap(blockIdx.x, gridDim.x);
  const int blk = (int)(item % a.nblk);
  const int64_t ck = item / a.nblk;
  const int k = (int)(ck % a.K);
  const int64_t c = ck / a.K;
  const int64_t lb = a.off[k], le = a.off[k + 1];
  const int64_t p_begin = lb + c * a.chp;
  if (p_begin >= le) return;
  const int64_t p_end = min(le, p_begin + a.chp);
  const int ci0 = (blk / a.nco) * 64, co0 = (blk % a.nco) * 64;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n16 = lane & 15, q = lane >> 4;
  // this thread's channel (V4: channel quad) of each operand, clamped into
  // the layer; out-of-layer channels are zeroed on store
  const int ch = V4 ? 4 * (tid & 15) : lane;
  const bool xin = ci0 + ch < a.Cin, din = co0 + ch < a.Cout;
  const int cx = xin ? ci0 + ch : 0, cd = din ? co0 + ch : 0;
  const float gsub = (!V4 && xin) ? a.g_in[cx] : 0.f;
  const float4 gsub4 = (V4 && xin) ? *reinterpret_cast<const float4*>(a.g_in + cx)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
  const int pq = tid >> 4;  // V4: pair quad

  // index loaders: threads 0..63 input rows, 64..127 output rows of one stage
  auto load_index = [&](int64_t p0) -> int {
    const int64_t pp = min(p0 + (tid & 63), p_end - 1);
    return tid < 64 ? a.in_rows[pp] : a.out_rows[pp];
  };
  if (tid < 128) {
    idx[0][tid >> 6][tid & 63] = load_index(p_begin);
    idx[1][tid >> 6][tid & 63] = load_index(p_begin + DW_SC);
  }
  __syncthreads();
  DwRows R;
  DwRows4 R4;
  if (V4)
    dw_rows4(a, idx[0][0], idx[0][1], cx >> 2, cd >> 2, pq, R4);
  else
    dw_rows(a, idx[0][0], idx[0][1], cx, cd, w, R);

  v4f acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = (v4f){0.f, 0.f, 0.f, 0.f};
  float tsum = 0.f;
  const int tcol = 16 * w + n16;

  int buf = 0;
  for (int64_t p0 = p_begin; p0 < p_end; p0 += DW_SC) {
    const int n = (int)min<int64_t>(DW_SC, p_end - p0);
    // stage rows -> LDS, transposed; pairs past the chunk and channels past
    // the layer are zero; x is shifted by the ground state
    if (V4) {
      const int pb = 4 * pq;
      float xe[4][4], de[4][4];  // [channel][pair]
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bool lx = pb + u < n && xin, ld = pb + u < n && din;
        xe[0][u] = lx ? R4.x[u].x - gsub4.x : 0.f;
        xe[1][u] = lx ? R4.x[u].y - gsub4.y : 0.f;
        xe[2][u] = lx ? R4.x[u].z - gsub4.z : 0.f;
        xe[3][u] = lx ? R4.x[u].w - gsub4.w : 0.f;
        de[0][u] = ld ? R4.d[u].x : 0.f;
        de[1][u] = ld ? R4.d[u].y : 0.f;
        de[2][u] = ld ? R4.d[u].z : 0.f;
        de[3][u] = ld ? R4.d[u].w : 0.f;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int sq = 4 * (pq ^ ((ch + e) >> 4));  // swizzled pair quad
        *reinterpret_cast<float4*>(&xsT[(ch + e) * DW_LD + sq]) =
            make_float4(xe[e][0], xe[e][1], xe[e][2], xe[e][3]);
        *reinterpret_cast<float4*>(&dsT[(ch + e) * DW_LD + sq]) =
            make_float4(de[e][0], de[e][1], de[e][2], de[e][3]);
      }
    } else {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int pb = 4 * (w + 4 * v);
        float xe[4], de[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const bool live = pb + u < n;
          xe[u] = (live && xin) ? R.x[4 * v + u] - gsub : 0.f;
          de[u] = (live && din) ? R.d[4 * v + u] : 0.f;
        }
        const int sq = 4 * ((pb >> 2) ^ (ch >> 4));  // swizzled pair quad
        *reinterpret_cast<float4*>(&xsT[ch * DW_LD + sq]) = make_float4(xe[0], xe[1], xe[2], xe[3]);
        *reinterpret_cast<float4*>(&dsT[ch * DW_LD + sq]) = make_float4(de[0], de[1], de[2], de[3]);
      }
    }
    int nidx = 0;
    if (tid < 128) nidx = load_index(p0 + 2 * DW_SC);  // stage s+2 indices in flight
    __syncthreads();
    // stage s+1 rows while the matrix cores work on stage s
    if (V4)
      dw_rows4(a, idx[buf ^ 1][0], idx[buf ^ 1][1], cx >> 2, cd >> 2, pq, R4);
    else
      dw_rows(a, idx[buf ^ 1][0], idx[buf ^ 1][1], cx, cd, w, R);
    // keep those loads ahead of the matrix-core section (left to itself the
    // scheduler sinks them below it to reuse their registers, and the next
    // stage then waits for the full memory latency)
    __builtin_amdgcn_sched_barrier(0);
    // A(m = ci, kk = pair) = xsT[16w + m][pair];  B(kk = pair, n = co) = dsT[16j + n][pair]
    const float* ar = xsT + (16 * w + n16) * DW_LD + 4 * (q ^ w);
#pragma unroll
    for (int t = 0; t < DW_SC / 16; ++t) {
      const float4 av = *reinterpret_cast<const float4*>(ar + 16 * t);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 bv =
            *reinterpret_cast<const float4*>(dsT + (16 * j + n16) * DW_LD + 4 * (q ^ j) + 16 * t);
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
        const float4 v = *reinterpret_cast<const float4*>(tr + 4 * (i ^ w));
        tsum += ((v.x + v.y) + v.z) + v.w;
      }
    }
    if (tid < 128) idx[buf][tid >> 6][tid & 63] = nidx;  // stage s's slot is free
    buf ^= 1;
    __syncthreads();
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

// dW[k][ci][co] = sum_c part + g_in[ci] * u0[co];  T[k][co] = sum_c partT.
// A block covers RED_E consecutive elements; thread group g (of RED_G) sums
// the chunks c = g (mod RED_G) in ascending order, and the group sums are
// added in group order (a fixed order, so the result is deterministic).
constexpr int RED_E = 32, RED_G = 8;
__global__ void __launch_bounds__(RED_E * RED_G) dw_reduce_kernel(
    const float* __restrict__ part, const float* __restrict__ partT,
    const int64_t* __restrict__ off, int K, int Cin, int Cout, int64_t chp, int64_t maxc,
    const float* __restrict__ g_in, const float* __restrict__ u0, float* __restrict__ dW,
    float* __restrict__ T) {
  __shared__ float red[2][RED_G][RED_E];
  const int le = threadIdx.x % RED_E, g = threadIdx.x / RED_E;
  const int64_t i = (int64_t)blockIdx.x * RED_E + le;
  const int64_t per = (int64_t)Cin * Cout;
  float s = 0.f, t = 0.f;
  if (i < (int64_t)K * per) {
    const int k = (int)(i / per);
    const int64_t e = i - k * per;
    const int64_t nch = ceil_div(off[k + 1] - off[k], chp);
    const float* p = part + (int64_t)k * maxc * per + e;
#pragma unroll 4
    for (int64_t c = g; c < nch; c += RED_G) s += p[c * per];
  }
  if (i < (int64_t)K * Cout) {
    const int k = (int)(i / Cout), co = (int)(i % Cout);
    const int64_t nch = ceil_div(off[k + 1] - off[k], chp);
    for (int64_t c = g; c < nch; c += RED_G) t += partT[((int64_t)k * maxc + c) * Cout + co];
  }
  red[0][g][le] = s;
  red[1][g][le] = t;
  __syncthreads();
  if (g != 0) return;
  s = red[0][0][le];
  t = red[1][0][le];
#pragma unroll
  for (int h = 1; h < RED_G; ++h) {
    s += red[0][h][le];
    t += red[1][h][le];
  }
  if (i < (int64_t)K * per && dW) {
    const int64_t e = i % per;
    const int ci = (int)(e / Cout), co = (int)(e - (int64_t)ci * Cout);
    dW[i] = s + g_in[ci] * u0[co];
  }
  if (i < (int64_t)K * Cout) T[i] = t;
}

// dg_in[ci] = sum_k sum_co W[k][ci][co] * (u0[co] - T[k][co]); one block per ci,
// fixed-order tree over the block.
__global__ void __launch_bounds__(256) dgin_kernel(const float* __restrict__ W,
                                                   const float* __restrict__ u0,
                                                   const float* __restrict__ T, int K, int Cin,
                                                   int Cout, float* __restrict__ dg_in) {
  __shared__ float red[256];
  const int ci = blockIdx.x;
  const int64_t n = (int64_t)K * Cout;
  float s = 0.f;
  for (int64_t i = threadIdx.x; i < n; i += 256) {
    const int k = (int)(i / Cout), co = (int)(i - (int64_t)k * Cout);
    s = fmaf(W[((int64_t)k * Cin + ci) * Cout + co], u0[co] - T[i], s);
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) dg_in[ci] = red[0];
}

// Work-groups of the weight-gradient kernel that run at once on the current
// device (per-CU occupancy times CUs), cached per device.
int dw_slots() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev]) return cached[dev];
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per_cu, reinterpret_cast<const void*>(dw_partial_kernel<true>), NT, 0) != hipSuccess ||
      per_cu < 1)
    per_cu = 1;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus < 1)
    cus = 1;
  (void)hipGetLastError();
  cached[dev] = per_cu * cus;
  return cached[dev];
}

// The (offset, chunk, column block) work items fill DW_ROUNDS whole rounds of
// the concurrent work-groups: each offset's list is cut into at most
// DW_ROUNDS * slots / (K * blocks) chunks, so the last round is nearly full
// instead of holding a few stragglers that would take a round's time alone.
constexpr int DW_ROUNDS = 4;

struct BwdLayout {
  int64_t chp, maxc, nblk;
  size_t o_dyb, o_part, o_partT, o_partS, o_S, o_u0, o_T, o_wp, o_gz, total;
};

BwdLayout bwd_layout(const scn_rulebook* rb, int Cin, int Cout, uint32_t flags) {
  BwdLayout L{};
  int64_t pmax = 0;
  for (int k = 0; k < rb->K; ++k) pmax = std::max(pmax, rb->off_host[k + 1] - rb->off_host[k]);
  const int64_t blocks = ceil_div(Cin, 64) * ceil_div(Cout, 64);
  const int64_t target = std::max<int64_t>(1, DW_ROUNDS * (int64_t)dw_slots() / (rb->K * blocks));
  const int64_t per = ceil_div(std::max<int64_t>(pmax, 1), target);
  L.chp = std::max<int64_t>(DW_SC, ceil_div(per, DW_SC) * DW_SC);
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
  L.o_wp = cur;
  cur += al((size_t)rb->K * ceil_div(Cin, 64) * 64 * ceil_div(Cout, 16) * 16 * 4);
  L.o_gz = cur;
  cur += al((size_t)rb->K * ceil_div(Cin, 64) * 64 * 4);
  L.total = cur;
  return L;
}

}  // namespace
}  // namespace scn

using namespace scn;

// Measurement hook (scn_set_kernel_timer): per host thread, pairs of the
// caller's events recorded on the call's stream around the contraction
// kernels: [0, 1] the forward, [2, 3] the input gradient, [4, 5] the weight
// gradient's partial products.
enum TimedKernel { TK_FWD = 0, TK_DX = 1, TK_DW = 2 };
static thread_local hipEvent_t g_kernel_timer[6] = {};

static scn_status timer_mark(TimedKernel k, int end, hipStream_t st) {
  hipEvent_t e = g_kernel_timer[2 * k + end];
  if (e) SCN_HIP(hipEventRecord(e, st));
  return SCN_OK;
}

// The forward's scratch: gw [K][NcP] and g_pre [NcP] (256-byte aligned),
// then the packed weights [K][NcP][RkP].  Every element is written by the
// forward's first kernels before any is read.
struct FwdScratch {
  int RkP, NcP;
  size_t gw_bytes, total;
};

static FwdScratch fwd_scratch(const scn_rulebook* rb, int Cin, int Cout) {
  FwdScratch f;
  f.RkP = (int)ceil_div(Cin, 16) * 16;
  f.NcP = (int)ceil_div(Cout, 64) * 64;
  f.gw_bytes = ((size_t)(rb->K + 1) * f.NcP * sizeof(float) + 255) & ~size_t(255);
  f.total = f.gw_bytes + (size_t)rb->K * f.NcP * f.RkP * sizeof(float);
  return f;
}

static scn_status fwd_check(const char* who, const scn_rulebook* rb, const float* x,
                            const float* g_in, const float* W, int32_t Cin, int32_t Cout,
                            float* y, float* g_out) {
  if (!rb || !g_in || !W || !g_out || Cin < 1 || Cout < 1 || (rb->a_in > 0 && !x) ||
      (rb->a_out > 0 && !y)) {
    set_error("%s: invalid argument", who);
    return SCN_ERR_INVALID;
  }
  if (Cin > 256) {
    set_error("%s: Cin %d > 256 is not supported", who, Cin);
    return SCN_ERR_UNSUPPORTED;
  }
  return SCN_OK;
}

// Steps 2-3 with the ground state, on a scratch block laid out as FwdScratch.
static scn_status fwd_run(const scn_rulebook* rb, const float* x, const float* g_in,
                          const float* W, const float* bias, int32_t Cin, int32_t Cout,
                          uint32_t flags, float* y, float* g_out, hipStream_t st,
                          const FwdScratch& fs, float* gw) {
  const int relu = (flags & SCN_RELU) ? 1 : 0;
  const int RkP = fs.RkP, NcP = fs.NcP;
  float* const gpre = gw + (size_t)rb->K * NcP;
  float* Wp = reinterpret_cast<float*>(reinterpret_cast<char*>(gw) + fs.gw_bytes);
  hipLaunchKernelGGL(pack_w_kernel, dim3((unsigned)ceil_div((int64_t)rb->K * NcP * RkP, 256)),
                     dim3(256), 0, st, W, rb->K, Cin, Cout, 1, RkP, NcP, Wp);
  SCN_LAUNCH_CHECK();
  hipLaunchKernelGGL(ground_w_kernel, dim3((unsigned)(rb->K * (NcP / 64))), dim3(256), 0, st,
                     g_in, W, rb->K, Cin, Cout, NcP, gw);
  SCN_LAUNCH_CHECK();
  hipLaunchKernelGGL(ground_pre_kernel, dim3((unsigned)ceil_div(Cout, 64)), dim3(64), 0, st, gw,
                     NcP, bias, rb->K, Cout, relu, gpre, g_out);
  SCN_LAUNCH_CHECK();
  if (rb->fnb) {
    DenseArgs d{};
    d.x = x;
    d.g_in = g_in;
    d.Wp = Wp;
    d.add = gpre;
    d.nb = rb->fnb;
    d.nb_off = rb->fnb_off;
    d.fperm = rb->fperm;
    d.fmask = rb->fmask;
    d.y = y;
    d.a_out = rb->a_out;
    d.nblk = rb->n_fblocks;
    d.K = rb->K;
    d.Cin = Cin;
    d.Cout = Cout;
    d.NcP = NcP;
    d.relu = relu;
    scn_status rc;
    if ((rc = timer_mark(TK_FWD, 0, st)) || (rc = launch_dense(d, st))) return rc;
    return timer_mark(TK_FWD, 1, st);
  }
  GatherArgs a{};
  a.src = x;
  a.gidx = rb->in_rows;
  a.aidx = rb->out_rows;
  a.tpos = rb->otile;
  a.ntile = rb->n_otiles;
  a.Wp = Wp;
  a.gwp = gw;
  a.NcP = NcP;
  a.Rk = Cin;
  a.Nc = Cout;
  a.add = gpre;
  a.relu = relu;
  a.dst = y;
  a.wmap = nullptr;
  a.nrows = rb->a_out;
  a.K = rb->K;
  scn_status rc;
  if ((rc = timer_mark(TK_FWD, 0, st)) || (rc = launch_gather(a, st))) return rc;
  return timer_mark(TK_FWD, 1, st);
}

// Scratch of scn_conv_fwd_noalloc: one array per GPU the library runs on,
// held until the process ends.  In host code its name is not a device
// address; the address each device gives it (hipGetSymbolAddress, once per
// device) is what kernels and copies get.
constexpr size_t NOALLOC_SCRATCH_BYTES = size_t(8) << 20;
static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

static std::mutex g_scratch_mutex;
static void* g_scratch_ptr[64] = {};

static scn_status noalloc_scratch(void** out) {
  int dev = 0;
  SCN_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) {
    set_error("scn_conv_fwd_noalloc: device %d out of range", dev);
    return SCN_ERR_HIP;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    SCN_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) {
      set_error("scn_conv_fwd_noalloc: no device address for the scratch array");
      return SCN_ERR_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SCN_OK;
}

extern "C" {

scn_status scn_conv_fwd(const scn_rulebook* rb, const float* x, const float* g_in,
                        const float* W, const float* bias, int32_t Cin, int32_t Cout,
                        uint32_t flags, float* y, float* g_out, hipStream_t st) {
  clear_error();
  if (scn_status rc0 = after_build(rb, st)) return rc0;
  if (scn_status rc0 = fwd_check("scn_conv_fwd", rb, x, g_in, W, Cin, Cout, y, g_out))
    return rc0;
  const FwdScratch fs = fwd_scratch(rb, Cin, Cout);
  float* gw = nullptr;
  const Allocator al = current_allocator();
  scn_status rc = dalloc(reinterpret_cast<void**>(&gw), fs.total, st, al);
  if (rc) return rc;
  struct Free {
    float* p;
    hipStream_t s;
    Allocator al;
    ~Free() { dfree(p, s, al); }
  } free_gw{gw, st, al};
  return fwd_run(rb, x, g_in, W, bias, Cin, Cout, flags, y, g_out, st, fs, gw);
}

size_t scn_conv_fwd_noalloc_max_bytes(void) { return NOALLOC_SCRATCH_BYTES; }

scn_status scn_set_kernel_timer(const hipEvent_t* events) {
  for (int i = 0; i < 6; ++i) g_kernel_timer[i] = events ? events[i] : nullptr;
  return SCN_OK;
}

scn_status scn_conv_fwd_noalloc(const scn_rulebook* rb, const float* x, const float* g_in,
                                const float* W, const float* bias, int32_t Cin, int32_t Cout,
                                uint32_t flags, float* y, float* g_out, hipStream_t st) {
  clear_error();
  if (scn_status rc0 = after_build(rb, st)) return rc0;
  if (scn_status rc0 = fwd_check("scn_conv_fwd_noalloc", rb, x, g_in, W, Cin, Cout, y, g_out))
    return rc0;
  const FwdScratch fs = fwd_scratch(rb, Cin, Cout);
  if (fs.total > NOALLOC_SCRATCH_BYTES) {
    set_error("scn_conv_fwd_noalloc: K=%d Cin=%d Cout=%d needs %zu bytes of scratch, more than "
              "the %zu the library holds",
              rb->K, Cin, Cout, fs.total, NOALLOC_SCRATCH_BYTES);
    return SCN_ERR_WORKSPACE;
  }
  void* base = nullptr;
  if (scn_status rc0 = noalloc_scratch(&base)) return rc0;
  return fwd_run(rb, x, g_in, W, bias, Cin, Cout, flags, y, g_out, st, fs,
                 static_cast<float*>(base));
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
  if (scn_status rc0 = after_build(rb, st)) return rc0;
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
  float* wpack = reinterpret_cast<float*>(base + L.o_wp);
  float* gzero = reinterpret_cast<float*>(base + L.o_gz);
  const int K = rb->K;

  // dȳ and S (column sums over active outputs)
  if (rb->a_out > 0) {
    const bool v4 = (Cout % 4 == 0) && Cout <= 4 * NT &&
                    ((reinterpret_cast<uintptr_t>(dy) | reinterpret_cast<uintptr_t>(y) |
                      reinterpret_cast<uintptr_t>(ws)) & 15) == 0;
    if (v4)
      hipLaunchKernelGGL(colsum_vec_kernel, dim3((unsigned)L.nblk), dim3(NT), 0, st,
                         reinterpret_cast<const float4*>(dy), reinterpret_cast<const float4*>(y),
                         relu, rb->a_out, Cout / 4, reinterpret_cast<float4*>(dyb),
                         reinterpret_cast<float4*>(partS));
    else
      hipLaunchKernelGGL(colsum_kernel, dim3((unsigned)L.nblk), dim3(NT), 0, st, dy, y, relu,
                         rb->a_out, Cout, dyb, partS);
    SCN_LAUNCH_CHECK();
  }
  hipLaunchKernelGGL(finish_vec_kernel, dim3((unsigned)Cout), dim3(NT), 0, st, partS,
                     rb->a_out > 0 ? L.nblk : 0, Cout, g_out, dg_out, relu, S, u0, dbias);
  SCN_LAUNCH_CHECK();

  // input gradient: accumulate over input ranks with W_k^T
  if (dx && rb->a_in > 0) {
    GatherArgs a{};
    a.src = dyb;
    a.gidx = rb->out_rows;
    a.aidx = rb->in_rank;
    a.tpos = rb->itile;
    a.ntile = rb->n_itiles;
    const int RkP = (int)ceil_div(Cout, 16) * 16, NcP = (int)ceil_div(Cin, 64) * 64;
    hipLaunchKernelGGL(pack_w_kernel, dim3((unsigned)ceil_div((int64_t)K * NcP * RkP, 256)),
                       dim3(256), 0, st, W, K, Cin, Cout, 0, RkP, NcP, wpack);
    SCN_LAUNCH_CHECK();
    hipLaunchKernelGGL(zero_kernel, dim3((unsigned)ceil_div((int64_t)K * NcP, 256)), dim3(256), 0,
                       st, gzero, (int64_t)K * NcP);
    SCN_LAUNCH_CHECK();
    a.Wp = wpack;  // W_k(j = output channel, n = input channel) = W[k][n][j]
    a.gwp = gzero;
    a.NcP = NcP;
    a.Rk = Cout;
    a.Nc = Cin;
    a.add = nullptr;
    a.relu = 0;
    a.dst = dx;
    a.wmap = rb->input_sorted ? nullptr : rb->perm;
    a.nrows = rb->a_in;
    a.K = K;
    scn_status rc;
    if ((rc = timer_mark(TK_DX, 0, st)) || (rc = launch_gather(a, st)) ||
        (rc = timer_mark(TK_DX, 1, st)))
      return rc;
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
    d.K = K;
    d.Cin = Cin;
    d.Cout = Cout;
    d.nco = (int)ceil_div(Cout, 64);
    d.nblk = (int)ceil_div(Cin, 64) * d.nco;
    d.chp = L.chp;
    d.maxc = L.maxc;
    d.part = part;
    d.partT = partT;
    if (rb->n_pairs > 0) {
      const int64_t nwg = L.maxc * K * d.nblk;
      const bool v4 = Cin % 4 == 0 && Cout % 4 == 0 &&
                      ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(dyb) |
                        reinterpret_cast<uintptr_t>(g_in)) & 15) == 0;
      if (scn_status rc = timer_mark(TK_DW, 0, st)) return rc;
      if (v4)
        hipLaunchKernelGGL(dw_partial_kernel<true>, dim3((unsigned)nwg), dim3(NT), 0, st, d);
      else
        hipLaunchKernelGGL(dw_partial_kernel<false>, dim3((unsigned)nwg), dim3(NT), 0, st, d);
      SCN_LAUNCH_CHECK();
      if (scn_status rc = timer_mark(TK_DW, 1, st)) return rc;
    }
    const int64_t nred = std::max<int64_t>((int64_t)K * Cin * Cout, (int64_t)K * Cout);
    hipLaunchKernelGGL(dw_reduce_kernel, dim3((unsigned)ceil_div(nred, RED_E)),
                       dim3(RED_E * RED_G), 0, st,
                       part, partT, rb->off_dev, K, Cin, Cout, L.chp, L.maxc, g_in, u0, dW, T);
    SCN_LAUNCH_CHECK();
    if (dg_in) {
      hipLaunchKernelGGL(dgin_kernel, dim3((unsigned)Cin), dim3(256), 0, st, W, u0, T, K, Cin,
                         Cout, dg_in);
      SCN_LAUNCH_CHECK();
    }
  }
  return SCN_OK;
}

}  // extern "C"
