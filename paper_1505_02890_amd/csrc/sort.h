// Stable LSD radix sort of (key, int32 value) pairs by the low `bits` bits of
// the key (uint32 or uint64), 9 bits (512 digits) per pass.  The dense
// forward view uses it to order output rows by their neighbour masks, the
// keyed rulebook builder to order site keys.
//
// Each pass, over tiles of 2048 pairs:
//   upsweep    digit histogram of every tile -> hist[digit][tile]
//   colscan    one work-group per digit: exclusive prefix of its row of
//              hist over the tiles, and the digit's total
//   downsweep  every pair's place inside its tile, a local sort of the tile
//              in LDS, then contiguous runs out to the digits' places.
// Inside a tile, wave w owns the 512 consecutive pairs [512w, 512w + 512)
// and takes them 64 at a time in order.  The lanes holding one digit find
// each other with nine ballots (one per digit bit); the lowest of them reads
// and advances the wave's running count of that digit in LDS.  A pair's place
// in the tile is then (pairs of smaller digits in the tile) + (pairs of its
// digit in earlier waves) + (earlier pairs of the wave with its digit), so
// pairs with equal digits keep their input order: the sort is stable and
// deterministic.  The tile's run of digit d goes to the output at
// (pairs of smaller digits overall) + (pairs of digit d in earlier tiles).
#pragma once

#include "scan.h"
#include "scn_internal.h"

namespace scn {

constexpr int RS_BITS = 9;
constexpr int RS_DIGITS = 1 << RS_BITS;
constexpr int RS_THREADS = 256;
constexpr int RS_WAVES = RS_THREADS / 64;
constexpr int RS_ROUNDS = 8;                         // rounds of 64 pairs per wave
constexpr int RS_TILE = RS_THREADS * RS_ROUNDS;      // 2048 pairs per tile

inline int64_t rs_tiles(int64_t n) { return std::max<int64_t>(1, ceil_div(n, RS_TILE)); }
inline int rs_passes(int bits) { return std::max(1, (bits + RS_BITS - 1) / RS_BITS); }

// lanes of the wave whose (valid) digit equals this lane's
__device__ inline uint64_t rs_peers(uint32_t d, bool valid) {
  uint64_t m = __ballot(valid);
#pragma unroll
  for (int b = 0; b < RS_BITS; ++b) {
    const uint64_t bal = __ballot((d >> b) & 1u);
    m &= ((d >> b) & 1u) ? bal : ~bal;
  }
  return m;
}

__device__ inline uint32_t rs_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

template <typename KT>
__global__ void __launch_bounds__(RS_THREADS) rs_upsweep_kernel(const KT* __restrict__ keys,
                                                                int64_t n, int shift,
                                                                int64_t ntiles,
                                                                uint32_t* __restrict__ hist) {
  __shared__ uint32_t h[RS_DIGITS];
  for (int i = threadIdx.x; i < RS_DIGITS; i += RS_THREADS) h[i] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * RS_TILE;
  const int lane = threadIdx.x & 63;
  KT k[RS_ROUNDS];
#pragma unroll
  for (int j = 0; j < RS_ROUNDS; ++j) {
    const int64_t i = base + (int64_t)j * RS_THREADS + threadIdx.x;
    k[j] = i < n ? keys[i] : KT(0);
  }
#pragma unroll
  for (int j = 0; j < RS_ROUNDS; ++j) {
    const bool valid = base + (int64_t)j * RS_THREADS + threadIdx.x < n;
    const uint32_t d = (uint32_t)(k[j] >> shift) & (RS_DIGITS - 1);
    const uint64_t peers = rs_peers(d, valid);
    // one LDS add per digit group of the wave
    if (valid && lane == __builtin_ctzll(peers)) atomicAdd(&h[d], (uint32_t)__popcll(peers));
  }
  __syncthreads();
  for (int i = threadIdx.x; i < RS_DIGITS; i += RS_THREADS)
    hist[(int64_t)i * ntiles + blockIdx.x] = h[i];
}

// One work-group per digit d: pre[d][t] = sum of hist[d][t'] for t' < t, and
// tot[d] = the digit's count.  Each thread adds a contiguous run of the row,
// one block scan places the runs, and each thread writes its run's prefixes
// (a block scan per 256 entries, as before, made a 2150-tile row cost 10 us).
static __global__ void __launch_bounds__(RS_THREADS) rs_colscan_kernel(const uint32_t* __restrict__ hist,
                                                                int64_t ntiles,
                                                                uint32_t* __restrict__ pre,
                                                                uint32_t* __restrict__ tot) {
  const int64_t row = (int64_t)blockIdx.x * ntiles;
  const int64_t per = (ntiles + RS_THREADS - 1) / RS_THREADS;
  const int64_t t0 = min<int64_t>(ntiles, (int64_t)threadIdx.x * per),
                t1 = min<int64_t>(ntiles, t0 + per);
  uint32_t s = 0;
  for (int64_t t = t0; t < t1; ++t) s += hist[row + t];
  uint32_t all;
  uint32_t ex = block_exclusive_scan<uint32_t>(s, &all);
  for (int64_t t = t0; t < t1; ++t) {
    const uint32_t v = hist[row + t];
    pre[row + t] = ex;
    ex += v;
  }
  if (threadIdx.x == 0) tot[blockIdx.x] = all;
}

// FIRST: the values are the pairs' input positions (vin is not read)
template <typename KT, bool FIRST>
__global__ void __launch_bounds__(RS_THREADS) rs_downsweep_kernel(
    const KT* __restrict__ kin, const int32_t* __restrict__ vin,
    KT* __restrict__ kout, int32_t* __restrict__ vout, int64_t n, int shift,
    int64_t ntiles, const uint32_t* __restrict__ pre, const uint32_t* __restrict__ tot) {
  __shared__ uint32_t cnt[RS_WAVES][RS_DIGITS];  // per-wave running counts
  __shared__ uint32_t toff[RS_DIGITS];           // tile: pairs of smaller digits
  __shared__ uint32_t gbase[RS_DIGITS];          // output place of the tile's run, less toff
  __shared__ KT skey[RS_TILE];
  __shared__ int32_t sval[RS_TILE];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int i = lane; i < RS_DIGITS; i += 64) cnt[w][i] = 0;
  __builtin_amdgcn_wave_barrier();
  const int64_t tbase = (int64_t)blockIdx.x * RS_TILE;
  const int64_t base = tbase + (int64_t)w * (64 * RS_ROUNDS);
  KT key[RS_ROUNDS];
  uint32_t rank[RS_ROUNDS];
  int32_t val[RS_ROUNDS];
#pragma unroll
  for (int j = 0; j < RS_ROUNDS; ++j) {
    const int64_t i = base + j * 64 + lane;
    key[j] = i < n ? kin[i] : KT(0);
    val[j] = FIRST ? (int32_t)i : (i < n ? vin[i] : 0);
  }
#pragma unroll
  for (int j = 0; j < RS_ROUNDS; ++j) {
    const bool valid = base + j * 64 + lane < n;
    const uint32_t d = (uint32_t)(key[j] >> shift) & (RS_DIGITS - 1);
    const uint64_t peers = rs_peers(d, valid);
    const int leader = valid ? __builtin_ctzll(peers) : lane;
    uint32_t c = 0;
    if (valid && lane == leader) {
      c = cnt[w][d];
      cnt[w][d] = c + (uint32_t)__popcll(peers);
    }
    c = (uint32_t)__shfl((int)c, leader, 64);
    rank[j] = c + rs_below(peers);
  }
  __syncthreads();
  // Per digit: pairs in earlier waves (cnt, in place), the tile's count, and
  // the run's output place.  Thread t owns digits 2t and 2t + 1.
  constexpr int PER = RS_DIGITS / RS_THREADS;
  uint32_t tcount[PER], dtot[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int dd = threadIdx.x * PER + u;
    uint32_t run = 0;
#pragma unroll
    for (int v = 0; v < RS_WAVES; ++v) {
      const uint32_t t = cnt[v][dd];
      cnt[v][dd] = run;
      run += t;
    }
    tcount[u] = run;
    dtot[u] = tot[dd];
  }
  {
    uint32_t s_t = 0, s_g = 0;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      s_t += tcount[u];
      s_g += dtot[u];
    }
    uint32_t all;
    uint32_t ex_t = block_exclusive_scan<uint32_t>(s_t, &all);
    uint32_t ex_g = block_exclusive_scan<uint32_t>(s_g, &all);
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int dd = threadIdx.x * PER + u;
      toff[dd] = ex_t;
      gbase[dd] = ex_g + pre[(int64_t)dd * ntiles + blockIdx.x] - ex_t;
      ex_t += tcount[u];
      ex_g += dtot[u];
    }
  }
  __syncthreads();
  // the tile sorted by digit in LDS
#pragma unroll
  for (int j = 0; j < RS_ROUNDS; ++j) {
    if (base + j * 64 + lane < n) {
      const uint32_t d = (uint32_t)(key[j] >> shift) & (RS_DIGITS - 1);
      const uint32_t q = toff[d] + cnt[w][d] + rank[j];
      skey[q] = key[j];
      sval[q] = val[j];
    }
  }
  __syncthreads();
  // runs of equal digits go out contiguously: local place q of digit d goes
  // to gbase[d] + q
  const int64_t valid_n = n - tbase < RS_TILE ? n - tbase : RS_TILE;
#pragma unroll
  for (int j = 0; j < RS_ROUNDS; ++j) {
    const int q = j * RS_THREADS + threadIdx.x;
    if (q < valid_n) {
      const KT k = skey[q];
      const uint32_t dst = gbase[(uint32_t)(k >> shift) & (RS_DIGITS - 1)] + (uint32_t)q;
      if (dst < n) {  // always, when histogram and ranks agree
        kout[dst] = k;
        vout[dst] = sval[q];
      }
    }
  }
}

// Scratch of radix_sort_pairs, in 32-bit words: two key and two value
// buffers of n, the histogram, its column prefix and the digit totals.
template <typename KT = uint32_t>
inline int64_t radix_sort_words(int64_t n) {
  const int64_t h = (int64_t)RS_DIGITS * rs_tiles(n);
  auto al = [](int64_t w) { return (w + 63) & ~int64_t(63); };  // 256-byte pieces
  const int64_t kw = (int64_t)(sizeof(KT) / 4);
  return 2 * (kw + 1) * al(std::max<int64_t>(n, 1)) + 2 * al(h) + al(RS_DIGITS);
}

// Sorts (keys_in[i], i) by the low `bits` bits of keys_in into
// (keys_out, vals_out), stably.  tmp: radix_sort_words(n) 32-bit words,
// 256-byte aligned.  All arrays device, n < 2^31.
template <typename KT>
inline scn_status radix_sort_pairs(const KT* keys_in, KT* keys_out, int32_t* vals_out, int64_t n,
                                   int bits, uint32_t* tmp, hipStream_t st) {
  if (n <= 0) return SCN_OK;
  const int64_t ntiles = rs_tiles(n), h = (int64_t)RS_DIGITS * ntiles;
  auto al = [](int64_t w) { return (w + 63) & ~int64_t(63); };
  const int64_t kw = (int64_t)(sizeof(KT) / 4);  // 32-bit words per key
  KT* ka = reinterpret_cast<KT*>(tmp);
  int32_t* va = reinterpret_cast<int32_t*>(tmp + kw * al(n));
  KT* kb = reinterpret_cast<KT*>(va + al(n));
  int32_t* vb = reinterpret_cast<int32_t*>(tmp + (kw + 1) * al(n) + kw * al(n));
  uint32_t* hist = reinterpret_cast<uint32_t*>(vb + al(n));
  uint32_t* pre = hist + al(h);
  uint32_t* tot = pre + al(h);
  const int passes = rs_passes(bits);
  const KT* kin = keys_in;
  const int32_t* vin = nullptr;
  for (int p = 0; p < passes; ++p) {
    const bool last = p == passes - 1;
    // passes ping-pong between the two buffers and end in the outputs
    KT* ko = last ? keys_out : ((passes - 1 - p) % 2 ? ka : kb);
    int32_t* vo = last ? vals_out : ((passes - 1 - p) % 2 ? va : vb);
    const int shift = p * RS_BITS;
    hipLaunchKernelGGL(rs_upsweep_kernel<KT>, dim3((unsigned)ntiles), dim3(RS_THREADS), 0, st, kin, n,
                       shift, ntiles, hist);
    SCN_LAUNCH_CHECK();
    hipLaunchKernelGGL(rs_colscan_kernel, dim3(RS_DIGITS), dim3(RS_THREADS), 0, st,
                       (const uint32_t*)hist, ntiles, pre, tot);
    SCN_LAUNCH_CHECK();
    if (p == 0)
      hipLaunchKernelGGL((rs_downsweep_kernel<KT, true>), dim3((unsigned)ntiles), dim3(RS_THREADS), 0,
                         st, kin, vin, ko, vo, n, shift, ntiles, (const uint32_t*)pre,
                         (const uint32_t*)tot);
    else
      hipLaunchKernelGGL((rs_downsweep_kernel<KT, false>), dim3((unsigned)ntiles), dim3(RS_THREADS), 0,
                         st, kin, vin, ko, vo, n, shift, ntiles, (const uint32_t*)pre,
                         (const uint32_t*)tot);
    SCN_LAUNCH_CHECK();
    kin = ko;
    vin = vo;
  }
  return SCN_OK;
}

}  // namespace scn
