// Rulebook construction on the GPU: step 1 of the sparse convolution of
// section 1.3 (iterate over H_in, find and number the active output sites,
// H_out) and the per-offset (input row, output row) lists that stand for the
// non-ground-state blocks of the matrix Q of step 2.
//
// Data structure.  The paper keeps H_in / H_out as a map or hash table from
// site to row.  Here the grids are bounded, so the map is an occupancy bitmap
// (one bit per lattice site, x-rows padded to whole 32-bit words) plus an
// exclusive prefix sum of the word popcounts: the rank of an active site in
// key order is prefix[word] + popcount(word & bits below it).  This is a
// minimal perfect hash of the active set that is ordered by key, so the output
// numbering (ascending key) needs no sort, no hash probing and no atomics on
// the output side, and every result is deterministic.
//
// Lattices (section 1.2, Figure 2).  The cubic lattice uses the grid
// [0, m)^3 and the f^3 offsets of a cube.  The tetrahedral lattice is held in
// skewed integer coordinates: its grid of size m is the sites x + y + z < m
// of a cube with equal extents m, a filter of size f covers the C(f+2, 3)
// offsets kx + ky + kz < f (numbered in the cube's scan order restricted to
// them), and output o exists where its whole window lies in the grid, i.e.
// where ox + oy + oz < (m - f) / s + 1.  The square and triangular lattices
// are their 2D counterparts on grids with one z plane (mz = 1, z = 0): f^2
// offsets (kx, ky, 0), or the C(f+1, 2) offsets kx + ky < f on the sites
// x + y < m.  All lattices share every phase below; the simplex ones
// (tetrahedral, triangular) mask the dilated rows to their output grid and
// visit only their own offsets.
//
// Phases (one stream, two host synchronisations):
//   1 mark inputs            bitmap OR per input; range / duplicate checks
//   2 scan input words       rank of every input site
//   3 rank -> caller row     perm[rank] = row
//   4 dilate                 output word = OR over the window of input bits
//                            (second active-site rule of section 1.3)
//   5 scan output words      a_out and output numbering          [sync 1]
//   6 output sites           coordinates and K-bit neighbour mask per output
//   7 tile counts            pairs per (offset, tile of 64 outputs)
//   8 scan of tile counts    list boundaries and per-tile pair ranges
//   9 emit pairs             in_row / out_row (+ rank; pool maps)
//  10 input-tile ranges      per (offset, tile of 64 input ranks)   [sync 2]
//
// The output layer's bitmap and its prefix (phases 4-5) stay with the
// rulebook: they are H_out, and a build from this rulebook's output sites
// (scn_rulebook_build_next) takes them as its H_in and skips phases 1-3.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <memory>
#include <vector>

#include "scan.h"
#include "scn_internal.h"
#include "sort.h"

namespace scn {
namespace {

enum : uint32_t { F_RANGE = 1, F_DUP = 2, F_UNSORTED = 4 };

struct GridDev {
  int32_t B, mx, my, mz;  // grid extents
  int32_t rw;             // 32-bit words per x-row
  int32_t simplex;        // 1: sites with x + y + z < mx only (tetrahedral, triangular)
};

// Window offsets of a filter of size F on lattice LAT: the cube [0, F)^3, its
// corner kx + ky + kz < F (tetrahedral), the square [0, F)^2 x {0}, or its
// corner kx + ky < F (triangular).  FZ is the window's extent along z;
// row_len(ky, kz) offsets of x-row (ky, kz) are in the window (0 or fewer:
// none); offsets are counted in scan order (x fastest).
template <int F, int LAT>
struct Win {
  static constexpr bool SIMPLEX = LAT == SCN_LATTICE_TETRAHEDRAL || LAT == SCN_LATTICE_TRIANGULAR;
  static constexpr bool PLANAR = LAT == SCN_LATTICE_SQUARE || LAT == SCN_LATTICE_TRIANGULAR;
  static constexpr int FZ = PLANAR ? 1 : F;
  static constexpr int K = LAT == SCN_LATTICE_CUBIC         ? F * F * F
                           : LAT == SCN_LATTICE_TETRAHEDRAL ? F * (F + 1) * (F + 2) / 6
                           : LAT == SCN_LATTICE_SQUARE      ? F * F
                                                            : F * (F + 1) / 2;
  static constexpr int row_len(int ky, int kz) { return SIMPLEX ? F - ky - kz : F; }
};

__device__ inline uint64_t site_key(const GridDev& g, int64_t b, int64_t x, int64_t y,
                                    int64_t z) {
  return (uint64_t)(((b * g.mz + z) * g.my + y) * g.mx + x);
}

__device__ inline int64_t row_base(const GridDev& g, int64_t b, int64_t y, int64_t z) {
  return ((b * g.mz + z) * g.my + y) * g.rw;
}

// 32 bits of an x-row starting at bit position p (bits past the row read 0).
__device__ inline uint32_t extract32(const uint32_t* __restrict__ bm, int64_t base, int rw,
                                     int64_t p) {
  const int64_t w = p >> 5;
  const int sh = (int)(p & 31);
  const uint32_t lo = w < rw ? bm[base + w] : 0u;
  if (sh == 0) return lo;
  const uint32_t hi = w + 1 < rw ? bm[base + w + 1] : 0u;
  return (lo >> sh) | (hi << (32 - sh));
}

__device__ inline uint32_t lane_rank(uint64_t ballot) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(ballot >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)ballot, 0u));
}

// even bits of a 64-bit word packed into 32 bits
__device__ inline uint32_t compress_even(uint64_t x) {
  x &= 0x5555555555555555ull;
  x = (x | (x >> 1)) & 0x3333333333333333ull;
  x = (x | (x >> 2)) & 0x0F0F0F0F0F0F0F0Full;
  x = (x | (x >> 4)) & 0x00FF00FF00FF00FFull;
  x = (x | (x >> 8)) & 0x0000FFFF0000FFFFull;
  x = (x | (x >> 16)) & 0x00000000FFFFFFFFull;
  return (uint32_t)x;
}

// ---- phase 1: mark the input sites ----------------------------------------
__global__ void __launch_bounds__(256) mark_inputs_kernel(const int32_t* __restrict__ coords,
                                                          int64_t n, GridDev g,
                                                          uint32_t* __restrict__ bm,
                                                          uint32_t* __restrict__ flags) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint32_t f = 0;
  if (i < n) {
    const int4 c = reinterpret_cast<const int4*>(coords)[i];
    const bool ok = c.x >= 0 && c.x < g.B && c.y >= 0 && c.y < g.mx && c.z >= 0 &&
                    c.z < g.my && c.w >= 0 && c.w < g.mz &&
                    (!g.simplex || (int64_t)c.y + c.z + c.w < g.mx);
    if (!ok) {
      f |= F_RANGE;
    } else {
      const int64_t w = row_base(g, c.x, c.z, c.w) + (c.y >> 5);
      const uint32_t bit = 1u << (c.y & 31);
      const uint32_t old = atomicOr(&bm[w], bit);
      if (old & bit) f |= F_DUP;
      if (i > 0) {
        const int4 p = reinterpret_cast<const int4*>(coords)[i - 1];
        // an out-of-range predecessor is reported by its own thread
        if (site_key(g, c.x, c.y, c.z, c.w) <= site_key(g, p.x, p.y, p.z, p.w)) f |= F_UNSORTED;
      }
    }
  }
  // one atomic per block at most
  __shared__ uint32_t sf;
  if (threadIdx.x == 0) sf = 0;
  __syncthreads();
  if (f) atomicOr(&sf, f);
  __syncthreads();
  // every block of an unsorted list raises F_UNSORTED: read the word first,
  // so the blocks do not all queue atomics on one address
  if (threadIdx.x == 0 && sf &&
      (__hip_atomic_load(flags, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & sf) != sf)
    atomicOr(flags, sf);
}

struct PopcountLoad {
  const uint32_t* bm;
  __device__ uint32_t operator()(int64_t i) const { return (uint32_t)__popc(bm[i]); }
  __device__ void chunk(int64_t i, uint32_t (&v)[SCAN_ITEMS]) const {
    load16<uint32_t>(bm + i, v);
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j) v[j] = (uint32_t)__popc(v[j]);
  }
};

// ---- phase 3: rank -> caller row ------------------------------------------
__global__ void __launch_bounds__(256) perm_kernel(const int32_t* __restrict__ coords, int64_t n,
                                                   GridDev g, const uint32_t* __restrict__ bm,
                                                   const uint32_t* __restrict__ pref,
                                                   int32_t* __restrict__ perm) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int4 c = reinterpret_cast<const int4*>(coords)[i];
  // it runs before the list's errors are read back: sites outside the grid
  // are skipped (the build then fails with SCN_ERR_RANGE)
  if (c.x < 0 || c.x >= g.B || c.y < 0 || c.y >= g.mx || c.z < 0 || c.z >= g.my || c.w < 0 ||
      c.w >= g.mz)
    return;
  const int64_t w = row_base(g, c.x, c.z, c.w) + (c.y >> 5);
  const uint32_t below = (1u << (c.y & 31)) - 1u;
  const uint32_t rank = pref[w] + (uint32_t)__popc(bm[w] & below);
  if (rank < n) perm[rank] = (int32_t)i;
}

// Output word wo of the output grid -> (b, z, y, word-in-row).  32-bit:
// bitmaps hold at most 2^26 words.
struct WordPos {
  int b, z, y, wx;
};

__device__ inline WordPos word_pos(int wo, const GridDev& g) {
  WordPos p;
  p.wx = wo % g.rw;
  int r = wo / g.rw;
  p.y = r % g.my;
  r /= g.my;
  p.z = r % g.mz;
  p.b = r / g.mz;
  return p;
}

// ---- phase 4: output occupancy (dilation of the input bitmap) -------------
// SM: 1 stride 1 (funnel shifts), 2 stride 2 (even-bit compression), 0 any.
// On the simplex lattices the bits past the output grid (x + y + z >= mx)
// are cleared and rows wholly past it are not read.
template <int F, int LAT, int SM>
__global__ void __launch_bounds__(256) dilate_kernel(const uint32_t* __restrict__ inb, GridDev gi,
                                                     uint32_t* __restrict__ outb, GridDev go,
                                                     int nw_out, int s) {
  using W = Win<F, LAT>;
  const int wo = blockIdx.x * blockDim.x + threadIdx.x;
  if (wo >= nw_out) return;
  const WordPos wp = word_pos(wo, go);
  const int x0 = wp.wx * 32;
  const int lim = W::SIMPLEX ? go.mx - wp.y - wp.z : go.mx;  // x < lim on this row
  const int nvalid = min(32, lim - x0);
  if (nvalid <= 0) {
    outb[wo] = 0u;
    return;
  }
  const uint32_t valid = nvalid >= 32 ? 0xFFFFFFFFu : ((1u << nvalid) - 1u);
  uint32_t v = 0;
#pragma unroll
  for (int kz = 0; kz < W::FZ; ++kz)
#pragma unroll
    for (int ky = 0; ky < F; ++ky) {
      const int nx = W::row_len(ky, kz);
      if (nx <= 0) continue;
      const int64_t base = row_base(gi, wp.b, (int64_t)s * wp.y + ky, (int64_t)s * wp.z + kz);
      if (SM == 1) {
#pragma unroll
        for (int kx = 0; kx < F; ++kx)
          if (kx < nx) v |= extract32(inb, base, gi.rw, (int64_t)x0 + kx);
      } else if (SM == 2) {
        const int64_t p = 2 * (int64_t)x0;  // multiple of 64
        const uint64_t lo = extract32(inb, base, gi.rw, p);
        const uint64_t hi = extract32(inb, base, gi.rw, p + 32);
        const uint64_t w64 = lo | (hi << 32);
        uint64_t t = w64;
        if (nx >= 2) t |= w64 >> 1;
        if (nx >= 3) {
          const uint64_t nxt = extract32(inb, base, gi.rw, p + 64) & 1u;
          t |= (w64 >> 2) | (nxt << 62);
        }
        v |= compress_even(t);
      } else {
        const uint32_t fm = (1u << nx) - 1u;
        for (int j = 0; j < nvalid; ++j)
          if (extract32(inb, base, gi.rw, (int64_t)s * (x0 + j)) & fm) v |= 1u << j;
      }
    }
  outb[wo] = v & valid;
}

// ---- phase 6: output coordinates and neighbour masks ----------------------
// One thread per output word; its sites take consecutive ranks.  A block's
// 256 words hold one contiguous rank range: when it fits OUT_STAGE entries
// the sites are staged in LDS and written out as one coalesced run (stored
// straight from the lanes, every store touched up to 64 lines, each only
// partly); a denser block writes directly.
constexpr int OUT_STAGE = 1024;
template <int F, int LAT, bool S1>
__global__ void __launch_bounds__(256) out_sites_kernel(const uint32_t* __restrict__ inb, GridDev gi,
                                                        const uint32_t* __restrict__ outb,
                                                        const uint32_t* __restrict__ opref,
                                                        GridDev go, int nw_out, int s,
                                                        int32_t* __restrict__ out_coords,
                                                        uint32_t* __restrict__ masks, int chunk) {
  using W = Win<F, LAT>;
  __shared__ int4 st_c[OUT_STAGE];
  __shared__ uint32_t st_m[OUT_STAGE];
  // runs of blocks per XCD: neighbouring output rows read the same input
  // bitmap words (70.9 -> 58.7 us for 4.4M outputs with runs of 64 blocks)
  const int wb0 = (int)xcd_block(blockIdx.x, chunk) * blockDim.x;
  if (wb0 >= nw_out) return;  // the whole block: a launch rounded up to whole runs
  const int wb1 = min(nw_out, wb0 + (int)blockDim.x);
  // opref[nw_out] is the total
  const uint32_t first = opref[wb0], cnt = opref[wb1] - first;
  const bool staged = cnt <= (uint32_t)OUT_STAGE;
  const int wo = wb0 + threadIdx.x;
  uint32_t v = wo < nw_out ? outb[wo] : 0u;
  auto put = [&](uint32_t rank, int4 c, uint32_t m) {
    if (staged) {
      st_c[rank - first] = c;
      st_m[rank - first] = m;
    } else {
      reinterpret_cast<int4*>(out_coords)[rank] = c;
      masks[rank] = m;
    }
  };
  if (v) {
    const WordPos wp = word_pos(wo, go);
    const int x0 = wp.wx * 32;
    uint32_t rank = opref[wo];
    if (S1) {
      // R[r] bit j + kx: input site (x0 + j + kx, y + ky, z + kz) of window row
      // r = (ky, kz) is active; the row's offsets are consecutive mask bits
      constexpr int NR = W::FZ * F;
      uint64_t R[NR];
#pragma unroll
      for (int kz = 0; kz < W::FZ; ++kz)
#pragma unroll
        for (int ky = 0; ky < F; ++ky) {
          R[kz * F + ky] = 0;
          if (W::row_len(ky, kz) <= 0) continue;
          const int64_t base = row_base(gi, wp.b, wp.y + ky, wp.z + kz);
          const int64_t w = x0 >> 5;
          const uint32_t lo = w < gi.rw ? inb[base + w] : 0u;
          const uint32_t hi = w + 1 < gi.rw ? inb[base + w + 1] : 0u;
          R[kz * F + ky] = (uint64_t)lo | ((uint64_t)hi << 32);
        }
      while (v) {
        const int j = __builtin_ctz(v);
        v &= v - 1;
        uint32_t m = 0;
        int k = 0;
#pragma unroll
        for (int kz = 0; kz < W::FZ; ++kz)
#pragma unroll
          for (int ky = 0; ky < F; ++ky) {
            const int len = W::row_len(ky, kz);
            if (len <= 0) continue;
            m |= (uint32_t)((R[kz * F + ky] >> j) & ((1u << len) - 1u)) << k;
            k += len;
          }
        put(rank++, make_int4(wp.b, x0 + j, wp.y, wp.z), m);
      }
    } else {
      while (v) {
        const int j = __builtin_ctz(v);
        v &= v - 1;
        const int64_t xi = (int64_t)s * (x0 + j);
        uint32_t m = 0;
        int k = 0;
#pragma unroll
        for (int kz = 0; kz < W::FZ; ++kz)
#pragma unroll
          for (int ky = 0; ky < F; ++ky) {
            if (W::row_len(ky, kz) <= 0) continue;
            const int64_t base =
                row_base(gi, wp.b, (int64_t)s * wp.y + ky, (int64_t)s * wp.z + kz);
            const uint32_t bits = extract32(inb, base, gi.rw, xi);
#pragma unroll
            for (int kx = 0; kx < F; ++kx)
              if (kx < W::row_len(ky, kz)) m |= ((bits >> kx) & 1u) << k++;
          }
        put(rank++, make_int4(wp.b, x0 + j, wp.y, wp.z), m);
      }
    }
  }
  if (!staged) return;  // block-uniform
  __syncthreads();
  int4* oc = reinterpret_cast<int4*>(out_coords) + first;
  for (uint32_t i = threadIdx.x; i < cnt; i += blockDim.x) {
    oc[i] = st_c[i];
    masks[first + i] = st_m[i];
  }
}

// ---- phase 7: pairs per (offset, output tile) ------------------------------
// one wave per tile of 64 output rows; cnt[k * nt + t]
template <int K>
__global__ void __launch_bounds__(256) tile_count_kernel(const uint32_t* __restrict__ masks,
                                                         int64_t a_out, int64_t nt,
                                                         uint64_t* __restrict__ cnt) {
  const int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t t = o >> 6;
  const uint32_t m = o < a_out ? masks[o] : 0u;
  const int lane = threadIdx.x & 63;
  uint64_t c = 0;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const uint64_t n = (uint64_t)__popcll(__ballot((m >> k) & 1u));
    if (lane == k) c = n;
  }
  if (lane < K && t < nt) cnt[lane * nt + t] = c;
}

// ---- phase 9: output-major tables --------------------------------------------
// One thread per output, one wave per tile of 64 outputs: the window table
// nbr[o][k] of a pooling rulebook, or the output-major neighbour list fnb of
// the dense forward view (a stride-1 rulebook); the per-offset pair lists are
// emitted input-major (emit_in_kernel).  The rows come from rank lookups in
// the input bitmap and perm, which stay in L2 (reading them back from the
// pair lists, long evicted, took 1.55 times as long).  All K rank lookups
// are issued before any dependent load so they overlap.
constexpr int EMIT_NB_STAGE = 12;  // staged neighbour-list entries per output
template <int F, int LAT>
__global__ void __launch_bounds__(256) emit_out_kernel(
    const uint32_t* __restrict__ masks, const int32_t* __restrict__ out_coords, int64_t a_out,
    int s, const uint32_t* __restrict__ inb, const uint32_t* __restrict__ ipref, GridDev gi,
    const int32_t* __restrict__ perm, int32_t* __restrict__ nbr,
    const uint32_t* __restrict__ fnb_off, int32_t* __restrict__ fnb, int chunk) {
  using W = Win<F, LAT>;
  constexpr int K = W::K;
  // runs of blocks per XCD, as in out_sites_kernel
  const int64_t blk = xcd_block(blockIdx.x, chunk);
  if (blk * 256 >= (a_out + 63) / 64 * 64) return;  // the whole block: past the last tile
  const int64_t o = blk * blockDim.x + threadIdx.x;
  const bool live = o < a_out;
  const uint32_t m = live ? masks[o] : 0u;
  int4 c = make_int4(0, 0, 0, 0);
  if (live) c = reinterpret_cast<const int4*>(out_coords)[o];
  // Rank lookups one window row (ky, kz) at a time: its inputs sit at bits
  // sh .. sh + len - 1 counted from word w of the input bitmap, so the row
  // needs w's prefix and bits and, when it runs past bit 31, the next word's
  // bits (that word's prefix is w's plus popcount(w)).  Words are read only
  // for rows with an active input, so every read word holds a site.
  uint32_t rank[K];
  {
    const int64_t x0 = (int64_t)s * c.y;
    const int sh = (int)(x0 & 31);
    int k = 0;
#pragma unroll
    for (int kz = 0; kz < W::FZ; ++kz)
#pragma unroll
      for (int ky = 0; ky < F; ++ky) {
        const int len = W::row_len(ky, kz);
        if (len <= 0) continue;
        const uint32_t rbits = (m >> k) & ((1u << len) - 1u);
        const uint32_t high = sh + len > 32 ? rbits >> (32 - sh) : 0u;
        const int64_t w =
            row_base(gi, c.x, (int64_t)s * c.z + ky, (int64_t)s * c.w + kz) + (x0 >> 5);
        uint32_t p0 = 0u, b0 = 0u, b1 = 0u;
        if (rbits) {
          p0 = ipref[w];
          b0 = inb[w];
        }
        if (high) b1 = inb[w + 1];
#pragma unroll
        for (int kx = 0; kx < F; ++kx)
          if (kx < len) {
            const int xb = sh + kx;
            rank[k + kx] = xb < 32 ? p0 + (uint32_t)__popc(b0 & ((1u << xb) - 1u))
                                   : p0 + (uint32_t)__popc(b0) +
                                         (uint32_t)__popc(b1 & ((1u << (xb - 32)) - 1u));
          }
        k += len;
      }
  }
  // A lane's entries are up to K words apart, so the wave stages its 64
  // outputs' entries in LDS (dynamic: 64*K words per wave for the table,
  // 64*EMIT_NB_STAGE for the list) and writes them out as one contiguous run.
  // Stored straight from the lanes, every store instruction touched up to 64
  // cache lines, each only partly.  A wave whose list run is longer than its
  // stage writes it directly.
  extern __shared__ int4 emit_lds[];
  int32_t* stage = reinterpret_cast<int32_t*>(emit_lds) +
                   (threadIdx.x >> 6) * (64 * (nbr ? K : EMIT_NB_STAGE));
  const int lane = threadIdx.x & 63;
  const int64_t o0 = o & ~(int64_t)63;  // the wave's first output
  uint32_t nb_at = 0, nb0 = 0, nb_len = 0;
  bool nb_lds = false;
  if (fnb) {
    // the wave's run of the neighbour list starts at fnb_off[o0]
    nb_at = live ? fnb_off[o] : 0u;
    nb0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)nb_at);
    const int last = a_out - 1 - o0 < 63 ? (int)(a_out - 1 - o0) : 63;
    nb_len = (uint32_t)__shfl((int)(nb_at + (uint32_t)__popc(m)), last < 0 ? 0 : last, 64) - nb0;
    nb_lds = nb_len <= 64 * EMIT_NB_STAGE;
    if (nb_lds) nb_at -= nb0;
  }
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const bool bit = (m >> k) & 1u;
    // sorted input: rank order is the caller's row order (no perm table)
    const int32_t row = bit ? (perm ? perm[rank[k]] : (int32_t)rank[k]) : -1;
    if (fnb && bit) {
      if (nb_lds)
        stage[nb_at++] = row;
      else
        fnb[nb_at++] = row;
    }
    if (nbr) stage[lane * K + k] = row;
  }
  if (nb_lds && o0 < a_out) {
    // the stage is this wave's alone: LDS accesses of one wave complete in order
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    for (uint32_t i = lane; i < nb_len; i += 64) __builtin_nontemporal_store(stage[i], fnb + nb0 + i);
  }
  if (nbr) {
    __syncthreads();
    if (o0 < a_out) {
      // 64-output runs start 256-byte aligned in nbr
      const int64_t n = ((o0 + 64 < a_out ? o0 + 64 : a_out) - o0) * K, n4 = n >> 2;
      const int4* src = reinterpret_cast<const int4*>(stage);
      int4* dst = reinterpret_cast<int4*>(nbr + o0 * K);
      for (int64_t i = lane; i < n4; i += 64) dst[i] = src[i];
      for (int64_t i = 4 * n4 + lane; i < n; i += 64) nbr[o0 * K + i] = stage[i];
    }
  }
}

// ---- phase 9b (pooling, stride >= 2): the windows of each input ----------
// One thread per input row r (the caller's order).  Along each axis an input
// at x lies in the window starting at s*floor(x/s) (offset x mod s < s) and,
// when f > s, possibly in the one before it (offset x mod s + s); slot bit a
// says which.  inv[r*slots + slot] = o*K + k for window o at offset k, or -1.
// Every window that holds an active input inside the output grid is active,
// so its row is its rank in the output bitmap.  The row of 4 or 32 bytes is
// written at once instead of scattered from the pair emission.
template <int F, int LAT>
__device__ inline int window_index(int kx, int ky, int kz) {
  using W = Win<F, LAT>;
  int k = 0;
  for (int z = 0; z < kz; ++z)
    for (int y = 0; y < F; ++y) k += W::row_len(y, z);
  for (int y = 0; y < ky; ++y) k += W::row_len(y, kz);
  return k + kx;
}

// With `homeless` given, inputs outside their home window (slot 0 empty:
// the window starting at s*floor(x/s) along each axis lies outside the output
// grid) are appended to homeless[], counted in *n_homeless (in no particular
// order).
template <int F, int LAT, int SLOTS>
__global__ void __launch_bounds__(256) inv_windows_kernel(
    const int32_t* __restrict__ coords, int64_t n, int s, GridDev go,
    const uint32_t* __restrict__ outb, const uint32_t* __restrict__ opref,
    int32_t* __restrict__ inv, int32_t* __restrict__ homeless, int32_t* __restrict__ n_homeless) {
  using W = Win<F, LAT>;
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n) return;
  const int4 c = reinterpret_cast<const int4*>(coords)[r];
  const int p[3] = {c.y, c.z, c.w};
  const int m[3] = {go.mx, go.my, go.mz};
  int v[SLOTS];
#pragma unroll
  for (int slot = 0; slot < SLOTS; ++slot) {
    int o[3], k[3];
    bool ok = true;
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      const int j = (slot >> a) & 1;
      o[a] = p[a] / s - j;
      k[a] = p[a] - s * o[a];
      ok = ok && o[a] >= 0 && o[a] < m[a] && k[a] < F;
    }
    if (W::SIMPLEX) ok = ok && k[0] + k[1] + k[2] < F && o[0] + o[1] + o[2] < go.mx;
    if (W::PLANAR) ok = ok && k[2] == 0;
    v[slot] = -1;
    if (ok) {
      const int64_t w = row_base(go, c.x, o[1], o[2]) + (o[0] >> 5);
      const uint32_t rank =
          opref[w] + (uint32_t)__popc(outb[w] & ((1u << (o[0] & 31)) - 1u));
      v[slot] = (int32_t)((int64_t)rank * W::K + window_index<F, LAT>(k[0], k[1], k[2]));
    }
  }
  if (homeless && v[0] < 0) homeless[atomicAdd(n_homeless, 1)] = (int32_t)r;
  if (SLOTS == 8) {
    int4* d = reinterpret_cast<int4*>(inv + r * 8);
    d[0] = make_int4(v[0], v[1], v[2], v[3]);
    d[1] = make_int4(v[4 % SLOTS], v[5 % SLOTS], v[6 % SLOTS], v[7 % SLOTS]);
  } else {
    inv[r] = v[0];
  }
}

// ---- phase 9c (3-wide windows of stride 2, cubic lattice): the cells ------
// Window h's home cell is the 2x2x2 block of inputs at offsets {0,1}^3 of
// it.  Those inputs also lie in the windows h - b (b in {0,1}^3, bit a: one
// step down along axis a, x y z), at offset +2 along the axes of b.  The
// backward walks windows and computes the dx of each one's home cell from
// the dy rows of these 8 windows.  low[h*8 + b] = row of window h - b, or -1
// when it is outside the grid or inactive (low[h*8] = h).  Thread 0 also
// zeroes the homeless count that inv_windows_kernel fills next.
__global__ void __launch_bounds__(256) lower_windows_kernel(
    const int32_t* __restrict__ out_coords, int64_t a_out, GridDev go,
    const uint32_t* __restrict__ outb, const uint32_t* __restrict__ opref,
    int32_t* __restrict__ low, int32_t* __restrict__ n_homeless) {
  const int64_t h = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (h == 0) *n_homeless = 0;
  if (h >= a_out) return;
  const int4 c = reinterpret_cast<const int4*>(out_coords)[h];
  int32_t v[8];
  v[0] = (int32_t)h;
#pragma unroll
  for (int b = 1; b < 8; ++b) {
    const int x = c.y - (b & 1), y = c.z - ((b >> 1) & 1), z = c.w - (b >> 2);
    v[b] = -1;
    if (x >= 0 && y >= 0 && z >= 0) {
      const int64_t w = row_base(go, c.x, y, z) + (x >> 5);
      const uint32_t bits = outb[w], bit = 1u << (x & 31);
      if (bits & bit) v[b] = (int32_t)(opref[w] + (uint32_t)__popc(bits & (bit - 1u)));
    }
  }
  int4* d = reinterpret_cast<int4*>(low + h * 8);
  d[0] = make_int4(v[0], v[1], v[2], v[3]);
  d[1] = make_int4(v[4], v[5], v[6], v[7]);
}

// The first read-back: flags[1] = number of active inputs, flags[2] =
// number of active outputs and, when the lists are already emitted, their
// boundaries off[k] = itile[k * nit] (also kept in the rulebook's off_dev).
__global__ void pack_totals_kernel(uint32_t* __restrict__ flags, const uint32_t* __restrict__ a_in,
                                   const uint32_t* __restrict__ a_out,
                                   const int64_t* __restrict__ itile, int64_t nit, int K,
                                   int64_t* __restrict__ off, int64_t* __restrict__ off_dev) {
  const int k = threadIdx.x;
  if (k == 0) {
    flags[1] = *a_in;
    flags[2] = *a_out;
  }
  if (itile && k <= K) {
    const int64_t v = itile[(int64_t)k * nit];
    off[k] = v;
    off_dev[k] = v;
  }
}

// list boundaries from the input tiles (lists emitted after the first wait)
__global__ void list_offsets_kernel(const int64_t* __restrict__ itile, int64_t nit, int K,
                                    int64_t* __restrict__ off) {
  const int k = threadIdx.x;
  if (k <= K) off[k] = itile[(int64_t)k * nit];
}

// ---- phase 10: pair counts per (offset, tile of input ranks) --------------
// One wave per tile of 64 input ranks.  Input i pairs at offset k with the
// output o = (i - k) / s when the division is exact and o lies in the output
// grid: that output is active, since input i lies in its window.  So the
// count needs only the input's coordinates, and the exclusive scan of
// cnt[k * nit + t] gives itile[k * nit + t], the position in list k of the
// first pair whose input rank is >= t * TILE (lists ascend by input rank).
template <int F, int LAT, int SM>
__global__ void __launch_bounds__(256) in_tile_count_kernel(
    const int32_t* __restrict__ coords, const int32_t* __restrict__ perm, int64_t n,
    int64_t nit, int s, GridDev go, uint64_t* __restrict__ cnt) {
  using W = Win<F, LAT>;
  constexpr int K = W::K;
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t t = r >> 6;
  const int lane = threadIdx.x & 63;
  int4 c = make_int4(0, 0, 0, 0);
  bool live = r < n;
  if (live) {
    // a list with errors leaves ranks unwritten (the build then fails)
    const int64_t row = perm ? perm[r] : r;
    live = row >= 0 && row < n;
    if (live) c = reinterpret_cast<const int4*>(coords)[row];
  }
  uint64_t mine = 0;
  int k = 0;
#pragma unroll
  for (int kz = 0; kz < W::FZ; ++kz)
#pragma unroll
    for (int ky = 0; ky < F; ++ky)
#pragma unroll
      for (int kx = 0; kx < F; ++kx) {
        if (kx >= W::row_len(ky, kz)) continue;
        const int dx = c.y - kx, dy = c.z - ky, dz = c.w - kz;
        // SM: stride 1, stride 2, or any (a division)
        bool ok = live && dx >= 0 && dy >= 0 && dz >= 0;
        int ox = dx, oy = dy, oz = dz;
        if (SM == 2) {
          ok = ok && !((dx | dy | dz) & 1);
          ox = dx >> 1;
          oy = dy >> 1;
          oz = dz >> 1;
        } else if (SM != 1) {
          ok = ok && dx % s == 0 && dy % s == 0 && dz % s == 0;
          ox = dx / s;
          oy = dy / s;
          oz = dz / s;
        }
        ok = ok && ox < go.mx && oy < go.my && oz < go.mz;
        if (W::SIMPLEX) ok = ok && ox + oy + oz < go.mx;
        const uint64_t c_k = (uint64_t)__popcll(__ballot(ok));
        if (lane == k) mine = c_k;
        ++k;
      }
  if (lane < K && t < nit) cnt[lane * nit + t] = mine;
}

// ---- phase 10b: the pair lists, input-major ------------------------------
// One thread per input rank r, one wave per tile of 64 ranks (the tiles of
// in_tile_count_kernel).  Input i pairs at window offset k with output
// o = (i - k) / s when that is exact and in the output grid; o's row is its
// rank in the output bitmap.  The pair's place in list k is itile[k*nit + t]
// plus the tile's earlier ranks that pair at offset k, so every list ascends
// by input rank and, the window map keeping key order, by output row.  Where
// every input of the tile pairs at k, the wave's stores of that list are one
// contiguous 256-byte run.  The kernel tolerates an input list with errors
// (out-of-grid sites and unwritten ranks are skipped; the build then fails),
// and no store goes past the lists' capacity.
template <int F, int LAT, int SM>
__global__ void __launch_bounds__(256) emit_in_kernel(
    const int32_t* __restrict__ coords, const int32_t* __restrict__ perm, int64_t n,
    int64_t nit, int s, GridDev go, const uint32_t* __restrict__ outb,
    const uint32_t* __restrict__ opref, const int64_t* __restrict__ itile, int64_t cap,
    int32_t* __restrict__ in_rows, int32_t* __restrict__ out_rows,
    int32_t* __restrict__ in_rank) {
  using W = Win<F, LAT>;
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int tw = __builtin_amdgcn_readfirstlane((int)(r >> 6));
  if (tw >= nit) return;  // a whole padding wave
  int4 c = make_int4(0, 0, 0, 0);
  int32_t row = 0;
  bool live = r < n;
  if (live) {
    row = perm ? perm[r] : (int32_t)r;
    live = row >= 0 && row < n;
    if (live) {
      c = reinterpret_cast<const int4*>(coords)[row];
      live = c.x >= 0 && c.x < go.B;  // the other coordinates are checked per offset
    }
  }
  int k = 0;
#pragma unroll
  for (int kz = 0; kz < W::FZ; ++kz)
#pragma unroll
    for (int ky = 0; ky < F; ++ky) {
      const int len = W::row_len(ky, kz);
      if (len <= 0) continue;
      // stride 1: the row's outputs x - len + 1 .. x lie in at most two words
      // of one output x-row
      uint32_t pa = 0, ba = 0, bb = 0;
      int wa = 0;
      if (SM == 1) {
        const int oy = c.z - ky, oz = c.w - kz;
        const int xl = c.y - (len - 1) > 0 ? c.y - (len - 1) : 0;
        const bool row_ok = live && oy >= 0 && oz >= 0 && oy < go.my && oz < go.mz && xl < go.mx;
        if (row_ok) {
          const int64_t base = row_base(go, c.x, oy, oz);
          wa = xl >> 5;
          pa = opref[base + wa];
          ba = outb[base + wa];
          const int wb = c.y >> 5;
          if (wb != wa && wb < go.rw) bb = outb[base + wb];
        }
      }
#pragma unroll
      for (int kx = 0; kx < F; ++kx) {
        if (kx >= len) continue;
        const int dx = c.y - kx, dy = c.z - ky, dz = c.w - kz;
        bool ok = live && dx >= 0 && dy >= 0 && dz >= 0;
        int ox = dx, oy = dy, oz = dz;
        if (SM == 2) {
          ok = ok && !((dx | dy | dz) & 1);
          ox = dx >> 1;
          oy = dy >> 1;
          oz = dz >> 1;
        } else if (SM != 1) {
          ok = ok && dx % s == 0 && dy % s == 0 && dz % s == 0;
          ox = dx / s;
          oy = dy / s;
          oz = dz / s;
        }
        ok = ok && ox < go.mx && oy < go.my && oz < go.mz;
        if (W::SIMPLEX) ok = ok && ox + oy + oz < go.mx;
        uint32_t orank = 0;
        if (ok) {
          const uint32_t below = (1u << (ox & 31)) - 1u;
          if (SM == 1) {
            orank = (ox >> 5) == wa ? pa + (uint32_t)__popc(ba & below)
                                    : pa + (uint32_t)__popc(ba) + (uint32_t)__popc(bb & below);
          } else {
            const int64_t w = row_base(go, c.x, oy, oz) + (ox >> 5);
            orank = opref[w] + (uint32_t)__popc(outb[w] & below);
          }
        }
        const uint64_t bal = __ballot(ok);
        const int64_t p0 = itile[(int64_t)k * nit + tw];
        if (ok) {
          const int64_t p = p0 + lane_rank(bal);
          if (p < cap) {
            // streaming stores: the lists are read only by later calls, and
            // the bitmap words this build looks up keep the cache (build
            // 0.657 -> 0.599 ms on 1M sites, with the neighbour lists')
            __builtin_nontemporal_store(row, in_rows + p);
            __builtin_nontemporal_store((int32_t)orank, out_rows + p);
            if (in_rank) __builtin_nontemporal_store((int32_t)r, in_rank + p);
          }
        }
        ++k;
      }
    }
}

inline unsigned blocks_for(int64_t n, int threads) {
  return (unsigned)std::max<int64_t>(1, ceil_div(n, threads));
}

// Build temporaries.  reserve(bytes) takes one block from the allocator and
// get() carves 256-byte-aligned pieces from it, so a build phase costs one
// allocation and one free (each is a host call of tens of microseconds); a
// request that does not fit gets a block of its own.
struct Temps {
  hipStream_t s = nullptr;
  Allocator al;
  void* p[16] = {nullptr};
  int n = 0;
  char* cur = nullptr;
  size_t left = 0;
  Temps() = default;
  Temps(hipStream_t st, const Allocator& a) : s(st), al(a) {}
  static size_t round(size_t b) { return (std::max<size_t>(b, 1) + 255) & ~size_t(255); }
  scn_status take(void** q, size_t bytes) {
    if (n >= 16) {
      set_error("scn_rulebook_build: too many temporary blocks");
      return SCN_ERR_NOMEM;
    }
    scn_status st = dalloc(q, bytes, s, al);
    if (st == SCN_OK) p[n++] = *q;
    return st;
  }
  scn_status reserve(size_t bytes) {
    void* q = nullptr;
    scn_status st = take(&q, bytes);
    if (st != SCN_OK) return st;
    cur = static_cast<char*>(q);
    left = bytes;
    return SCN_OK;
  }
  template <typename T>
  scn_status get(T** out, size_t count) {
    const size_t b = round(count * sizeof(T));
    if (b <= left) {
      *out = reinterpret_cast<T*>(cur);
      cur += b;
      left -= b;
      return SCN_OK;
    }
    void* q = nullptr;
    scn_status st = take(&q, b);
    *out = static_cast<T*>(q);
    return st;
  }
  ~Temps() {
    for (int i = 0; i < n; ++i) dfree(p[i], s, al);
  }
};

// Kernel variants by filter size and lattice.
template <int F, int LAT>
struct Kernels {
  static constexpr int K = Win<F, LAT>::K;
  static void dilate(int sm, dim3 g, hipStream_t st, const uint32_t* inb, GridDev gi, uint32_t* outb,
                     GridDev go, int nw_out, int s) {
    if (sm == 1)
      hipLaunchKernelGGL((dilate_kernel<F, LAT, 1>), g, dim3(256), 0, st, inb, gi, outb, go, nw_out, s);
    else if (sm == 2)
      hipLaunchKernelGGL((dilate_kernel<F, LAT, 2>), g, dim3(256), 0, st, inb, gi, outb, go, nw_out, s);
    else
      hipLaunchKernelGGL((dilate_kernel<F, LAT, 0>), g, dim3(256), 0, st, inb, gi, outb, go, nw_out, s);
  }
  template <typename... A>
  static void out_sites(bool s1, dim3 g, hipStream_t st, A... a) {
    if (s1)
      hipLaunchKernelGGL((out_sites_kernel<F, LAT, true>), g, dim3(256), 0, st, a...);
    else
      hipLaunchKernelGGL((out_sites_kernel<F, LAT, false>), g, dim3(256), 0, st, a...);
  }
  template <typename... A>
  static void tile_count(dim3 g, hipStream_t st, A... a) {
    hipLaunchKernelGGL((tile_count_kernel<K>), g, dim3(256), 0, st, a...);
  }
  template <typename... A>
  static void emit_out(dim3 g, size_t lds, hipStream_t st, A... a) {
    hipLaunchKernelGGL((emit_out_kernel<F, LAT>), g, dim3(256), lds, st, a...);
  }
  template <typename... A>
  static void emit_in(int sm, dim3 g, hipStream_t st, A... a) {
    if (sm == 1)
      hipLaunchKernelGGL((emit_in_kernel<F, LAT, 1>), g, dim3(256), 0, st, a...);
    else if (sm == 2)
      hipLaunchKernelGGL((emit_in_kernel<F, LAT, 2>), g, dim3(256), 0, st, a...);
    else
      hipLaunchKernelGGL((emit_in_kernel<F, LAT, 0>), g, dim3(256), 0, st, a...);
  }
  template <typename... A>
  static void in_tile_count(int sm, dim3 g, hipStream_t st, A... a) {
    if (sm == 1)
      hipLaunchKernelGGL((in_tile_count_kernel<F, LAT, 1>), g, dim3(256), 0, st, a...);
    else if (sm == 2)
      hipLaunchKernelGGL((in_tile_count_kernel<F, LAT, 2>), g, dim3(256), 0, st, a...);
    else
      hipLaunchKernelGGL((in_tile_count_kernel<F, LAT, 0>), g, dim3(256), 0, st, a...);
  }
  template <typename... A>
  static void inv_windows(int slots, dim3 g, hipStream_t st, A... a) {
    if (slots == 8)
      hipLaunchKernelGGL((inv_windows_kernel<F, LAT, 8>), g, dim3(256), 0, st, a...);
    else
      hipLaunchKernelGGL((inv_windows_kernel<F, LAT, 1>), g, dim3(256), 0, st, a...);
  }
};

// calls fn(Kernels<F, LAT>{}) for the runtime filter size and lattice
template <int LAT, typename Fn>
void with_filter(int f, Fn fn) {
  if (f == 1) fn(Kernels<1, LAT>{});
  else if (f == 2) fn(Kernels<2, LAT>{});
  else fn(Kernels<3, LAT>{});
}

template <typename Fn>
void with_kernels(int f, int lattice, Fn fn) {
  switch (lattice) {
    case SCN_LATTICE_TETRAHEDRAL: with_filter<SCN_LATTICE_TETRAHEDRAL>(f, fn); break;
    case SCN_LATTICE_SQUARE: with_filter<SCN_LATTICE_SQUARE>(f, fn); break;
    case SCN_LATTICE_TRIANGULAR: with_filter<SCN_LATTICE_TRIANGULAR>(f, fn); break;
    default: with_filter<SCN_LATTICE_CUBIC>(f, fn); break;
  }
}

// Host-pinned read-back area of one layer: flags and totals after phase 1,
// the list boundaries after phase 2.
struct Readback {
  uint32_t flags, a_in, a_out, pad;
  int64_t off[MAX_K + 1];
};
constexpr int MAX_CHAIN = 64;  // layers of one scn_rulebook_build_chain call

// One pinned array of read-back slots per host thread, kept for the life of
// the process.
scn_status readback_slots(Readback** out) {
  static thread_local Readback* hb = nullptr;
  if (!hb) SCN_HIP(hipHostMalloc((void**)&hb, MAX_CHAIN * sizeof(Readback), hipHostMallocDefault));
  *out = hb;
  return SCN_OK;
}

// The event recorded after a build's list-boundary copy (one per host thread
// and device).
scn_status copy_event(hipEvent_t* out) {
  static thread_local hipEvent_t ev[64] = {};
  int dev = 0;
  SCN_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) {
    set_error("scn_rulebook_build: device %d out of range", dev);
    return SCN_ERR_HIP;
  }
  if (!ev[dev]) SCN_HIP(hipEventCreateWithFlags(&ev[dev], hipEventDisableTiming));
  *out = ev[dev];
  return SCN_OK;
}

// A second stream per device and host thread, at the default priority like
// the caller's, for build stages that do not depend on each other: fork()
// orders it after the work queued so far on st, join() orders st after it.
struct AuxStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};

scn_status aux_stream(AuxStream** out) {
  static thread_local AuxStream aux[64];
  int dev = 0;
  SCN_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) {
    set_error("scn_rulebook_build: device %d out of range", dev);
    return SCN_ERR_HIP;
  }
  AuxStream& a = aux[dev];
  if (!a.s) {
    SCN_HIP(hipStreamCreateWithFlags(&a.s, hipStreamNonBlocking));
    SCN_HIP(hipEventCreateWithFlags(&a.fork, hipEventDisableTiming));
    SCN_HIP(hipEventCreateWithFlags(&a.join, hipEventDisableTiming));
  }
  *out = &a;
  return SCN_OK;
}

scn_status fork(hipStream_t st, AuxStream* a) {
  SCN_HIP(hipEventRecord(a->fork, st));
  SCN_HIP(hipStreamWaitEvent(a->s, a->fork, 0));
  return SCN_OK;
}

scn_status join(hipStream_t st, AuxStream* a) {
  SCN_HIP(hipEventRecord(a->join, a->s));
  SCN_HIP(hipStreamWaitEvent(st, a->join, 0));
  return SCN_OK;
}

// The build of one layer, in steps:
//   check()   host only: arguments, output grid, bitmap sizes;
//   phase1()  device: mark the caller's sites (first layer only), rank them,
//             the input side (rank -> row, pair counts per tile of input
//             ranks), dilate, rank the outputs; queues the copy of the
//             flags, totals and list boundaries to the layer's read-back
//             slot, then the pair lists;
//   sized()   after the host has waited for that copy (a single build waits
//             for the copy alone, so the pair lists run meanwhile): errors,
//             a_out, the rest of the rulebook's storage;
//   phase2()  device: output sites and masks, per-tile pair ranges, the
//             output-major tables (window table of a pooling rulebook, or the
//             dense forward view and its mask sort), pooling windows;
//   finish()  the pair count.
// A layer of scn_rulebook_build_chain built from the previous layer's
// outputs learns its sites only after the first wait: its input side and
// lists move to sized() / phase2(), whose list boundaries are copied out
// (then `copied` is recorded) for a second wait.
// A layer built from the previous layer's outputs (`chained`) uses that
// layer's output rank bitmap (its H_out) as its H_in and skips marking (its
// sites are valid, distinct and in key order by construction).
struct LayerBuild {
  // inputs
  const int32_t* coords = nullptr;
  int64_t n = 0;
  int64_t grid[4] = {0, 0, 0, 0};
  int32_t f = 0, s = 0, lattice = 0;
  hipStream_t st = nullptr;
  bool chained = false;
  const uint32_t* prev_bits = nullptr;
  const uint32_t* prev_rank = nullptr;
  Readback* hb = nullptr;
  hipEvent_t ready = nullptr;  // when set: recorded once the first read-back has landed
  // derived
  bool planar = false, simplex = false;
  int K = 0;
  int64_t go4[4] = {0, 0, 0, 0};
  int64_t nw_in = 0, nw_out = 0, nsb = 0;
  GridDev gi{}, go{};
  Allocator mem;
  Temps tmp;
  // the output layer's rank bitmap (H_out) outlives the build: the rulebook
  // keeps it for a following chained build
  struct Hout {
    uint32_t *bits = nullptr, *rank = nullptr;
    hipStream_t s = nullptr;
    Allocator al;
    ~Hout() {
      if (bits) dfree(bits, s, al);
    }
  } hout;
  uint32_t *inb = nullptr, *ipref = nullptr, *sc32 = nullptr;
  // input side of the rulebook, built before the first wait (it needs only
  // the input sites): rank -> caller row and the pair ranges per tile of
  // input ranks, in one allocation the rulebook adopts
  void* inblock = nullptr;
  int32_t* perm = nullptr;
  int64_t* itile = nullptr;
  // the pair lists (capacity: inputs x windows per input) and their bounds,
  // in the same allocation
  int32_t *in_rows = nullptr, *out_rows = nullptr, *in_rank_arr = nullptr;
  int64_t* off_dev = nullptr;
  int64_t pcap = 0;
  bool early = false;  // input side and lists before the first wait
  const uint32_t *obits = nullptr, *orank = nullptr;  // this layer's H_out
  Readback* drb = nullptr;                             // device side of the read-back
  // after phase 1
  int64_t a_out = 0, nt = 0, nit = 0, pmax = 0, nfb = 0;
  bool sorted = true, pool = false, dense = false, cells = false;
  int inv_slots = 0;
  scn_rulebook* rb = nullptr;
  bool keep = false;
  uint32_t* masks = nullptr;
  uint64_t *cnt = nullptr, *sc64 = nullptr;
  int64_t ncnt = 0;
  size_t sort_bytes = 0;

  ~LayerBuild() {
    if (!keep && rb) {
      dfree(rb->block, st, rb->alloc);      // stream-ordered: after any queued kernel
      dfree(rb->hout_bits, st, rb->alloc);  // also holds hout_rank
      dfree(rb->inblock, st, rb->alloc);
      if (rb->done) (void)hipEventDestroy(rb->done);
      delete rb;
    }
    if (inblock) dfree(inblock, st, mem);  // not adopted by a rulebook
  }

  scn_status check() {
    if (n < 0 || (n > 0 && !coords) || f < 1 || s < 1 ||
        (reinterpret_cast<uintptr_t>(coords) & 15) != 0 || lattice < SCN_LATTICE_CUBIC ||
        lattice > SCN_LATTICE_TRIANGULAR) {
      set_error("scn_rulebook_build: invalid argument (n=%lld f=%d s=%d lattice=%d)",
                (long long)n, f, s, lattice);
      return SCN_ERR_INVALID;
    }
    for (int a = 0; a < 4; ++a)
      if (grid[a] < 1 || grid[a] > INT32_MAX) {
        set_error("scn_rulebook_build: grid extent %d is %lld", a, (long long)grid[a]);
        return SCN_ERR_INVALID;
      }
    planar = lattice == SCN_LATTICE_SQUARE || lattice == SCN_LATTICE_TRIANGULAR;
    simplex = lattice == SCN_LATTICE_TETRAHEDRAL || lattice == SCN_LATTICE_TRIANGULAR;
    if (planar && grid[3] != 1) {
      set_error("scn_rulebook_build: a 2D lattice needs mz = 1 (got %lld)", (long long)grid[3]);
      return SCN_ERR_INVALID;
    }
    if (simplex && (grid[2] != grid[1] || (!planar && grid[3] != grid[1]))) {
      set_error("scn_rulebook_build: a simplex grid has one size (got %lld, %lld, %lld)",
                (long long)grid[1], (long long)grid[2], (long long)grid[3]);
      return SCN_ERR_INVALID;
    }
    if (f > 3) {
      set_error("scn_rulebook_build: filter %d > 3 is not supported", f);
      return SCN_ERR_UNSUPPORTED;
    }
    if (n > INT32_MAX) {
      set_error("scn_rulebook_build: %lld sites exceed INT32_MAX", (long long)n);
      return SCN_ERR_OVERFLOW;
    }
    with_kernels(f, lattice, [&](auto k) { K = decltype(k)::K; });
    // the window's extent is f on every axis, except 1 along z on a 2D lattice
    go4[0] = grid[0];
    for (int a = 1; a < 4; ++a) {
      const int fa = (a == 3 && planar) ? 1 : f;
      go4[a] = grid[a] >= fa ? (grid[a] - fa) / s + 1 : 0;
    }
    // bitmap words of each grid; bound them (2^26 words = 2^31 sites each)
    const int64_t rw_in = ceil_div(grid[1], 32),
                  rw_out = ceil_div(std::max<int64_t>(go4[1], 1), 32);
    const double nwi_d = (double)grid[0] * grid[3] * grid[2] * rw_in;
    const double nwo_d = (double)go4[0] * go4[3] * go4[2] * rw_out;
    const double LIMW = (double)(int64_t(1) << 26);
    if (nwi_d > LIMW || nwo_d > LIMW) {
      set_error("scn_rulebook_build: grid too large for the occupancy bitmap (%.3g / %.3g words)",
                nwi_d, nwo_d);
      return SCN_ERR_UNSUPPORTED;
    }
    nw_in = (int64_t)nwi_d;
    nw_out = (int64_t)nwo_d;
    gi = GridDev{(int32_t)grid[0], (int32_t)grid[1], (int32_t)grid[2], (int32_t)grid[3],
                 (int32_t)rw_in, simplex ? 1 : 0};
    go = GridDev{(int32_t)go4[0], (int32_t)std::max<int64_t>(go4[1], 0), (int32_t)go4[2],
                 (int32_t)go4[3], (int32_t)rw_out, simplex ? 1 : 0};
    return SCN_OK;
  }

  // The rulebook's input side, which needs only the input sites: perm
  // (rank -> caller row; not for a chained layer, whose sites are in key
  // order by construction) and itile (pair ranges per tile of input ranks:
  // counts from the inputs' sites, then a scan), in one allocation the
  // rulebook adopts.  Queued before the first wait when the sites are known;
  // the kernels tolerate an input list with errors (the build then fails).
  bool in_done = false;
  AuxStream* aux = nullptr;
  // xs: the stream its kernels run on (allocations stay tagged with st)
  scn_status input_side(hipStream_t xs) {
    scn_status rc;
    nit = std::max<int64_t>(1, ceil_div(n, TILE));
    // windows per input: at most ceil(f/s) per axis of the window
    int per = 1;
    for (int a = 0; a < (planar ? 2 : 3); ++a) per *= (f + s - 1) / s;
    pcap = std::min<int64_t>((int64_t)n * std::min(per, K), INT32_MAX);
    const size_t perm_bytes = chained ? 0 : Temps::round(std::max<int64_t>(n, 1) * 4);
    const size_t list_bytes = Temps::round(std::max<int64_t>(pcap, 1) * 4);
    if ((rc = dalloc(&inblock,
                     perm_bytes + Temps::round((K * nit + 1) * 8) +
                         (chained ? 2 : 3) * list_bytes + Temps::round((K + 1) * 8),
                     st, mem)))
      return rc;
    char* cur = static_cast<char*>(inblock);
    perm = chained ? nullptr : reinterpret_cast<int32_t*>(cur);
    cur += perm_bytes;
    itile = reinterpret_cast<int64_t*>(cur);
    cur += Temps::round((K * nit + 1) * 8);
    in_rows = reinterpret_cast<int32_t*>(cur);
    cur += list_bytes;
    out_rows = reinterpret_cast<int32_t*>(cur);
    cur += list_bytes;
    // a chained layer's sites are in key order: ranks are rows
    in_rank_arr = chained ? nullptr : reinterpret_cast<int32_t*>(cur);
    cur += chained ? 0 : list_bytes;
    off_dev = reinterpret_cast<int64_t*>(cur);
    if (!chained && n > 0) {
      hipLaunchKernelGGL(perm_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, xs, coords, n, gi,
                         (const uint32_t*)inb, (const uint32_t*)ipref, perm);
      SCN_LAUNCH_CHECK();
    }
    uint64_t *icnt = nullptr, *isc = nullptr;
    if ((rc = tmp.get(&icnt, K * nit)) || (rc = tmp.get(&isc, scan_blocks(K * nit)))) return rc;
    with_kernels(f, lattice, [&](auto k) {
      k.in_tile_count(s == 1 ? 1 : (s == 2 ? 2 : 0), dim3(blocks_for(nit * TILE, 256)), xs,
                      coords, (const int32_t*)perm, n, nit, s, go, icnt);
    });
    SCN_LAUNCH_CHECK();
    if ((rc = exclusive_scan<uint64_t>(PlainLoad<uint64_t>{icnt}, K * nit, (uint64_t*)itile,
                                       (uint64_t*)itile + K * nit, isc, xs)))
      return rc;
    in_done = true;
    return SCN_OK;
  }

  // The pair lists, input-major, from the input side and this layer's H_out.
  scn_status emit_lists() {
    if (n > 0) {
      with_kernels(f, lattice, [&](auto k) {
        k.emit_in(s == 1 ? 1 : (s == 2 ? 2 : 0), dim3(blocks_for(nit * TILE, 256)), st, coords,
                  (const int32_t*)perm, n, nit, s, go, obits, orank, (const int64_t*)itile, pcap,
                  in_rows, out_rows, in_rank_arr);
      });
      SCN_LAUNCH_CHECK();
    }
    return SCN_OK;
  }

  scn_status phase1() {
    mem = current_allocator();  // every array of this build comes from it
    tmp.s = st;
    tmp.al = mem;
    hout.s = st;
    hout.al = mem;
    scn_status rc;
    nsb = std::max(scan_blocks(nw_in), scan_blocks(nw_out));
    // bits and their prefix in one block (freed through its start, bits)
    const size_t hbits_bytes = Temps::round((size_t)std::max<int64_t>(nw_out, 1) * 4);
    if ((rc = dalloc((void**)&hout.bits, hbits_bytes + Temps::round((nw_out + 1) * 4), st, mem)))
      return rc;
    hout.rank = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(hout.bits) + hbits_bytes);
    obits = hout.bits;
    orank = hout.rank;
    // a chained layer of scn_rulebook_build_chain learns its sites only after
    // the first wait; every other build has them now
    const bool in_early = !(chained && !coords);
    early = in_early;
    const int64_t nit_early = std::max<int64_t>(1, ceil_div(n, TILE));
    if ((rc = tmp.reserve((chained ? 0 : Temps::round(nw_in * 4) + Temps::round((nw_in + 1) * 4)) +
                          Temps::round(sizeof(Readback)) + Temps::round(nsb * 4) +
                          (in_early ? Temps::round(K * nit_early * 8) +
                                          Temps::round(scan_blocks(K * nit_early) * 8)
                                    : 0))))
      return rc;
    if (chained) {
      inb = const_cast<uint32_t*>(prev_bits);
      ipref = const_cast<uint32_t*>(prev_rank);
    } else {
      if ((rc = tmp.get(&inb, nw_in)) || (rc = tmp.get(&ipref, nw_in + 1))) return rc;
      SCN_HIP(hipMemsetAsync(inb, 0, std::max<int64_t>(nw_in, 1) * 4, st));
    }
    char* drb_bytes = nullptr;
    if ((rc = tmp.get(&drb_bytes, sizeof(Readback))) || (rc = tmp.get(&sc32, nsb))) return rc;
    drb = reinterpret_cast<Readback*>(drb_bytes);
    uint32_t* const flags = &drb->flags;
    SCN_HIP(hipMemsetAsync(drb, 0, sizeof(Readback), st));
    std::memset(hb, 0, sizeof(Readback));
    // phases 1-5 (1-2 only for the caller's sites)
    if (!chained) {
      if (n > 0) {
        hipLaunchKernelGGL(mark_inputs_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, st, coords,
                           n, gi, inb, flags);
        SCN_LAUNCH_CHECK();
      }
      if ((rc = exclusive_scan<uint32_t>(PopcountLoad{inb}, nw_in, ipref, ipref + nw_in, sc32,
                                         st)))
        return rc;
    }
    // the input side overlaps the host's first wait
    // the input side (it needs only the input bitmap: every output of an
    // active input is active) beside the output bitmap's dilation and scan
    if (in_early &&
        ((rc = aux_stream(&aux)) || (rc = fork(st, aux)) || (rc = input_side(aux->s))))
      return rc;
    {
      const int sm = s == 1 ? 1 : (s == 2 ? 2 : 0);
      with_kernels(f, lattice, [&](auto k) {
        k.dilate(sm, dim3(blocks_for(nw_out, 256)), st, inb, gi, hout.bits, go, (int)nw_out, s);
      });
      SCN_LAUNCH_CHECK();
    }
    if ((rc = exclusive_scan<uint32_t>(PopcountLoad{hout.bits}, nw_out, hout.rank,
                                       hout.rank + nw_out, sc32, st)))
      return rc;
    if (in_early && (rc = join(st, aux))) return rc;
    // flags, both totals and (input side known) the list boundaries in one
    // read-back; the lists are emitted after it, so a host that waits for
    // `ready` (not for the stream) sizes the rest of the build while they run
    hipLaunchKernelGGL(pack_totals_kernel, dim3(1), dim3(64), 0, st, flags, ipref + nw_in,
                       hout.rank + nw_out, in_early ? (const int64_t*)itile : nullptr, nit, K,
                       drb->off, off_dev);
    SCN_LAUNCH_CHECK();
    SCN_HIP(hipMemcpyAsync(hb, drb, sizeof(Readback), hipMemcpyDeviceToHost, st));
    if (ready) SCN_HIP(hipEventRecord(ready, st));
    if (in_early && (rc = emit_lists())) return rc;
    return SCN_OK;
  }

  scn_status sized() {
    scn_status rc;
    if (hb->flags & F_RANGE) {
      set_error("scn_rulebook_build: a site lies outside the grid (%lld,%lld,%lld,%lld)",
                (long long)grid[0], (long long)grid[1], (long long)grid[2], (long long)grid[3]);
      return SCN_ERR_RANGE;
    }
    if ((hb->flags & F_DUP) || (int64_t)hb->a_in != n) {
      set_error("scn_rulebook_build: duplicate site in the input list");
      return SCN_ERR_DUPLICATE;
    }
    a_out = hb->a_out;
    sorted = !(hb->flags & F_UNSORTED);
    if (!in_done && (rc = input_side(st))) return rc;
    // pooling tables (window rows per output, windows per input) for stride >= 2
    pool = s >= 2;
    inv_slots = pool ? (f > s ? 8 : 1) : 0;
    nt = std::max<int64_t>(1, ceil_div(a_out, TILE));
    pmax = pcap;
    if (pool && a_out * K > INT32_MAX) {
      set_error("scn_rulebook_build: %lld pooling windows exceed the supported count",
                (long long)a_out);
      return SCN_ERR_OVERFLOW;
    }
    // persistent rulebook storage in one block
    auto al = [](int64_t bytes) { return (bytes + 255) & ~int64_t(255); };
    // dense forward view for large stride-1 rulebooks (see scn_rulebook)
    dense = s == 1 && dense_forward_for(a_out, K);
    const int64_t sz_oc = al(a_out * 16), sz_ot = dense ? 0 : al((K * nt + 1) * 8),
                  sz_nbr = pool ? al(a_out * K * 4) : 0,
                  sz_inv = pool ? al(n * 4 * inv_slots) : 0,
                  sz_pmask = pool ? al(a_out * 4) : 0;
    // cell tables of 3-wide windows of stride 2 on the cubic lattice
    cells = pool && lattice == SCN_LATTICE_CUBIC && f == 3 && s == 2;
    const int64_t sz_low = cells ? al(a_out * 8 * 4) : 0,
                  sz_homeless = cells ? al(std::max<int64_t>(n, 1) * 4) + 256 : 0;
    nfb = dense ? ceil_div(a_out, DENSE_ROWS) : 0;
    const int64_t sz_fnb = al((pmax + 1) * 4), sz_fnboff = al((a_out + 1) * 4),
                  sz_fperm = al(a_out * 4), sz_fmask = al(a_out * 4);
    const int64_t total = sz_oc + sz_ot + sz_nbr + sz_inv + sz_pmask + sz_low + sz_homeless +
                          (dense ? sz_fnb + sz_fnboff + sz_fperm + sz_fmask : 0);
    rb = new scn_rulebook();
    rb->alloc = mem;
    rb->stream = st;
    if ((rc = dalloc(&rb->block, (size_t)total, st, mem))) return rc;
    char* cur = static_cast<char*>(rb->block);
    auto take = [&](int64_t bytes) {
      char* p = bytes ? cur : nullptr;
      cur += bytes;
      return p;
    };
    rb->out_coords = (int32_t*)take(sz_oc);
    rb->in_rows = in_rows;
    rb->out_rows = out_rows;
    rb->in_rank = sorted || !in_rank_arr ? in_rows : in_rank_arr;
    rb->perm = sorted ? nullptr : perm;  // identity when sorted
    rb->off_dev = off_dev;
    rb->otile = dense ? nullptr : (int64_t*)take(sz_ot);  // the dense view replaces it
    rb->itile = itile;
    rb->inblock = inblock;  // owned by rb from here (freed with it)
    inblock = nullptr;
    rb->nbr = pool ? (int32_t*)take(sz_nbr) : nullptr;
    rb->inv = pool ? (int32_t*)take(sz_inv) : nullptr;
    rb->inv_slots = inv_slots;
    rb->pmask = pool ? (uint32_t*)take(sz_pmask) : nullptr;
    rb->lowwin = cells ? (int32_t*)take(sz_low) : nullptr;
    rb->n_homeless = cells ? (int32_t*)take(256) : nullptr;
    rb->homeless = cells ? (int32_t*)take(sz_homeless - 256) : nullptr;
    rb->n_fblocks = nfb;
    rb->fnb = dense ? (int32_t*)take(sz_fnb) : nullptr;
    rb->fnb_off = dense ? (uint32_t*)take(sz_fnboff) : nullptr;
    rb->fperm = dense ? (int32_t*)take(sz_fperm) : nullptr;
    rb->fmask = dense ? (uint32_t*)take(sz_fmask) : nullptr;
    rb->f = f;
    rb->s = s;
    rb->K = K;
    rb->lattice = lattice;
    rb->hout_bits = hout.bits;
    rb->hout_rank = hout.rank;
    rb->hout_words = nw_out;
    hout.bits = hout.rank = nullptr;  // owned by rb from here (freed with it)
    for (int a = 0; a < 4; ++a) {
      rb->gin[a] = rb->gin_nd[a] = grid[a];
      rb->gout[a] = rb->gout_nd[a] = go4[a];
    }
    rb->a_in = n;
    rb->a_out = a_out;
    rb->input_sorted = sorted ? 1 : 0;
    rb->n_otiles = nt;
    rb->n_itiles = nit;

    ncnt = dense ? 0 : K * nt;  // tile counts only for the pair-list forward
    // the mask sort's scratch
    if (dense) sort_bytes = (size_t)radix_sort_words(a_out) * 4;
    // a pooling rulebook keeps its windows' masks (pmask); others use scratch
    if ((rc = tmp.reserve((pool ? 0 : Temps::round(a_out * 4)) + Temps::round(ncnt * 8) +
                          Temps::round(scan_blocks(ncnt) * 8) +
                          (dense ? Temps::round(scan_blocks(a_out) * 4) +
                                       Temps::round(sort_bytes)
                                 : 0))))
      return rc;
    if (pool) masks = rb->pmask;
    if ((!pool && (rc = tmp.get(&masks, a_out))) || (rc = tmp.get(&cnt, ncnt)) ||
        (rc = tmp.get(&sc64, scan_blocks(ncnt))))
      return rc;
    return SCN_OK;
  }

  scn_status phase2(hipEvent_t copied) {
    scn_status rc;
    const uint32_t* outb = rb->hout_bits;
    const uint32_t* opref = rb->hout_rank;
    if (!early) {
      // the lists of a layer whose sites arrived after the first wait; the
      // host waits for their boundaries
      if ((rc = emit_lists())) return rc;
      hipLaunchKernelGGL(list_offsets_kernel, dim3(1), dim3(64), 0, st, (const int64_t*)itile,
                         nit, K, off_dev);
      SCN_LAUNCH_CHECK();
      SCN_HIP(hipMemcpyAsync(hb->off, off_dev, (K + 1) * 8, hipMemcpyDeviceToHost, st));
      SCN_HIP(hipEventRecord(copied, st));
    }
    const int os_chunk = xcd_chunk(blocks_for(nw_out, 256), 64);
    if (a_out > 0) {
      with_kernels(f, lattice, [&](auto k) {
        k.out_sites(s == 1, dim3(xcd_grid(blocks_for(nw_out, 256), os_chunk)), st,
                    (const uint32_t*)inb, gi, outb, opref, go, (int)nw_out, s, rb->out_coords,
                    masks, os_chunk);
      });
      SCN_LAUNCH_CHECK();
    }
    if (!dense) {
      // pair ranges per output tile, for the pair-list forward (a rulebook
      // with the dense view forwards through it instead):
      // otile[k*nt + t] = off[k] + pairs of list k in tiles < t
      with_kernels(f, lattice, [&](auto k) {
        k.tile_count(dim3(blocks_for(nt * TILE, 256)), st, (const uint32_t*)masks, a_out, nt,
                     cnt);
      });
      SCN_LAUNCH_CHECK();
      if ((rc = exclusive_scan<uint64_t>(PlainLoad<uint64_t>{cnt}, ncnt, (uint64_t*)rb->otile,
                                         (uint64_t*)rb->otile + ncnt, sc64, st)))
        return rc;
    }
    // the mask sort (it needs only the masks) beside the neighbour lists:
    // the lists go to the second stream, which waits for the masks here, and
    // are queued first, so they start while the host still queues the sort;
    // the sort, the longer of the two, stays on the main stream, which then
    // seldom waits at the join (a wait for work still running there left the
    // device idle for about 40 us)
    const bool side_sort = dense && a_out > 0;
    uint32_t* sort_tmp = nullptr;
    if (side_sort &&
        ((rc = tmp.get(&sort_tmp, sort_bytes / 4)) || (rc = aux_stream(&aux)) ||
         (rc = fork(st, aux))))
      return rc;
    const hipStream_t ls = side_sort ? aux->s : st;  // the output-major tables' stream
    if (dense) {
      // start of each output's neighbour list: exclusive sum of mask popcounts
      uint32_t* sc_nb = nullptr;
      if ((rc = tmp.get(&sc_nb, scan_blocks(a_out))) ||
          (rc = exclusive_scan<uint32_t>(PopcountLoad{masks}, a_out, rb->fnb_off,
                                         rb->fnb_off + a_out, sc_nb, ls)))
        return rc;
    }
    if (a_out > 0 && (rb->nbr || rb->fnb)) {
      with_kernels(f, lattice, [&](auto k) {
        // LDS stages the window table or the neighbour list
        const int eo_chunk = xcd_chunk(blocks_for(nt * TILE, 256), 64);
        k.emit_out(dim3(xcd_grid(blocks_for(nt * TILE, 256), eo_chunk)),
                   rb->nbr ? (size_t)256 * K * 4 : (size_t)256 * EMIT_NB_STAGE * 4, ls,
                   (const uint32_t*)masks, (const int32_t*)rb->out_coords, a_out, s,
                   (const uint32_t*)inb, (const uint32_t*)ipref, gi, (const int32_t*)rb->perm,
                   rb->nbr, (const uint32_t*)rb->fnb_off, rb->fnb, eo_chunk);
      });
      SCN_LAUNCH_CHECK();
    }
    if (side_sort &&
        ((rc = radix_sort_pairs(masks, rb->fmask, rb->fperm, a_out, K, sort_tmp, st)) ||
         (rc = join(st, aux))))
      return rc;
    if (cells) {
      // (also zeroes the homeless count before inv_windows fills it)
      hipLaunchKernelGGL(lower_windows_kernel, dim3(blocks_for(std::max<int64_t>(a_out, 1), 256)),
                         dim3(256), 0, st, (const int32_t*)rb->out_coords, a_out, go,
                         (const uint32_t*)outb, (const uint32_t*)opref, rb->lowwin,
                         rb->n_homeless);
      SCN_LAUNCH_CHECK();
    }
    if (pool && n > 0) {
      with_kernels(f, lattice, [&](auto k) {
        k.inv_windows(inv_slots, dim3(blocks_for(n, 256)), st, coords, n, s, go, outb, opref,
                      rb->inv, rb->homeless, rb->n_homeless);
      });
      SCN_LAUNCH_CHECK();
    }
    SCN_HIP(hipEventCreateWithFlags(&rb->done, hipEventDisableTiming));
    SCN_HIP(hipEventRecord(rb->done, st));
    return SCN_OK;
  }

  scn_status finish(scn_rulebook** out) {
    rb->n_pairs = hb->off[K];
    if (rb->n_pairs > INT32_MAX || rb->n_pairs > pcap) {
      set_error("scn_rulebook_build: %lld pairs exceed the supported count",
                (long long)rb->n_pairs);
      return SCN_ERR_OVERFLOW;
    }
    for (int k = 0; k <= K; ++k) rb->off_host[k] = hb->off[k];
    keep = true;
    *out = rb;
    return SCN_OK;
  }
};

// Builds from the caller's sites, or (prev != null) from the active output
// sites of prev: then coords/n/grid/lattice are prev's output layer, whose
// rank bitmap (prev's H_out) serves as this build's H_in.
// Whether a cubic-lattice layer's occupancy bitmaps fit (at most 2^26 words
// per grid); valid arguments assumed (others are reported by check()).
bool bitmaps_fit(const int64_t* grid, int32_t f, int32_t s) {
  for (int a = 0; a < 4; ++a)
    if (grid[a] < 1 || grid[a] > INT32_MAX) return true;
  if (f < 1 || s < 1) return true;
  double words_in = (double)grid[0] * grid[2] * grid[3] * (double)ceil_div(grid[1], 32);
  int64_t go[4] = {grid[0], 0, 0, 0};
  for (int a = 1; a < 4; ++a) go[a] = grid[a] >= f ? (grid[a] - f) / s + 1 : 0;
  double words_out =
      (double)go[0] * go[2] * go[3] * (double)ceil_div(std::max<int64_t>(go[1], 1), 32);
  const double LIMW = (double)(int64_t(1) << 26);
  return words_in <= LIMW && words_out <= LIMW;
}

scn_status build(const int32_t* coords, int64_t n, const int64_t* grid, int32_t f, int32_t s,
                 int32_t lattice, hipStream_t st, scn_rulebook** out,
                 const scn_rulebook* prev = nullptr) {
  if (!out) {
    set_error("scn_rulebook_build: out is NULL");
    return SCN_ERR_INVALID;
  }
  *out = nullptr;
  if (!grid) {
    set_error("scn_rulebook_build: grid is NULL");
    return SCN_ERR_INVALID;
  }
  // past the bitmaps' reach, the cubic lattice goes to the keyed builder
  if (lattice == SCN_LATTICE_CUBIC && !bitmaps_fit(grid, f, s))
    return keyed_build(coords, n, 3, grid, f, s, st, out);
  LayerBuild L;
  L.coords = coords;
  L.n = n;
  for (int a = 0; a < 4; ++a) L.grid[a] = grid[a];
  L.f = f;
  L.s = s;
  L.lattice = lattice;
  L.st = st;
  if (prev) {
    L.chained = true;
    L.prev_bits = prev->hout_bits;
    L.prev_rank = prev->hout_rank;
  }
  scn_status rc;
  hipEvent_t copied = nullptr;
  // arguments first: no device call before they are known to be valid
  if ((rc = L.check()) || (rc = readback_slots(&L.hb)) || (rc = copy_event(&copied)))
    return rc;
  L.ready = copied;  // recorded after the read-back, ahead of the pair emission
  if ((rc = L.phase1())) return rc;
  SCN_HIP(hipEventSynchronize(copied));
  if ((rc = L.sized()) || (rc = L.phase2(copied))) return rc;
  // The build's last kernels read prev's output bitmap and sites after the
  // call returns.  prev is freed on its own stream, so that stream waits
  // for them: a free of prev after this call is then ordered after them.
  if (prev && prev->stream != st) SCN_HIP(hipStreamWaitEvent(prev->stream, L.rb->done, 0));
  if (!L.early) SCN_HIP(hipEventSynchronize(copied));
  return L.finish(out);
}

// Layers 0 .. nl-1: layer 0 from the caller's sites, layer i from the active
// outputs of layer i-1.  Phase 1 of every layer is queued before the host's
// first wait, and phase 2 of every layer before its second, so the chain
// waits twice in all.  On an error no rulebook is returned.
scn_status build_chain(const int32_t* coords, int64_t n, const int64_t* grid, int32_t lattice,
                       int32_t nl, const int32_t* filters, const int32_t* strides,
                       hipStream_t st, scn_rulebook** out) {
  if (!out || !grid || !filters || !strides || nl < 1 || nl > MAX_CHAIN) {
    set_error("scn_rulebook_build_chain: invalid argument (%d layers, at most %d)", nl,
              MAX_CHAIN);
    return SCN_ERR_INVALID;
  }
  for (int i = 0; i < nl; ++i) out[i] = nullptr;
  if (lattice == SCN_LATTICE_CUBIC && !bitmaps_fit(grid, filters[0], strides[0])) {
    // keyed builds one after the other, each from the previous one's
    // outputs, until a layer's grids fit the bitmaps: the rest of the chain
    // is then a bitmap chain (same results, faster)
    std::vector<scn_rulebook*> res(nl, nullptr);
    scn_status rc = SCN_OK;
    for (int i = 0; i < nl && rc == SCN_OK; ++i) {
      if (i == 0) {
        rc = keyed_build(coords, n, 3, grid, filters[0], strides[0], st, &res[0]);
      } else if (bitmaps_fit(res[i - 1]->gout_nd, filters[i], strides[i])) {
        rc = build_chain(res[i - 1]->out_coords, res[i - 1]->a_out, res[i - 1]->gout_nd,
                         lattice, nl - i, filters + i, strides + i, st, res.data() + i);
        break;
      } else {
        rc = keyed_build(res[i - 1]->out_coords, res[i - 1]->a_out, 3, res[i - 1]->gout_nd,
                         filters[i], strides[i], st, &res[i]);
      }
    }
    if (rc != SCN_OK) {
      for (int i = 0; i < nl; ++i) scn_rulebook_free(res[i]);
      return rc;
    }
    for (int i = 0; i < nl; ++i) out[i] = res[i];
    return SCN_OK;
  }
  std::vector<std::unique_ptr<LayerBuild>> Ls;
  Readback* hb = nullptr;
  hipEvent_t copied = nullptr;
  scn_status rc;
  for (int i = 0; i < nl; ++i) {
    Ls.emplace_back(new LayerBuild());
    LayerBuild& L = *Ls.back();
    L.f = filters[i];
    L.s = strides[i];
    L.lattice = lattice;
    L.st = st;
    if (i == 0) {
      L.coords = coords;
      L.n = n;
      for (int a = 0; a < 4; ++a) L.grid[a] = grid[a];
    } else {
      const LayerBuild& P = *Ls[i - 1];
      for (int a = 0; a < 4; ++a) {
        if (a > 0 && P.go4[a] < 1) {
          set_error("scn_rulebook_build_chain: layer %d's output grid is empty", i - 1);
          return SCN_ERR_INVALID;
        }
        L.grid[a] = P.go4[a];
      }
      L.chained = true;
      L.prev_bits = P.hout.bits;
      L.prev_rank = P.hout.rank;
    }
    if ((rc = L.check())) return rc;
    // arguments first: no device call before layer 0's are known to be valid
    if (i == 0 && ((rc = readback_slots(&hb)) || (rc = copy_event(&copied)))) return rc;
    L.hb = hb + i;
    if ((rc = L.phase1())) return rc;
  }
  SCN_HIP(hipStreamSynchronize(st));
  for (int i = 0; i < nl; ++i) {
    LayerBuild& L = *Ls[i];
    if (i > 0) {
      // this layer's sites: the previous layer's outputs
      L.n = Ls[i - 1]->a_out;
      L.coords = Ls[i - 1]->rb->out_coords;
    }
    if ((rc = L.sized()) || (rc = L.phase2(copied))) return rc;
  }
  // the last deferred layer's copy, so every layer's boundaries are known
  bool deferred = false;
  for (int i = 0; i < nl; ++i) deferred = deferred || !Ls[i]->early;
  if (deferred) SCN_HIP(hipEventSynchronize(copied));
  std::vector<scn_rulebook*> res(nl, nullptr);
  for (int i = 0; i < nl; ++i)
    if ((rc = Ls[i]->finish(&res[i]))) {
      for (int j = 0; j < i; ++j) Ls[j]->keep = false;  // freed with their builders
      return rc;
    }
  for (int i = 0; i < nl; ++i) out[i] = res[i];
  return SCN_OK;
}

}  // namespace
}  // namespace scn

extern "C" {

scn_status scn_rulebook_build(const int32_t* coords, int64_t n, const int64_t* grid,
                              int32_t filter, int32_t stride, hipStream_t stream,
                              scn_rulebook** out) {
  scn::clear_error();
  return scn::build(coords, n, grid, filter, stride, SCN_LATTICE_CUBIC, stream, out);
}

scn_status scn_rulebook_build_lattice(const int32_t* coords, int64_t n, const int64_t* grid,
                                      int32_t filter, int32_t stride, int32_t lattice,
                                      hipStream_t stream, scn_rulebook** out) {
  scn::clear_error();
  return scn::build(coords, n, grid, filter, stride, lattice, stream, out);
}

scn_status scn_rulebook_build_chain(const int32_t* coords, int64_t n, const int64_t* grid,
                                   int32_t lattice, int32_t n_layers, const int32_t* filters,
                                   const int32_t* strides, hipStream_t stream,
                                   scn_rulebook** out) {
  scn::clear_error();
  return scn::build_chain(coords, n, grid, lattice, n_layers, filters, strides, stream, out);
}

scn_status scn_rulebook_build_next(const scn_rulebook* prev, int32_t filter, int32_t stride,
                                   hipStream_t stream, scn_rulebook** out) {
  scn::clear_error();
  if (!prev || !out) {
    if (out) *out = nullptr;
    scn::set_error("scn_rulebook_build_next: NULL argument");
    return SCN_ERR_INVALID;
  }
  for (int a = 1; a <= prev->ndim; ++a)
    if (prev->gout_nd[a] < 1) {
      *out = nullptr;
      scn::set_error("scn_rulebook_build_next: the previous layer's output grid is empty");
      return SCN_ERR_INVALID;
    }
  if (scn_status rc = scn::after_build(prev, stream)) {
    *out = nullptr;
    return rc;
  }
  if (prev->keyed) {
    // 3D sites whose next grids fit the bitmaps take the bitmap builder
    // (same result); the sites, in key order, are read by kernels queued here
    if (prev->ndim == 3 && scn::bitmaps_fit(prev->gout_nd, filter, stride)) {
      scn_status rc = scn::build(prev->out_coords, prev->a_out, prev->gout_nd, filter, stride,
                                 SCN_LATTICE_CUBIC, stream, out);
      if (rc == SCN_OK && prev->stream != stream)
        rc = (hipStreamWaitEvent(prev->stream, (*out)->done, 0) == hipSuccess) ? SCN_OK
                                                                              : SCN_ERR_HIP;
      return rc;
    }
    return scn::keyed_build(prev->out_coords, prev->a_out, prev->ndim, prev->gout_nd, filter,
                            stride, stream, out);
  }
  return scn::build(prev->out_coords, prev->a_out, prev->gout, filter, stride, prev->lattice,
                    stream, out, prev);
}

scn_status scn_rulebook_get_info(const scn_rulebook* rb, scn_rulebook_info* info) {
  if (!rb || !info) {
    scn::set_error("scn_rulebook_get_info: NULL argument");
    return SCN_ERR_INVALID;
  }
  info->a_in = rb->a_in;
  info->a_out = rb->a_out;
  info->n_pairs = rb->n_pairs;
  info->K = rb->K;
  info->filter = rb->f;
  info->stride = rb->s;
  info->input_sorted = rb->input_sorted;
  info->lattice = rb->lattice;
  info->dense_view = rb->fnb ? 1 : 0;
  for (int a = 0; a < 4; ++a) {
    info->in_grid[a] = rb->gin[a];
    info->out_grid[a] = rb->gout[a];
  }
  info->ndim = rb->ndim;
  info->keyed = rb->keyed;
  for (int a = 0; a < 5; ++a) {
    info->in_grid_nd[a] = a <= rb->ndim ? rb->gin_nd[a] : 0;
    info->out_grid_nd[a] = a <= rb->ndim ? rb->gout_nd[a] : 0;
  }
  return SCN_OK;
}

const int32_t* scn_rulebook_out_coords(const scn_rulebook* rb) { return rb ? rb->out_coords : nullptr; }
const int32_t* scn_rulebook_in_rows(const scn_rulebook* rb) { return rb ? rb->in_rows : nullptr; }
const int32_t* scn_rulebook_out_rows(const scn_rulebook* rb) { return rb ? rb->out_rows : nullptr; }
const int64_t* scn_rulebook_offsets(const scn_rulebook* rb) { return rb ? rb->off_host : nullptr; }

scn_status scn_rulebook_export(const scn_rulebook* rb, int32_t* out_coords, int32_t* in_rows,
                               int32_t* out_rows, hipStream_t stream) {
  scn::clear_error();
  if (!rb) {
    scn::set_error("scn_rulebook_export: rb is NULL");
    return SCN_ERR_INVALID;
  }
  if (scn_status rc = scn::after_build(rb, stream)) return rc;
  if (out_coords && rb->a_out > 0)
    SCN_HIP(hipMemcpyAsync(out_coords, rb->out_coords, rb->a_out * (rb->ndim + 1) * 4,
                           hipMemcpyDeviceToDevice, stream));
  if (in_rows && rb->n_pairs > 0)
    SCN_HIP(hipMemcpyAsync(in_rows, rb->in_rows, rb->n_pairs * 4, hipMemcpyDeviceToDevice, stream));
  if (out_rows && rb->n_pairs > 0)
    SCN_HIP(hipMemcpyAsync(out_rows, rb->out_rows, rb->n_pairs * 4, hipMemcpyDeviceToDevice,
                           stream));
  return SCN_OK;
}

void scn_rulebook_free(scn_rulebook* rb) {
  if (!rb) return;
  scn::dfree(rb->block, rb->stream, rb->alloc);
  scn::dfree(rb->hout_bits, rb->stream, rb->alloc);  // also holds hout_rank
  scn::dfree(rb->inblock, rb->stream, rb->alloc);
  if (rb->done) (void)hipEventDestroy(rb->done);
  delete rb;
}

}  // extern "C"
