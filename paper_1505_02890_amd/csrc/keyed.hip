// Rulebooks from sorted site keys and open-addressing hash tables (section
// 1.3, step 1: the map H_in from active locations to rows of the feature
// matrix, the active output sites numbered in H_out, and the rules that say
// which input row feeds which output row at each filter offset).
//
// The main builder (rulebook.hip) keeps one occupancy bit per grid site.
// Past 2^26 bitmap words per grid, and for sites with other than three
// coordinates (the hypercubic lattice in 1 to 4 dimensions, section 1.2),
// this builder takes over.  It produces the same arrays in the same order:
// outputs numbered in ascending key order, and each offset's pairs in
// ascending input key order (a fixed offset moves every input by the same
// amount, so its pairs are then in ascending output order too).
//
//   keys       one thread per site: the key ((b*m_D + x_D)*m_{D-1} + ...)*m_1
//              + x_1 (x_1 fastest, as the 3D key ((b*mz + z)*my + y)*mx + x)
//              and the range check
//   sort       stable radix sort of (key, row): rank -> caller row
//   ranked     duplicates (equal neighbouring keys), whether the caller's
//              rows were in key order, the sites' coordinates by rank
//   H_in       open-addressing table key -> rank, linear probing, capacity a
//              power of two at least twice the sites
//   outputs    one thread per (input, offset) candidate output site.  A wave
//              takes the 64 inputs of one tile of ranks at one offset, so its
//              candidates are distinct and go straight to an insert into
//              H_out (a read, then an atomicCAS if the slot is empty); a
//              ballot over the wave's valid candidates gives the tile's pair
//              count at that offset, and a scan of those counts each tile's
//              place in the pair lists (the per-input-tile ranges)
//   compact    the occupied slots of H_out, in slot order, by a prefix scan
//   -- one host wait: the output count, the list boundaries, the flags --
//   sort       the output keys, into canonical order; rank written into H_out
//   pairs      per (offset, input tile) one wave: the ballot again places
//              each pair; output rows are looked up in H_out
//   tiles      per (offset, tile of output rows): a binary search in the list
//   pooling    window tables from H_in lookups, each input's windows from
//              H_out lookups
#include <algorithm>
#include <cstring>

#include "scan.h"
#include "scn_internal.h"
#include "sort.h"

namespace scn {
namespace {

constexpr uint64_t HK_EMPTY = ~uint64_t(0);
// Probe bound of the output table's inserts.  The table is first sized from
// an estimate of the output count; an insert that finds no place within the
// bound (or a table more than half full) sends the build back to insert into
// a table sized for every candidate being distinct.
constexpr int KD_PROBES = 256;
enum : uint32_t { KF_RANGE = 1, KF_DUP = 2, KF_UNSORTED = 4 };

struct KGeo {
  int32_t D, f, s, K;
  int32_t B, pad;
  int32_t m[KD_MAX];     // input extents, axis 0 fastest in the key
  int32_t mo[KD_MAX];    // output extents floor((m - f) / s) + 1
  int32_t fpow[KD_MAX];  // f^a: offset k = sum_a k_a f^a
};

// The 64-bit finaliser of MurmurHash3 (Appleby): a slot spread for the keys.
__device__ inline uint64_t hmix(uint64_t k) {
  k ^= k >> 33;
  k *= 0xff51afd7ed558ccdull;
  k ^= k >> 33;
  k *= 0xc4ceb9fe1a85ec53ull;
  k ^= k >> 33;
  return k;
}

__device__ inline uint64_t kd_key(int64_t b, const int32_t (&x)[KD_MAX], const int32_t* m, int D) {
  uint64_t k = (uint64_t)b;
#pragma unroll
  for (int a = KD_MAX - 1; a >= 0; --a)
    if (a < D) k = k * (uint64_t)m[a] + (uint64_t)x[a];
  return k;
}

// A slot of a hash table: the key (HK_EMPTY when free) and the rank stored
// with it, side by side, so a probe that finds its key reads one 16-byte
// piece of memory.
struct alignas(16) HSlot {
  uint64_t key;
  int32_t val;
  int32_t pad;
};

// The rank stored with key k, or -1 when k is absent.  The table is at most
// half full, so the probe meets an empty slot.
__device__ inline int32_t h_find(const HSlot* __restrict__ h, uint64_t mask, uint64_t k) {
  for (uint64_t i = hmix(k) & mask;; i = (i + 1) & mask) {
    const uint4 v = *reinterpret_cast<const uint4*>(h + i);
    const uint64_t t = ((uint64_t)v.y << 32) | v.x;
    if (t == k) return (int32_t)v.z;
    if (t == HK_EMPTY) return -1;
  }
}

// The output site that input x (batch b) feeds at offset k, if any: o_a =
// (x_a - k_a) / s when that divides and lies in the output grid.
__device__ inline bool kd_out_site(int32_t b, int4 xv, int k, const KGeo& g, uint64_t* key) {
  const int32_t x[KD_MAX] = {xv.x, xv.y, xv.z, xv.w};
  int32_t o[KD_MAX] = {0, 0, 0, 0};
  bool ok = true;
#pragma unroll
  for (int a = 0; a < KD_MAX; ++a)
    if (a < g.D) {
      const int32_t d = x[a] - (k / g.fpow[a]) % g.f;
      ok = ok && d >= 0 && d % g.s == 0 && d / g.s < g.mo[a];
      o[a] = d / g.s;
    }
  if (ok) *key = kd_key(b, o, g.mo, g.D);
  return ok;
}

// wave-wide OR of f, at most one atomic per wave: the word is read first, so
// the waves of an unsorted list (each of which raises the same flag) do not
// all queue atomics on one address
__device__ inline void flag_or(uint32_t* flags, uint32_t f) {
  uint32_t all = 0;
#pragma unroll
  for (int bit = 0; bit < 3; ++bit)
    if (__ballot((f >> bit) & 1u)) all |= 1u << bit;
  if (all && (threadIdx.x & 63) == 0 &&
      (__hip_atomic_load(flags, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & all) != all)
    atomicOr(flags, all);
}

// one thread per site in caller order: its key and the range check
__global__ void __launch_bounds__(256) kd_keys_kernel(const int32_t* __restrict__ coords, int64_t n,
                                                      KGeo g, uint64_t* __restrict__ keys,
                                                      uint32_t* __restrict__ flags) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint32_t f = 0;
  if (i < n) {
    const int32_t* c = coords + i * (g.D + 1);
    const int32_t b = c[0];
    int32_t x[KD_MAX] = {0, 0, 0, 0};
    bool bad = b < 0 || b >= g.B;
#pragma unroll
    for (int a = 0; a < KD_MAX; ++a)
      if (a < g.D) {
        x[a] = c[1 + a];
        bad = bad || x[a] < 0 || x[a] >= g.m[a];
      }
    keys[i] = bad ? 0 : kd_key(b, x, g.m, g.D);
    if (bad) f = KF_RANGE;
  }
  flag_or(flags, f);
}

// one thread per rank: the site's batch and coordinates by rank, duplicates,
// and whether rank order is the caller's row order
__global__ void __launch_bounds__(256) kd_ranked_kernel(const int32_t* __restrict__ coords,
                                                        const uint64_t* __restrict__ skeys,
                                                        const int32_t* __restrict__ perm,
                                                        int64_t n, KGeo g,
                                                        int32_t* __restrict__ sb,
                                                        int4* __restrict__ sx,
                                                        uint32_t* __restrict__ flags) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint32_t f = 0;
  if (r < n) {
    const int64_t row = perm[r];
    const int32_t* c = coords + row * (g.D + 1);
    int32_t x[KD_MAX] = {0, 0, 0, 0};
#pragma unroll
    for (int a = 0; a < KD_MAX; ++a)
      if (a < g.D) x[a] = c[1 + a];
    sb[r] = c[0];
    sx[r] = make_int4(x[0], x[1], x[2], x[3]);
    if (r > 0 && skeys[r] == skeys[r - 1]) f |= KF_DUP;
    if (row != r) f |= KF_UNSORTED;
  }
  flag_or(flags, f);
}

// H_in: key -> rank, one thread per rank
__global__ void __launch_bounds__(256) kd_insert_kernel(const uint64_t* __restrict__ skeys,
                                                        int64_t n, HSlot* __restrict__ h,
                                                        uint64_t mask) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n) return;
  const uint64_t k = skeys[r];
  for (uint64_t i = hmix(k) & mask;; i = (i + 1) & mask) {
    const uint64_t prev = atomicCAS(reinterpret_cast<unsigned long long*>(&h[i].key),
                                    (unsigned long long)HK_EMPTY, (unsigned long long)k);
    if (prev == HK_EMPTY || prev == k) {
      h[i].val = (int32_t)r;
      return;
    }
  }
}

// Candidate output sites: input rank r = 64 blockIdx.x + lane (one wave per
// tile of TILE = 64 ranks), offset k = blockIdx.y.  cnt[k*nit + tile] = the
// tile's pairs at offset k; *full set when an insert found no place within
// KD_PROBES slots.  Most candidates repeat a key already in the table (a
// window holds several active inputs), so a slot is read before any atomic:
// a slot changes once, from empty to its key, so a stale read can only show
// it empty, and the atomicCAS then decides.
__global__ void __launch_bounds__(64) kd_candidates_kernel(
    const int32_t* __restrict__ sb, const int4* __restrict__ sx, int64_t n, KGeo g, int64_t nit,
    HSlot* __restrict__ h, uint64_t mask, uint64_t* __restrict__ cnt,
    uint32_t* __restrict__ full) {
  const int64_t r = (int64_t)blockIdx.x * 64 + threadIdx.x;
  const int k = blockIdx.y;
  uint64_t key = 0;
  const bool valid = r < n && kd_out_site(sb[r], sx[r], k, g, &key);
  bool placed = !valid;
  if (valid) {
    uint64_t i = hmix(key) & mask;
    for (int t = 0; t < KD_PROBES; ++t, i = (i + 1) & mask) {
      const uint64_t cur = h[i].key;
      if (cur == key) {
        placed = true;
        break;
      }
      if (cur != HK_EMPTY) continue;
      const uint64_t prev = atomicCAS(reinterpret_cast<unsigned long long*>(&h[i].key),
                                      (unsigned long long)HK_EMPTY, (unsigned long long)key);
      if (prev == HK_EMPTY || prev == key) {
        placed = true;
        break;
      }
    }
  }
  const uint64_t vb = __ballot(valid);
  const bool lost = __ballot(!placed) != 0;
  if (threadIdx.x == 0) {
    cnt[(int64_t)k * nit + blockIdx.x] = (uint64_t)__popcll(vb);
    if (lost) atomicOr(full, 1u);
  }
}

// Occupied slots of the output table per chunk of SCAN_BLOCK slots
__global__ void __launch_bounds__(SCAN_THREADS) kd_occupied_kernel(const HSlot* __restrict__ h,
                                                                   uint64_t cap,
                                                                   uint32_t* __restrict__ bcnt) {
  const uint64_t base = (uint64_t)blockIdx.x * SCAN_BLOCK;
  uint32_t c = 0;
  for (int j = threadIdx.x; j < SCAN_BLOCK; j += SCAN_THREADS)
    c += (base + j < cap && h[base + j].key != HK_EMPTY) ? 1u : 0u;
  uint32_t all;
  block_exclusive_scan<uint32_t>(c, &all);
  if (threadIdx.x == 0) bcnt[blockIdx.x] = all;
}

// The occupied slots' keys to list[], in slot order: chunk b starts at
// bpre[b]; inside it, ballots place the wave's keys
__global__ void __launch_bounds__(SCAN_THREADS) kd_compact_kernel(const HSlot* __restrict__ h,
                                                                  uint64_t cap,
                                                                  const uint32_t* __restrict__ bpre,
                                                                  uint64_t* __restrict__ list) {
  __shared__ uint32_t wsum[SCAN_THREADS / 64];
  const uint64_t base = (uint64_t)blockIdx.x * SCAN_BLOCK;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t out = bpre[blockIdx.x];
  for (int j0 = 0; j0 < SCAN_BLOCK; j0 += SCAN_THREADS) {
    const uint64_t i = base + j0 + threadIdx.x;
    const uint64_t key = i < cap ? h[i].key : HK_EMPTY;
    const bool occ = key != HK_EMPTY;
    const uint64_t bal = __ballot(occ);
    if (lane == 0) wsum[w] = (uint32_t)__popcll(bal);
    __syncthreads();
    uint32_t before = 0, all = 0;
#pragma unroll
    for (int v = 0; v < SCAN_THREADS / 64; ++v) {
      if (v < w) before += wsum[v];
      all += wsum[v];
    }
    if (occ)
      list[out + before + __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                    __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u))] =
          key;
    out += all;
    __syncthreads();
  }
}

// rank i of the sorted output keys: its row into H_out and its coordinates
__global__ void __launch_bounds__(256) kd_assign_kernel(const uint64_t* __restrict__ okeys,
                                                        int64_t a_out, KGeo g,
                                                        HSlot* __restrict__ h, uint64_t mask,
                                                        int32_t* __restrict__ out_coords) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a_out) return;
  uint64_t key = okeys[i];
  for (uint64_t j = hmix(key) & mask;; j = (j + 1) & mask)
    if (h[j].key == key) {
      h[j].val = (int32_t)i;
      break;
    }
  int32_t* c = out_coords + i * (g.D + 1);
#pragma unroll
  for (int a = 0; a < KD_MAX; ++a)
    if (a < g.D) {
      c[1 + a] = (int32_t)(key % (uint64_t)g.mo[a]);
      key /= (uint64_t)g.mo[a];
    }
  c[0] = (int32_t)key;
}

// The pairs: list k holds, in input rank order, (caller row, output row) of
// every input with an output at offset k.  itile[k*nit + t] = place of the
// first pair of list k from input tile t.
__global__ void __launch_bounds__(64) kd_emit_kernel(
    const int32_t* __restrict__ sb, const int4* __restrict__ sx, int64_t n, KGeo g, int64_t nit,
    const uint64_t* __restrict__ itile, const int32_t* __restrict__ perm,
    const HSlot* __restrict__ h, uint64_t mask,
    int32_t* __restrict__ in_rows, int32_t* __restrict__ out_rows,
    int32_t* __restrict__ in_rank) {
  const int64_t r = (int64_t)blockIdx.x * 64 + threadIdx.x;
  const int k = blockIdx.y;
  uint64_t key = 0;
  const bool valid = r < n && kd_out_site(sb[r], sx[r], k, g, &key);
  const uint64_t vb = __ballot(valid);
  if (!valid) return;
  const uint64_t pos = itile[(int64_t)k * nit + blockIdx.x] +
                       __builtin_amdgcn_mbcnt_hi((uint32_t)(vb >> 32),
                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)vb, 0u));
  // streaming stores, as for the bitmap builder's lists
  __builtin_nontemporal_store(perm ? perm[r] : (int32_t)r, in_rows + pos);
  __builtin_nontemporal_store(h_find(h, mask, key), out_rows + pos);
  if (in_rank) __builtin_nontemporal_store((int32_t)r, in_rank + pos);
}

// list boundaries off[k] = itile[k*nit] (off[K] = the pair count)
__global__ void kd_offsets_kernel(const uint64_t* __restrict__ itile, int64_t nit, int K,
                                  int64_t* __restrict__ off) {
  const int k = threadIdx.x;
  if (k <= K) off[k] = (int64_t)itile[(int64_t)k * nit];
}

// the output count: the compaction's total
__global__ void kd_total_kernel(const uint32_t* __restrict__ bpre, int64_t nb,
                                const uint32_t* __restrict__ bcnt, unsigned long long* out) {
  *out = nb > 0 ? (unsigned long long)bpre[nb - 1] + bcnt[nb - 1] : 0ull;
}

// otile[k*nt + t] = place of the first pair of list k whose output row is at
// least t*TILE (the list is in output order); otile[K*nt] = the pair count
__global__ void __launch_bounds__(256) kd_otile_kernel(const int32_t* __restrict__ out_rows,
                                                       const int64_t* __restrict__ off, int K,
                                                       int64_t nt, int64_t* __restrict__ otile) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) otile[(int64_t)K * nt] = off[K];
  if (i >= (int64_t)K * nt) return;
  const int k = (int)(i / nt);
  const int64_t t = i - (int64_t)k * nt;
  int64_t lo = off[k], hi = off[k + 1];
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (out_rows[mid] < t * TILE)
      lo = mid + 1;
    else
      hi = mid;
  }
  otile[i] = lo;
}

// Pooling window table: nbr[o*K + k] = caller row of the input at s*o + k
// (offset k = sum_a k_a f^a) or -1; pmask[o] bit k = that input is active.
// A window per 32 lanes (lane k < K looks up offset k, K <= 27): the K hash
// lookups of a window run side by side, its row of the table is one
// contiguous store, and its mask is a ballot.
__global__ void __launch_bounds__(256) kd_windows_kernel(const int32_t* __restrict__ out_coords,
                                                         int64_t a_out, KGeo g,
                                                         const HSlot* __restrict__ h,
                                                         uint64_t mask,
                                                         const int32_t* __restrict__ perm,
                                                         int32_t* __restrict__ nbr,
                                                         uint32_t* __restrict__ pmask) {
  const int64_t o = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 5;
  const int k = threadIdx.x & 31;
  const bool live = o < a_out && k < g.K;
  int32_t row = -1;
  if (live) {
    const int32_t* c = out_coords + o * (g.D + 1);
    int32_t x[KD_MAX] = {0, 0, 0, 0};
#pragma unroll
    for (int a = 0; a < KD_MAX; ++a)
      if (a < g.D) x[a] = g.s * c[1 + a] + (k / g.fpow[a]) % g.f;
    const int32_t rank = h_find(h, mask, kd_key(c[0], x, g.m, g.D));
    row = rank < 0 ? -1 : (perm ? perm[rank] : rank);
    nbr[o * g.K + k] = row;
  }
  const uint64_t bal = __ballot(row >= 0);
  if (live && k == 0) pmask[o] = (uint32_t)(bal >> (threadIdx.x & 32));
}

// Each input's windows: slot j (bit a: the window one step down along axis a,
// used when f > s) of input rank r is window o_a = x_a / s - j_a at offset
// k_a = x_a - s*o_a < f; inv[row*slots + j] = (output row)*K + k or -1.  A
// thread per (input, slot), so an input's lookups run side by side.
__global__ void __launch_bounds__(256) kd_inv_kernel(const int32_t* __restrict__ sb,
                                                     const int4* __restrict__ sx, int64_t n,
                                                     KGeo g, int slots,
                                                     const int32_t* __restrict__ perm,
                                                     const HSlot* __restrict__ h, uint64_t mask,
                                                     int32_t* __restrict__ inv) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t r = i / slots;
  const int j = (int)(i - r * slots);
  if (r >= n) return;
  const int4 xv = sx[r];
  const int32_t x[KD_MAX] = {xv.x, xv.y, xv.z, xv.w};
  const int64_t row = perm ? perm[r] : r;
  int32_t o[KD_MAX] = {0, 0, 0, 0};
  int kidx = 0;
  bool ok = true;
#pragma unroll
  for (int a = 0; a < KD_MAX; ++a)
    if (a < g.D) {
      o[a] = x[a] / g.s - ((j >> a) & 1);
      const int32_t ka = x[a] - g.s * o[a];
      ok = ok && o[a] >= 0 && o[a] < g.mo[a] && ka < g.f;
      kidx += ka * g.fpow[a];
    }
  int32_t v = -1;
  if (ok) {
    const int32_t orow = h_find(h, mask, kd_key(sb[r], o, g.mo, g.D));
    if (orow >= 0) v = (int32_t)((int64_t)orow * g.K + kidx);
  }
  inv[row * slots + j] = v;
}

inline unsigned kd_blocks(int64_t n, int t) {
  return (unsigned)std::max<int64_t>(1, ceil_div(n, t));
}

inline uint64_t pow2_at_least(uint64_t v) {
  uint64_t p = 1;
  while (p < v) p <<= 1;
  return p;
}

inline int bits_for(uint64_t v) {  // bits of the largest key below v
  int b = 1;
  while (b < 64 && (uint64_t(1) << b) < v) ++b;
  return b;
}

// Read-back of the host wait (pinned, one per host thread).
struct KReadback {
  uint32_t flags, full;
  unsigned long long a_out;
  int64_t off[MAX_K + 1];
};

scn_status kd_readback(KReadback** out) {
  static thread_local KReadback* hb = nullptr;
  if (!hb) SCN_HIP(hipHostMalloc((void**)&hb, sizeof(KReadback), hipHostMallocDefault));
  *out = hb;
  return SCN_OK;
}

// Device temporaries of one build, freed on its stream (in stream order).
struct KTemps {
  static constexpr int CAP = 32;
  hipStream_t st;
  Allocator al;
  void* p[CAP] = {nullptr};
  int n = 0;
  KTemps(hipStream_t s, const Allocator& a) : st(s), al(a) {}
  ~KTemps() {
    for (int i = 0; i < n; ++i) dfree(p[i], st, al);
  }
  template <typename T>
  scn_status get(T** out, int64_t count) {
    if (n >= CAP) {
      set_error("scn_rulebook_build_nd: too many temporary blocks");
      return SCN_ERR_NOMEM;
    }
    void* q = nullptr;
    scn_status rc = dalloc(&q, (size_t)std::max<int64_t>(count, 1) * sizeof(T), st, al);
    if (rc) return rc;
    p[n++] = q;
    *out = static_cast<T*>(q);
    return SCN_OK;
  }
};

}  // namespace

scn_status keyed_build(const int32_t* coords, int64_t n, int D, const int64_t* grid, int f, int s,
                       hipStream_t st, scn_rulebook** out) {
  if (!out) {
    set_error("scn_rulebook_build_nd: out is NULL");
    return SCN_ERR_INVALID;
  }
  *out = nullptr;
  if (D < 1 || D > KD_MAX || !grid || n < 0 || (n > 0 && !coords) || f < 1 || s < 1) {
    set_error("scn_rulebook_build_nd: invalid argument (ndim %d, filter %d, stride %d, n %lld)",
              D, f, s, (long long)n);
    return SCN_ERR_INVALID;
  }
  if (n > 0 && (reinterpret_cast<uintptr_t>(coords) & 3)) {
    set_error("scn_rulebook_build_nd: coords must be 4-byte aligned");
    return SCN_ERR_INVALID;
  }
  if (n > INT32_MAX) {
    set_error("scn_rulebook_build_nd: %lld sites exceed INT32_MAX", (long long)n);
    return SCN_ERR_OVERFLOW;
  }
  KGeo g{};
  g.D = D;
  g.f = f;
  g.s = s;
  g.B = 0;
  int64_t K = 1;
  for (int a = 0; a < D; ++a) K *= f;
  if (f > 3 || K > MAX_K) {
    set_error("scn_rulebook_build_nd: a filter of %d^%d = %lld offsets (at most %d)", f, D,
              (long long)K, MAX_K);
    return SCN_ERR_UNSUPPORTED;
  }
  g.K = (int32_t)K;
  if (grid[0] < 1 || grid[0] > INT32_MAX) {
    set_error("scn_rulebook_build_nd: batch extent %lld", (long long)grid[0]);
    return SCN_ERR_INVALID;
  }
  g.B = (int32_t)grid[0];
  // key ranges: B * prod m_a sites in, B * prod mo_a out, below 2^63
  uint64_t sites_in = (uint64_t)grid[0], sites_out = (uint64_t)grid[0];
  bool too_many = false;
  int64_t fp = 1;
  for (int a = 0; a < KD_MAX; ++a) {
    g.m[a] = g.mo[a] = 1;
    g.fpow[a] = (int32_t)fp;
    if (a < D) fp *= f;
  }
  for (int a = 0; a < D; ++a) {
    const int64_t m = grid[1 + a];
    if (m < 1 || m > INT32_MAX) {
      set_error("scn_rulebook_build_nd: grid extent %d is %lld", a, (long long)m);
      return SCN_ERR_INVALID;
    }
    g.m[a] = (int32_t)m;
    g.mo[a] = m >= f ? (int32_t)((m - f) / s + 1) : 0;
    too_many = too_many || sites_in > (uint64_t(1) << 63) / (uint64_t)m;
    if (!too_many) sites_in *= (uint64_t)m;
    sites_out *= (uint64_t)g.mo[a];  // at most sites_in
  }
  if (too_many || sites_in > (uint64_t(1) << 63)) {
    set_error("scn_rulebook_build_nd: the grid's sites do not fit a 63-bit key");
    return SCN_ERR_OVERFLOW;
  }
  // pooling tables for stride >= 2; windows wider than their stride (up to
  // twice it: f <= 3 <= 2s) only on 3D sites, whose inputs have 8 window slots
  const bool pool = s >= 2 && (f <= s || D == 3);
  const int slots = pool ? (f > s ? 8 : 1) : 0;
  const Allocator mem = current_allocator();
  KTemps tmp(st, mem);
  KReadback* hb = nullptr;
  scn_status rc;
  if ((rc = kd_readback(&hb))) return rc;

  const uint64_t cap_in = pow2_at_least(2 * (uint64_t)std::max<int64_t>(n, 1));
  // unique outputs: at most the output grid's sites, and per input at most
  // ceil(f/s) windows along each axis
  uint64_t per_in = 1;
  for (int a = 0; a < D; ++a) per_in *= (uint64_t)ceil_div(f, s);
  const uint64_t ucap = std::max<uint64_t>(
      1, std::min<uint64_t>((uint64_t)std::max<int64_t>(n, 1) * per_in, sites_out));
  // the output table: first sized for 8 outputs per input (a surface under a
  // 3x3x3 filter gives about 4.4), at most for every candidate distinct
  const uint64_t cap_full = pow2_at_least(2 * ucap);
  uint64_t cap_out = std::min(cap_full, pow2_at_least(2 * std::min<uint64_t>(
                                            ucap, 8 * (uint64_t)std::max<int64_t>(n, 1))));
  const int64_t nit = std::max<int64_t>(1, ceil_div(n, TILE));
  HSlot *h_in = nullptr, *h_out = nullptr;
  uint64_t *keys = nullptr, *skeys = nullptr,
           *list = nullptr, *cnt = nullptr, *scan_tmp = nullptr;
  int32_t* sb = nullptr;
  int4* sx = nullptr;
  uint32_t *flags = nullptr, *sort_tmp = nullptr, *bcnt = nullptr, *bpre = nullptr,
           *bscan = nullptr;
  int64_t* off_tmp = nullptr;
  unsigned long long* aout_dev = nullptr;
  const int bits_in = bits_for(sites_in);
  if ((rc = tmp.get(&keys, n)) || (rc = tmp.get(&skeys, n)) || (rc = tmp.get(&sb, n)) ||
      (rc = tmp.get(&sx, n)) || (rc = tmp.get(&h_in, (int64_t)cap_in)) ||
      (rc = tmp.get(&list, (int64_t)ucap)) ||
      (rc = tmp.get(&flags, 64)) || (rc = tmp.get(&off_tmp, MAX_K + 1)) ||
      (rc = tmp.get(&aout_dev, 1)) || (rc = tmp.get(&cnt, K * nit)) ||
      (rc = tmp.get(&scan_tmp, scan_blocks(K * nit))) ||
      (rc = tmp.get(&sort_tmp, radix_sort_words<uint64_t>(n))))
    return rc;
  // The input block, adopted by the rulebook: rank -> caller row (perm, used
  // when the rows were unsorted) and the per-input-tile pair ranges (itile,
  // K*nit + 1 entries: the scan of the candidates' tile counts).
  const size_t perm_bytes = (size_t)((std::max<int64_t>(n, 1) * 4 + 255) & ~int64_t(255));
  void* in_block = nullptr;
  if ((rc = dalloc(&in_block, perm_bytes + (size_t)(K * nit + 1) * 8, st, mem))) return rc;
  int32_t* perm = static_cast<int32_t*>(in_block);
  uint64_t* itile = reinterpret_cast<uint64_t*>(static_cast<char*>(in_block) + perm_bytes);
  struct BlockGuard {
    void*& p;
    hipStream_t st;
    Allocator al;
    ~BlockGuard() {
      if (p) dfree(p, st, al);
    }
  } in_guard{in_block, st, mem};

  SCN_HIP(hipMemsetAsync(flags, 0, 8, st));
  SCN_HIP(hipMemsetAsync(h_in, 0xFF, cap_in * sizeof(HSlot), st));
  if (n > 0) {
    hipLaunchKernelGGL(kd_keys_kernel, dim3(kd_blocks(n, 256)), dim3(256), 0, st, coords, n, g,
                       keys, flags);
    SCN_LAUNCH_CHECK();
    if ((rc = radix_sort_pairs<uint64_t>(keys, skeys, perm, n, bits_in, sort_tmp, st))) return rc;
    hipLaunchKernelGGL(kd_ranked_kernel, dim3(kd_blocks(n, 256)), dim3(256), 0, st, coords,
                       (const uint64_t*)skeys, (const int32_t*)perm, n, g, sb, sx, flags);
    SCN_LAUNCH_CHECK();
    hipLaunchKernelGGL(kd_insert_kernel, dim3(kd_blocks(n, 256)), dim3(256), 0, st,
                       (const uint64_t*)skeys, n, h_in, cap_in - 1);
    SCN_LAUNCH_CHECK();
  } else {
    SCN_HIP(hipMemsetAsync(cnt, 0, K * nit * 8, st));
  }
  // the output table: the candidates' inserts, the tile counts and their
  // scan, the compaction of the occupied slots and the read-back; again with
  // the largest table when the first one overflowed
  auto outputs = [&]() -> scn_status {
    scn_status rc2;
    const int64_t nb = (int64_t)ceil_div((int64_t)cap_out, SCAN_BLOCK);
    if ((rc2 = tmp.get(&h_out, (int64_t)cap_out)) || (rc2 = tmp.get(&bcnt, nb)) ||
        (rc2 = tmp.get(&bpre, nb + 1)) || (rc2 = tmp.get(&bscan, scan_blocks(nb))))
      return rc2;
    SCN_HIP(hipMemsetAsync(flags + 1, 0, 4, st));
    SCN_HIP(hipMemsetAsync(h_out, 0xFF, cap_out * sizeof(HSlot), st));
    if (n > 0) {
      hipLaunchKernelGGL(kd_candidates_kernel, dim3((unsigned)nit, (unsigned)K), dim3(64), 0, st,
                         (const int32_t*)sb, (const int4*)sx, n, g, nit, h_out, cap_out - 1, cnt,
                         flags + 1);
      SCN_LAUNCH_CHECK();
    }
    if ((rc2 = exclusive_scan<uint64_t>(PlainLoad<uint64_t>{cnt}, K * nit, itile,
                                        itile + K * nit, scan_tmp, st)))
      return rc2;
    hipLaunchKernelGGL(kd_offsets_kernel, dim3(1), dim3(64), 0, st, (const uint64_t*)itile, nit,
                       (int)K, off_tmp);
    SCN_LAUNCH_CHECK();
    hipLaunchKernelGGL(kd_occupied_kernel, dim3((unsigned)nb), dim3(SCAN_THREADS), 0, st,
                       (const HSlot*)h_out, cap_out, bcnt);
    SCN_LAUNCH_CHECK();
    if ((rc2 = exclusive_scan<uint32_t>(PlainLoad<uint32_t>{bcnt}, nb, bpre, bpre + nb, bscan,
                                        st)))
      return rc2;
    hipLaunchKernelGGL(kd_compact_kernel, dim3((unsigned)nb), dim3(SCAN_THREADS), 0, st,
                       (const HSlot*)h_out, cap_out, (const uint32_t*)bpre, list);
    SCN_LAUNCH_CHECK();
    hipLaunchKernelGGL(kd_total_kernel, dim3(1), dim3(1), 0, st, (const uint32_t*)bpre, nb,
                       (const uint32_t*)bcnt, aout_dev);
    SCN_LAUNCH_CHECK();
    SCN_HIP(hipMemcpyAsync(&hb->flags, flags, 8, hipMemcpyDeviceToHost, st));
    SCN_HIP(hipMemcpyAsync(&hb->a_out, aout_dev, 8, hipMemcpyDeviceToHost, st));
    SCN_HIP(hipMemcpyAsync(hb->off, off_tmp, (K + 1) * 8, hipMemcpyDeviceToHost, st));
    SCN_HIP(hipStreamSynchronize(st));
    return SCN_OK;
  };
  if ((rc = outputs())) return rc;
  if ((hb->full || hb->a_out > cap_out / 2) && !(hb->flags & (KF_RANGE | KF_DUP)) &&
      cap_out < cap_full) {
    cap_out = cap_full;
    if ((rc = outputs())) return rc;
  }
  if (hb->flags & KF_RANGE) {
    set_error("scn_rulebook_build_nd: a site lies outside the grid");
    return SCN_ERR_RANGE;
  }
  if (hb->flags & KF_DUP) {
    set_error("scn_rulebook_build_nd: duplicate site in the input list");
    return SCN_ERR_DUPLICATE;
  }
  if (hb->full || hb->a_out > cap_out / 2) {  // cannot happen with the largest table
    set_error("scn_rulebook_build_nd: output table overflow (%llu outputs)",
              (unsigned long long)hb->a_out);
    return SCN_ERR_HIP;
  }
  const bool sorted = !(hb->flags & KF_UNSORTED);
  const int64_t a_out = (int64_t)hb->a_out;
  int64_t off[MAX_K + 1];
  for (int k = 0; k <= K; ++k) off[k] = hb->off[k];
  const int64_t P = off[K];
  if (a_out > INT32_MAX || P > INT32_MAX) {
    set_error("scn_rulebook_build_nd: %lld outputs / %lld pairs exceed INT32_MAX",
              (long long)a_out, (long long)P);
    return SCN_ERR_OVERFLOW;
  }
  const int64_t nt = std::max<int64_t>(1, ceil_div(a_out, TILE));

  // the rulebook: one block for everything but the input block
  auto al = [](int64_t bytes) { return (bytes + 255) & ~int64_t(255); };
  const int64_t sz_oc = al(a_out * (D + 1) * 4), sz_p = al(P * 4),
                sz_rank = sorted ? 0 : al(P * 4), sz_off = al((K + 1) * 8),
                sz_ot = al((K * nt + 1) * 8), sz_nbr = pool ? al(a_out * K * 4) : 0,
                sz_inv = pool ? al(n * slots * 4) : 0, sz_pm = pool ? al(a_out * 4) : 0;
  const int64_t total =
      sz_oc + 2 * sz_p + sz_rank + sz_off + sz_ot + sz_nbr + sz_inv + sz_pm;
  scn_rulebook* rb = new scn_rulebook();
  struct RbGuard {
    scn_rulebook*& rb;
    bool keep = false;
    ~RbGuard() {
      if (!keep && rb) scn_rulebook_free(rb);
    }
  } rb_guard{rb};
  rb->alloc = mem;
  rb->stream = st;
  rb->inblock = in_block;  // owned by rb from here
  in_block = nullptr;
  if ((rc = dalloc(&rb->block, (size_t)total, st, mem))) return rc;
  char* cur = static_cast<char*>(rb->block);
  auto take = [&](int64_t bytes) {
    char* p = bytes ? cur : nullptr;
    cur += bytes;
    return p;
  };
  rb->out_coords = (int32_t*)take(sz_oc);
  rb->in_rows = (int32_t*)take(sz_p);
  rb->out_rows = (int32_t*)take(sz_p);
  int32_t* in_rank_arr = (int32_t*)take(sz_rank);
  rb->in_rank = sorted ? rb->in_rows : in_rank_arr;
  rb->off_dev = (int64_t*)take(sz_off);
  rb->otile = (int64_t*)take(sz_ot);
  rb->itile = reinterpret_cast<int64_t*>(itile);
  rb->nbr = pool ? (int32_t*)take(sz_nbr) : nullptr;
  rb->inv = pool ? (int32_t*)take(sz_inv) : nullptr;
  rb->pmask = pool ? (uint32_t*)take(sz_pm) : nullptr;
  rb->inv_slots = slots;
  rb->perm = sorted ? nullptr : perm;
  const int32_t* perm_or_null = rb->perm;
  rb->f = f;
  rb->s = s;
  rb->K = (int32_t)K;
  rb->lattice = SCN_LATTICE_CUBIC;
  rb->ndim = D;
  rb->keyed = 1;
  rb->gin_nd[0] = rb->gout_nd[0] = grid[0];
  for (int a = 0; a < D; ++a) {
    rb->gin_nd[1 + a] = g.m[a];
    rb->gout_nd[1 + a] = g.mo[a];
  }
  for (int a = 0; a < 4; ++a) {
    rb->gin[a] = a <= D ? rb->gin_nd[a] : 1;
    rb->gout[a] = a <= D ? rb->gout_nd[a] : 1;
  }
  rb->a_in = n;
  rb->a_out = a_out;
  rb->n_pairs = P;
  rb->input_sorted = sorted ? 1 : 0;
  rb->n_otiles = nt;
  rb->n_itiles = nit;
  for (int k = 0; k <= K; ++k) rb->off_host[k] = off[k];
  SCN_HIP(hipMemcpyAsync(rb->off_dev, off_tmp, (K + 1) * 8, hipMemcpyDeviceToDevice, st));

  // outputs in canonical order, their rows into H_out
  uint64_t* okeys = nullptr;
  int32_t* oval = nullptr;
  uint32_t* sort_tmp2 = nullptr;
  if ((rc = tmp.get(&okeys, a_out)) || (rc = tmp.get(&oval, a_out)) ||
      (rc = tmp.get(&sort_tmp2, radix_sort_words<uint64_t>(a_out))))
    return rc;
  const int bits_out = bits_for(std::max<uint64_t>(sites_out, 1));
  if (a_out > 0) {
    if ((rc = radix_sort_pairs<uint64_t>(list, okeys, oval, a_out, bits_out, sort_tmp2, st)))
      return rc;
    hipLaunchKernelGGL(kd_assign_kernel, dim3(kd_blocks(a_out, 256)), dim3(256), 0, st,
                       (const uint64_t*)okeys, a_out, g, h_out,
                       cap_out - 1, rb->out_coords);
    SCN_LAUNCH_CHECK();
  }
  if (n > 0 && P > 0) {
    hipLaunchKernelGGL(kd_emit_kernel, dim3((unsigned)nit, (unsigned)K), dim3(64), 0, st,
                       (const int32_t*)sb, (const int4*)sx, n, g, nit, (const uint64_t*)itile,
                       perm_or_null, (const HSlot*)h_out,
                       cap_out - 1, rb->in_rows, rb->out_rows, sorted ? nullptr : in_rank_arr);
    SCN_LAUNCH_CHECK();
  }
  hipLaunchKernelGGL(kd_otile_kernel, dim3(kd_blocks(K * nt, 256)), dim3(256), 0, st,
                     (const int32_t*)rb->out_rows, (const int64_t*)rb->off_dev, (int)K, nt,
                     rb->otile);
  SCN_LAUNCH_CHECK();
  if (pool && a_out > 0) {
    hipLaunchKernelGGL(kd_windows_kernel, dim3(kd_blocks(a_out * 32, 256)), dim3(256), 0, st,
                       (const int32_t*)rb->out_coords, a_out, g, (const HSlot*)h_in,
                       cap_in - 1, perm_or_null, rb->nbr, rb->pmask);
    SCN_LAUNCH_CHECK();
  }
  if (pool && n > 0) {
    hipLaunchKernelGGL(kd_inv_kernel, dim3(kd_blocks(n * slots, 256)), dim3(256), 0, st,
                       (const int32_t*)sb, (const int4*)sx, n, g, slots, perm_or_null,
                       (const HSlot*)h_out, cap_out - 1, rb->inv);
    SCN_LAUNCH_CHECK();
  }
  SCN_HIP(hipEventCreateWithFlags(&rb->done, hipEventDisableTiming));
  SCN_HIP(hipEventRecord(rb->done, st));
  rb_guard.keep = true;
  *out = rb;
  return SCN_OK;
}

}  // namespace scn

extern "C" scn_status scn_rulebook_build_nd(const int32_t* coords, int64_t n, int32_t ndim,
                                            const int64_t* grid, int32_t filter, int32_t stride,
                                            hipStream_t stream, scn_rulebook** out) {
  scn::clear_error();
  return scn::keyed_build(coords, n, ndim, grid, filter, stride, stream, out);
}
