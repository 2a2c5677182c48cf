// Internal definitions shared by the library's translation units (never by the
// CPU oracle).
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <string>

#include "scn.h"

namespace scn {

// Rows of a rulebook tile: pair ranges are stored per (offset, tile of TILE
// output rows) and per (offset, tile of TILE input ranks).
constexpr int TILE = 64;
constexpr int MAX_K = 27;  // f <= 3 (the tetrahedral lattice needs at most 10)
constexpr int KD_MAX = 4;  // coordinates per site of the keyed builder (keyed.hip)
constexpr int DENSE_ROWS = 32;  // output rows per block of the dense forward view
// Default policy for the dense forward view (scn_set_dense_forward): stride-1
// rulebooks with at least this many output rows and offsets.  Below them the
// view's sort and extra launches cost more than the forward saves (measured
// on the paper's networks, whose 2x2x2 layers never gain).
constexpr int64_t DENSE_MIN_ROWS = int64_t(1) << 19;
constexpr int DENSE_MIN_K = 8;

void set_error(const char* fmt, ...);
void clear_error();

struct DeviceBuffer {
  void* p = nullptr;
};

// Device allocation: the caller's hooks (scn_set_allocator) or, by default,
// the library's caching allocator (common.hip).  A value
// is a snapshot: memory goes back through the allocator that produced it.
struct Allocator {
  void* (*alloc)(size_t bytes, hipStream_t s, void* ctx) = nullptr;  // null: the library's cache
  void (*free)(void* p, hipStream_t s, void* ctx) = nullptr;
  void* ctx = nullptr;
};
Allocator current_allocator();
// whether a stride-1 rulebook with a_out outputs and K offsets gets the dense
// forward view (scn_set_dense_forward)
bool dense_forward_for(int64_t a_out, int K);
scn_status dalloc(void** p, size_t bytes, hipStream_t s, const Allocator& a);
void dfree(void* p, hipStream_t s, const Allocator& a);

#define SCN_HIP(call)                                                                  \
  do {                                                                                 \
    hipError_t e_ = (call);                                                            \
    if (e_ != hipSuccess) {                                                            \
      ::scn::set_error("%s failed: %s (%s:%d)", #call, hipGetErrorString(e_), __FILE__, \
                       __LINE__);                                                      \
      return SCN_ERR_HIP;                                                              \
    }                                                                                  \
  } while (0)

#define SCN_LAUNCH_CHECK()                                                             \
  do {                                                                                 \
    hipError_t e_ = hipGetLastError();                                                 \
    if (e_ != hipSuccess) {                                                            \
      ::scn::set_error("kernel launch failed: %s (%s:%d)", hipGetErrorString(e_),      \
                       __FILE__, __LINE__);                                            \
      return SCN_ERR_HIP;                                                              \
    }                                                                                  \
  } while (0)

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace scn

// Device layout of a rulebook.  All arrays are owned by the rulebook.
struct scn_rulebook {
  int32_t f = 0, s = 0, K = 0;
  int32_t lattice = SCN_LATTICE_CUBIC;
  int64_t gin[4] = {0, 0, 0, 0};   // B, mx, my, mz
  int64_t gout[4] = {0, 0, 0, 0};
  // Sites of ndim coordinates (out_coords rows of ndim + 1 int32: b, x_1 ..);
  // the extents (B, m_1 .. m_ndim) in gin_nd / gout_nd.  keyed: built from
  // sorted keys and hash tables (keyed.hip), without the occupancy bitmaps.
  int32_t ndim = 3;
  int32_t keyed = 0;
  int64_t gin_nd[scn::KD_MAX + 1] = {0, 0, 0, 0, 0};
  int64_t gout_nd[scn::KD_MAX + 1] = {0, 0, 0, 0, 0};
  int64_t a_in = 0, a_out = 0, n_pairs = 0;
  int32_t input_sorted = 0;
  hipStream_t stream = nullptr;    // stream the rulebook was built on (frees go there)

  int64_t off_host[scn::MAX_K + 1] = {0};  // list boundaries (host copy)

  int32_t* out_coords = nullptr;  // [a_out][4]
  int32_t* in_rows = nullptr;     // [P] caller row of the input of each pair
  int32_t* out_rows = nullptr;    // [P] output row of each pair
  int32_t* in_rank = nullptr;     // [P] rank of the input in key order (== in_rows if sorted)
  int32_t* perm = nullptr;        // [a_in] rank -> caller row (null when sorted: identity)
  int64_t* off_dev = nullptr;     // [K+1] list boundaries (device copy)

  // Pair ranges per tile.  otile[k*n_otiles + t] = global position of the first
  // pair of list k whose output row is >= t*TILE (t in [0, n_otiles]); the last
  // entry of list k equals the start of list k+1.  Length K*n_otiles + 1.
  // Null in a rulebook with the dense forward view (its forward does not use it).
  int64_t n_otiles = 0;
  int64_t* otile = nullptr;
  // Same per tile of TILE input ranks (for the input-gradient pass).
  int64_t n_itiles = 0;
  int64_t* itile = nullptr;

  // Pool helpers (stride >= 2 only): nbr[o*K + k] = input row at s*o+k or -1;
  // inv[r*inv_slots + j] = o*K + k of a window containing input r, or -1.  With
  // filter <= stride an input lies in at most one window (inv_slots = 1); with
  // filter > stride (3 over 2) in at most two per axis, slot j = sum over axes
  // of [k_axis >= s] << axis (inv_slots = 8).
  // pmask[o] bit k: position k of window o holds an active input
  // (nbr[o*K + k] >= 0), for the backward's ground-state test.
  int32_t* nbr = nullptr;
  int32_t* inv = nullptr;
  int inv_slots = 0;
  uint32_t* pmask = nullptr;
  // 3-wide windows of stride 2 on the cubic lattice: the backward goes cell by
  // cell.  Window h's home cell is its 2x2x2 corner of inputs (offsets
  // {0,1}^3); they also lie in the windows h - b, b in {0,1}^3 (bit a: one
  // step down along axis a).  lowwin[h*8 + b] = row of window h - b or -1
  // (lowwin[h*8] = h).  Inputs without a home window (at the upper grid edge)
  // are listed in homeless[0 .. *n_homeless) (device count, any order).
  int32_t* lowwin = nullptr;
  int32_t* homeless = nullptr;
  int32_t* n_homeless = nullptr;

  // Dense forward view (stride-1 rulebooks with outputs).  fnb holds, for
  // each output row o in key order, the caller rows of its active inputs in
  // ascending offset order, starting at fnb_off[o] (fnb_off[a_out] = P; fnb
  // has one spare entry).  fperm lists the output rows sorted by neighbour
  // mask (bit k: the input at offset k is active), a stable sort, so rows with
  // equal masks stay in key order; fmask[pos] is the mask of row fperm[pos].
  // The forward cuts the sorted order into blocks of DENSE_ROWS rows, whose
  // masks mostly agree.
  int64_t n_fblocks = 0;
  int32_t* fnb = nullptr;
  uint32_t* fnb_off = nullptr;
  int32_t* fperm = nullptr;
  uint32_t* fmask = nullptr;

  // Recorded on `stream` after the build's last kernel.  The build returns
  // once the host fields are known, with its last kernels possibly still
  // running; entry points called on another stream wait for this event.
  hipEvent_t done = nullptr;

  void* block = nullptr;    // one allocation holding the arrays above but perm and itile
  void* inblock = nullptr;  // one allocation holding perm and itile
  scn::Allocator alloc;   // the allocator every array of the rulebook came from

  // The output layer's rank bitmap (H_out): occupancy words of the output grid
  // and their exclusive popcount prefix (hout_rank[hout_words] = a_out); the
  // H_in of a rulebook built from this one's output sites.  One allocation,
  // starting at hout_bits.
  uint32_t* hout_bits = nullptr;
  uint32_t* hout_rank = nullptr;
  int64_t hout_words = 0;
};

namespace scn {
// The keyed builder (keyed.hip): a rulebook of the hypercubic lattice over
// sites of D coordinates, coords int32[n][D + 1], grid (B, m_1 .. m_D).
scn_status keyed_build(const int32_t* coords, int64_t n, int D, const int64_t* grid, int f, int s,
                       hipStream_t st, scn_rulebook** out);

// Work-groups go to the eight XCDs in turn (work-group b to XCD b mod 8), and
// each XCD has its own L2.  Kernels whose nearby blocks read the same lines
// give each XCD runs of `chunk` consecutive blocks: launched block b, the
// (b / 8)-th on XCD b mod 8, does block xcd_block(b, chunk) of the list.
// The grid is rounded up to whole rounds of 8 * chunk blocks; the blocks past
// the list return at once.
__device__ inline int64_t xcd_block(int64_t b, int chunk) {
  const int64_t x = b & 7, s = b >> 3;
  return ((s / chunk) * 8 + x) * chunk + s % chunk;
}

// runs of at most `want` blocks, and at most an eighth of the list (else
// the first XCDs would take every block of a short list)
inline int xcd_chunk(int64_t nblk, int want) {
  return (int)std::max<int64_t>(1, std::min<int64_t>(want, nblk / 8));
}

inline unsigned xcd_grid(int64_t nblk, int chunk) {
  const int64_t r = 8 * (int64_t)chunk;
  return (unsigned)std::max<int64_t>(1, (nblk + r - 1) / r * r);
}

// Orders work on stream st after the rulebook's build (a no-op on the build's
// own stream, where the order already holds).
inline scn_status after_build(const scn_rulebook* rb, hipStream_t st) {
  if (rb && rb->done && st != rb->stream && hipStreamWaitEvent(st, rb->done, 0) != hipSuccess) {
    set_error("HIP error ordering after the rulebook's build: %s",
              hipGetErrorString(hipGetLastError()));
    return SCN_ERR_HIP;
  }
  return SCN_OK;
}
}  // namespace scn
