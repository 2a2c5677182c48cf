/*
 * scn.h -- C ABI of the sparse 3D convolution library for AMD Instinct MI355X
 * (gfx950).
 *
 * The library implements the sparse operations of Graham, "Sparse 3D
 * convolutional neural networks" (section 1.3, "Sparse operations"): the
 * active-site rules, the per-layer ground state, the three-step sparse
 * convolution (active output set and hash H_out; the matrix Q; Q W + B) and
 * sparse max-pooling, plus their gradients (the paper trains these networks but
 * does not spell out the backward pass; the gradients here are those of the
 * dense-equivalent function, see scn_conv_bwd).
 *
 * Conventions for every call:
 *  - Lattice: cubic, 3D, unless a rulebook is built on the tetrahedral
 *    lattice (scn_rulebook_build_lattice).  A site is (b, x, y, z) with b the
 *    sample in the batch.  Its key is ((b*mz + z)*my + y)*mx + x for a grid
 *    (B, mx, my, mz).
 *  - Output extent of a filter (or pooling window) of size f and stride s is
 *    "valid": m_out = floor((m - f)/s) + 1 per axis (0 if m < f), as in the
 *    worked example of Figure 3 (a 2x2 filter on a 6x6 grid gives 5x5).
 *    Output site o sees input sites s*o + (kx, ky, kz), k in [0, f)^3; the
 *    offset index is k = (kz*f + ky)*f + kx.
 *  - Active sites: the inputs are the caller's list of sites (each listed site
 *    is active).  An output site is active iff some active input site lies in
 *    its window (second active-site rule of section 1.3).  Output rows are
 *    numbered 0..a_out-1 in ascending key order.
 *  - Feature matrices are fp32, row-major [rows][channels], channels innermost,
 *    one row per active site (the matrix M of section 1.3).  Weights are fp32
 *    [K][Cin][Cout] with K = f^3, i.e. the (f^3 n_in) x n_out matrix W of
 *    section 1.3 with row k*Cin + ci (K = C(f+2, 3) on the tetrahedral
 *    lattice: the rulebook's K).
 *  - Ground state: every inactive site of a layer holds the same vector g
 *    (section 1.3).  The input layer's ground state is normally 0.
 *  - All pointers named x, y, W, g_*, d*, coords, argmax are DEVICE pointers
 *    owned by the caller and never retained.  Host pointers are marked "host".
 *  - Calls are asynchronous on the given HIP stream unless stated otherwise;
 *    only the rulebook builds wait for the device (twice: to read back the
 *    number of output sites, then the per-offset list boundaries).  A build
 *    returns once its host-side sizes are known; its last kernels may still
 *    be running on its stream.  Every entry point that takes a rulebook and
 *    a different stream orders that stream after them (hipStreamWaitEvent);
 *    raw array pointers of a rulebook (scn_rulebook_out_coords and the like)
 *    are valid in the build stream's order.
 *  - No call allocates the caller's outputs.  Status codes are returned; no
 *    exception crosses the ABI.  scn_last_error() gives a message for the last
 *    failing call on the calling thread.
 *  - A rulebook is immutable after it is built and may be used from several
 *    streams; the caller orders its free after all work that uses it.
 */
#ifndef SCN_H_
#define SCN_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum scn_status {
  SCN_OK = 0,
  SCN_ERR_INVALID = 1,     /* null pointer, negative size, bad filter/stride/channels */
  SCN_ERR_RANGE = 2,       /* an input site outside its grid (or b outside [0, B)) */
  SCN_ERR_DUPLICATE = 3,   /* the same site listed twice */
  SCN_ERR_OVERFLOW = 4,    /* a count exceeds INT32_MAX, or a key exceeds 64 bits */
  SCN_ERR_UNSUPPORTED = 5, /* valid request outside what this version implements */
  SCN_ERR_WORKSPACE = 6,   /* workspace pointer null or smaller than required */
  SCN_ERR_HIP = 7,         /* a HIP runtime call failed */
  SCN_ERR_NOMEM = 8        /* device allocation failed */
} scn_status;

/* lattices of scn_rulebook_build_lattice (section 1.2, Figure 2) */
#define SCN_LATTICE_CUBIC 0
#define SCN_LATTICE_TETRAHEDRAL 1
#define SCN_LATTICE_SQUARE 2
#define SCN_LATTICE_TRIANGULAR 3

/* flags of scn_conv_fwd / scn_conv_bwd */
#define SCN_RELU 1u /* y = max(pre, 0) on active rows and on the ground state */

typedef struct scn_rulebook scn_rulebook;

typedef struct scn_rulebook_info {
  int64_t a_in;        /* active input sites */
  int64_t a_out;       /* active output sites */
  int64_t n_pairs;     /* P = total (input row, output row) incidences */
  int32_t K;           /* filter offsets: f^3, C(f+2, 3), f^2 or C(f+1, 2) by lattice */
  int32_t filter;      /* f */
  int32_t stride;      /* s */
  int32_t input_sorted;/* 1 if the caller's rows were already in ascending key order */
  int64_t in_grid[4];  /* B, mx, my, mz */
  int64_t out_grid[4]; /* B, floor((m-f)/s)+1 per axis */
  int32_t lattice;     /* SCN_LATTICE_* */
  int32_t dense_view;  /* 1 if the rulebook carries the dense forward view
                          (scn_set_dense_forward), else 0 */
  int32_t ndim;        /* coordinates per site (3 but for scn_rulebook_build_nd);
                          out_coords rows hold ndim + 1 int32 */
  int32_t keyed;       /* 1 if built from sorted keys and hash tables (grids past
                          the occupancy bitmaps, scn_rulebook_build_nd), else 0 */
  int64_t in_grid_nd[5];  /* B, m_1 .. m_ndim (then 0) */
  int64_t out_grid_nd[5]; /* B, floor((m_a - f)/s) + 1 (then 0) */
} scn_rulebook_info;

/*
 * Step 1 of the sparse convolution (section 1.3): build the map H_in from
 * active input site to row, find the active output sites of a filter of size
 * `filter` and stride `stride` and number them (H_out), and list for every
 * filter offset k which active input feeds which active output (the rulebook:
 * the blocks of the matrix Q of step 2 that are not the ground state).  A
 * rulebook with stride >= 2 also serves max-pooling (it then keeps the
 * window tables pooling uses: 4*K bytes per output and 4 bytes per input, 32
 * when windows overlap).
 *
 *  coords  device int32[n][4] rows (b, x, y, z); row i is row i of the
 *          layer's feature matrix.  Not retained, but read by kernels the
 *          call queues on `stream` (some after it returns): keep it valid in
 *          stream order (free it on `stream`, or after synchronising it).
 *  n       number of active input sites (>= 0; 0 gives an empty rulebook).
 *  grid    host int64[4] = (B, mx, my, mz), all >= 1.
 *  filter  f in {1, 2, 3};  stride s >= 1 (s <= f not required).
 *  stream  HIP stream for all device work; the call waits for it twice (the
 *          second time only for the list boundaries, with the build's last
 *          kernels queued behind them).
 *  out     receives a library-owned rulebook, freed by scn_rulebook_free.
 *
 * Output ordering is canonical: output rows ascend by key, and each
 * per-offset pair list ascends by output row (hence also by input key), so the
 * result is deterministic and independent of the input row order.
 * Grids whose occupancy bitmaps fit (2^26 32-bit words per grid, i.e.
 * B*my*mz*ceil(mx/32) <= 2^26 for the input and the output grid) take the
 * bitmap builder; larger ones the keyed builder of scn_rulebook_build_nd
 * (same results; it needs B*mx*my*mz < 2^63, and one host wait).
 * Errors: SCN_ERR_INVALID, SCN_ERR_RANGE, SCN_ERR_DUPLICATE, SCN_ERR_OVERFLOW,
 * SCN_ERR_UNSUPPORTED (f > 3), SCN_ERR_NOMEM, SCN_ERR_HIP.  coords must be
 * 16-byte aligned.  On error *out is NULL.
 */
scn_status scn_rulebook_build(const int32_t* coords, int64_t n, const int64_t* grid,
                              int32_t filter, int32_t stride, hipStream_t stream,
                              scn_rulebook** out);

/*
 * The rulebook of a hypercubic lattice in ndim = 1 .. 4 dimensions (section
 * 1.2: the method is the same in any dimension; its smallest filter has 2^d
 * sites), built from sorted site keys and open-addressing hash tables
 * (section 1.3 step 1 keeps H_in and H_out in "a map or hash table"), with
 * no occupancy bitmap, so any grid with B * prod m_a < 2^63 is accepted.
 *
 *  coords  device int32[n][ndim + 1] rows (b, x_1, .., x_ndim), 4-byte
 *          aligned; lifetime as for scn_rulebook_build.
 *  grid    host int64[ndim + 1] = (B, m_1, .., m_ndim), all >= 1.
 *  filter, stride   as for scn_rulebook_build, with f^ndim <= 27 offsets
 *          (f <= 2 in 4D); offset k = sum_a k_a f^(a-1), k_1 fastest.
 *
 * The site key is ((b*m_ndim + x_ndim)*m_(ndim-1) + ..)*m_1 + x_1 (in 3D the
 * key of scn_rulebook_build, whose results this reproduces); outputs are
 * numbered and pairs ordered as there.  The out_coords rows have ndim + 1
 * int32.  A rulebook with stride >= 2 serves pooling when filter <= stride,
 * and on 3D sites also when filter > stride (other such rulebooks serve
 * convolution only; scn_maxpool_* then return SCN_ERR_UNSUPPORTED).  The
 * call waits for `stream` once.  Errors: SCN_ERR_INVALID (ndim outside 1..4,
 * null or misaligned arguments), SCN_ERR_RANGE, SCN_ERR_DUPLICATE,
 * SCN_ERR_OVERFLOW (n, a_out or the pair count above INT32_MAX, or a key
 * above 63 bits), SCN_ERR_UNSUPPORTED (f > 3, or more than 27 offsets),
 * SCN_ERR_NOMEM, SCN_ERR_HIP.  On error *out is NULL.
 */
scn_status scn_rulebook_build_nd(const int32_t* coords, int64_t n, int32_t ndim,
                                 const int64_t* grid, int32_t filter, int32_t stride,
                                 hipStream_t stream, scn_rulebook** out);

/*
 * scn_rulebook_build on a chosen lattice (section 1.2, "CNNs on different
 * lattices").  SCN_LATTICE_CUBIC is scn_rulebook_build.  SCN_LATTICE_TETRAHEDRAL
 * holds the tetrahedral lattice in skewed integer coordinates:
 *  - the grid must have equal extents mx = my = mz = m; its sites are
 *    x + y + z < m (a site past it is SCN_ERR_RANGE);
 *  - a filter (or pooling region) of size f covers the C(f+2, 3) offsets
 *    kx + ky + kz < f: 4 for f = 2, 10 for f = 3.  They are numbered in the
 *    cubic scan order restricted to them (f = 2: (0,0,0), (1,0,0), (0,1,0),
 *    (0,0,1)), and W of a convolution on this rulebook is [K][Cin][Cout] in
 *    that order;
 *  - output o exists where its whole window lies in the grid:
 *    ox + oy + oz < floor((m - f)/s) + 1, the output grid of the same size
 *    (out_grid holds the cube's extents, as for the cubic lattice).
 * SCN_LATTICE_SQUARE and SCN_LATTICE_TRIANGULAR are the 2D lattices of
 * Figure 2 (i) and (ii): grid (B, mx, my, 1), every site with z = 0.  The
 * square filter covers the f^2 offsets (kx, ky, 0); the triangular lattice,
 * held in skewed coordinates like the tetrahedral one, has the sites
 * x + y < m (mx = my = m) and the C(f+1, 2) offsets kx + ky < f (3 for
 * f = 2, 6 for f = 3), numbered in the square scan order restricted to them.
 * out_grid[3] is 1.
 * Convolution and pooling on such a rulebook behave as on the cubic lattice
 * with these windows.  Another lattice value, unequal simplex extents or a
 * 2D grid with mz != 1 is SCN_ERR_INVALID; all other arguments and errors
 * as scn_rulebook_build.
 */
scn_status scn_rulebook_build_lattice(const int32_t* coords, int64_t n, const int64_t* grid,
                                      int32_t filter, int32_t stride, int32_t lattice,
                                      hipStream_t stream, scn_rulebook** out);

/*
 * The rulebook of the layer that follows prev (section 1.3: the active output
 * sites of one layer are the active input sites of the next).  Its input
 * sites are prev's active output sites, with their rows in prev's output
 * order, on prev's output grid and lattice; filter and stride as in
 * scn_rulebook_build.  The result equals scn_rulebook_build (or
 * scn_rulebook_build_lattice) called with scn_rulebook_out_coords(prev),
 * prev's a_out and out_grid, but reuses prev's output rank bitmap (every
 * rulebook keeps it: 8 bytes per 32 sites of its output grid) instead of
 * marking and ranking the sites again.  prev is only read, by kernels queued
 * on `stream` (some after the call returns).  If `stream` is not the stream
 * prev was built on, that stream is made to wait for them, so prev may be
 * freed (scn_rulebook_free, ordered on prev's stream) once this call
 * returns.  A keyed prev (grids past the bitmaps, or scn_rulebook_build_nd)
 * gives a keyed result over prev's ndim, built from prev's output sites.
 * Errors: SCN_ERR_INVALID (NULL, or prev's output grid is empty), and as
 * scn_rulebook_build.  It waits for stream as scn_rulebook_build does, and
 * orders stream after prev's build.
 */
scn_status scn_rulebook_build_next(const scn_rulebook* prev, int32_t filter, int32_t stride,
                                   hipStream_t stream, scn_rulebook** out);

/*
 * The rulebooks of a chain of layers in one call: layer 0 is built from the
 * caller's sites as by scn_rulebook_build_lattice (coords, n, grid, lattice),
 * and layer i > 0 from the active output sites of layer i - 1, as by
 * scn_rulebook_build_next, with filters[i] and strides[i] (host int32
 * [n_layers], 1 <= n_layers <= 64).  out is a host array of n_layers
 * handles, each freed by scn_rulebook_free.  Every layer's first phase is
 * queued before the call's first wait and every layer's second phase before
 * its second, so the whole chain waits for the device twice (a network of L
 * layers built one by one waits 2L times).  The rulebooks equal those of
 * the layer-by-layer builds.  Errors: as scn_rulebook_build_lattice for any
 * layer, and SCN_ERR_INVALID for a bad n_layers or a layer whose input grid
 * would be empty; on an error every out[i] is NULL.
 */
scn_status scn_rulebook_build_chain(const int32_t* coords, int64_t n, const int64_t* grid,
                                   int32_t lattice, int32_t n_layers, const int32_t* filters,
                                   const int32_t* strides, hipStream_t stream,
                                   scn_rulebook** out);

/* Sizes and grids of a rulebook (host struct).  SCN_ERR_INVALID on null. */
scn_status scn_rulebook_get_info(const scn_rulebook* rb, scn_rulebook_info* info);

/* Device int32[a_out][ndim + 1] (b, x, y, z for 3D) of the active output sites, ascending by
 * key: the input coordinates of the next layer.  Owned by rb. */
const int32_t* scn_rulebook_out_coords(const scn_rulebook* rb);

/* Device int32[n_pairs]: the per-offset pair lists, concatenated in offset
 * order; list k occupies [offsets[k], offsets[k+1]).  Owned by rb. */
const int32_t* scn_rulebook_in_rows(const scn_rulebook* rb);
const int32_t* scn_rulebook_out_rows(const scn_rulebook* rb);

/* Host int64[K+1] list boundaries.  Owned by rb. */
const int64_t* scn_rulebook_offsets(const scn_rulebook* rb);

/* Copies the active output sites and the pair lists into caller device
 * buffers (each may be NULL): out_coords int32[a_out][ndim + 1], in_rows and out_rows
 * int32[n_pairs].  Asynchronous on `stream`.  Errors: SCN_ERR_INVALID, SCN_ERR_HIP. */
scn_status scn_rulebook_export(const scn_rulebook* rb, int32_t* out_coords, int32_t* in_rows,
                               int32_t* out_rows, hipStream_t stream);

/* Frees a rulebook (stream-ordered on the stream it was built on). NULL is a no-op. */
void scn_rulebook_free(scn_rulebook* rb);

/*
 * Sparse convolution forward, steps 2 and 3 of section 1.3 (M_out = Q W + B)
 * over the rulebook rb, together with the output ground state.
 *   g_out = act(B + sum_k g_in W_k)               (the "pre-computed" g, section 1.3)
 *   y[o]  = act(B + sum_k v_k(o) W_k),  v_k(o) = x[row of s*o+k] if that site is
 *           active, else g_in
 * computed as y[o] = act(g_pre + sum_{pairs (r,o) of offset k} (x[r] - g_in) W_k),
 * which is the same sum regrouped.  act is ReLU if (flags & SCN_RELU), else
 * the identity.
 *
 *  x     [a_in][Cin];  g_in [Cin];  W [K][Cin][Cout];  bias [Cout] or NULL (= 0)
 *  y     [a_out][Cout] (written);  g_out [Cout] (written)
 * Errors: SCN_ERR_INVALID (null, Cin or Cout < 1, rb NULL), SCN_ERR_HIP.
 */
scn_status scn_conv_fwd(const scn_rulebook* rb, const float* x, const float* g_in,
                        const float* W, const float* bias, int32_t Cin, int32_t Cout,
                        uint32_t flags, float* y, float* g_out, hipStream_t stream);

/*
 * scn_conv_fwd for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation and result, bit for bit, with the
 * forward's scratch (the ground-state terms and the packed weights) in a
 * static device array of scn_conv_fwd_noalloc_max_bytes() bytes (8 MiB) that
 * the library holds on each GPU it runs on until the process ends.  The call
 * allocates nothing; the caller still passes every input and output.
 * Scratch needed: 4*((K+1)*NcP rounded up to 64 floats + K*NcP*RkP) bytes
 * with NcP = 64*ceil(Cout/64) and RkP = 16*ceil(Cin/16); every 3x3x3 layer
 * with Cin, Cout <= 256 fits.  Larger shapes return SCN_ERR_WORKSPACE before
 * any device work.  All calls on one GPU share its array: calls that overlap
 * on a GPU (on different streams, or from several threads without stream
 * order between them) race and give undefined results; calls ordered on one
 * stream do not.  Errors: as scn_conv_fwd, and SCN_ERR_WORKSPACE.
 */
scn_status scn_conv_fwd_noalloc(const scn_rulebook* rb, const float* x, const float* g_in,
                                const float* W, const float* bias, int32_t Cin, int32_t Cout,
                                uint32_t flags, float* y, float* g_out, hipStream_t stream);

/* Size in bytes of the static scratch array of scn_conv_fwd_noalloc. */
size_t scn_conv_fwd_noalloc_max_bytes(void);

/* Bytes of device workspace scn_conv_bwd needs for this rulebook and shape. */
size_t scn_conv_bwd_workspace_bytes(const scn_rulebook* rb, int32_t Cin, int32_t Cout,
                                    uint32_t flags);

/*
 * Gradients of scn_conv_fwd for the loss L = sum_o <dy[o], y[o]> + <dg_out, g_out>
 * (derivative of the dense-equivalent function; ReLU'(0) = 0).  With
 * dȳ = dy * [y > 0] and dḡ = dg_out * [g_out > 0] under ReLU (else dy, dg_out):
 *   dx[r]    = sum_{pairs (r,o) of k} dȳ[o] W_k^T
 *   dW_k     = sum_{pairs (r,o) of k} (x[r] - g_in)^T dȳ[o] + g_in^T (S + dḡ),  S = sum_o dȳ[o]
 *   dbias    = S + dḡ
 *   dg_in    = sum_k W_k (S - T_k + dḡ)^T,  T_k = sum_{pairs (r,o) of k} dȳ[o]
 * Outputs are overwritten (not accumulated); a NULL output is not computed.
 *  x [a_in][Cin], g_in [Cin], W [K][Cin][Cout], y [a_out][Cout] and g_out
 *  [Cout] (post-activation; read only under SCN_RELU, may be NULL otherwise),
 *  dy [a_out][Cout], dg_out [Cout] or NULL (= 0).
 *  dx [a_in][Cin], dg_in [Cin], dW [K][Cin][Cout], dbias [Cout].
 *  ws/ws_bytes: device workspace of at least scn_conv_bwd_workspace_bytes().
 * Errors: SCN_ERR_INVALID, SCN_ERR_WORKSPACE, SCN_ERR_HIP.  Deterministic:
 * every reduction runs in a fixed order, so repeated calls are bitwise equal.
 */
scn_status scn_conv_bwd(const scn_rulebook* rb, const float* x, const float* g_in,
                        const float* W, const float* y, const float* g_out, const float* dy,
                        const float* dg_out, int32_t Cin, int32_t Cout, uint32_t flags,
                        float* dx, float* dg_in, float* dW, float* dbias, void* ws,
                        size_t ws_bytes, hipStream_t stream);

/*
 * Sparse max-pooling forward (section 1.3, end: pooling "is similar" to the
 * convolution).  rb must have stride >= 2; windows may overlap (filter >
 * stride: 3 over 2, the pooling the paper's networks use) or leave gaps.
 * For each active output o and channel c, y[o][c] is the maximum over the K
 * positions of the window (the rulebook's K: f^3 on the cubic lattice, 10 for
 * MP3/2 on the tetrahedral one), an active position holding x[row][c] and an inactive one
 * g_in[c]; ties keep the first position in ascending k.
 * argmax[o][c] receives that k.  g_out = g_in.
 *  x [a_in][C], g_in [C] -> y [a_out][C], g_out [C], argmax uint8 [a_out][C].
 * Errors: SCN_ERR_INVALID, SCN_ERR_UNSUPPORTED (stride 1), SCN_ERR_HIP.
 */
scn_status scn_maxpool_fwd(const scn_rulebook* rb, const float* x, const float* g_in,
                           int32_t C, float* y, float* g_out, uint8_t* argmax,
                           hipStream_t stream);

/* Bytes of device workspace scn_maxpool_bwd needs. */
size_t scn_maxpool_bwd_workspace_bytes(const scn_rulebook* rb, int32_t C);

/*
 * Gradient of scn_maxpool_fwd: dy[o][c] flows to the winning position; a
 * winning inactive position passes it to the ground state, and g_out = g_in
 * passes dg_out through:
 *   dx[r][c] = sum over the windows o containing r of dy[o][c] if r is the
 *              active position argmax[o][c] of window o (one window at most
 *              when filter <= stride, up to 8 when 3 over 2; summed in a
 *              fixed order)
 *   dg_in[c] = dg_out[c] + sum_{o: argmax[o][c] inactive} dy[o][c]
 *  argmax [a_out][C] from scn_maxpool_fwd, dy [a_out][C], dg_out [C] or NULL.
 *  dx [a_in][C] (every row written), dg_in [C] (NULL: not computed).
 * Errors: SCN_ERR_INVALID, SCN_ERR_UNSUPPORTED (stride 1), SCN_ERR_WORKSPACE,
 *         SCN_ERR_HIP.
 */
scn_status scn_maxpool_bwd(const scn_rulebook* rb, const uint8_t* argmax, const float* dy,
                           const float* dg_out, int32_t C, float* dx, float* dg_in, void* ws,
                           size_t ws_bytes, hipStream_t stream);

/*
 * Device memory the library allocates for itself: rulebook storage and the
 * temporaries of scn_rulebook_build* and scn_conv_fwd (workspaces of the
 * backward passes are the caller's).  By default it comes from the library's
 * caching allocator: blocks from hipMalloc, kept by the library after they are
 * freed (never returned to the driver before the process ends, except when
 * hipMalloc fails) and reused in stream order, or on another stream once the
 * work queued before their free has completed.  Callers that manage
 * device memory themselves (a framework's caching allocator) install
 *   alloc(bytes, stream, ctx) -> 256-byte-aligned device pointer or NULL
 *   free(ptr, stream, ctx)
 * and the library calls them, ordered on the stream of the call that
 * allocates or frees; a NULL from alloc is SCN_ERR_NOMEM.  NULL alloc or
 * free restores the default.  Process-wide; it applies to calls that start
 * after it returns.  A rulebook is freed with the allocator that built it.
 */
void scn_set_allocator(void* (*alloc)(size_t bytes, hipStream_t stream, void* ctx),
                       void (*free)(void* ptr, hipStream_t stream, void* ctx), void* ctx);

/*
 * Which stride-1 rulebooks carry the dense forward view, used by
 * scn_conv_fwd instead of the per-offset pair lists: the output rows sorted
 * by their neighbour masks (the set of active offsets) so that blocks of 32
 * rows share one offset set, and each output's input rows in offset order.
 * Building the view costs a radix sort and one more list per rulebook; it
 * pays back when the layer is large and has many offsets.  A stride-1
 * rulebook built after this call carries the view when it has at least
 * min_rows output rows and at least min_offsets offsets (K).  Defaults:
 * min_rows = 524288, min_offsets = 8 (set with negative arguments).
 * Process-wide.  Results agree with the pair-list forward to rounding (each
 * output sums its active offsets in ascending order either way).
 * Errors: none (always SCN_OK).
 */
scn_status scn_set_dense_forward(int64_t min_rows, int32_t min_offsets);

/*
 * Measurement hook.  On the calling thread, later calls record the caller's
 * events on their stream around their contraction kernels: events[0] before
 * and events[1] after the forward's (scn_conv_fwd, scn_conv_fwd_noalloc),
 * events[2] / events[3] around the input gradient's and events[4] / events[5]
 * around the weight gradient's partial products (scn_conv_bwd).  A NULL entry
 * records nothing; events = NULL (host array of 6) turns the hook off.  The
 * events stay the caller's and must outlive the calls that record them.
 * Errors: none (SCN_OK); a failing record makes that call return SCN_ERR_HIP.
 */
scn_status scn_set_kernel_timer(const hipEvent_t* events);

/*
 * Measured ceilings for roofline fractions (not part of the convolution):
 * scn_ceiling_copy copies `bytes` (a multiple of 16, both pointers 16-byte
 * aligned) from src to dst with a plain streaming kernel (the HBM ceiling and
 * the reference of the memory counters); scn_ceiling_mfma_f32 runs
 * `workgroups` work-groups of 4 waves, each wave issuing `iters` x 8
 * independent v_mfma_f32_16x16x4f32 products on registers only (the fp32
 * matrix-core ceiling), writes one value per wave to out (device float
 * [4 * workgroups]) and stores its flop count in *flops (host).
 * Errors: SCN_ERR_INVALID, SCN_ERR_HIP.
 */
scn_status scn_ceiling_copy(const void* src, void* dst, size_t bytes, hipStream_t stream);
scn_status scn_ceiling_mfma_f32(float* out, int64_t workgroups, int32_t iters, double* flops,
                                hipStream_t stream);

/* Message describing the last failing call on this thread ("" if none). */
const char* scn_last_error(void);

/* Library version string. */
const char* scn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SCN_H_ */
