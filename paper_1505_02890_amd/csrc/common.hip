// Error reporting, device allocation and version string.
#include <cstdarg>
#include <cstdio>
#include <atomic>
#include <mutex>

#include "scn_internal.h"

namespace scn {

static thread_local char g_err[512] = {0};

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

void clear_error() { g_err[0] = 0; }

// The default stream-ordered pool returns freed memory to the driver at every
// synchronisation unless its release threshold is raised; the rulebook build
// synchronises, so without this every build would re-allocate from scratch.
// Memory freed into the pool stays reserved for the process's later calls.
static void keep_pool_memory() {
  static bool done[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64 || done[dev]) return;
  hipMemPool_t pool;
  if (hipDeviceGetDefaultMemPool(&pool, dev) == hipSuccess) {
    uint64_t keep = UINT64_MAX;
    (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
  }
  (void)hipGetLastError();
  done[dev] = true;
}

static std::mutex g_alloc_mutex;
static Allocator g_alloc;  // hooks set by scn_set_allocator (none: default pool)

Allocator current_allocator() {
  std::lock_guard<std::mutex> lock(g_alloc_mutex);
  return g_alloc;
}

void set_allocator(const Allocator& a) {
  std::lock_guard<std::mutex> lock(g_alloc_mutex);
  g_alloc = a;
}

static std::atomic<int64_t> g_dense_rows{DENSE_MIN_ROWS};
static std::atomic<int32_t> g_dense_k{DENSE_MIN_K};

bool dense_forward_for(int64_t a_out, int K) {
  return a_out > 0 && a_out >= g_dense_rows.load(std::memory_order_relaxed) &&
         K >= g_dense_k.load(std::memory_order_relaxed);
}

scn_status dalloc(void** p, size_t bytes, hipStream_t s, const Allocator& a) {
  *p = nullptr;
  if (bytes == 0) return SCN_OK;
  if (a.alloc) {
    *p = a.alloc(bytes, s, a.ctx);
    if (!*p || (reinterpret_cast<uintptr_t>(*p) & 255) != 0) {
      if (*p) a.free(*p, s, a.ctx);
      *p = nullptr;
      set_error("the caller's allocator gave no 256-byte-aligned block of %zu bytes", bytes);
      return SCN_ERR_NOMEM;
    }
    return SCN_OK;
  }
  keep_pool_memory();
  hipError_t e = hipMallocAsync(p, bytes, s);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    *p = nullptr;
    set_error("device allocation of %zu bytes failed: %s", bytes, hipGetErrorString(e));
    return SCN_ERR_NOMEM;
  }
  return SCN_OK;
}

void dfree(void* p, hipStream_t s, const Allocator& a) {
  if (!p) return;
  if (a.alloc)
    a.free(p, s, a.ctx);
  else
    (void)hipFreeAsync(p, s);
}

}  // namespace scn

extern "C" const char* scn_last_error(void) { return scn::g_err; }

extern "C" void scn_set_allocator(void* (*alloc)(size_t, hipStream_t, void*),
                                  void (*free)(void*, hipStream_t, void*), void* ctx) {
  scn::Allocator a;
  if (alloc && free) {
    a.alloc = alloc;
    a.free = free;
    a.ctx = ctx;
  }
  scn::set_allocator(a);
}

extern "C" scn_status scn_set_dense_forward(int64_t min_rows, int32_t min_offsets) {
  scn::g_dense_rows.store(min_rows < 0 ? scn::DENSE_MIN_ROWS : min_rows,
                          std::memory_order_relaxed);
  scn::g_dense_k.store(min_offsets < 0 ? scn::DENSE_MIN_K : min_offsets,
                       std::memory_order_relaxed);
  return SCN_OK;
}

extern "C" const char* scn_version(void) { return "scn-mi355x 0.1 (gfx950)"; }
