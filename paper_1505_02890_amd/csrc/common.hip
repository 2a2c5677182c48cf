// Error reporting, device allocation and version string.
#include <cstdarg>
#include <cstdio>
#include <atomic>
#include <map>
#include <mutex>
#include <unordered_map>
#include <vector>

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

// The library's own device memory, when the caller installed no hooks: a
// caching allocator.  Blocks come from hipMalloc and are never returned to
// the driver; a freed block goes to its device's free list, tagged with the
// stream it was freed on and an event recorded there.  A later request takes
// the smallest free block that fits (at most twice the request) and is safe
// to reuse: freed on the requesting stream (stream order covers the work
// that used it) or with its event complete.  Sizes are rounded up to an
// eighth of their power of two, so requests of varying size reuse blocks.
// (The device's stream-ordered pool spent 50-350 us per hipMallocAsync or
// hipFreeAsync call here, while the device waited for the host.)
namespace {

struct CachedBlock {
  void* p;
  size_t bytes;
  hipStream_t stream;
  hipEvent_t ready;
};

struct DeviceCache {
  std::multimap<size_t, CachedBlock> free_blocks;
  std::unordered_map<void*, size_t> live;  // allocated block -> its size
  std::vector<hipEvent_t> spare_events;
};

std::mutex g_cache_mutex;
DeviceCache g_cache[64];

size_t size_class(size_t b) {
  if (b <= 4096) return (b + 255) & ~size_t(255);
  size_t top = size_t(1) << (63 - __builtin_clzll(b));  // highest power of two <= b
  const size_t step = top / 8;
  return (b + step - 1) / step * step;
}

// Returns every cached block whose event has completed to the driver (on an
// allocation failure).  Caller holds the mutex.
void trim(DeviceCache& c) {
  for (auto it = c.free_blocks.begin(); it != c.free_blocks.end();) {
    if (hipEventQuery(it->second.ready) == hipSuccess) {
      (void)hipFree(it->second.p);
      c.spare_events.push_back(it->second.ready);
      it = c.free_blocks.erase(it);
    } else {
      ++it;
    }
  }
  (void)hipGetLastError();
}

scn_status cache_alloc(void** out, size_t bytes, hipStream_t s) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    set_error("device allocation: no current device");
    return SCN_ERR_NOMEM;
  }
  const size_t want = size_class(bytes);
  std::lock_guard<std::mutex> lock(g_cache_mutex);
  DeviceCache& c = g_cache[dev];
  for (auto it = c.free_blocks.lower_bound(want);
       it != c.free_blocks.end() && it->first <= 2 * want; ++it) {
    const CachedBlock& b = it->second;
    hipError_t q = b.stream == s ? hipSuccess : hipEventQuery(b.ready);
    if (q == hipSuccess) {
      *out = b.p;
      c.spare_events.push_back(b.ready);
      c.live[b.p] = it->first;
      c.free_blocks.erase(it);
      return SCN_OK;
    }
  }
  (void)hipGetLastError();  // hipEventQuery's hipErrorNotReady
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, want);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    trim(c);
    e = hipMalloc(&p, want);
  }
  if (e != hipSuccess) {
    (void)hipGetLastError();
    set_error("device allocation of %zu bytes failed: %s", want, hipGetErrorString(e));
    return SCN_ERR_NOMEM;
  }
  c.live[p] = want;
  *out = p;
  return SCN_OK;
}

void cache_free(void* p, hipStream_t s) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return;
  }
  std::lock_guard<std::mutex> lock(g_cache_mutex);
  DeviceCache& c = g_cache[dev];
  auto it = c.live.find(p);
  if (it == c.live.end()) return;  // not a block of this device's cache
  const size_t bytes = it->second;
  c.live.erase(it);
  hipEvent_t ev = nullptr;
  if (!c.spare_events.empty()) {
    ev = c.spare_events.back();
    c.spare_events.pop_back();
  } else if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) {
    (void)hipGetLastError();
    ev = nullptr;
  }
  if (!ev || hipEventRecord(ev, s) != hipSuccess) {
    // without an event the block can only be reused after a full wait
    (void)hipGetLastError();
    (void)hipStreamSynchronize(s);
    if (!ev && hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) {
      (void)hipGetLastError();
      (void)hipFree(p);
      return;
    }
    (void)hipEventRecord(ev, nullptr);
  }
  c.free_blocks.emplace(bytes, CachedBlock{p, bytes, s, ev});
}

}  // namespace

static std::mutex g_alloc_mutex;
static Allocator g_alloc;  // hooks set by scn_set_allocator (none: the cache below)

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
  return cache_alloc(p, bytes, s);
}

void dfree(void* p, hipStream_t s, const Allocator& a) {
  if (!p) return;
  if (a.alloc)
    a.free(p, s, a.ctx);
  else
    cache_free(p, s);
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
