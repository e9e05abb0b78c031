// Error reporting, allocation and field tables shared by the SS-Conv entry points.
#include "common.hpp"

#include <atomic>
#include <mutex>
#include <unordered_map>
#include <utility>
#include <vector>

namespace ssconv {

namespace {
thread_local std::string g_error;
std::atomic<int64_t> g_debug_hash_cap{0};
std::atomic<int64_t> g_debug_fail_alloc{0};
std::atomic<int64_t> g_debug_gather_variant{0};
std::atomic<int64_t> g_debug_timing{0};
// event pairs of the kernel timing hook, reused from call to call on this thread
constexpr size_t kMaxTimed = 4096;
struct TimingLog {
  std::vector<std::pair<hipEvent_t, hipEvent_t>> ev;
  size_t used = 0;
};
thread_local TimingLog g_timing;
}  // namespace

void set_error(const char* fmt, ...) {
  char buf[1024];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
}

int fail(int code, const char* fmt, ...) {
  char buf[1024];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
  return code;
}

// Device memory cache.  A block the library frees is kept with its freeing stream and handed out
// again: reuse on the same stream needs nothing (stream order), reuse on another stream first
// records an event on the freeing stream and makes the new stream wait for it.  A stream-ordered allocation costs
// tens of microseconds of host time after a synchronisation and can block the host while the
// device is busy; a cache hit costs a lock and a short search.  Blocks come in 64 KB steps; a
// request takes the smallest free block of at least its size and at most twice it (+ 1 MB).
// Free blocks beyond kCacheLimit bytes are released, oldest first.
namespace {
struct Block {
  void* p = nullptr;
  size_t bytes = 0;
  int dev = 0;
  hipStream_t stream = nullptr;
  hipEvent_t ev = nullptr;
};
constexpr size_t kCacheLimit = (size_t)8 << 30;
std::mutex g_cache_mu;
std::vector<Block> g_free_blocks;                // oldest first
std::unordered_map<void*, Block> g_live_blocks;  // handed out
size_t g_free_bytes = 0;

void release_block(Block& b) {  // caller holds the lock; the block is stream-ordered after its event
  (void)hipFreeAsync(b.p, b.stream);
  if (b.ev) (void)hipEventDestroy(b.ev);
  (void)hipGetLastError();
}
}  // namespace

int dev_alloc(void** p, size_t bytes, hipStream_t stream) {
  *p = nullptr;
  if (bytes == 0) bytes = 256;
  int64_t n = g_debug_fail_alloc.load();
  if (n > 0) {
    if (n == 1) {
      g_debug_fail_alloc.store(0);
      return fail(SSCONV_E_NOMEM, "device allocation of %zu bytes failed (forced by test hook)", bytes);
    }
    g_debug_fail_alloc.store(n - 1);
  }
  const size_t want = (bytes + 65535) & ~(size_t)65535;
  int dev = 0;
  SSC_HIP(hipGetDevice(&dev));
  {
    std::lock_guard<std::mutex> lk(g_cache_mu);
    size_t best = g_free_blocks.size();
    for (size_t i = 0; i < g_free_blocks.size(); ++i) {
      const Block& b = g_free_blocks[i];
      if (b.dev == dev && b.bytes >= want && b.bytes <= 2 * want + ((size_t)1 << 20) &&
          (best == g_free_blocks.size() || b.bytes < g_free_blocks[best].bytes))
        best = i;
    }
    if (best < g_free_blocks.size()) {
      Block& b = g_free_blocks[best];
      if (b.stream != stream) {
        // ordered after the block's last use: an event recorded now on the freeing stream covers
        // everything queued there so far, the free included (no system-scope fence: device-side
        // ordering only)
        hipError_t e = b.ev ? hipSuccess : hipEventCreateWithFlags(&b.ev, hipEventDisableTiming | hipEventDisableSystemFence);
        if (e == hipSuccess) e = hipEventRecord(b.ev, b.stream);
        if (e == hipSuccess) e = hipStreamWaitEvent(stream, b.ev, 0);
        if (e != hipSuccess) {
          (void)hipGetLastError();
          return fail(SSCONV_E_HIP, "ordering a cached block after its freeing stream: %s", hipGetErrorString(e));
        }
      }
      Block got = b;
      g_free_blocks.erase(g_free_blocks.begin() + (std::ptrdiff_t)best);
      g_free_bytes -= got.bytes;
      got.stream = stream;
      g_live_blocks[got.p] = got;
      *p = got.p;
      return SSCONV_OK;
    }
  }
  hipError_t e = hipMallocAsync(p, want, stream);
  if (e != hipSuccess || !*p) {
    (void)hipGetLastError();
    {  // give the cached blocks of this device back and try once more
      std::lock_guard<std::mutex> lk(g_cache_mu);
      for (size_t i = 0; i < g_free_blocks.size();) {
        if (g_free_blocks[i].dev == dev) {
          g_free_bytes -= g_free_blocks[i].bytes;
          release_block(g_free_blocks[i]);
          g_free_blocks.erase(g_free_blocks.begin() + (std::ptrdiff_t)i);
        } else {
          ++i;
        }
      }
    }
    *p = nullptr;
    e = hipMallocAsync(p, want, stream);
    if (e != hipSuccess || !*p) {
      *p = nullptr;
      (void)hipGetLastError();
      return fail(SSCONV_E_NOMEM, "device allocation of %zu bytes failed: %s", bytes, hipGetErrorString(e));
    }
  }
  std::lock_guard<std::mutex> lk(g_cache_mu);
  Block b;
  b.p = *p;
  b.bytes = want;
  b.dev = dev;
  b.stream = stream;
  g_live_blocks[b.p] = b;
  return SSCONV_OK;
}

int scratch_take(CallScratch* sc, void** p, size_t bytes, hipStream_t stream) {
  if (!sc || !sc->fixed()) return dev_alloc(p, bytes, stream);
  const size_t at = (sc->used + 255) & ~(size_t)255;
  if (at > sc->cap || bytes > sc->cap - at) {
    *p = nullptr;
    return fail(SSCONV_E_INVALID, "the call needs %zu more bytes of scratch; %zu of %zu are left", bytes,
                sc->cap > at ? sc->cap - at : (size_t)0, sc->cap);
  }
  *p = sc->base + at;
  sc->used = at + bytes;
  return SSCONV_OK;
}

void scratch_give(CallScratch* sc, void* p, hipStream_t stream) {
  if (!sc || !sc->fixed()) dev_free(p, stream);
}

void dev_free(void* p, hipStream_t stream) {
  if (!p) return;
  std::lock_guard<std::mutex> lk(g_cache_mu);
  auto it = g_live_blocks.find(p);
  if (it == g_live_blocks.end()) {
    (void)hipFreeAsync(p, stream);
    (void)hipGetLastError();
    return;
  }
  Block b = it->second;
  g_live_blocks.erase(it);
  // Kept with the freeing stream and nothing recorded: reuse on that stream is ordered by the
  // stream itself, and reuse on another one records its event then (dev_alloc).  An event
  // recorded here would sit between two kernels of the stream on every free, and each such
  // record holds the next kernel's start back by microseconds.
  b.stream = stream;
  g_free_blocks.push_back(b);
  g_free_bytes += b.bytes;
  while (g_free_bytes > kCacheLimit && !g_free_blocks.empty()) {
    g_free_bytes -= g_free_blocks.front().bytes;
    release_block(g_free_blocks.front());
    g_free_blocks.erase(g_free_blocks.begin());
  }
}

int64_t debug_hash_capacity() { return g_debug_hash_cap.load(); }
int64_t debug_gather_variant() { return g_debug_gather_variant.load(); }

bool debug_timing_events(hipEvent_t* start, hipEvent_t* stop) {
  if (g_debug_timing.load() == 0 || g_timing.used == kMaxTimed) return false;
  if (g_timing.used == g_timing.ev.size()) {
    hipEvent_t a = nullptr, b = nullptr;
    // timestamps only (read after the last stop event completes): no system-scope fence, which
    // would write back and invalidate the caches around every timed launch
    if (hipEventCreateWithFlags(&a, hipEventDisableSystemFence) != hipSuccess ||
        hipEventCreateWithFlags(&b, hipEventDisableSystemFence) != hipSuccess) {
      if (a) (void)hipEventDestroy(a);
      (void)hipGetLastError();
      return false;
    }
    g_timing.ev.emplace_back(a, b);
  }
  *start = g_timing.ev[g_timing.used].first;
  *stop = g_timing.ev[g_timing.used].second;
  ++g_timing.used;
  return true;
}

int make_fieldtab(const ssconv_fields* f, FieldTab* t) {
  if (!f || f->n < 1 || f->n > SSCONV_MAX_ENTRIES) return fail(SSCONV_E_INVALID, "bad field list");
  t->n = f->n;
  int ch = 0, fi = 0;
  for (int e = 0; e < f->n; ++e) {
    if (f->l[e] < 0 || f->l[e] > SSCONV_MAX_L || f->mult[e] < 1) return fail(SSCONV_E_INVALID, "bad field entry");
    t->l[e] = f->l[e];
    t->mult[e] = f->mult[e];
    t->ch0[e] = ch;
    t->f0[e] = fi;
    ch += f->mult[e] * (2 * f->l[e] + 1);
    fi += f->mult[e];
  }
  for (int e = f->n; e <= SSCONV_MAX_ENTRIES; ++e) {
    t->ch0[e] = ch;
    t->f0[e] = fi;
    if (e < SSCONV_MAX_ENTRIES) t->l[e] = 0, t->mult[e] = 0;
  }
  return SSCONV_OK;
}

}  // namespace ssconv

extern "C" const char* ssconv_last_error(void) { return ssconv::g_error.c_str(); }

extern "C" const char* ssconv_version(void) { return "ssconv-gfx950 0.1"; }

extern "C" int ssconv_debug_set(int option, int64_t value) {
  if (option == 1) {
    ssconv::g_debug_hash_cap.store(value < 0 ? 0 : value);
    return SSCONV_OK;
  }
  if (option == 2) {
    ssconv::g_debug_fail_alloc.store(value < 0 ? 0 : value);
    return SSCONV_OK;
  }
  if (option == 3) {
    ssconv::g_debug_gather_variant.store(value < 0 ? 0 : value);
    return SSCONV_OK;
  }
  if (option == 4) {
    ssconv::g_debug_timing.store(value != 0 ? 1 : 0);
    if (value != 0) ssconv::g_timing.used = 0;
    return SSCONV_OK;
  }
  return ssconv::fail(SSCONV_E_INVALID, "unknown debug option %d", option);
}

extern "C" int ssconv_empty_cache(void) {
  using namespace ssconv;
  std::lock_guard<std::mutex> lk(g_cache_mu);
  int cur = 0;
  (void)hipGetDevice(&cur);
  for (Block& b : g_free_blocks) {
    (void)hipSetDevice(b.dev);
    (void)hipStreamSynchronize(b.stream);  // the block's last use is queued there
    (void)hipFree(b.p);
    if (b.ev) (void)hipEventDestroy(b.ev);
  }
  (void)hipSetDevice(cur);
  (void)hipGetLastError();
  g_free_blocks.clear();
  g_free_bytes = 0;
  return SSCONV_OK;
}

extern "C" int64_t ssconv_cached_bytes(void) {
  using namespace ssconv;
  std::lock_guard<std::mutex> lk(g_cache_mu);
  return (int64_t)g_free_bytes;
}

extern "C" int ssconv_debug_kernel_ms(int64_t* count, float* total_ms) {
  using namespace ssconv;
  if (!count || !total_ms) return fail(SSCONV_E_INVALID, "count or total_ms is NULL");
  *count = 0;
  *total_ms = 0.f;
  if (g_timing.used == 0) return fail(SSCONV_E_INVALID, "no timed kernel on this thread");
  SSC_HIP(hipEventSynchronize(g_timing.ev[g_timing.used - 1].second));
  double sum = 0.0;
  for (size_t i = 0; i < g_timing.used; ++i) {
    float ms = 0.f;
    SSC_HIP(hipEventElapsedTime(&ms, g_timing.ev[i].first, g_timing.ev[i].second));
    sum += ms;
  }
  *count = (int64_t)g_timing.used;
  *total_ms = (float)sum;
  return SSCONV_OK;
}

namespace ssconv {

// A second stream per device (default priority, non-blocking) and a pair of events per calling
// thread, for work the library forks off the caller's stream and joins back before returning.
namespace {
std::mutex g_aux_mu;
hipStream_t g_aux[64] = {};
struct AuxEvents {
  hipEvent_t fork = nullptr, join = nullptr;
};
thread_local AuxEvents g_aux_ev[64];
}  // namespace

int aux_fork(hipStream_t caller, hipStream_t* side) {
  int dev = 0;
  SSC_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return fail(SSCONV_E_INVALID, "device index %d out of range", dev);
  {
    std::lock_guard<std::mutex> lk(g_aux_mu);
    if (!g_aux[dev]) SSC_HIP(hipStreamCreateWithFlags(&g_aux[dev], hipStreamNonBlocking));
  }
  AuxEvents& e = g_aux_ev[dev];
  // stream-to-stream ordering on one device: no system-scope fence needed
  if (!e.fork) SSC_HIP(hipEventCreateWithFlags(&e.fork, hipEventDisableTiming | hipEventDisableSystemFence));
  if (!e.join) SSC_HIP(hipEventCreateWithFlags(&e.join, hipEventDisableTiming | hipEventDisableSystemFence));
  SSC_HIP(hipEventRecord(e.fork, caller));
  SSC_HIP(hipStreamWaitEvent(g_aux[dev], e.fork, 0));
  *side = g_aux[dev];
  return SSCONV_OK;
}

int aux_join(hipStream_t caller, hipStream_t side) {
  int dev = 0;
  SSC_HIP(hipGetDevice(&dev));
  AuxEvents& e = g_aux_ev[dev];
  SSC_HIP(hipEventRecord(e.join, side));
  SSC_HIP(hipStreamWaitEvent(caller, e.join, 0));
  return SSCONV_OK;
}

}  // namespace ssconv
