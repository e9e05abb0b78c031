// Shared host/device helpers of the SS-Conv library (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/ssconv.h"

namespace ssconv {

// ---------------------------------------------------------------------------
// errors: thread-local message, negative status codes, no exceptions across the ABI
// ---------------------------------------------------------------------------
void set_error(const char* fmt, ...);
int fail(int code, const char* fmt, ...);

#define SSC_HIP(expr)                                                                       \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return ::ssconv::fail(SSCONV_E_HIP, "%s failed: %s (%s:%d)", #expr,                   \
                            hipGetErrorString(e_), __FILE__, __LINE__);                     \
  } while (0)

#define SSC_TRY(expr)            \
  do {                           \
    int rc_ = (expr);            \
    if (rc_ != SSCONV_OK) return rc_; \
  } while (0)

// stream-ordered device allocation with the test hook for forced failures
int dev_alloc(void** p, size_t bytes, hipStream_t stream);
void dev_free(void* p, hipStream_t stream);
// Device scratch of one call, handed down to the kernels that need it.  base == nullptr: every
// request is a block of the device memory cache (dev_alloc / dev_free).  Otherwise requests are
// carved, 256-byte aligned, from [base, base + cap) in order and never freed (the
// allocation-free entry points pass their fixed per-device region this way); a request that
// does not fit fails with SSCONV_E_INVALID.
struct CallScratch {
  char* base = nullptr;
  size_t cap = 0, used = 0;
  bool fixed() const { return base != nullptr; }
  size_t left() const { return cap > ((used + 255) & ~(size_t)255) ? cap - ((used + 255) & ~(size_t)255) : 0; }
};
int scratch_take(CallScratch* sc, void** p, size_t bytes, hipStream_t stream);
void scratch_give(CallScratch* sc, void* p, hipStream_t stream);
int64_t debug_hash_capacity();
int64_t debug_gather_variant();
// Fork / join of work onto the library's second stream of the current device: aux_fork makes
// the side stream wait for everything queued on caller so far; aux_join makes caller wait for
// everything queued on the side stream so far.  Not reentrant across overlapping forks of one
// thread.
int aux_fork(hipStream_t caller, hipStream_t* side);
int aux_join(hipStream_t caller, hipStream_t side);
// Kernel timing hook (ssconv_debug_set option 4): returns the event pair to record around the
// next timed kernel, or false when timing is off.
bool debug_timing_events(hipEvent_t* start, hipEvent_t* stop);

// ---------------------------------------------------------------------------
// field tables (channel -> field, order, component) passed by value to kernels
// ---------------------------------------------------------------------------
struct FieldTab {
  int n;                         // entries
  int l[SSCONV_MAX_ENTRIES];     // order per entry
  int mult[SSCONV_MAX_ENTRIES];  // fields per entry
  int ch0[SSCONV_MAX_ENTRIES + 1];  // first channel of each entry (ch0[n] = channels)
  int f0[SSCONV_MAX_ENTRIES + 1];   // first field index of each entry
};

int make_fieldtab(const ssconv_fields* f, FieldTab* t);

// Position of dW[s][o][i] in the field-pair-blocked layout of the kernel gradient: the
// K*(2k+1)*(2l+1) values of each (out field, in field) pair are contiguous, in (s, a, b) order
// (a, b = component in the out and in field), and the pair of out field rows [ro, ro+dk) and in
// field columns [cc, cc+dl) starts at K*(ro*cin + dk*cc), so the layout is a permutation of
// [K][cout][cin].  The coefficient gradient then reads each pair's block contiguously.
__device__ __forceinline__ int64_t dw_block_pos(const FieldTab& fout, const FieldTab& fin, int K, int cin, int s,
                                                int o, int i) {
  int eo = 0, ei = 0;
  while (eo + 1 < fout.n && o >= fout.ch0[eo + 1]) ++eo;
  while (ei + 1 < fin.n && i >= fin.ch0[ei + 1]) ++ei;
  const int dk = 2 * fout.l[eo] + 1, dl = 2 * fin.l[ei] + 1;
  const int ro = fout.ch0[eo] + (o - fout.ch0[eo]) / dk * dk, cc = fin.ch0[ei] + (i - fin.ch0[ei]) / dl * dl;
  return (int64_t)K * ((int64_t)ro * cin + (int64_t)dk * cc) + ((int64_t)s * dk + (o - ro)) * dl + (i - cc);
}

// ---------------------------------------------------------------------------
// bf16 helpers (storage as uint16, round-to-nearest-even from fp32)
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

template <typename T> struct DT;
template <> struct DT<float> {
  static constexpr int bytes = 4;
  __device__ static __forceinline__ float to_f(float v) { return v; }
  __device__ static __forceinline__ float from_f(float v) { return v; }
};
template <> struct DT<uint16_t> {
  static constexpr int bytes = 2;
  __device__ static __forceinline__ float to_f(uint16_t v) { return bf16_to_f32(v); }
  __device__ static __forceinline__ uint16_t from_f(float v) { return f32_to_bf16_rne(v); }
};

inline size_t dtype_bytes(ssconv_dtype d) { return d == SSCONV_BF16 ? 2 : 4; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline unsigned cdiv(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

}  // namespace ssconv

// The rule book handle (opaque to callers).
struct ssconv_rulebook {
  int ksize = 0, K = 0, stride = 1, submanifold = 1;
  int grid[3] = {0, 0, 0}, grid_out[3] = {0, 0, 0};
  int64_t n_in = 0, n_out = 0, n_pairs = 0, nbatch = 0;
  hipStream_t stream = nullptr;
  // device buffers (owned)
  uint64_t* hash_in = nullptr;
  int64_t cap_in = 0;
  uint64_t* hash_out = nullptr;  // == hash_in for submanifold
  int64_t cap_out = 0;
  bool hash_out_built = false;    // generated output sets: hash_out is filled on first request
  int32_t* out_coords = nullptr;  // [n_out, 4]
  int32_t* nbr = nullptr;         // [K, n_out]
  int32_t* pairs = nullptr;       // [n_pairs, 2] grouped by offset
  int64_t* pair_off_dev = nullptr;  // [K + 1], followed by the build flags
  void* mem[3] = {nullptr, nullptr, nullptr};  // the allocations every buffer above lives in
  // host copies
  int64_t* pair_off = nullptr;  // [K + 1] (host)
  // An asynchronous submanifold build returns before its pair counts and flags reach the host:
  // they arrive in `stage` (pinned, from the library's pool) when `ready` has passed, and
  // rulebook_settle() reads them on first need; `status` then holds the build's result.
  bool pending = false;
  int status = 0;
  char error[192] = {0};
  hipEvent_t ready = nullptr;
  int64_t* stage = nullptr;
};

namespace ssconv {
// Completes an asynchronous build (waits for its read-back, fills pair_off / n_pairs, turns the
// device-detected errors into the build's status); returns that status on every call.  A build
// made synchronously is settled already.
int rulebook_settle(ssconv_rulebook* rb);
}  // namespace ssconv
