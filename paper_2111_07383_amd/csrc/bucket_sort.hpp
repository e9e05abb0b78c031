// Ascending sort of many small buckets of int32 (the per-site entry lists of the voxelisation and
// interpolation adjoints): one wavefront per bucket, a 64-lane bitonic network on cross-lane
// shuffles for buckets of up to 64 entries (padding sorts last), an in-place insertion sort by
// lane 0 beyond that.  The order of a bucket on exit is independent of the order it was filled in,
// which makes the sums over buckets deterministic.
#pragma once

#include "common.hpp"

namespace ssconv {
namespace {  // one copy per translation unit that includes this header

// Bucket r = a[start[r] .. start[r] + cnt[r]) for r < *n_rows (n_rows read on the device, or
// n_rows_host when n_rows is null); four buckets per 256-thread workgroup.
__global__ __launch_bounds__(256) void bucket_sort_kernel(const int64_t* __restrict__ n_rows, int64_t n_rows_host,
                                                          const int64_t* __restrict__ start,
                                                          const int32_t* __restrict__ cnt, int32_t* __restrict__ a) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t nr = n_rows ? *n_rows : n_rows_host;
  if (r >= nr) return;  // uniform per wavefront: no cross-wavefront barrier below
  int32_t* b = a + start[r];
  const int m = cnt[r];
  if (m <= 1) return;
  if (m <= 64) {
    int32_t v = lane < m ? b[lane] : 0x7fffffff;
#pragma unroll
    for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
      for (int j = k >> 1; j > 0; j >>= 1) {
        const int32_t p = __shfl_xor(v, j, 64);
        const bool asc = (lane & k) == 0, lower = (lane & j) == 0;
        v = (lower == asc) ? min(v, p) : max(v, p);
      }
    }
    if (lane < m) b[lane] = v;
    return;
  }
  if (lane == 0) {
    for (int j = 1; j < m; ++j) {
      const int32_t v = b[j];
      int k = j - 1;
      while (k >= 0 && b[k] > v) {
        b[k + 1] = b[k];
        --k;
      }
      b[k + 1] = v;
    }
  }
}

}  // namespace
}  // namespace ssconv
