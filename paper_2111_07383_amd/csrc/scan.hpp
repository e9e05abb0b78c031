// Wave64 / block prefix sums and a device-wide exclusive scan (int32 counts -> int64 offsets).
#pragma once

#include "common.hpp"

namespace ssconv {

// Inclusive scan across the 64 lanes of a wavefront.
template <typename V>
__device__ __forceinline__ V wave_incl_scan(V v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    V o = __shfl_up(v, d, 64);
    if (lane >= d) v += o;
  }
  return v;
}

// Exclusive scan over a block of NT threads; *total receives the block sum.
template <int NT, typename V>
__device__ __forceinline__ V block_excl_scan(V v, V* total) {
  __shared__ V wsum[NT / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  V inc = wave_incl_scan(v);
  if (lane == 63) wsum[w] = inc;
  __syncthreads();
  V base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) {
    V x = wsum[i];
    if (i < w) base += x;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return base + inc - v;
}

// out[i] = sum_{j < i} in[j] for i < n, and *total = sum of all in.  in and out
// may not alias.  tmp must hold scan_tmp_elems(n) int64 values.
int64_t scan_tmp_elems(int64_t n);
int exclusive_scan(const int32_t* in, int64_t n, int64_t* out, int64_t* total, int64_t* tmp, hipStream_t stream);
// The same over the population counts of n bitmap words.
int exclusive_scan_popc(const uint32_t* words, int64_t n, int64_t* out, int64_t* total, int64_t* tmp,
                        hipStream_t stream);
// The scan of K*nblk offset-major counts, followed by pair_off[s] = out[s*nblk] (s < K) and
// pair_off[K] = *total.
int exclusive_scan_pair_off(const int32_t* counts, int K, int nblk, int64_t* out, int64_t* total, int64_t* tmp,
                            int64_t* pair_off, hipStream_t stream);

}  // namespace ssconv
