// Ascending sort of many buckets of int32 (the per-site entry lists of the voxelisation and
// interpolation adjoints).  The order of a bucket on exit is independent of the order it was
// filled in, which makes the sums over buckets deterministic.
//
// Buckets of up to 64 entries are sorted by bitonic networks on cross-lane shuffles (padding
// sorts last).  For lists of mostly tiny buckets (voxelisation: a few points per site) a
// wavefront takes eight consecutive buckets, those of up to 8 entries on eight lanes each and
// those of 9 to 64 entries then one at a time on the whole wavefront (a wavefront per bucket left
// most lanes sorting padding there: 59 -> 14 us for 158k sites); otherwise (interpolation
// adjoint: ~32 entries per site) a wavefront takes one bucket, the 64-lane network.
// Larger buckets are appended to a list on the device and sorted
// by a second kernel, one workgroup per bucket: the bitonic network in its all-ascending form
// (each merge starts by comparing i with its mirror i ^ (k - 1) in the block of k, then halves
// with i ^ j; every comparator puts the smaller value at the lower index).  In that form entries
// past the bucket's end behave as +infinity and their comparators never swap, so they are simply
// skipped: up to kBigLds entries the network runs in LDS, beyond that in place in global memory
// (O(m log^2 m) either way).
#pragma once

#include "common.hpp"

namespace ssconv {
namespace {  // one copy per translation unit that includes this header

constexpr int kBigLds = 8192;  // largest bucket sorted in LDS (32 KB)

// Bucket r = a[start[r] .. start[r] + cnt[r]) for r < *n_rows (n_rows read on the device, or
// n_rows_host when n_rows is null); BPW buckets per wavefront (1 or 8), 4 BPW per 256-thread
// workgroup.  A bucket of more than 64 entries is appended to big[1 ..] (big[0] counts them; zero
// at launch).
template <int BPW>
__global__ __launch_bounds__(256) void bucket_sort_kernel(const int64_t* __restrict__ n_rows, int64_t n_rows_host,
                                                          const int64_t* __restrict__ start,
                                                          const int32_t* __restrict__ cnt, int32_t* __restrict__ a,
                                                          int32_t* __restrict__ big) {
  constexpr int GW = 64 / BPW;  // lanes per bucket in the first pass
  const int lane = threadIdx.x & 63, grp = lane / GW, sub = lane % GW;
  const int64_t nr = n_rows ? *n_rows : n_rows_host;
  const int64_t r0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * BPW;
  if (r0 >= nr) return;  // uniform per wavefront: no cross-wavefront barrier below
  const int64_t r = r0 + grp;
  const int m = r < nr ? cnt[r] : 0;
  const bool small = m > 1 && m <= GW;
  int32_t* b = small ? a + start[r] : nullptr;
  {
    int32_t v = small && sub < m ? b[sub] : 0x7fffffff;
#pragma unroll
    for (int k = 2; k <= GW; k <<= 1) {
#pragma unroll
      for (int j = k >> 1; j > 0; j >>= 1) {
        const int32_t p = __shfl_xor(v, j, 64);  // j < GW: the partner is in the same group
        const bool asc = (sub & k) == 0, lower = (sub & j) == 0;
        v = (lower == asc) ? min(v, p) : max(v, p);
      }
    }
    if (small && sub < m) b[sub] = v;
  }
  if (sub == 0 && m > 64) big[1 + atomicAdd(big, 1)] = (int32_t)r;
  if constexpr (BPW == 1) return;
  uint64_t mid = __ballot(sub == 0 && m > GW && m <= 64);
  while (mid) {  // uniform: the ballot is the same in every lane
    const int g = (__ffsll((unsigned long long)mid) - 1) / GW;
    mid &= mid - 1;
    const int64_t rr = r0 + g;
    const int mm = cnt[rr];
    int32_t* bb = a + start[rr];
    int32_t v = lane < mm ? bb[lane] : 0x7fffffff;
#pragma unroll
    for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
      for (int j = k >> 1; j > 0; j >>= 1) {
        const int32_t p = __shfl_xor(v, j, 64);
        const bool asc = (lane & k) == 0, lower = (lane & j) == 0;
        v = (lower == asc) ? min(v, p) : max(v, p);
      }
    }
    if (lane < mm) bb[lane] = v;
  }
}

// Comparator t (0 <= t < p2 / 2) of the stage (k, j) of the all-ascending network over p2
// entries: j == k / 2 is the mirror stage, smaller j the half-cleaners.  Returns the pair (lo, hi).
__device__ __forceinline__ void bitonic_pair(int64_t t, int64_t k, int64_t j, int64_t* lo, int64_t* hi) {
  if (j == k / 2) {
    const int64_t base = (t / j) * k, o = t % j;
    *lo = base + o;
    *hi = base + k - 1 - o;
  } else {
    *lo = (t / j) * 2 * j + t % j;
    *hi = *lo + j;
  }
}

// The listed large buckets, one workgroup each (the grid strides over the list).
__global__ __launch_bounds__(256) void bucket_sort_big_kernel(const int32_t* __restrict__ big,
                                                              const int64_t* __restrict__ start,
                                                              const int32_t* __restrict__ cnt, int32_t* __restrict__ a) {
  __shared__ int32_t s[kBigLds];
  const int tid = threadIdx.x;
  const int nbig = big[0];
  for (int q = blockIdx.x; q < nbig; q += gridDim.x) {
    const int64_t r = big[1 + q];
    int32_t* b = a + start[r];
    const int64_t m = cnt[r];
    int64_t p2 = 128;
    while (p2 < m) p2 <<= 1;
    if (m <= kBigLds) {
      for (int64_t i = tid; i < p2; i += 256) s[i] = i < m ? b[i] : 0x7fffffff;
      __syncthreads();
      for (int64_t k = 2; k <= p2; k <<= 1)
        for (int64_t j = k >> 1; j > 0; j >>= 1) {
          for (int64_t t = tid; t < p2 / 2; t += 256) {
            int64_t lo, hi;
            bitonic_pair(t, k, j, &lo, &hi);
            const int32_t x = s[lo], y = s[hi];
            if (y < x) s[lo] = y, s[hi] = x;
          }
          __syncthreads();
        }
      for (int64_t i = tid; i < m; i += 256) b[i] = s[i];
    } else {
      for (int64_t k = 2; k <= p2; k <<= 1)
        for (int64_t j = k >> 1; j > 0; j >>= 1) {
          for (int64_t t = tid; t < p2 / 2; t += 256) {
            int64_t lo, hi;
            bitonic_pair(t, k, j, &lo, &hi);
            if (hi < m) {  // a comparator with an entry past the end never swaps
              const int32_t x = b[lo], y = b[hi];
              if (y < x) b[lo] = y, b[hi] = x;
            }
          }
          __syncthreads();  // also orders this workgroup's global writes before the next stage
        }
    }
    __syncthreads();  // LDS reuse by the next bucket
  }
}

// Sorts every bucket: big must hold n_max + 1 int32 (n_max = the largest number of buckets);
// tiny: most buckets hold at most 8 entries (eight buckets per wavefront).
inline int sort_buckets(const int64_t* n_rows, int64_t n_rows_host, int64_t n_max, const int64_t* start,
                        const int32_t* cnt, int32_t* a, int32_t* big, bool tiny, hipStream_t st) {
  if (n_max <= 0) return SSCONV_OK;
  SSC_HIP(hipMemsetAsync(big, 0, 4, st));
  if (tiny)
    bucket_sort_kernel<8><<<cdiv(n_max, 32), 256, 0, st>>>(n_rows, n_rows_host, start, cnt, a, big);
  else
    bucket_sort_kernel<1><<<cdiv(n_max, 4), 256, 0, st>>>(n_rows, n_rows_host, start, cnt, a, big);
  bucket_sort_big_kernel<<<256, 256, 0, st>>>(big, start, cnt, a);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

}  // namespace
}  // namespace ssconv
