// Device-wide exclusive scan: one workgroup for up to 32 768 elements, else three passes (per-tile
// sums, one-block scan of the tile sums, per-tile rescan with the tile offset).  Deterministic.
#include <algorithm>

#include "scan.hpp"

namespace ssconv {

namespace {
constexpr int kNT = 256;
constexpr int kPer = 16;                 // elements per thread
constexpr int kTile = kNT * kPer;        // elements per block

// Element i of the scanned sequence: a count, or the population count of a bitmap word.
template <bool kPopc>
__device__ __forceinline__ int64_t elem(const void* in, int64_t i) {
  if (kPopc) return __popc(reinterpret_cast<const uint32_t*>(in)[i]);
  return reinterpret_cast<const int32_t*>(in)[i];
}

// pair_off[s] = out[s * nblk] for s < K, pair_off[K] = total (the offsets of the pair lists of
// the rule book, whose counts are laid out offset-major in blocks of nblk).
__device__ __forceinline__ void write_pair_off(const int64_t* out, int64_t total, int K, int nblk,
                                               int64_t* __restrict__ pair_off) {
  for (int s = threadIdx.x; s <= K; s += blockDim.x) pair_off[s] = s < K ? out[(int64_t)s * nblk] : total;
}

constexpr int kSmallNT = 1024;
constexpr int64_t kSmallMax = 32768;  // elements staged in LDS (128 KB)

// The whole scan in one workgroup (n <= kSmallMax).  The elements are staged in LDS with coalesced
// loads, at index i + i/32 so that the contiguous runs [t*per, (t+1)*per) that thread t sums and
// rescans fall in different banks; each run's local exclusive offsets go back into LDS in place (a
// run's sum stays below 2^32 for every caller: popcounts, and counts bounded by a block's rows or
// the point count), and the results leave with coalesced stores of run base + local offset.
__device__ __forceinline__ int lds_pad(int i) { return i + (i >> 5); }

template <bool kPopc>
__global__ __launch_bounds__(kSmallNT) void scan_small(const void* __restrict__ in, int64_t n,
                                                       int64_t* __restrict__ out, int64_t* __restrict__ total,
                                                       int K, int nblk, int64_t* __restrict__ pair_off) {
  __shared__ uint32_t sh[kSmallMax + kSmallMax / 32];
  __shared__ int64_t base[kSmallNT];
  const int t = threadIdx.x, nn = (int)n;
  // 16-byte loads where the input allows, so a thread has all its loads in flight at once
  const int n4 = (reinterpret_cast<uintptr_t>(in) & 15u) == 0 ? nn >> 2 : 0;
#pragma unroll 8
  for (int q = t; q < n4; q += kSmallNT) {
    const uint4 w = reinterpret_cast<const uint4*>(in)[q];
    const uint32_t v[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) sh[lds_pad(4 * q + k)] = kPopc ? (uint32_t)__popc(v[k]) : v[k];
  }
  for (int i = 4 * n4 + t; i < nn; i += kSmallNT) sh[lds_pad(i)] = (uint32_t)elem<kPopc>(in, i);
  __syncthreads();
  const int per = (nn + kSmallNT - 1) / kSmallNT;
  const int b0 = t * per, e0 = min(b0 + per, nn);
  int64_t s = 0;
  for (int i = b0; i < e0; ++i) s += sh[lds_pad(i)];
  int64_t tot;
  base[t] = block_excl_scan<kSmallNT>(s, &tot);
  uint32_t loc = 0;
  for (int i = b0; i < e0; ++i) {
    const uint32_t v = sh[lds_pad(i)];
    sh[lds_pad(i)] = loc;
    loc += v;
  }
  __syncthreads();
#pragma unroll 8
  for (int i = t; i < nn; i += kSmallNT) out[i] = base[i / per] + (int64_t)sh[lds_pad(i)];
  if (t == 0) *total = tot;
  if (pair_off) {
    __syncthreads();  // out[] of every thread is visible to the block after the barrier
    write_pair_off(out, tot, K, nblk, pair_off);
  }
}

__global__ void pair_off_kernel(const int64_t* __restrict__ out, const int64_t* __restrict__ total, int K, int nblk,
                                int64_t* __restrict__ pair_off) {
  write_pair_off(out, *total, K, nblk, pair_off);
}

template <bool kPopc>
__global__ __launch_bounds__(kNT) void tile_sums(const void* __restrict__ in, int64_t n,
                                                 int64_t* __restrict__ sums) {
  const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kPer;
  int64_t s = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i)
    if (base + i < n) s += elem<kPopc>(in, base + i);
  int64_t tot;
  block_excl_scan<kNT>(s, &tot);
  if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

// Single block: exclusive scan of nb tile sums in place; total written to *total.
__global__ __launch_bounds__(1024) void scan_sums(int64_t* __restrict__ sums, int64_t nb,
                                                  int64_t* __restrict__ total) {
  const int64_t per = (nb + 1023) / 1024;
  const int64_t b0 = (int64_t)threadIdx.x * per;
  int64_t s = 0;
  for (int64_t i = 0; i < per; ++i)
    if (b0 + i < nb) s += sums[b0 + i];
  int64_t tot;
  int64_t run = block_excl_scan<1024>(s, &tot);
  for (int64_t i = 0; i < per; ++i)
    if (b0 + i < nb) {
      int64_t v = sums[b0 + i];
      sums[b0 + i] = run;
      run += v;
    }
  if (threadIdx.x == 0) *total = tot;
}

template <bool kPopc>
__global__ __launch_bounds__(kNT) void tile_apply(const void* __restrict__ in, int64_t n,
                                                  const int64_t* __restrict__ offs, int64_t* __restrict__ out) {
  const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kPer;
  int64_t v[kPer];
  int64_t s = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    v[i] = (base + i < n) ? elem<kPopc>(in, base + i) : 0;
    s += v[i];
  }
  int64_t tot;
  int64_t run = block_excl_scan<kNT>(s, &tot) + offs[blockIdx.x];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    if (base + i < n) out[base + i] = run;
    run += v[i];
  }
}
}  // namespace

int64_t scan_tmp_elems(int64_t n) { return (n + kTile - 1) / kTile + 1; }

// One workgroup up to small_max elements (at most kSmallMax): measured, it beats the three
// passes on the 32 768 bitmap words of a 32^3 x 32 output grid but loses on 20 250 pair counts.
template <bool kPopc>
static int scan_impl(const void* in, int64_t n, int64_t* out, int64_t* total, int64_t* tmp, int K, int nblk,
                     int64_t* pair_off, int64_t small_max, hipStream_t stream) {
  if (n <= 0) {
    SSC_HIP(hipMemsetAsync(total, 0, sizeof(int64_t), stream));
    if (pair_off) SSC_HIP(hipMemsetAsync(pair_off, 0, (size_t)(K + 1) * sizeof(int64_t), stream));
    return SSCONV_OK;
  }
  if (n <= std::min(small_max, kSmallMax)) {
    scan_small<kPopc><<<1, kSmallNT, 0, stream>>>(in, n, out, total, K, nblk, pair_off);
  } else {
    const int64_t nb = (n + kTile - 1) / kTile;
    tile_sums<kPopc><<<(unsigned)nb, kNT, 0, stream>>>(in, n, tmp);
    scan_sums<<<1, 1024, 0, stream>>>(tmp, nb, total);
    tile_apply<kPopc><<<(unsigned)nb, kNT, 0, stream>>>(in, n, tmp, out);
    if (pair_off) pair_off_kernel<<<1, 256, 0, stream>>>(out, total, K, nblk, pair_off);
  }
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

int exclusive_scan(const int32_t* in, int64_t n, int64_t* out, int64_t* total, int64_t* tmp, hipStream_t stream) {
  return scan_impl<false>(in, n, out, total, tmp, 0, 0, nullptr, 16384, stream);
}

int exclusive_scan_popc(const uint32_t* words, int64_t n, int64_t* out, int64_t* total, int64_t* tmp,
                        hipStream_t stream) {
  return scan_impl<true>(words, n, out, total, tmp, 0, 0, nullptr, kSmallMax, stream);
}

int exclusive_scan_pair_off(const int32_t* counts, int K, int nblk, int64_t* out, int64_t* total, int64_t* tmp,
                            int64_t* pair_off, hipStream_t stream) {
  return scan_impl<false>(counts, (int64_t)K * nblk, out, total, tmp, K, nblk, pair_off, 16384, stream);
}

}  // namespace ssconv
