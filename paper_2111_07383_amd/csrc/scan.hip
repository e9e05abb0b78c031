// Device-wide exclusive scan in three passes: per-tile sums, one-block scan of
// the tile sums, per-tile rescan with the tile offset.  Deterministic.
#include "scan.hpp"

namespace ssconv {

namespace {
constexpr int kNT = 256;
constexpr int kPer = 16;                 // elements per thread
constexpr int kTile = kNT * kPer;        // elements per block

__global__ __launch_bounds__(kNT) void tile_sums(const int32_t* __restrict__ in, int64_t n,
                                                 int64_t* __restrict__ sums) {
  const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kPer;
  int64_t s = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i)
    if (base + i < n) s += in[base + i];
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

__global__ __launch_bounds__(kNT) void tile_apply(const int32_t* __restrict__ in, int64_t n,
                                                  const int64_t* __restrict__ offs, int64_t* __restrict__ out) {
  const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kPer;
  int64_t v[kPer];
  int64_t s = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    v[i] = (base + i < n) ? in[base + i] : 0;
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

int exclusive_scan(const int32_t* in, int64_t n, int64_t* out, int64_t* total, int64_t* tmp, hipStream_t stream) {
  if (n <= 0) {
    SSC_HIP(hipMemsetAsync(total, 0, sizeof(int64_t), stream));
    return SSCONV_OK;
  }
  const int64_t nb = (n + kTile - 1) / kTile;
  tile_sums<<<(unsigned)nb, kNT, 0, stream>>>(in, n, tmp);
  scan_sums<<<1, 1024, 0, stream>>>(tmp, nb, total);
  tile_apply<<<(unsigned)nb, kNT, 0, stream>>>(in, n, tmp, out);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

}  // namespace ssconv
