// Voxelisation of point clouds with per-cell feature averaging (Sec. 4.1: a site is active when
// its grid cell encloses a point, and its feature is the average over the enclosed points; the
// Feature-Steering module of Sec. 4.1 re-voxelises transformed sites the same way).
//
// The cell of a point is floor((p - origin) / voxel), subtraction and division in fp32 with
// round-to-nearest; points whose cell is outside the grid (or not finite) are dropped.  The active
// cells are marked in a bitmap over (batch, grid), whose popcount scan gives every cell its row
// in lexicographic (b, x, y, z) order.  Averages are deterministic without floating-point
// atomics: per-row point counts (integer atomics, whose returned values give each point a slot in
// its row's bucket), a scan to bucket offsets, a bucket fill (a plain scatter; the order inside a
// bucket is arbitrary), a pass that sorts every bucket by point index, and a pass that adds each
// site's points in that order and divides by the count.
#include <algorithm>
#include <cmath>

#include "bucket_sort.hpp"
#include "scan.hpp"

namespace ssconv {
namespace {

constexpr uint32_t kDropped = 0xFFFFFFFFu;
constexpr int kFlagBadBatch = 1;

// Cell key of every point ((b*G0 + x)*G1 + y)*G2 + z, or kDropped; marks the cell's bit.
__global__ void vox_cell_kernel(const float* __restrict__ pts, const int32_t* __restrict__ batch, int64_t n,
                                float ox, float oy, float oz, float voxel, int g0, int g1, int g2, int nbatch,
                                uint32_t* __restrict__ key, uint32_t* __restrict__ bits, int* __restrict__ flags) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool bad = false;
  if (i < n) {
    const float tx = __fdiv_rn(__fsub_rn(pts[3 * i + 0], ox), voxel);
    const float ty = __fdiv_rn(__fsub_rn(pts[3 * i + 1], oy), voxel);
    const float tz = __fdiv_rn(__fsub_rn(pts[3 * i + 2], oz), voxel);
    const int b = batch ? batch[i] : 0;
    bad = b < 0 || b >= nbatch;
    uint32_t k = kDropped;
    // NaN fails every comparison, so non-finite points are dropped here too
    if (!bad && tx >= 0.f && ty >= 0.f && tz >= 0.f && tx < (float)g0 && ty < (float)g1 && tz < (float)g2) {
      const uint32_t x = (uint32_t)floorf(tx), y = (uint32_t)floorf(ty), z = (uint32_t)floorf(tz);
      k = (((uint32_t)b * (uint32_t)g0 + x) * (uint32_t)g1 + y) * (uint32_t)g2 + z;
      atomicOr(&bits[k >> 5], 1u << (k & 31u));
    }
    key[i] = k;
  }
  const uint64_t any_bad = __ballot(bad);
  if (any_bad && (threadIdx.x & 63) == __ffsll((unsigned long long)any_bad) - 1) atomicOr(flags, kFlagBadBatch);
}

// Row of every point (rank of its cell's bit), the per-row point counts and each point's slot in
// its row's bucket (the count before its own increment).
__global__ void vox_row_kernel(const uint32_t* __restrict__ key, int64_t n, const uint32_t* __restrict__ bits,
                               const int64_t* __restrict__ woff, int32_t* __restrict__ point_row,
                               int32_t* __restrict__ cnt, int32_t* __restrict__ slot) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint32_t k = key[i];
  int32_t r = -1;
  if (k != kDropped) {
    const uint32_t w = k >> 5, b = k & 31u;
    r = (int32_t)(woff[w] + __popc(bits[w] & ((1u << b) - 1u)));
    slot[i] = atomicAdd(&cnt[r], 1);
  }
  point_row[i] = r;
}

// One thread per bitmap word: its set bits, in ascending order, write their sites' coordinates at
// consecutive ranks from the word's offset (only bits of cells inside the grid are ever set).
__global__ void vox_emit_kernel(const uint32_t* __restrict__ bits, int64_t nw, const int64_t* __restrict__ woff,
                                int g0, int g1, int g2, int32_t* __restrict__ coords) {
  const int64_t wd = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (wd >= nw) return;
  uint32_t m = bits[wd];
  int64_t r = woff[wd];
  const uint32_t g12 = (uint32_t)g1 * (uint32_t)g2, per_b = (uint32_t)g0 * g12;
  while (m) {
    const uint32_t k = (uint32_t)(wd * 32) + (uint32_t)(__ffs(m) - 1);
    m &= m - 1u;
    const uint32_t bb = k / per_b, rem = k - bb * per_b;
    const uint32_t x = rem / g12, yz = rem - x * g12;
    const uint32_t y = yz / (uint32_t)g2, z = yz - y * (uint32_t)g2;
    reinterpret_cast<int4*>(coords)[r++] = make_int4((int)bb, (int)x, (int)y, (int)z);
  }
}

// Bucket fill: point i goes to slot slot[i] of its row's bucket [start[r], start[r]+cnt[r]).
__global__ void vox_fill_kernel(const int32_t* __restrict__ point_row, int64_t n, const int64_t* __restrict__ start,
                                const int32_t* __restrict__ slot, int32_t* __restrict__ idx) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t r = point_row[i];
  if (r < 0) return;
  idx[start[r] + slot[i]] = (int32_t)i;
}


// feats_out[r][c] = (sum over the sorted bucket of feats[i][c], in point order) / count; one
// thread per (site, channel), so the threads of a site read its points' rows together.
__global__ void vox_mean_kernel(const float* __restrict__ feats, int C, const int64_t* __restrict__ n_rows,
                                const int64_t* __restrict__ start, const int32_t* __restrict__ cnt,
                                const int32_t* __restrict__ idx, float* __restrict__ out) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t r = e / C;
  if (r >= *n_rows) return;
  const int c = (int)(e - r * C);
  const int32_t* a = idx + start[r];
  const int m = cnt[r];
  float s = 0.f;
  for (int j = 0; j < m; ++j) s += feats[(int64_t)a[j] * C + c];
  out[r * C + c] = s / (float)m;
}

}  // namespace
}  // namespace ssconv

using namespace ssconv;

extern "C" int ssconv_voxelize(const float* points, const int32_t* batch, const float* feats, int64_t n, int channels,
                               const float* origin, float voxel, const int32_t* grid, int nbatch, int32_t* coords_out,
                               float* feats_out, int32_t* point_row, int64_t* n_sites, hipStream_t stream) {
  if (!origin || !grid || !n_sites) return fail(SSCONV_E_INVALID, "origin, grid and n_sites are required");
  *n_sites = 0;
  if (n < 0 || n > 0x7fffffffll) return fail(SSCONV_E_INVALID, "n must be in [0, 2^31)");
  if (channels < 0) return fail(SSCONV_E_INVALID, "channels must be >= 0");
  if (!(voxel > 0.f) || !std::isfinite(voxel)) return fail(SSCONV_E_INVALID, "voxel must be positive and finite");
  for (int a = 0; a < 3; ++a) {
    if (grid[a] < 1) return fail(SSCONV_E_INVALID, "grid extents must be positive");
    if (!std::isfinite(origin[a])) return fail(SSCONV_E_INVALID, "origin must be finite");
  }
  if (nbatch < 1) return fail(SSCONV_E_INVALID, "nbatch must be >= 1");
  const int64_t nbits = (int64_t)nbatch * grid[0] * grid[1] * grid[2];
  if (nbits > 0xFFFFFFFFll) return fail(SSCONV_E_BOUNDS, "nbatch * grid volume exceeds the 32-bit key space");
  if (n == 0) return SSCONV_OK;
  if (!points || !coords_out || (channels > 0 && (!feats || !feats_out)))
    return fail(SSCONV_E_INVALID, "NULL buffer");
  if (!aligned16(coords_out)) return fail(SSCONV_E_INVALID, "coords_out must be 16-byte aligned");

  const hipStream_t st = stream;
  const int64_t nw = (nbits + 31) / 32;
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t o_bits = 0, o_woff = o_bits + up(nw * 4), o_stmp = o_woff + up(nw * 8);
  const size_t o_key = o_stmp + up((size_t)(scan_tmp_elems(std::max<int64_t>(nw, n)) + 2) * 8);
  const size_t o_row = o_key + up(n * 4), o_cnt = o_row + up(n * 4), o_fill = o_cnt + up(n * 4);
  const size_t o_start = o_fill + up(n * 4), o_idx = o_start + up(n * 8), o_flags = o_idx + up(n * 4);
  const size_t o_big = o_flags + 256, total_b = o_big + up((n + 1) * 4);
  char* ws = nullptr;
  SSC_TRY(dev_alloc((void**)&ws, total_b, st));
  uint32_t* bits = (uint32_t*)(ws + o_bits);
  int64_t* woff = (int64_t*)(ws + o_woff);
  int64_t* stmp = (int64_t*)(ws + o_stmp);
  int64_t* d_sites = stmp + scan_tmp_elems(std::max<int64_t>(nw, n));
  int64_t* d_pts = d_sites + 1;
  uint32_t* key = (uint32_t*)(ws + o_key);
  int32_t* prow = point_row ? point_row : (int32_t*)(ws + o_row);
  int32_t* cnt = (int32_t*)(ws + o_cnt);
  int32_t* slot = (int32_t*)(ws + o_fill);  // each point's slot in its row's bucket
  int64_t* start = (int64_t*)(ws + o_start);
  int32_t* idx = (int32_t*)(ws + o_idx);
  int* flags = (int*)(ws + o_flags);
  int32_t* big = (int32_t*)(ws + o_big);

  int rc = SSCONV_OK;
  auto run = [&]() -> int {
    SSC_HIP(hipMemsetAsync(bits, 0, (size_t)nw * 4, st));
    SSC_HIP(hipMemsetAsync(cnt, 0, (size_t)n * 4, st));
    SSC_HIP(hipMemsetAsync(flags, 0, 4, st));
    vox_cell_kernel<<<cdiv(n, 256), 256, 0, st>>>(points, batch, n, origin[0], origin[1], origin[2], voxel, grid[0],
                                                  grid[1], grid[2], nbatch, key, bits, flags);
    SSC_TRY(exclusive_scan_popc(bits, nw, woff, d_sites, stmp, st));
    vox_row_kernel<<<cdiv(n, 256), 256, 0, st>>>(key, n, bits, woff, prow, cnt, slot);
    vox_emit_kernel<<<cdiv(nw, 256), 256, 0, st>>>(bits, nw, woff, grid[0], grid[1], grid[2], coords_out);
    if (channels > 0) {
      // rows past the site count have zero counts, so the scan over n rows is exact
      SSC_TRY(exclusive_scan(cnt, n, start, d_pts, stmp, st));
      vox_fill_kernel<<<cdiv(n, 256), 256, 0, st>>>(prow, n, start, slot, idx);
      SSC_TRY(sort_buckets(d_sites, 0, n, start, cnt, idx, big, true, st));
      vox_mean_kernel<<<cdiv(n * channels, 256), 256, 0, st>>>(feats, channels, d_sites, start, cnt, idx, feats_out);
    }
    SSC_HIP(hipGetLastError());
    int64_t host[2] = {0, 0};
    SSC_HIP(hipMemcpyAsync(&host[0], d_sites, 8, hipMemcpyDeviceToHost, st));
    SSC_HIP(hipMemcpyAsync(&host[1], flags, 4, hipMemcpyDeviceToHost, st));
    SSC_HIP(hipStreamSynchronize(st));
    if ((int)host[1] & kFlagBadBatch) return fail(SSCONV_E_BOUNDS, "a batch index lies outside [0, nbatch)");
    *n_sites = host[0];
    return SSCONV_OK;
  };
  rc = run();
  dev_free(ws, st);
  return rc;
}
