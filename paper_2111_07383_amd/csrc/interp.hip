// Tensor-to-Point: trilinear interpolation of a sparse tensor at points, and its adjoint (Sec. 4.1
// interpolates point-wise features from the sparse backbone maps).
//
// The features live at the cell centres origin + (x + 1/2) voxel of the active sites and are zero
// elsewhere; a point is the trilinear blend of the 8 site centres around it.  With
// u = (p - origin) / voxel - 1/2 (fp32, rounded to nearest in that order: floor(u) decides which
// sites are read), x0 = floor(u), w = u - x0, corner x0 + c (c in {0,1}^3, index 4 cx + 2 cy + cz)
// has weight prod_a (c_a ? w_a : 1 - w_a).  Corners are found in the rule book's coordinate hash;
// corners outside the grid or inactive contribute nothing, and points never read sites of
// another batch entry.  The backward pass is the exact adjoint, deterministic: the (point,
// corner) entries of every site are bucketed (integer-atomic counts, whose returned values are the
// entries' slots in their buckets, a scan, a plain scatter), each bucket is sorted by entry index,
// and every site adds weight * grad over its bucket in that order.
#include <algorithm>
#include <cmath>

#include "hash.hpp"
#include "bucket_sort.hpp"
#include "scan.hpp"

namespace ssconv {
namespace {

// Per point: the site row (or -1) and weight of each of its 8 corners.
__global__ void interp_corners_kernel(const float* __restrict__ pts, const int32_t* __restrict__ batch, int64_t m,
                                      float ox, float oy, float oz, float voxel, int g0, int g1, int g2, int bmax,
                                      const uint64_t* __restrict__ slots, uint64_t mask, int32_t* __restrict__ rows,
                                      float* __restrict__ wts) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= m) return;
  const float o[3] = {ox, oy, oz};
  const int g[3] = {g0, g1, g2};
  float w[3];
  int x0[3];
  bool ok = true;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    const float u = __fsub_rn(__fdiv_rn(__fsub_rn(pts[3 * i + a], o[a]), voxel), 0.5f);
    ok = ok && isfinite(u) && fabsf(u) < 1e9f;
    const float f = floorf(u);
    x0[a] = ok ? (int)f : 0;
    w[a] = __fsub_rn(u, f);  // exact: u - floor(u)
  }
  const int b = batch ? batch[i] : 0;
  ok = ok && b >= 0 && b <= bmax;  // larger b would wrap the 32-bit key onto other sites
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int cx = (k >> 2) & 1, cy = (k >> 1) & 1, cz = k & 1;
    const int x = x0[0] + cx, y = x0[1] + cy, z = x0[2] + cz;
    int r = -1;
    if (ok && x >= 0 && y >= 0 && z >= 0 && x < g[0] && y < g[1] && z < g[2])
      r = hash_find(slots, mask, site_key(b, x, y, z, g0, g1, g2));
    rows[i * 8 + k] = r;
    wts[i * 8 + k] = (cx ? w[0] : 1.f - w[0]) * (cy ? w[1] : 1.f - w[1]) * (cz ? w[2] : 1.f - w[2]);
  }
}

// out[i][c..c+V) = sum over the corners, in corner order, of weight * feats[row][c..c+V)
// (V = 4 with 16-byte accesses when C % 4 == 0).
template <int V>
__global__ void interp_fwd_kernel(const float* __restrict__ feats, int C, const int32_t* __restrict__ rows,
                                  const float* __restrict__ wts, int64_t m, float* __restrict__ out) {
  const int nv = C / V;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= m * nv) return;
  const int64_t i = e / nv;
  const int c = (int)(e - i * nv) * V;
  float s[V];
#pragma unroll
  for (int v = 0; v < V; ++v) s[v] = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int32_t r = rows[i * 8 + k];
    if (r < 0) continue;
    const float w = wts[i * 8 + k];
    if constexpr (V == 4) {
      const float4 f = *reinterpret_cast<const float4*>(feats + (int64_t)r * C + c);
      s[0] = fmaf(w, f.x, s[0]);
      s[1] = fmaf(w, f.y, s[1]);
      s[2] = fmaf(w, f.z, s[2]);
      s[3] = fmaf(w, f.w, s[3]);
    } else {
      s[0] = fmaf(w, feats[(int64_t)r * C + c], s[0]);
    }
  }
  if constexpr (V == 4)
    *reinterpret_cast<float4*>(out + i * C + c) = make_float4(s[0], s[1], s[2], s[3]);
  else
    out[i * C + c] = s[0];
}

// Per-site entry counts; slot[e] = the count before entry e's own increment (its bucket slot).
__global__ void interp_count_kernel(const int32_t* __restrict__ rows, int64_t ne, int32_t* __restrict__ cnt,
                                    int32_t* __restrict__ slot) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < ne && rows[e] >= 0) slot[e] = atomicAdd(&cnt[rows[e]], 1);
}

// Bucket fill: entry e = 8 * point + corner goes to slot slot[e] of its site's bucket (the order
// inside a bucket is that of the atomics, sorted afterwards).
__global__ void interp_fill_kernel(const int32_t* __restrict__ rows, int64_t ne, const int64_t* __restrict__ start,
                                   const int32_t* __restrict__ slot, int32_t* __restrict__ ent) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= ne) return;
  const int32_t r = rows[e];
  if (r >= 0) ent[start[r] + slot[e]] = (int32_t)e;
}

// grad_feats[r][c..c+V) = sum over the sorted bucket of weight * grad[point][c..c+V); every site
// row written (V = 4 with 16-byte accesses when C % 4 == 0).
template <int V>
__global__ void interp_bwd_kernel(const float* __restrict__ grad, int C, const float* __restrict__ wts,
                                  const int64_t* __restrict__ start, const int32_t* __restrict__ cnt,
                                  const int32_t* __restrict__ ent, int64_t n, float* __restrict__ gf) {
  const int nv = C / V;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n * nv) return;
  const int64_t r = e / nv;
  const int c = (int)(e - r * nv) * V;
  const int32_t* a = ent + start[r];
  const int mcount = cnt[r];
  float s[V];
#pragma unroll
  for (int v = 0; v < V; ++v) s[v] = 0.f;
  for (int j = 0; j < mcount; ++j) {
    const int32_t en = a[j];
    const float w = wts[en];
    const float* g = grad + (int64_t)(en >> 3) * C + c;
    if constexpr (V == 4) {
      const float4 x = *reinterpret_cast<const float4*>(g);
      s[0] = fmaf(w, x.x, s[0]);
      s[1] = fmaf(w, x.y, s[1]);
      s[2] = fmaf(w, x.z, s[2]);
      s[3] = fmaf(w, x.w, s[3]);
    } else {
      s[0] = fmaf(w, g[0], s[0]);
    }
  }
  if constexpr (V == 4)
    *reinterpret_cast<float4*>(gf + r * C + c) = make_float4(s[0], s[1], s[2], s[3]);
  else
    gf[r * C + c] = s[0];
}

int interp_args(ssconv_rulebook_t rb, int C, const float* points, int64_t m, const float* origin, float voxel) {
  if (!rb) return fail(SSCONV_E_INVALID, "NULL rule book");
  SSC_TRY(rulebook_settle(rb));
  if (C < 1) return fail(SSCONV_E_INVALID, "channels must be positive");
  if (m < 0 || m > 0x0fffffffll) return fail(SSCONV_E_INVALID, "m must be in [0, 2^28)");
  if (!origin || !(voxel > 0.f) || !std::isfinite(voxel)) return fail(SSCONV_E_INVALID, "bad origin / voxel");
  for (int a = 0; a < 3; ++a)
    if (!std::isfinite(origin[a])) return fail(SSCONV_E_INVALID, "origin must be finite");
  if (m > 0 && !points) return fail(SSCONV_E_INVALID, "NULL points");
  return SSCONV_OK;
}

// Fills the corner table: rows [m*8] int32 (site row or -1) and weights [m*8] fp32.
void launch_corners(ssconv_rulebook_t rb, const float* points, const int32_t* batch, int64_t m, const float* origin,
                    float voxel, int32_t* rows, float* wts, hipStream_t st) {
  // the largest batch index whose keys fit 32 bits (key ~0 is reserved), as in the rule book
  const int64_t cells = (int64_t)rb->grid[0] * rb->grid[1] * rb->grid[2];
  const int bmax = (int)std::min<int64_t>(0xFFFFFFFFll / cells - 1, 0x7fffffff);
  interp_corners_kernel<<<cdiv(m, 256), 256, 0, st>>>(points, batch, m, origin[0], origin[1], origin[2], voxel,
                                                      rb->grid[0], rb->grid[1], rb->grid[2], bmax, rb->hash_in,
                                                      (uint64_t)(rb->cap_in - 1), rows, wts);
}

}  // namespace
}  // namespace ssconv

using namespace ssconv;

extern "C" int ssconv_interpolate(ssconv_rulebook_t rb, const float* feats, int channels, const float* points,
                                  const int32_t* batch, int64_t m, const float* origin, float voxel, float* out,
                                  hipStream_t stream) {
  SSC_TRY(interp_args(rb, channels, points, m, origin, voxel));
  if (m == 0) return SSCONV_OK;
  if (!out || (rb->n_in > 0 && !feats)) return fail(SSCONV_E_INVALID, "NULL feature buffer");
  if (rb->n_in == 0) {
    SSC_HIP(hipMemsetAsync(out, 0, (size_t)m * channels * 4, stream));
    return SSCONV_OK;
  }
  char* ws = nullptr;
  const size_t o_w = ((size_t)m * 32 + 255) & ~(size_t)255;
  SSC_TRY(dev_alloc((void**)&ws, o_w + (size_t)m * 32, stream));
  int32_t* rows = (int32_t*)ws;
  float* wts = (float*)(ws + o_w);
  launch_corners(rb, points, batch, m, origin, voxel, rows, wts, stream);
  if (channels % 4 == 0 && aligned16(feats) && aligned16(out))
    interp_fwd_kernel<4><<<cdiv(m * channels / 4, 256), 256, 0, stream>>>(feats, channels, rows, wts, m, out);
  else
    interp_fwd_kernel<1><<<cdiv(m * channels, 256), 256, 0, stream>>>(feats, channels, rows, wts, m, out);
  int rc = SSCONV_OK;
  if (hipGetLastError() != hipSuccess) rc = fail(SSCONV_E_HIP, "interpolation launch failed");
  dev_free(ws, stream);
  return rc;
}

extern "C" int ssconv_interpolate_backward(ssconv_rulebook_t rb, const float* grad, int channels, const float* points,
                                           const int32_t* batch, int64_t m, const float* origin, float voxel,
                                           float* grad_feats, hipStream_t stream) {
  SSC_TRY(interp_args(rb, channels, points, m, origin, voxel));
  const int64_t n = rb->n_in;
  if (n == 0) return SSCONV_OK;
  if (!grad_feats || (m > 0 && !grad)) return fail(SSCONV_E_INVALID, "NULL gradient buffer");
  if (m == 0) {
    SSC_HIP(hipMemsetAsync(grad_feats, 0, (size_t)n * channels * 4, stream));
    return SSCONV_OK;
  }
  const int64_t ne = m * 8;
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t o_w = up(ne * 4), o_cnt = o_w + up(ne * 4), o_fill = o_cnt + up(n * 4), o_start = o_fill + up(ne * 4);
  const size_t o_ent = o_start + up(n * 8), o_tmp = o_ent + up(ne * 4);
  const size_t o_big = o_tmp + up((size_t)(scan_tmp_elems(n) + 1) * 8), total = o_big + up((n + 1) * 4);
  char* ws = nullptr;
  SSC_TRY(dev_alloc((void**)&ws, total, stream));
  int32_t* rows = (int32_t*)ws;
  float* wts = (float*)(ws + o_w);
  int32_t* cnt = (int32_t*)(ws + o_cnt);
  int32_t* slot = (int32_t*)(ws + o_fill);  // each entry's slot in its site's bucket
  int64_t* start = (int64_t*)(ws + o_start);
  int32_t* ent = (int32_t*)(ws + o_ent);
  int64_t* tmp = (int64_t*)(ws + o_tmp);
  int32_t* big = (int32_t*)(ws + o_big);
  auto run = [&]() -> int {
    SSC_HIP(hipMemsetAsync(cnt, 0, (size_t)n * 4, stream));
    launch_corners(rb, points, batch, m, origin, voxel, rows, wts, stream);
    interp_count_kernel<<<cdiv(ne, 256), 256, 0, stream>>>(rows, ne, cnt, slot);
    SSC_TRY(exclusive_scan(cnt, n, start, tmp + scan_tmp_elems(n), tmp, stream));
    interp_fill_kernel<<<cdiv(ne, 256), 256, 0, stream>>>(rows, ne, start, slot, ent);
    SSC_TRY(sort_buckets(nullptr, n, n, start, cnt, ent, big, false, stream));
    if (channels % 4 == 0 && aligned16(grad) && aligned16(grad_feats))
      interp_bwd_kernel<4><<<cdiv(n * channels / 4, 256), 256, 0, stream>>>(grad, channels, wts, start, cnt, ent, n,
                                                                            grad_feats);
    else
      interp_bwd_kernel<1><<<cdiv(n * channels, 256), 256, 0, stream>>>(grad, channels, wts, start, cnt, ent, n,
                                                                        grad_feats);
    SSC_HIP(hipGetLastError());
    return SSCONV_OK;
  };
  const int rc = run();
  dev_free(ws, stream);
  return rc;
}
