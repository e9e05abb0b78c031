// Feature-Steering of a sparse tensor by a rigid motion (r, t) (Sec. 4.1): every field of order l
// is rotated by its Wigner-D matrix D^l(r) (the block-diagonal rho(r) of Eq. 5, applied as a
// matrix product), every site is taken to the centre of its cell, origin + (x + 1/2) voxel, moved
// to r p + t, and the moved points are re-voxelised with the features of sites that land in one
// cell averaged (the voxelisation of voxel.hip).  The centre and the moved point are computed in
// fp32 with every product and sum rounded to nearest in a fixed order, because they decide the
// integer cells.
#include <algorithm>
#include <cmath>

#include "common.hpp"

namespace ssconv {

void wigner_d(int l, const double* r, double* D);

namespace {

constexpr int kDFloats = 1 + 9 + 25 + 49 + 81;  // D^0 .. D^4, row-major, concatenated

struct SteerArgs {
  FieldTab f;
  float D[kDFloats];
  float r[9], t[3], origin[3], voxel;
};

__host__ __device__ constexpr int d_offset(int l) { return l == 0 ? 0 : l == 1 ? 1 : l == 2 ? 10 : l == 3 ? 35 : 84; }

// One thread per site: its moved cell centre and its batch index.
__global__ void steer_points_kernel(SteerArgs a, const int32_t* __restrict__ coords, int64_t n,
                                    float* __restrict__ pts, int32_t* __restrict__ batch) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int4 c = reinterpret_cast<const int4*>(coords)[i];
  const float p[3] = {__fadd_rn(__fmul_rn(__fadd_rn((float)c.y, 0.5f), a.voxel), a.origin[0]),
                      __fadd_rn(__fmul_rn(__fadd_rn((float)c.z, 0.5f), a.voxel), a.origin[1]),
                      __fadd_rn(__fmul_rn(__fadd_rn((float)c.w, 0.5f), a.voxel), a.origin[2])};
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const float s = __fadd_rn(__fadd_rn(__fmul_rn(a.r[3 * k], p[0]), __fmul_rn(a.r[3 * k + 1], p[1])),
                              __fmul_rn(a.r[3 * k + 2], p[2]));
    pts[3 * i + k] = __fadd_rn(s, a.t[k]);
  }
  batch[i] = c.x;
}

// One thread per (site, field): out field = D^l(r) x field.
__global__ void steer_rotate_kernel(SteerArgs a, const float* __restrict__ f, int64_t n, float* __restrict__ out) {
  const int n_fields = a.f.f0[a.f.n], C = a.f.ch0[a.f.n];
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n * n_fields) return;
  const int64_t row = i / n_fields;
  const int field = (int)(i - row * n_fields);
  int e = 0;
  while (e + 1 < a.f.n && field >= a.f.f0[e + 1]) ++e;
  const int l = a.f.l[e], d = 2 * l + 1;
  const int c0 = a.f.ch0[e] + (field - a.f.f0[e]) * d;
  const float* x = f + row * C + c0;
  float* y = out + row * C + c0;
  const float* D = a.D + d_offset(l);
  float v[2 * SSCONV_MAX_L + 1];
  for (int k = 0; k < d; ++k) v[k] = x[k];
  for (int r = 0; r < d; ++r) {
    float s = 0.f;
    for (int k = 0; k < d; ++k) s = fmaf(D[r * d + k], v[k], s);
    y[r] = s;
  }
}

}  // namespace
}  // namespace ssconv

using namespace ssconv;

extern "C" int ssconv_steer(const int32_t* coords, const float* feats, int64_t n, const ssconv_fields* fields,
                            const double* rot, const double* trans, const float* origin, float voxel,
                            const int32_t* grid, int nbatch, int32_t* coords_out, float* feats_out,
                            int32_t* site_row, int64_t* n_sites, hipStream_t stream) {
  if (!rot || !trans || !origin || !grid || !n_sites) return fail(SSCONV_E_INVALID, "NULL host argument");
  *n_sites = 0;
  SteerArgs a;
  SSC_TRY(make_fieldtab(fields, &a.f));
  const int C = a.f.ch0[a.f.n];
  // r must be a proper rotation (orthonormal, det +1)
  double dev = 0.0;
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 3; ++j) {
      double s = 0.0;
      for (int k = 0; k < 3; ++k) s += rot[3 * i + k] * rot[3 * j + k];
      dev = std::max(dev, std::fabs(s - (i == j ? 1.0 : 0.0)));
    }
  const double det = rot[0] * (rot[4] * rot[8] - rot[5] * rot[7]) - rot[1] * (rot[3] * rot[8] - rot[5] * rot[6]) +
                     rot[2] * (rot[3] * rot[7] - rot[4] * rot[6]);
  if (!(dev < 1e-6) || !(std::fabs(det - 1.0) < 1e-6)) return fail(SSCONV_E_INVALID, "rot is not a rotation");
  for (int k = 0; k < 3; ++k)
    if (!std::isfinite(trans[k])) return fail(SSCONV_E_INVALID, "trans must be finite");
  if (n < 0 || n > 0x7fffffffll) return fail(SSCONV_E_INVALID, "n must be in [0, 2^31)");
  if (n > 0 && (!coords || !feats || !aligned16(coords))) return fail(SSCONV_E_INVALID, "bad coords / feats");
  for (int l = 0; l <= SSCONV_MAX_L; ++l) {
    double D[81];
    wigner_d(l, rot, D);
    for (int k = 0; k < (2 * l + 1) * (2 * l + 1); ++k) a.D[d_offset(l) + k] = (float)D[k];
  }
  for (int k = 0; k < 9; ++k) a.r[k] = (float)rot[k];
  for (int k = 0; k < 3; ++k) {
    a.t[k] = (float)trans[k];
    a.origin[k] = origin[k];
  }
  a.voxel = voxel;
  if (n == 0) return ssconv_voxelize(nullptr, nullptr, nullptr, 0, C, origin, voxel, grid, nbatch, coords_out,
                                     feats_out, site_row, n_sites, stream);
  char* ws = nullptr;
  const size_t o_pts = 0, o_b = (n * 12 + 255) & ~(size_t)255, o_f = o_b + ((n * 4 + 255) & ~(size_t)255);
  SSC_TRY(dev_alloc((void**)&ws, o_f + (size_t)n * C * 4 + 256, stream));
  float* pts = (float*)(ws + o_pts);
  int32_t* bat = (int32_t*)(ws + o_b);
  float* rf = (float*)(ws + o_f);
  steer_points_kernel<<<cdiv(n, 256), 256, 0, stream>>>(a, coords, n, pts, bat);
  const int64_t work = n * a.f.f0[a.f.n];
  if (work > 0) steer_rotate_kernel<<<cdiv(work, 256), 256, 0, stream>>>(a, feats, n, rf);
  int rc = SSCONV_OK;
  if (hipGetLastError() != hipSuccess) rc = fail(SSCONV_E_HIP, "steering launch failed");
  if (rc == SSCONV_OK)
    rc = ssconv_voxelize(pts, bat, rf, n, C, origin, voxel, grid, nbatch, coords_out, feats_out, site_row, n_sites,
                         stream);
  dev_free(ws, stream);
  return rc;
}
