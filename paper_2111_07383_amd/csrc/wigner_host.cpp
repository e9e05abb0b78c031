// Wigner-D matrices of the real spherical-harmonic basis on the host (Sec. 3.1, Eq. 4-5: a
// feature field of order l transforms by D^l(r) under a rotation r).
//
// Real harmonics Y_l^m, m = -l..l, orthonormal on the sphere, without the Condon-Shortley phase
// (Y_1 is proportional to (y, z, x)):  Y_l^0 = N_l^0 P_l^0(cos t), Y_l^m = sqrt2 N_l^m P_l^m(cos t)
// cos(m p) for m > 0 and sqrt2 N_l^|m| P_l^|m|(cos t) sin(|m| p) for m < 0, with the associated
// Legendre functions P_l^m taken without the (-1)^m factor.  D^l(r) is defined by
// Y^l(r u) = D^l(r) Y^l(u); by orthonormality D^l(r)_{ab} = integral over the sphere of
// Y_a(r u) Y_b(u), a polynomial of degree 2l in u, which a product rule of 5 Gauss-Legendre nodes
// in cos t and 10 uniform angles in p integrates exactly for l <= 4.
#include <algorithm>
#include <cmath>
#include <vector>

#include "common.hpp"

namespace ssconv {

namespace {

constexpr int kNTheta = 5, kNPhi = 10;

// Gauss-Legendre nodes and weights on [-1, 1] by Newton's method on P_n.
void gauss_legendre(int n, double* x, double* w) {
  for (int i = 0; i < n; ++i) {
    double z = std::cos(M_PI * (i + 0.75) / (n + 0.5));
    for (int it = 0; it < 100; ++it) {
      double p0 = 1.0, p1 = z;
      for (int k = 2; k <= n; ++k) {
        const double p2 = ((2.0 * k - 1.0) * z * p1 - (k - 1.0) * p0) / k;
        p0 = p1;
        p1 = p2;
      }
      const double dp = n * (z * p1 - p0) / (z * z - 1.0);
      const double dz = p1 / dp;
      z -= dz;
      if (std::fabs(dz) < 1e-16) break;
    }
    double p0 = 1.0, p1 = z;
    for (int k = 2; k <= n; ++k) {
      const double p2 = ((2.0 * k - 1.0) * z * p1 - (k - 1.0) * p0) / k;
      p0 = p1;
      p1 = p2;
    }
    const double dp = n * (z * p1 - p0) / (z * z - 1.0);
    x[i] = z;
    w[i] = 2.0 / ((1.0 - z * z) * dp * dp);
  }
}

// Y_l^m(u), m = -l..l, for a unit vector u.
void real_harmonics(int l, const double u[3], double* y) {
  const double ct = std::max(-1.0, std::min(1.0, u[2]));
  const double st = std::sqrt(std::max(0.0, 1.0 - ct * ct));
  const double ph = std::atan2(u[1], u[0]);
  for (int m = 0; m <= l; ++m) {
    // P_l^m(ct) without the Condon-Shortley factor: P_m^m = (2m-1)!! st^m, then the l-recurrence
    double pmm = 1.0;
    for (int k = 1; k <= m; ++k) pmm *= (2.0 * k - 1.0) * st;
    double plm = pmm;
    if (l > m) {
      double pm1 = ct * (2.0 * m + 1.0) * pmm;  // P_{m+1}^m
      double a = pmm, b = pm1;
      for (int ll = m + 2; ll <= l; ++ll) {
        const double c = ((2.0 * ll - 1.0) * ct * b - (ll + m - 1.0) * a) / (ll - m);
        a = b;
        b = c;
      }
      plm = b;
    }
    double ratio = 1.0;  // (l - m)! / (l + m)!
    for (int k = l - m + 1; k <= l + m; ++k) ratio /= k;
    const double N = std::sqrt((2.0 * l + 1.0) / (4.0 * M_PI) * ratio);
    if (m == 0) {
      y[l] = N * plm;
    } else {
      y[l + m] = std::sqrt(2.0) * N * plm * std::cos(m * ph);
      y[l - m] = std::sqrt(2.0) * N * plm * std::sin(m * ph);
    }
  }
}

}  // namespace

// D^l(r) row-major [(2l+1) x (2l+1)] for l <= SSCONV_MAX_L; r row-major 3x3 (applied as r u).
void wigner_d(int l, const double* r, double* D) {
  const int d = 2 * l + 1;
  for (int i = 0; i < d * d; ++i) D[i] = 0.0;
  double gx[kNTheta], gw[kNTheta];
  gauss_legendre(kNTheta, gx, gw);
  std::vector<double> ya(d), yb(d);
  for (int i = 0; i < kNTheta; ++i) {
    const double ct = gx[i], st = std::sqrt(1.0 - ct * ct);
    for (int j = 0; j < kNPhi; ++j) {
      const double ph = 2.0 * M_PI * j / kNPhi;
      const double u[3] = {st * std::cos(ph), st * std::sin(ph), ct};
      const double ru[3] = {r[0] * u[0] + r[1] * u[1] + r[2] * u[2], r[3] * u[0] + r[4] * u[1] + r[5] * u[2],
                            r[6] * u[0] + r[7] * u[1] + r[8] * u[2]};
      real_harmonics(l, ru, ya.data());
      real_harmonics(l, u, yb.data());
      const double w = gw[i] * 2.0 * M_PI / kNPhi;
      for (int a = 0; a < d; ++a)
        for (int b = 0; b < d; ++b) D[a * d + b] += w * ya[a] * yb[b];
    }
  }
}

}  // namespace ssconv

extern "C" int ssconv_wigner_d(int l, const double* rot, double* D) {
  using namespace ssconv;
  if (l < 0 || l > SSCONV_MAX_L) return fail(SSCONV_E_INVALID, "l must be in 0..%d", SSCONV_MAX_L);
  if (!rot || !D) return fail(SSCONV_E_INVALID, "NULL argument");
  wigner_d(l, rot, D);
  return SSCONV_OK;
}
