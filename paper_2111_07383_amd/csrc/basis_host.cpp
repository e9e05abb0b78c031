// Host construction of the steerable basis kernels (Sec. 3.2.1, Eq. 7-8).
//
// kappa^{kl,Jm}(s) = phi^m(|s|) sum_j Y^J_j(s/|s|) Q^{kl,J}_j,  phi^m(r) = exp(-(r-m)^2 / (2 eps^2)).
//
// Q^{kl,J} is the Clebsch-Gordan intertwiner of orders k (out) and l (in)
// into J.  Here it is computed from the complex Clebsch-Gordan coefficients
// (Racah's closed formula, Condon-Shortley convention) and carried to the real
// spherical-harmonic basis used for features (no Condon-Shortley phase,
// components m = -l..l, Y_1 ~ (y, z, x)) by the unitary complex-to-real change
// of basis A_l:
//     Q'_{j a b} = sum conj(A^J_{j j'}) A^k_{a a'} A^l_{b b'} <k a'; l b' | J j'>.
// Q' satisfies sum_j D^J_{j j'} Q'_j = D^k Q'_{j'} (D^l)^T for the real
// Wigner-D matrices of the features, which is the kernel constraint of Eq. 4;
// its real (or imaginary) part is the real solution, unique up to scale.
// Each element is then normalised to unit Frobenius norm over (offset, row,
// column) with its first entry above 1e-3 of its maximum made positive, so the
// result does not depend on phase or scale conventions.
#include <cmath>
#include <complex>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"

namespace ssconv {
namespace {

using cplx = std::complex<double>;
constexpr double kPi = 3.14159265358979323846;

double fact(int n) {
  double r = 1.0;
  for (int i = 2; i <= n; ++i) r *= i;
  return r;
}

// <j1 m1; j2 m2 | J M> by Racah's formula.
double clebsch_gordan(int j1, int m1, int j2, int m2, int J, int M) {
  if (M != m1 + m2) return 0.0;
  if (J < std::abs(j1 - j2) || J > j1 + j2) return 0.0;
  if (std::abs(m1) > j1 || std::abs(m2) > j2 || std::abs(M) > J) return 0.0;
  double pre = std::sqrt((2.0 * J + 1.0) * fact(j1 + j2 - J) * fact(j1 - j2 + J) * fact(-j1 + j2 + J) /
                         fact(j1 + j2 + J + 1));
  pre *= std::sqrt(fact(j1 + m1) * fact(j1 - m1) * fact(j2 + m2) * fact(j2 - m2) * fact(J + M) * fact(J - M));
  double sum = 0.0;
  for (int k = 0; k <= j1 + j2 + J; ++k) {
    int a = j1 + j2 - J - k, b = j1 - m1 - k, c = j2 + m2 - k, d = J - j2 + m1 + k, e = J - j1 - m2 + k;
    if (a < 0 || b < 0 || c < 0 || d < 0 || e < 0) continue;
    double den = fact(k) * fact(a) * fact(b) * fact(c) * fact(d) * fact(e);
    sum += ((k & 1) ? -1.0 : 1.0) / den;
  }
  return pre * sum;
}

// Associated Legendre P_l^m(x) without the Condon-Shortley phase, s = sqrt(1 - x^2).
double legendre(int l, int m, double x, double s) {
  double pmm = 1.0;
  for (int i = 1; i <= m; ++i) pmm *= (2.0 * i - 1.0) * s;
  if (l == m) return pmm;
  double pm1 = x * (2.0 * m + 1.0) * pmm;
  if (l == m + 1) return pm1;
  double pll = 0.0;
  for (int ll = m + 2; ll <= l; ++ll) {
    pll = ((2.0 * ll - 1.0) * x * pm1 - (ll + m - 1.0) * pmm) / (ll - m);
    pmm = pm1;
    pm1 = pll;
  }
  return pll;
}

// Real spherical harmonics Y^J_j(v/|v|), j = -J..J, into out[2J+1].  At v = 0 the
// direction is undefined: Y^0 = 1/(2 sqrt(pi)), Y^{J>0} = 0.
void real_sh(int J, const double v[3], double* out) {
  double r = std::sqrt(v[0] * v[0] + v[1] * v[1] + v[2] * v[2]);
  for (int j = 0; j < 2 * J + 1; ++j) out[j] = 0.0;
  if (r < 1e-12) {
    if (J == 0) out[0] = 0.5 / std::sqrt(kPi);
    return;
  }
  double ct = v[2] / r;
  double st = std::sqrt(std::max(0.0, 1.0 - ct * ct));
  double ph = std::atan2(v[1], v[0]);
  for (int m = 0; m <= J; ++m) {
    double nrm = std::sqrt((2.0 * J + 1.0) / (4.0 * kPi) * fact(J - m) / fact(J + m));
    double p = legendre(J, m, ct, st);
    if (m == 0) {
      out[J] = nrm * p;
    } else {
      out[J + m] = std::sqrt(2.0) * nrm * p * std::cos(m * ph);
      out[J - m] = std::sqrt(2.0) * nrm * p * std::sin(m * ph);
    }
  }
}

// Complex-to-real change of basis: Y_real[mu] = sum_m A[mu][m] Y_complex[m].
cplx c2r(int mu, int m) {
  const double h = 1.0 / std::sqrt(2.0);
  if (mu == 0) return m == 0 ? cplx(1.0, 0.0) : cplx(0.0, 0.0);
  if (mu > 0) {
    if (m == mu) return cplx(((mu & 1) ? -1.0 : 1.0) * h, 0.0);
    if (m == -mu) return cplx(h, 0.0);
    return cplx(0.0, 0.0);
  }
  int nu = -mu;
  if (m == nu) return cplx(0.0, -((nu & 1) ? -1.0 : 1.0) * h);
  if (m == -nu) return cplx(0.0, h);
  return cplx(0.0, 0.0);
}

// Real intertwiner Q[j][a][b] ((2J+1) x (2k+1) x (2l+1)), unnormalised.
std::vector<double> real_intertwiner(int k, int l, int J) {
  const int dJ = 2 * J + 1, dk = 2 * k + 1, dl = 2 * l + 1;
  std::vector<cplx> q(dJ * dk * dl);
  for (int j = -J; j <= J; ++j)
    for (int a = -k; a <= k; ++a)
      for (int b = -l; b <= l; ++b) {
        cplx acc(0.0, 0.0);
        for (int j2 = -J; j2 <= J; ++j2) {
          cplx aj = std::conj(c2r(j, j2));
          if (aj == cplx(0.0, 0.0)) continue;
          for (int a2 = -k; a2 <= k; ++a2) {
            cplx ak = c2r(a, a2);
            if (ak == cplx(0.0, 0.0)) continue;
            int b2 = j2 - a2;
            if (b2 < -l || b2 > l) continue;
            cplx al = c2r(b, b2);
            if (al == cplx(0.0, 0.0)) continue;
            acc += aj * ak * al * clebsch_gordan(k, a2, l, b2, J, j2);
          }
        }
        q[((j + J) * dk + (a + k)) * dl + (b + l)] = acc;
      }
  double nr = 0.0, ni = 0.0;
  for (auto& v : q) {
    nr += v.real() * v.real();
    ni += v.imag() * v.imag();
  }
  std::vector<double> out(q.size());
  for (size_t i = 0; i < q.size(); ++i) out[i] = nr >= ni ? q[i].real() : q[i].imag();
  return out;
}

bool valid_fields(const ssconv_fields& f) {
  if (f.n < 1 || f.n > SSCONV_MAX_ENTRIES) return false;
  for (int e = 0; e < f.n; ++e)
    if (f.l[e] < 0 || f.l[e] > SSCONV_MAX_L || f.mult[e] < 1) return false;
  return true;
}

}  // namespace

int validate_desc(const ssconv_basis_desc* d) {
  if (!d) return fail(SSCONV_E_INVALID, "basis descriptor is NULL");
  if (!valid_fields(d->in) || !valid_fields(d->out))
    return fail(SSCONV_E_INVALID, "field list: 1..%d entries, 0 <= l <= %d, mult >= 1", SSCONV_MAX_ENTRIES,
                SSCONV_MAX_L);
  if (d->ksize < 1 || d->ksize > 5 || (d->ksize & 1) == 0)
    return fail(SSCONV_E_INVALID, "ksize must be odd and in 1..5 (got %d)", d->ksize);
  if (d->n_shells < 1 || d->n_shells > SSCONV_MAX_SHELLS) return fail(SSCONV_E_INVALID, "n_shells out of range");
  if (!(d->eps > 0.0)) return fail(SSCONV_E_INVALID, "eps must be positive");
  return SSCONV_OK;
}

// Distinct orders of a field list, ascending; returns count.
int distinct_orders(const ssconv_fields& f, int* out) {
  bool seen[SSCONV_MAX_L + 1] = {};
  for (int e = 0; e < f.n; ++e) seen[f.l[e]] = true;
  int n = 0;
  for (int l = 0; l <= SSCONV_MAX_L; ++l)
    if (seen[l]) out[n++] = l;
  return n;
}

// Normalised elements of the (k, l) block in (J ascending, shell) order: [nq][K][2k+1][2l+1].
std::vector<double> pair_basis(const ssconv_basis_desc* d, int k, int l, int* nq) {
  const int ks = d->ksize, h = (ks - 1) / 2, K = ks * ks * ks, dk = 2 * k + 1, dl = 2 * l + 1;
  const int jtop = d->jmax < 0 ? k + l : std::min(k + l, d->jmax);
  std::vector<double> out;
  *nq = 0;
  std::vector<double> Y;
  for (int J = std::abs(k - l); J <= jtop; ++J) {
    std::vector<double> Q = real_intertwiner(k, l, J);
    const int dJ = 2 * J + 1;
    Y.assign(dJ, 0.0);
    for (int m = 0; m < d->n_shells; ++m) {
      std::vector<double> B((size_t)K * dk * dl, 0.0);
      for (int s = 0; s < K; ++s) {
        double v[3] = {double(s / (ks * ks) - h), double((s / ks) % ks - h), double(s % ks - h)};
        double r = std::sqrt(v[0] * v[0] + v[1] * v[1] + v[2] * v[2]);
        double phi = std::exp(-0.5 * (r - d->shells[m]) * (r - d->shells[m]) / (d->eps * d->eps));
        real_sh(J, v, Y.data());
        for (int a = 0; a < dk; ++a)
          for (int b = 0; b < dl; ++b) {
            double acc = 0.0;
            for (int j = 0; j < dJ; ++j) acc += Y[j] * Q[(j * dk + a) * dl + b];
            B[((size_t)s * dk + a) * dl + b] = phi * acc;
          }
      }
      double nrm = 0.0, mx = 0.0;
      for (double x : B) {
        nrm += x * x;
        mx = std::max(mx, std::fabs(x));
      }
      nrm = std::sqrt(nrm);
      if (nrm < 1e-12) continue;  // vanishes on the grid
      double sign = 1.0;
      for (double x : B)
        if (std::fabs(x) > 1e-3 * mx) {
          sign = x > 0 ? 1.0 : -1.0;
          break;
        }
      for (double x : B) out.push_back(sign * x / nrm);
      ++*nq;
    }
  }
  return out;
}

// Element count of a (k, l) block, memoised per (ksize, shells, eps, jmax, k, l): the
// synthesis and backward entry points need it on every call.
static int pair_count(const ssconv_basis_desc* d, int k, int l) {
  static std::mutex mu;
  static std::map<std::string, int> memo;
  std::string key(reinterpret_cast<const char*>(&d->ksize), sizeof(int));
  key.append(reinterpret_cast<const char*>(&d->n_shells), sizeof(int));
  key.append(reinterpret_cast<const char*>(d->shells), sizeof(double) * d->n_shells);
  key.append(reinterpret_cast<const char*>(&d->eps), sizeof(double));
  key.append(reinterpret_cast<const char*>(&d->jmax), sizeof(int));
  key.push_back((char)k);
  key.push_back((char)l);
  {
    std::lock_guard<std::mutex> g(mu);
    auto it = memo.find(key);
    if (it != memo.end()) return it->second;
  }
  int n = 0;
  pair_basis(d, k, l, &n);
  std::lock_guard<std::mutex> g(mu);
  memo[key] = n;
  return n;
}

int basis_nq_table(const ssconv_basis_desc* d, int nq[SSCONV_MAX_L + 1][SSCONV_MAX_L + 1],
                   int64_t base[SSCONV_MAX_L + 1][SSCONV_MAX_L + 1], int64_t* total_floats) {
  SSC_TRY(validate_desc(d));
  int ko[SSCONV_MAX_L + 1], lo[SSCONV_MAX_L + 1];
  int nk = distinct_orders(d->out, ko), nl = distinct_orders(d->in, lo);
  const int K = d->ksize * d->ksize * d->ksize;
  for (int a = 0; a <= SSCONV_MAX_L; ++a)
    for (int b = 0; b <= SSCONV_MAX_L; ++b) nq[a][b] = 0, base[a][b] = 0;
  int64_t off = 0;
  for (int i = 0; i < nk; ++i)
    for (int j = 0; j < nl; ++j) {
      int k = ko[i], l = lo[j];
      int n = pair_count(d, k, l);
      nq[k][l] = n;
      base[k][l] = off;
      off += (int64_t)n * K * (2 * k + 1) * (2 * l + 1);
    }
  *total_floats = off;
  return SSCONV_OK;
}

int64_t coeff_total(const ssconv_basis_desc* d, int nq[SSCONV_MAX_L + 1][SSCONV_MAX_L + 1]) {
  int64_t total = 0;
  for (int eo = 0; eo < d->out.n; ++eo)
    for (int ei = 0; ei < d->in.n; ++ei)
      total += (int64_t)d->out.mult[eo] * d->in.mult[ei] * nq[d->out.l[eo]][d->in.l[ei]];
  return total;
}

}  // namespace ssconv

using namespace ssconv;

extern "C" int ssconv_basis_info(const ssconv_basis_desc* desc, int64_t* basis_floats, int64_t* n_coeff) {
  if (!basis_floats || !n_coeff) return fail(SSCONV_E_INVALID, "NULL output pointer");
  int nq[SSCONV_MAX_L + 1][SSCONV_MAX_L + 1];
  int64_t base[SSCONV_MAX_L + 1][SSCONV_MAX_L + 1];
  SSC_TRY(basis_nq_table(desc, nq, base, basis_floats));
  *n_coeff = coeff_total(desc, nq);
  return SSCONV_OK;
}

extern "C" int ssconv_basis_build(const ssconv_basis_desc* desc, float* basis) {
  if (!basis) return fail(SSCONV_E_INVALID, "basis output pointer is NULL");
  SSC_TRY(validate_desc(desc));
  int ko[SSCONV_MAX_L + 1], lo[SSCONV_MAX_L + 1];
  int nk = distinct_orders(desc->out, ko), nl = distinct_orders(desc->in, lo);
  int64_t off = 0;
  for (int i = 0; i < nk; ++i)
    for (int j = 0; j < nl; ++j) {
      int n = 0;
      std::vector<double> B = pair_basis(desc, ko[i], lo[j], &n);
      for (double x : B) basis[off++] = (float)x;
    }
  return SSCONV_OK;
}
