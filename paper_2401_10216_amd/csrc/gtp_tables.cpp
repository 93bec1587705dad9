// Host-side fp64 construction of the change-of-basis tables (Sec. 3.2).
#include "gtp_tables.hpp"

#include <algorithm>
#include <cmath>
#include <stdexcept>

namespace gtp {

namespace {

constexpr double kPi = 3.14159265358979323846264338327950288;

// int_0^pi cos(n t) sin t dt (Clenshaw-Curtis moment).
double moment_sin(int n) {
  if (n == 1 || n == -1) return 0.0;
  return (n % 2 == 0) ? 2.0 / (1.0 - double(n) * double(n)) : 0.0;
}

// int_0^pi cos(n t) dt for integer n.
double moment_flat(int n) { return n == 0 ? kPi : 0.0; }

}  // namespace

void theta_factors(int L, double t, double* out) {
  // Normalised associated Legendre functions without the Condon-Shortley
  // phase, by the standard three-term recurrence in l at fixed m.
  const double c = std::cos(t), s = std::sin(t);
  double pmm = std::sqrt(1.0 / (4.0 * kPi));
  for (int m = 0; m <= L; ++m) {
    if (m > 0) pmm *= std::sqrt((2.0 * m + 1.0) / (2.0 * m)) * s;
    const double f = m > 0 ? std::sqrt(2.0) : 1.0;
    out[tri(m, m)] = f * pmm;
    if (m == L) continue;
    double p2 = pmm;
    double p1 = std::sqrt(2.0 * m + 3.0) * c * pmm;
    out[tri(m + 1, m)] = f * p1;
    for (int l = m + 2; l <= L; ++l) {
      const double a = std::sqrt((4.0 * l * l - 1.0) / (double(l) * l - double(m) * m));
      const double b = std::sqrt(((l - 1.0) * (l - 1.0) - double(m) * m) / (4.0 * (l - 1.0) * (l - 1.0) - 1.0));
      const double p = a * (c * p1 - b * p2);
      out[tri(l, m)] = f * p;
      p2 = p1;
      p1 = p;
    }
  }
}

Tables build_tables(int L1, int L2, int Lout) {
  if (L1 < 0 || L2 < 0 || Lout < 0 || L1 > 128 || L2 > 128 || Lout > 256)
    throw std::invalid_argument("degree out of range");
  Tables t;
  t.L1 = L1;
  t.L2 = L2;
  t.Lout = Lout;
  t.U = L1 + L2;
  t.Le = std::min(Lout, t.U);
  t.Lin = std::max(L1, L2);
  t.Lt = std::max(t.Lin, t.Le);
  // A phi moment of the product is a cos series (even m) of degree <= U, or a
  // sine series (odd m) of degree 1..U.  The uniform grid t_j = j pi / NT
  // (DCT-I on j = 0..NT, DST-I on j = 1..NT-1) represents both exactly for
  // NT = U + 1.
  t.NT = t.U + 1;
  t.NJ = t.NT + 1;
  // The product has phi frequencies <= U; reading moments m <= Le from NP
  // uniform samples is alias-free when NP > U + Le.  NP is rounded up to a
  // multiple of 4 so that the phi grid is closed under p -> -p, p -> pi +- p.
  t.NP = (t.U + t.Le + 1 + 3) / 4 * 4;
  t.ldT1 = t.Lt + 1;
  t.ldZ = t.NT + 1;

  // ---- T1: theta-Fourier series of Theta_lm by an exact DCT-II / DST-II of
  // Lt+1 samples (a degree-<=Lt series is determined by them).
  const int Lt = t.Lt;
  const int N = Lt + 1;
  t.T1.assign(size_t(ntri(Lt)) * t.ldT1, 0.0);
  {
    std::vector<double> samp(size_t(N) * ntri(Lt));
    for (int j = 0; j < N; ++j) theta_factors(Lt, (j + 0.5) * kPi / N, &samp[size_t(j) * ntri(Lt)]);
    for (int l = 0; l <= Lt; ++l)
      for (int m = 0; m <= l; ++m)
        for (int u = 0; u <= Lt; ++u) {
          if ((u + l) % 2) continue;  // Theta_lm has only u = l (mod 2)
          if (m % 2 == 1 && u == 0) continue;
          double acc = 0.0;
          for (int j = 0; j < N; ++j) {
            const double th = (j + 0.5) * kPi / N;
            const double b = (m % 2 == 0) ? std::cos(u * th) : std::sin(u * th);
            acc += samp[size_t(j) * ntri(Lt) + tri(l, m)] * b;
          }
          const double norm = (m % 2 == 0 && u == 0) ? 1.0 / N : 2.0 / N;
          t.T1[size_t(tri(l, m)) * t.ldT1 + u] = acc * norm;
        }
  }

  // ---- Zc, Zs: closed-form theta integrals of each series term against
  // {cos, sin}(u t) sin t on [0, pi], l <= Le, u = 0..NT.
  const int Le = t.Le;
  t.Zc.assign(size_t(ntri(Le)) * t.ldZ, 0.0);
  t.Zs.assign(size_t(ntri(Le)) * t.ldZ, 0.0);
  for (int l = 0; l <= Le; ++l)
    for (int m = 0; m <= l; ++m) {
      const double* c = &t.T1[size_t(tri(l, m)) * t.ldT1];
      for (int u = 0; u <= t.NT; ++u) {
        double zc = 0.0, zs = 0.0;
        for (int k = 0; k <= l; ++k) {
          if (c[k] == 0.0) continue;
          if (m % 2 == 0) {
            zc += c[k] * 0.5 * (moment_sin(u - k) + moment_sin(u + k));
            zs += c[k] * 0.25 *
                  (moment_flat(u - 1 - k) + moment_flat(u - 1 + k) - moment_flat(u + 1 - k) - moment_flat(u + 1 + k));
          } else {
            zc += c[k] * 0.25 *
                  (moment_flat(k - 1 - u) + moment_flat(k - 1 + u) - moment_flat(k + 1 - u) - moment_flat(k + 1 + u));
            zs += c[k] * 0.5 * (moment_sin(u - k) - moment_sin(u + k));
          }
        }
        t.Zc[size_t(tri(l, m)) * t.ldZ + u] = zc;
        t.Zs[size_t(tri(l, m)) * t.ldZ + u] = zs;
      }
    }

  // ---- S: Theta_lm at t_j (series of T1 evaluated on the grid), l <= Lin.
  const int NT = t.NT, NJ = t.NJ;
  t.S.assign(size_t(ntri(t.Lin)) * NJ, 0.0);
  for (int l = 0; l <= t.Lin; ++l)
    for (int m = 0; m <= l; ++m)
      for (int j = 0; j < NJ; ++j) {
        const double th = j * kPi / NT;
        double acc = 0.0;
        for (int u = 0; u <= l; ++u) {
          const double cu = t.T1[size_t(tri(l, m)) * t.ldT1 + u];
          if (cu == 0.0) continue;
          acc += cu * ((m % 2 == 0) ? std::cos(u * th) : std::sin(u * th));
        }
        if (m > 0 && (j == 0 || j == NT)) acc = 0.0;  // P_l^m(+-1) = 0 for m > 0
        t.S[size_t(tri(l, m)) * NJ + j] = acc;
      }

  // ---- W: analysis weights.  A moment g sampled at t_j has theta-Fourier
  // coefficients by the inverse DCT-I (even m) / DST-I (odd m); the SH
  // coefficient is sum_u coef_u Z[u].  The phi moment is taken as a plain sum
  // over the NP samples, so its 2 pi / NP quadrature factor is folded in too.
  t.W.assign(size_t(ntri(Le)) * NJ, 0.0);
  const double phiw = 2.0 * kPi / t.NP;
  for (int l = 0; l <= Le; ++l)
    for (int m = 0; m <= l; ++m)
      for (int j = 0; j < NJ; ++j) {
        const double th = j * kPi / NT;
        double acc = 0.0;
        if (m % 2 == 0) {
          const double wj = (j == 0 || j == NT) ? 0.5 : 1.0;
          for (int u = 0; u <= NT; ++u) {
            const double wu = (u == 0 || u == NT) ? 0.5 : 1.0;
            acc += t.Zc[size_t(tri(l, m)) * t.ldZ + u] * (2.0 / NT) * wu * wj * std::cos(u * th);
          }
        } else if (j != 0 && j != NT) {
          for (int u = 1; u < NT; ++u) acc += t.Zs[size_t(tri(l, m)) * t.ldZ + u] * (2.0 / NT) * std::sin(u * th);
        }
        t.W[size_t(tri(l, m)) * NJ + j] = acc * phiw;
      }

  // ---- Phi: trig(mp, k).
  t.Mphi = std::max(t.Lin, t.Le);
  const int nmp = 2 * t.Mphi + 1;
  t.Phi.assign(size_t(nmp) * t.NP, 0.0);
  for (int mp = 0; mp < nmp; ++mp)
    for (int k = 0; k < t.NP; ++k) {
      const int m = (mp + 1) / 2;
      // reduce m*k mod NP exactly before taking the angle
      const double ang = 2.0 * kPi * double((int64_t(m) * k) % t.NP) / t.NP;
      double v = 1.0;
      if (mp > 0) v = (mp % 2 == 1) ? std::cos(ang) : std::sin(ang);
      t.Phi[size_t(mp) * t.NP + k] = v;
    }
  return t;
}

void host_pipeline(const Tables& t, const double* x1, const double* x2, int64_t n, double* y) {
  const int K1 = nsh(t.L1), K2 = nsh(t.L2), KO = nsh(t.Lout);
  const int NJ = t.NJ, NP = t.NP;
  const int n1 = 2 * t.L1 + 1, n2 = 2 * t.L2 + 1, no = 2 * t.Le + 1;
  std::vector<double> A1(size_t(NJ) * n1), A2(size_t(NJ) * n2), F3(size_t(NJ) * NP), C(size_t(NJ) * no);
  auto coef_index = [](int l, int mp) {
    const int m = (mp + 1) / 2;
    return (mp == 0 || mp % 2 == 1) ? l * l + l + m : l * l + l - m;
  };
  for (int64_t p = 0; p < n; ++p) {
    const double* a = x1 + p * K1;
    const double* b = x2 + p * K2;
    for (int j = 0; j < NJ; ++j) {
      for (int mp = 0; mp < n1; ++mp) {
        const int m = (mp + 1) / 2;
        double s = 0.0;
        for (int l = m; l <= t.L1; ++l) s += t.S[size_t(tri(l, m)) * NJ + j] * a[coef_index(l, mp)];
        A1[size_t(j) * n1 + mp] = s;
      }
      for (int mp = 0; mp < n2; ++mp) {
        const int m = (mp + 1) / 2;
        double s = 0.0;
        for (int l = m; l <= t.L2; ++l) s += t.S[size_t(tri(l, m)) * NJ + j] * b[coef_index(l, mp)];
        A2[size_t(j) * n2 + mp] = s;
      }
      for (int k = 0; k < NP; ++k) {
        double f1 = 0.0, f2 = 0.0;
        for (int mp = 0; mp < n1; ++mp) f1 += A1[size_t(j) * n1 + mp] * t.Phi[size_t(mp) * NP + k];
        for (int mp = 0; mp < n2; ++mp) f2 += A2[size_t(j) * n2 + mp] * t.Phi[size_t(mp) * NP + k];
        F3[size_t(j) * NP + k] = f1 * f2;
      }
      for (int mp = 0; mp < no; ++mp) {
        double s = 0.0;
        for (int k = 0; k < NP; ++k) s += F3[size_t(j) * NP + k] * t.Phi[size_t(mp) * NP + k];
        C[size_t(j) * no + mp] = s;
      }
    }
    double* out = y + p * KO;
    for (int i = 0; i < KO; ++i) out[i] = 0.0;
    for (int l = 0; l <= t.Le; ++l)
      for (int mp = 0; mp < 2 * l + 1; ++mp) {
        const int m = (mp + 1) / 2;
        double s = 0.0;
        for (int j = 0; j < NJ; ++j) s += t.W[size_t(tri(l, m)) * NJ + j] * C[size_t(j) * no + mp];
        out[coef_index(l, mp)] = s;
      }
  }
}

}  // namespace gtp
