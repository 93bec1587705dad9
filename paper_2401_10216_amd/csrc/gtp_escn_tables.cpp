// Host-side fp64 tables of the rotated-frame equivariant convolution.
#include <cmath>
#include <vector>

#include "gtp_escn_tables.hpp"

namespace gtp {
namespace {

constexpr double kPi = 3.14159265358979323846264338327950288;

// Gauss-Legendre nodes and weights on [-1, 1] (Newton's method on P_n).
void gauss_legendre(int n, std::vector<double>& x, std::vector<double>& w) {
  x.assign(n, 0.0);
  w.assign(n, 0.0);
  for (int i = 0; i < n; ++i) {
    double z = std::cos(kPi * (i + 0.75) / (n + 0.5));
    double dp = 1.0;
    for (int it = 0; it < 100; ++it) {
      double p0 = 1.0, p1 = z;
      for (int k = 2; k <= n; ++k) {
        const double p2 = ((2.0 * k - 1.0) * z * p1 - (k - 1.0) * p0) / k;
        p0 = p1;
        p1 = p2;
      }
      const double pn = n == 0 ? 1.0 : (n == 1 ? z : p1);
      const double pm = n == 1 ? 1.0 : p0;
      dp = n * (z * pn - pm) / (z * z - 1.0);
      const double dz = pn / dp;
      z -= dz;
      if (std::fabs(dz) < 1e-16) break;
    }
    x[i] = z;
    w[i] = 2.0 / ((1.0 - z * z) * dp * dp);
  }
}

// Real SH Y_{l,m}(theta, phi), all l <= L, index l*l + l + m.
void real_sh(int L, double th, double ph, std::vector<double>& out) {
  std::vector<double> f(ntri(L));
  theta_factors(L, th, f.data());
  out.assign(nsh(L), 0.0);
  for (int l = 0; l <= L; ++l) {
    out[l * l + l] = f[tri(l, 0)];
    for (int m = 1; m <= l; ++m) {
      out[l * l + l + m] = f[tri(l, m)] * std::cos(m * ph);
      out[l * l + l - m] = f[tri(l, m)] * std::sin(m * ph);
    }
  }
}

}  // namespace

EscnHost build_escn_tables(const Tables& t) {
  EscnHost e;
  if (t.L1 != t.L2 || t.L2 != t.Lout || t.NT % 2 == 0) return e;
  e.LM = t.L1;
  // ---- J: real-SH matrices of Q = R_x(90 deg), (x, y, z) -> (x, -z, y), by a
  // quadrature exact for the degree-2l integrand (Gauss-Legendre in cos theta
  // with LM + 1 nodes, 2 LM + 1 uniform phi points).
  {
    const int L = e.LM;
    std::vector<double> gx, gw;
    gauss_legendre(L + 1, gx, gw);
    const int nph = 2 * L + 1;
    size_t tot = 0;
    for (int l = 0; l <= L; ++l) tot += size_t(2 * l + 1) * (2 * l + 1);
    e.J.assign(tot, 0.0);
    std::vector<double> y, yq;
    for (int i = 0; i < L + 1; ++i) {
      const double z = gx[i], s = std::sqrt(1.0 - z * z), th = std::acos(z);
      for (int k = 0; k < nph; ++k) {
        const double ph = 2.0 * kPi * k / nph, wq = gw[i] * 2.0 * kPi / nph;
        const double px = s * std::cos(ph), py = s * std::sin(ph), pz = z;
        const double qx = px, qy = -pz, qz = py;  // Q r
        real_sh(L, th, ph, y);
        real_sh(L, std::acos(qz < -1.0 ? -1.0 : (qz > 1.0 ? 1.0 : qz)), std::atan2(qy, qx), yq);
        size_t off = 0;
        for (int l = 0; l <= L; ++l) {
          const int d = 2 * l + 1;
          for (int a = 0; a < d; ++a)
            for (int b = 0; b < d; ++b) e.J[off + size_t(a) * d + b] += wq * yq[l * l + a] * y[l * l + b];
          off += size_t(d) * d;
        }
      }
    }
  }

  // ---- E: node-pair rows (j = 0 .. NT / 2; j = 0 is the pole pair), m-major
  // chunks padded to 4 floats.
  const int L = t.L1;
  auto pad4 = [](int n) { return (n + 3) / 4 * 4; };
  e.NPAIR = (t.NT + 1) / 2;
  e.ERL = pad4(L + 1);
  for (int m = 0; m <= L; ++m) e.ERL += 2 * pad4(L + 1 - m);
  e.E.assign(size_t(e.NPAIR) * e.ERL, 0.0);
  std::vector<double> f0(ntri(L)), fj(ntri(L));
  theta_factors(L, 0.0, f0.data());
  for (int j = 0; j < e.NPAIR; ++j) {
    double* row = e.E.data() + size_t(j) * e.ERL;
    theta_factors(L, kPi * j / t.NT, fj.data());
    for (int l = 0; l <= L; ++l) row[l] = f0[tri(l, 0)] * fj[tri(l, 0)];
    int off = pad4(L + 1);
    for (int m = 0; m <= L; ++m) {
      for (int l = m; l <= L; ++l) row[off + l - m] = t.S[size_t(tri(l, m)) * t.NJ + j];
      off += pad4(L + 1 - m);
    }
    for (int m = 0; m <= L; ++m) {
      const double cm = m == 0 ? double(t.NP) : 0.5 * t.NP;
      for (int l = m; l <= L; ++l) row[off + l - m] = cm * t.W[size_t(tri(l, m)) * t.NJ + j];
      off += pad4(L + 1 - m);
    }
  }

  // ---- A, Z: operand images of the matrix-core kernel (layouts in the header)
  if (L == kEscnWaveL && e.NPAIR == L + 1) {
    auto S = [&](int l, int m, int j) { return l <= L ? t.S[size_t(tri(l, m)) * t.NJ + j] : 0.0; };
    auto CW = [&](int l, int m, int j) {
      return l <= L ? (m == 0 ? double(t.NP) : 0.5 * t.NP) * t.W[size_t(tri(l, m)) * t.NJ + j] : 0.0;
    };
    e.A.assign(size_t(escn_wave_moff(L, L + 1)), 0.0);
    for (int m = 0; m <= L; ++m) {
      const int n = L + 1 - m, ne = (n + 1) / 2, no = n / 2, ke = (ne + 3) / 4, ko = (no + 3) / 4;
      const int nl = escn_wave_lane_floats(L, m);
      for (int lane = 0; lane < 64; ++lane) {
        const int k = lane / 16, i = lane % 16, pj = 4 * (i % 4) + i / 4 + 1;
        double* v = e.A.data() + escn_wave_moff(L, m) + size_t(lane) * nl;
        int q = 0;
        for (int s = 0; s < ke; ++s) v[q++] = S(m + 2 * (4 * s + k), m, pj);
        for (int s = 0; s < ko; ++s) v[q++] = S(m + 1 + 2 * (4 * s + k), m, pj);
        for (int r = 0; r < 4; ++r) v[q++] = i < ne ? CW(m + 2 * i, m, 4 * r + k + 1) : 0.0;
        if (no > 0)
          for (int r = 0; r < 4; ++r) v[q++] = i < no ? CW(m + 1 + 2 * i, m, 4 * r + k + 1) : 0.0;
      }
    }
    e.Z.assign(size_t(escn_wave_zfloats(L)), 0.0);
    for (int g = 0; g < 4; ++g)
      for (int r = 0; r < 4; ++r) {
        const int j = 4 * r + g + 1;
        for (int l = 0; l <= L; ++l) e.Z[size_t(4 * g + r) * (L + 1) + l] = e.E[size_t(j) * e.ERL + l];
      }
    double* zp = e.Z.data() + 16 * (L + 1);
    for (int l = 0; l <= L; ++l) {
      zp[l] = e.E[l];                // pole pair: the unit filter
      zp[L + 1 + l] = S(l, 0, 0);    // Theta_l0(0)
      zp[2 * (L + 1) + l] = CW(l, 0, 0);
    }
    e.JI.assign(size_t(2 * escn_wave_jtoff()), 0.0);
    size_t jo = 0;
    for (int l = 0; l <= L; ++l) {
      const int d = 2 * l + 1;
      for (int t = 0; t < escn_wave_jtiles(l); ++t) {
        const int nk4 = escn_wave_jnk4(l, t);
        for (int lane = 0; lane < 64; ++lane) {
          const int k = lane / 16, i = lane % 16, row = escn_wave_jtrow(l, t, i);
          // class tiles: rows of one lane-group parity meet only the columns
          // of the same parity (the other sub-blocks of J are zero)
          const bool same = l < kEscnClassL || ((i / 4) & 1) == (k & 1);
          for (int s = 0; s < escn_wave_jsteps(l, t); ++s) {
            const int col = escn_wave_jtcol(l, t, s, k);
            if (row < 0 || col < 0 || !same) continue;
            const size_t at = size_t(escn_wave_joff(l, t)) + size_t(lane) * nk4 + s;
            e.JI[at] = e.J[jo + size_t(row) * d + col];                          // J[row][col]
            e.JI[escn_wave_jtoff() + at] = e.J[jo + size_t(col) * d + row];      // J^T[row][col]
          }
        }
      }
      jo += size_t(d) * d;
    }
  }
  return e;
}

}  // namespace gtp
