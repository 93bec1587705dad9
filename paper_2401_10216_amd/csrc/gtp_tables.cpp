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
  if (L1 == L2 && L1 == Lout && (L1 == 16 || L1 == 32 || L1 == 64)) build_wave_tables(t);
  return t;
}

// Wave kernel geometry (L = L1 = L2 = Lout): lane = 16 g + i (g = 0..3,
// i = 8 h + pi); mirror pairs of theta nodes (jp, NT - jp), jp = 1..L, 8 per
// pass (PASSES = L / 8); phi samples k = 0..Q (Q = NP / 4) in NMB blocks of
// 16; the m-parts m = 1..L split into 4 classes {cos, sin} x {even m, odd m}
// of L / 2 values each, taken 4 at a time (one per lane group g) in NKS = L / 8
// K-steps: K-step s, group g holds m = 8s + 2g + 2 (even) and 8s + 2g + 1
// (odd).  Lane (g, 8h + pi) sums, for pair jp = 8 pass + pi + 1, the terms
// with l - m = h (mod 2).  Every table is a lane-permuted copy that the
// kernel reads as one 16-byte load per lane:
//
//   TWR[lane][TWRN]  seeds of the phi operands for rotation recurrences
//                    (NMBP = NMB rounded up to even; NMR = 16-row blocks of
//                    analysis m-rows per class, L / 32 at L = 64, else 1): per
//                    mb (k = 16 mb + 4 (i mod 4) + i / 4, zero for k > Q: the
//                    synthesis row i holds that sample, so that register r of
//                    lane group g of the result holds sample 16 mb + 4 r + g)
//                    cos/sin of (2g+2) phi_k, cos/sin of (2g+1) phi_k, cos/sin
//                    of 8 phi_k (entries 6 mb .. 6 mb + 5); from ASD = 6 NMBP,
//                    per (mr, mb) (k0 = 16 mb + g, m = 2(16 mr + i) + 2) fold
//                    times cos/sin of m phi_k0 and of (m - 1) phi_k0 (fold = 4
//                    below L = 64, where the kernel folds the sample products
//                    as class sums, else 1; entries
//                    ASD + 4 (mr NMBP + mb) ..); from AST = ASD + 4 NMR NMBP,
//                    per mr cos/sin of m phi_4 and of (m - 1) phi_4 (the step
//                    from register r to r + 1); zero where m > L.
//                    TWRN = AST + 4 NMR.
//   SMP[pass][s][u2][lane][4]  Theta_{mo+2u+h, mo}(t_jp),
//                    Theta_{me+2u-h, me}(t_jp) for u = 2 u2, then u = 2 u2 + 1
//                    (mo = 8s + 2g + 1, me = mo + 1; zero outside m <= l <= L);
//                    u2 < nu(s) / 2 with nu(s) = L/2 - 4s u-steps in K-step s.
//   SM0P[pass][lane][v]  m = 0 parts: Theta_{l,0}(t_jp), l = 8v + g + 4h
//                    (v < NV0 = ceil((L+1)/8), padded to 4 | NV0); pass = L/8
//                    holds the north pole (jp = 0).
//   WP               analysis weights W[row][j] of the rows a thread owns:
//                    step it < NIT: the (tid + NTH it)-th row with m > 0 in
//                    tri order, it = NIT: row tri(tid, 0); zero where the row
//                    does not exist.  NTH = 64 (L <= 32): [pass][it][lane][jj],
//                    j = 8 pass + jj + 1; NTH = 256 (L = 64, four waves per
//                    product): [it][tid][j - 1], j = 1..L.
//   XMAPP[tid][k]    LDS slot (4 * quad + (m' < 0)) of coefficient
//                    idx = tid + NTH k = l^2 + l + m' (k < NXK = ceil(K / NTH),
//                    padded to 4 | NXK with -1).  Quads: the m = 0 block
//                    (quad l), then for each m-pair c (m = 2c + 1, 2c + 2) 4
//                    quads per u-step (2c+1, l_a), (2c+1, l_b), (2c+2, l_a),
//                    (2c+2, l_b) with l_a = 2c + 1 + 2u, l_b = l_a + 1, for
//                    the nu(c / 4) - c % 4 u-steps that hold a coefficient,
//                    and one pad quad.  XQUADS also covers the reads of every
//                    group's nu(c / 4) u-steps (past its block: the next
//                    blocks, then a zero tail).
void build_wave_tables(Tables& t) {
  const int L = t.L1;
  if (t.L2 != L || t.Lout != L || (L != 16 && L != 32 && L != 64)) throw std::invalid_argument("wave tables: bad degree");
  const int NP = t.NP, Q = NP / 4, NMB = (Q + 1 + 15) / 16, NKS = L / 8;
  const int NMBP = (NMB + 1) / 2 * 2;                        // seed layout per lane
  const int NMR = L > 32 ? L / 32 : 1, ASD = 6 * NMBP, AST = ASD + 4 * NMR * NMBP, TWRN = AST + 4 * NMR;
  const int NTH = L > 32 ? 256 : 64;                         // threads per product
  // weight every phi sample shares in the analysis: the 4-point sets' products
  // enter as class sums (a quarter of the four sample products) below L = 64
  const double fold = L < 64 ? 4.0 : 1.0;
  auto trig = [&](bool is_sin, int m, int k) {
    const double ang = 2.0 * kPi * double((int64_t(m) * k) % NP) / NP;
    return is_sin ? std::sin(ang) : std::cos(ang);
  };
  t.waveL = L;
  // x scatter map; pair blocks hold nu(s) = L/2 - 4s u-steps (s = c / 4)
  std::vector<int> xb(L / 2 + 1);
  xb[0] = L + 1;
  for (int c = 0; c < L / 2; ++c) xb[c + 1] = xb[c] + 4 * (L / 2 - 4 * (c / 4) - c % 4) + 1;
  const int K = (L + 1) * (L + 1);
  std::vector<int> xmap(K, 0);
  for (int l = 0; l <= L; ++l)
    for (int ms = -l; ms <= l; ++ms) {
      const int m = ms < 0 ? -ms : ms;
      int quad = l;
      if (m > 0) {
        const int c = (m - 1) / 2, dl = l - (2 * c + 1);
        quad = xb[c] + 4 * (dl / 2) + (m % 2 == 1 ? 0 : 2) + (dl % 2);
      }
      xmap[size_t(l) * l + l + ms] = 4 * quad + (ms < 0 ? 1 : 0);
    }
  t.XQUADS = xb[L / 2];
  for (int c = 0; c < L / 2; ++c) t.XQUADS = std::max(t.XQUADS, xb[c] + 4 * (L / 2 - 4 * (c / 4)));
  const int NXK = (K + NTH - 1) / NTH, NXKP = (NXK + 3) / 4 * 4;
  t.XMAPP.assign(size_t(NTH) * NXKP, -1);
  for (int tid = 0; tid < NTH; ++tid)
    for (int k = 0; k < NXK; ++k)
      if (tid + NTH * k < K) t.XMAPP[size_t(tid) * NXKP + k] = xmap[tid + NTH * k];

  t.TWR.assign(size_t(64) * TWRN, 0.0);
  for (int lane = 0; lane < 64; ++lane) {
    const int g = lane / 16, i = lane % 16;
    double* o = &t.TWR[size_t(lane) * TWRN];
    for (int mb = 0; mb < NMB; ++mb) {
      const int k = 16 * mb + 4 * (i % 4) + i / 4;
      if (k <= Q) {
        o[6 * mb + 0] = trig(false, 2 * g + 2, k);
        o[6 * mb + 1] = trig(true, 2 * g + 2, k);
        o[6 * mb + 2] = trig(false, 2 * g + 1, k);
        o[6 * mb + 3] = trig(true, 2 * g + 1, k);
        o[6 * mb + 4] = trig(false, 8, k);
        o[6 * mb + 5] = trig(true, 8, k);
      }
      const int k0 = 16 * mb + g;
      for (int mr = 0; mr < NMR; ++mr) {
        const int me = 2 * (16 * mr + i) + 2, mo = me - 1;
        double* a = &o[ASD + 4 * (mr * NMBP + mb)];
        if (me <= L) {
          a[0] = fold * trig(false, me, k0);
          a[1] = fold * trig(true, me, k0);
        }
        if (mo <= L) {
          a[2] = fold * trig(false, mo, k0);
          a[3] = fold * trig(true, mo, k0);
        }
      }
    }
    for (int mr = 0; mr < NMR; ++mr) {
      const int me = 2 * (16 * mr + i) + 2, mo = me - 1;
      if (me <= L) {
        o[AST + 4 * mr + 0] = trig(false, me, 4);
        o[AST + 4 * mr + 1] = trig(true, me, 4);
      }
      if (mo <= L) {
        o[AST + 4 * mr + 2] = trig(false, mo, 4);
        o[AST + 4 * mr + 3] = trig(true, mo, 4);
      }
    }
  }

  // lane-permuted copies for 16-byte loads
  auto S = [&](int l, int m, int j) { return (m <= l && l <= L) ? t.S[size_t(tri(l, m)) * t.NJ + j] : 0.0; };
  const int PASSES = L / 8;
  int TU2 = 0;
  for (int s = 0; s < NKS; ++s) TU2 += (L / 2 - 4 * s) / 2;
  t.SMP.assign(size_t(PASSES) * TU2 * 64 * 4, 0.0);
  for (int pass = 0; pass < PASSES; ++pass) {
    int u2base = 0;
    for (int s = 0; s < NKS; ++s) {
      const int nu = L / 2 - 4 * s;
      for (int u2 = 0; u2 < nu / 2; ++u2)
        for (int lane = 0; lane < 64; ++lane) {
          const int g = lane / 16, h = (lane / 8) % 2, pi = lane % 8;
          const int mo = 2 * (4 * s + g) + 1, me = mo + 1, jp = 8 * pass + pi + 1;
          double* o = &t.SMP[((size_t(pass) * TU2 + u2base + u2) * 64 + lane) * 4];
          for (int e = 0; e < 2; ++e) {
            const int u = 2 * u2 + e;
            o[2 * e] = S(mo + 2 * u + h, mo, jp);
            o[2 * e + 1] = S(me + 2 * u - h, me, jp);
          }
        }
      u2base += nu / 2;
    }
  }
  const int NV0 = (L + 1 + 7) / 8, NV0P = (NV0 + 3) / 4 * 4;
  t.SM0P.assign(size_t(PASSES + 1) * 64 * NV0P, 0.0);
  for (int pass = 0; pass <= PASSES; ++pass)
    for (int lane = 0; lane < 64; ++lane) {
      const int g = lane / 16, h = (lane / 8) % 2, pi = lane % 8;
      const int jp = pass < PASSES ? 8 * pass + pi + 1 : 0;
      for (int v = 0; v < NV0; ++v) t.SM0P[(size_t(pass) * 64 + lane) * NV0P + v] = S(8 * v + g + 4 * h, 0, jp);
    }
  const int NROW = ntri(L) - (L + 1), NIT = (NROW + NTH - 1) / NTH;
  // row owned by thread tid in row step it (it = NIT: the m = 0 row), or -1
  auto owned_row = [&](int it, int tid) {
    if (it == NIT) return tid <= L ? tri(tid, 0) : -1;
    const int q = tid + NTH * it;
    if (q >= NROW) return -1;
    int l = 1;
    while ((l + 1) * l / 2 <= q) ++l;  // rows with m > 0: l rows of degree l
    return tri(l, q - l * (l - 1) / 2 + 1);
  };
  if (NTH == 64) {
    t.WP.assign(size_t(PASSES) * (NIT + 1) * 64 * 8, 0.0);
    for (int pass = 0; pass < PASSES; ++pass)
      for (int it = 0; it <= NIT; ++it)
        for (int lane = 0; lane < 64; ++lane) {
          const int row = owned_row(it, lane);
          if (row < 0) continue;
          for (int jj = 0; jj < 8; ++jj)
            t.WP[((size_t(pass) * (NIT + 1) + it) * 64 + lane) * 8 + jj] = t.W[size_t(row) * t.NJ + 8 * pass + jj + 1];
        }
  } else {
    t.WP.assign(size_t(NIT + 1) * NTH * L, 0.0);
    for (int it = 0; it <= NIT; ++it)
      for (int tid = 0; tid < NTH; ++tid) {
        const int row = owned_row(it, tid);
        if (row < 0) continue;
        for (int j = 1; j <= L; ++j) t.WP[(size_t(it) * NTH + tid) * L + j - 1] = t.W[size_t(row) * t.NJ + j];
      }
  }
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
