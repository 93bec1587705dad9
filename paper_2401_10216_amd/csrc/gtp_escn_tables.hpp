// Host fp64 tables of the rotated-frame equivariant convolution (Sec. 3.3
// "Equivariant Convolutions"; Appendix, eq. sh2fs-escn).
#pragma once

#include <vector>

#include "gtp_tables.hpp"

namespace gtp {

// Host fp64 tables of the rotated-frame path for a plan (L1, L2, Lout).
//   J  : per degree l <= LM = max(L1, Lout), the (2l+1) x (2l+1) real-SH
//        rotation matrix of Q = R_x(90 deg) (which maps the y axis to the z
//        axis), row-major, block l at offset sum_{l' < l} (2l'+1)^2;
//        J[a][b] = int Y_{l,a-l}(Q r) Y_{l,b-l}(r) dOmega, so that the
//        coefficients of F(Q^-1 r) are J x, and a rotation about y by t is
//        J^T Z(t) J with Z(t) the rotation about z.
//   E  : per mirror pair of theta nodes (j, NT - j), j = 0 .. NPAIR - 1 (j = 0
//        pairs the two poles), one row of length ERL in chunks padded to a
//        multiple of 4 floats (P(n) = n rounded up to 4), L = L1 = L2 = Lout:
//          [0, P(L+1))        Theta_l0(0) Theta_l0(t_j), l <= L: the zonal
//                             filter of unit radial weights at t_j
//          then for m = 0..L  Theta_lm(t_j), l = m..L          (P(L+1-m) each)
//          then for m = 0..L  c_m W[tri(l, m)][j], l = m..L    (P(L+1-m) each)
//        with c_0 = NP and c_m = NP / 2 (the phi moment of a band-limited
//        function is NP a_0, NP / 2 a_m).  The mirror node NT - j takes the
//        factor (-1)^(l + m) of both Theta and W.  Built for L1 = L2 = Lout
//        only (NT = 2L + 1 is odd: no equator node).
//   A, Z: the operand images of the matrix-core kernel (L = kEscnWaveL only;
//        empty otherwise).  A holds, per order m = 0..L, escn_wave_steps(L, m)
//        operands of the 16x16x4 contractions for each of the 64 lanes (lane
//        16 k + i, a block of escn_wave_lane_floats(L, m) floats per lane,
//        blocks at escn_wave_moff(L, m)):
//          synthesis, even then odd set (l - m even / odd; K-steps of four
//          degrees, lane row i = node pair 4 (i % 4) + i / 4 + 1, K index k =
//          the degree m + par + 2 (4 s + k)): Theta_lm(t_j);
//          analysis, even then odd set (4 K-steps each: row i = the degree
//          m + par + 2 i, K index k = node pair 4 r + k + 1): c_m W[tri(l, m)][j];
//        zero where the degree exceeds L.  Z holds the unit zonal filter
//        Theta_l0(0) Theta_l0(t_j) at the node pairs 4 r + g + 1 of lane
//        group g (Z[(g 4 + r)(L + 1) + l]), then three rows of L + 1 values
//        at the pole pair: the filter, Theta_l0(0) and c_0 W[tri(l, 0)][0].
//   JI : the A-operand images of J and J^T for that kernel's rotations
//        (the edge's D_b = J^T Z(-beta) J Z(-alpha) applied factor by
//        factor): per degree block l, 16-row tile mt and lane 16 k + i, the
//        K-steps s = 0 .. NK(l) - 1 (NK = ceil((2l+1) / 4), padded to a
//        multiple of 4) of J[16 mt + jrow(i)][4 s + k] at escn_wave_joff(l, mt)
//        (jrow = escn_wave_jrow, the block row of tile row i),
//        then the same for J^T at escn_wave_jtoff() + escn_wave_joff(l, mt);
//        zero outside the block.
struct EscnHost {
  int LM = 0, NPAIR = 0, ERL = 0;
  std::vector<double> J, E, A, Z, JI;
};

// Degree of the matrix-core rotated-frame kernel: 16 interior node pairs,
// one per row of a 16 x 16 tile.
constexpr int kEscnWaveL = 16;
// K-steps of order m: synthesis over the even and odd degree sets, then 4
// analysis steps per non-empty set.
constexpr int escn_wave_steps(int L, int m) {
  const int n = L + 1 - m, ne = (n + 1) / 2, no = n / 2;
  return (ne + 3) / 4 + (no + 3) / 4 + 4 + (no > 0 ? 4 : 0);
}
constexpr int escn_wave_lane_floats(int L, int m) { return (escn_wave_steps(L, m) + 3) / 4 * 4; }
constexpr int escn_wave_moff(int L, int m) {
  int o = 0;
  for (int k = 0; k < m; ++k) o += 64 * escn_wave_lane_floats(L, k);
  return o;
}
constexpr int escn_wave_zfloats(int L) { return 16 * (L + 1) + 3 * (L + 1); }
// K-steps of degree block l (padded to 4 per lane) and the image offsets
constexpr int escn_wave_nk4(int l) { return ((2 * l + 1 + 3) / 4 + 3) / 4 * 4; }
constexpr int escn_wave_nm(int l) { return (2 * l + 1 + 15) / 16; }
constexpr int escn_wave_joff(int l, int mt) {
  int o = 0;
  for (int k = 0; k < l; ++k) o += escn_wave_nm(k) * 64 * escn_wave_nk4(k);
  return o + mt * 64 * escn_wave_nk4(l);
}
constexpr int escn_wave_jtoff() { return escn_wave_joff(kEscnWaveL + 1, 0); }
// The block row held by row rho = 4 g + r of a 16-row output tile (register
// r of lane group g): 2 r + (g & 1) + 8 (g >> 1), so that lane groups 0 and
// 1 (and 2 and 3), which share a half-wave's LDS access, write rows one apart.
constexpr int escn_wave_jrow(int rho) { return 2 * (rho & 3) + ((rho >> 2) & 1) + 8 * (rho >> 3); }

// Builds the tables from a plan's tables; empty (NPAIR = 0) unless
// L1 = L2 = Lout; A and Z only for L1 = kEscnWaveL.
EscnHost build_escn_tables(const Tables& t);

}  // namespace gtp
