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
//        factor): per degree block l and output tile t (escn_wave_jtile),
//        for lane 16 k + i the K-steps s of the tile (escn_wave_jsteps,
//        padded to a multiple of 4 floats, escn_wave_jnk4) at
//        escn_wave_joff(l, t) + lane escn_wave_jnk4(l, t), then the same
//        for J^T at escn_wave_jtoff() + escn_wave_joff(l, t): the entry of
//        tile row i (escn_wave_jtrow) and tile column 4 s + k
//        (escn_wave_jtcol), zero where either lies outside the block.
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
// ---- The output tiles of J and J^T on degree block l (the K index of a
// 16x16x4 contraction over the block's columns, the M index over its rows;
// the block's index is l + m, m = -l..l).
//
// Degrees below kEscnClassL: one tile of the whole block (d = 2l + 1 <= 15
// rows, ceil(d / 4) K-steps): tile row i holds block row escn_wave_jrow(i)
// = 2 (i % 4) + (i / 4) % 2 + 8 (i / 8), so that lane groups 0 and 1 (and 2
// and 3), which share a half-wave's LDS access, write rows one apart; tile
// column 4 s + k is block column 4 s + k.
//
// Degrees kEscnClassL..16: J is zero outside four square sub-blocks.  The
// block's indices fall in four classes c (0: m >= 0 with |m| even, 1: m > 0
// odd, 2: m < 0 even, 3: m < 0 odd), each taken in ascending m (first index
// escn_cls_start, step 2, escn_cls_n of them), and J (so J^T) maps each row
// class onto one column class (escn_cls_map: even l 0-0, 1-2, 3-3; odd l
// 0-3, 1-1, 2-2).  Tile 0 holds the rows of class 0 in lane groups 0, 2 and
// those of class 3 in lane groups 1, 3; tile 1 classes 1 and 2; tile 2
// (degree 16 only, whose class 0 has 9 rows) the ninth row of class 0.  A
// tile row i = 4 g + r: class R of the lane-group parity g % 2, element p =
// first + 4 (g / 2) + r.  Tile column 4 s + k: class map(R) of the lane
// group parity k % 2, element q = 2 s + k / 2.  K-steps: half the larger of
// the two column classes, rounded up.
constexpr int kEscnClassL = 8;
constexpr int escn_cls_n(int l, int c) { return c == 0 ? l / 2 + 1 : c == 2 ? l / 2 : (l + 1) / 2; }
constexpr int escn_cls_start(int l, int c) { return c == 0 ? l : c == 1 ? l + 1 : c == 2 ? (l & 1) : 1 - (l & 1); }
constexpr int escn_cls_map(int l, int c) { return (l & 1) ? (c == 0 ? 3 : c == 3 ? 0 : c) : (c == 1 ? 2 : c == 2 ? 1 : c); }
constexpr int escn_wave_jtiles(int l) { return l < kEscnClassL ? 1 : (escn_cls_n(l, 0) > 8 ? 3 : 2); }
// row class of tile t for lane-group parity par (-1: none) and its first element
constexpr int escn_wave_jtcls(int l, int t, int par) { return t == 0 ? (par ? 3 : 0) : t == 1 ? (par ? 2 : 1) : (par ? -1 : 0); }
constexpr int escn_wave_jtfirst(int t) { return t == 2 ? 8 : 0; }
// rows of class cls from element first on, at most 8 (lane groups par, par + 2)
constexpr int escn_wave_jtrows(int l, int t, int par) {
  return escn_wave_jtcls(l, t, par) < 0 ? 0
         : (escn_cls_n(l, escn_wave_jtcls(l, t, par)) - escn_wave_jtfirst(t) < 8
                ? escn_cls_n(l, escn_wave_jtcls(l, t, par)) - escn_wave_jtfirst(t)
                : 8);
}
// columns of the tile's half par (the class its rows map to, every element)
constexpr int escn_wave_jtcols(int l, int t, int par) {
  return escn_wave_jtcls(l, t, par) < 0 ? 0 : escn_cls_n(l, escn_cls_map(l, escn_wave_jtcls(l, t, par)));
}
constexpr int escn_wave_jsteps(int l, int t) {
  return l < kEscnClassL ? (2 * l + 1 + 3) / 4
                         : ((escn_wave_jtcols(l, t, 0) > escn_wave_jtcols(l, t, 1) ? escn_wave_jtcols(l, t, 0)
                                                                                   : escn_wave_jtcols(l, t, 1)) + 1) / 2;
}
constexpr int escn_wave_jnk4(int l, int t) { return (escn_wave_jsteps(l, t) + 3) / 4 * 4; }
constexpr int escn_wave_joff(int l, int t) {
  int o = 0;
  for (int k = 0; k < l; ++k)
    for (int u = 0; u < escn_wave_jtiles(k); ++u) o += 64 * escn_wave_jnk4(k, u);
  for (int u = 0; u < t; ++u) o += 64 * escn_wave_jnk4(l, u);
  return o;
}
constexpr int escn_wave_jtoff() { return escn_wave_joff(kEscnWaveL + 1, 0); }
constexpr int escn_wave_jrow(int rho) { return 2 * (rho & 3) + ((rho >> 2) & 1) + 8 * (rho >> 3); }
// block-local row of tile row i = 4 g + r (-1: padding)
constexpr int escn_wave_jtrow(int l, int t, int i) {
  if (l < kEscnClassL) return escn_wave_jrow(i) < 2 * l + 1 ? escn_wave_jrow(i) : -1;
  const int g = i / 4, r = i % 4, par = g & 1, p = 4 * (g / 2) + r;
  return p < escn_wave_jtrows(l, t, par)
             ? escn_cls_start(l, escn_wave_jtcls(l, t, par)) + 2 * (escn_wave_jtfirst(t) + p)
             : -1;
}
// block-local column of tile column 4 s + k (-1: padding)
constexpr int escn_wave_jtcol(int l, int t, int s, int k) {
  if (l < kEscnClassL) return 4 * s + k < 2 * l + 1 ? 4 * s + k : -1;
  const int par = k & 1, q = 2 * s + k / 2;
  return q < escn_wave_jtcols(l, t, par)
             ? escn_cls_start(l, escn_cls_map(l, escn_wave_jtcls(l, t, par))) + 2 * q
             : -1;
}

// Builds the tables from a plan's tables; empty (NPAIR = 0) unless
// L1 = L2 = Lout; A and Z only for L1 = kEscnWaveL.
EscnHost build_escn_tables(const Tables& t);

}  // namespace gtp
