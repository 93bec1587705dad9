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
struct EscnHost {
  int LM = 0, NPAIR = 0, ERL = 0;
  std::vector<double> J, E;
};

// Builds the tables from a plan's tables; empty (NPAIR = 0) unless
// L1 = L2 = Lout.
EscnHost build_escn_tables(const Tables& t);

}  // namespace gtp
