// Host-side fp64 tables for the Gaunt Tensor Product (Sec. 3.2).
//
// Notation.  Theta_lm(t) is the theta factor of the real SH Y_l^{+-m}
// (Y_l^{+m} = Theta_lm cos(m p), Y_l^{-m} = Theta_lm sin(m p), Y_l^0 =
// Theta_l0), i.e. Theta_lm = (m > 0 ? sqrt2 : 1) * N_lm * P_l^m(cos t).
// On theta in [0, pi] Theta_lm is a cosine series (even m) or a sine series
// (odd m) of degree <= l with only u = l (mod 2) present; extended to
// [-pi, pi) by that series it gives the double-Fourier-sphere function the
// paper's 2D Fourier basis needs.  Pairs (l, m >= 0) are indexed
// tri(l, m) = l(l+1)/2 + m.
#pragma once

#include <cstdint>
#include <vector>

namespace gtp {

inline int tri(int l, int m) { return l * (l + 1) / 2 + m; }
inline int ntri(int L) { return (L + 1) * (L + 2) / 2; }
inline int nsh(int L) { return (L + 1) * (L + 1); }

struct Tables {
  int L1 = 0, L2 = 0, Lout = 0;
  int U = 0;    // L1 + L2: theta/phi degree of the product
  int Le = 0;   // min(Lout, U): highest output degree that can be non-zero
  int Lin = 0;  // max(L1, L2)
  int Lt = 0;   // max(Lin, Le): rows of T1
  int NT = 0;   // theta intervals of the sampling grid t_j = j pi / NT, j = 0..NT
  int NJ = 0;   // NT + 1 theta nodes
  int NP = 0;   // phi samples p_k = 2 pi k / NP
  int ldT1 = 0; // Lt + 1
  int ldZ = 0;  // NT + 1

  // Step 1 (eq. sh-fs): Theta_lm(t) = sum_u T1[tri][u] {cos|sin}(u t), l <= Lt.
  std::vector<double> T1;
  // Step 3 (eq. fs-sh): Zc = int_0^pi cos(u t) Theta_lm sin t dt,
  //                     Zs = int_0^pi sin(u t) Theta_lm sin t dt, l <= Le, u <= NT.
  std::vector<double> Zc, Zs;
  // Convolution-theorem path: S = Theta_lm at the theta nodes (T1 composed
  // with the inverse theta DFT), l <= Lin; W = weights that map the theta
  // samples of a band-limited phi moment to the SH coefficient (Zc/Zs
  // composed with the forward theta DFT, times 2 pi / NP), l <= Le.
  std::vector<double> S, W;
  // phi trigonometric table trig(mp, k): mp = 0 -> 1, mp = 2m-1 -> cos(m p_k),
  // mp = 2m -> sin(m p_k), for m <= Mphi = max(Lin, Le); layout [mp][k].
  int Mphi = 0;
  std::vector<double> Phi;

  // Lane-permuted tables of the wave-per-product kernel whose phi transforms
  // run on the matrix cores; built when L1 = L2 = Lout = L with L in {16, 32}
  // (waveL = L), empty otherwise.  Layouts are given in build_wave_tables.
  int waveL = 0;
  std::vector<double> TWR, SMP, SM0P, WP;
  std::vector<int> XMAPP;
  int XQUADS = 0;  // quads of the kernel's LDS image of one input pair
};

// Fills the wave-kernel tables (and t.waveL) from t.S, t.W and the phi grid;
// t must have L1 = L2 = Lout = L in {16, 32}.
void build_wave_tables(Tables& t);

// Builds every table for (L1, L2, Lout) in fp64.  Throws std::invalid_argument
// on a bad degree.
Tables build_tables(int L1, int L2, int Lout);

// Theta factors Theta_lm(t) for all l <= L, m >= 0 at one angle (own fp64
// recurrence), out[tri(l, m)].
void theta_factors(int L, double t, double* out);

// fp64 evaluation of the sampled three-step pipeline with the tables above
// (host check of the tables; never used by the device path).
void host_pipeline(const Tables& t, const double* x1, const double* x2, int64_t n, double* y);

}  // namespace gtp
