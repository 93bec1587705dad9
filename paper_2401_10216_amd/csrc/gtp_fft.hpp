// Radix-2 fast Fourier transforms held in one lane's registers, with
// compile-time twiddle factors, for the phi transforms of the matrix-core
// kernel's FFT variant (Sec. 3.2: the 2D convolution taken by the
// convolution theorem with FFTs).  A length-N transform is split as
// N = N1 N2 across lanes and LDS (the four-step decomposition); these are the
// in-register pieces of length N1 and N2.
#pragma once

#include "gtp_ct.hpp"

namespace gtp {

struct cpx {
  float re, im;
};

__host__ __device__ __forceinline__ cpx cadd(cpx a, cpx b) { return {a.re + b.re, a.im + b.im}; }
__host__ __device__ __forceinline__ cpx csub(cpx a, cpx b) { return {a.re - b.re, a.im - b.im}; }
__host__ __device__ __forceinline__ cpx cmul(cpx a, cpx b) {
  return {fmaf(a.re, b.re, -(a.im * b.im)), fmaf(a.re, b.im, a.im * b.re)};
}
__host__ __device__ __forceinline__ cpx cconj(cpx a) { return {a.re, -a.im}; }

// v exp(i 2 pi SIGN J / N) for compile-time J, N: multiples of a quarter
// turn are sign changes and swaps, odd multiples of an eighth turn take two
// adds and two multiplies, the rest a full complex multiply.
template <int J, int N, int SIGN>
__host__ __device__ __forceinline__ cpx twiddle(cpx v) {
  constexpr int j = ((J % N) + N) % N;
  if constexpr (j == 0) {
    return v;
  } else if constexpr (2 * j == N) {
    return {-v.re, -v.im};
  } else if constexpr (4 * j == N) {  // SIGN i
    return SIGN > 0 ? cpx{-v.im, v.re} : cpx{v.im, -v.re};
  } else if constexpr (4 * j == 3 * N) {  // -SIGN i
    return SIGN > 0 ? cpx{v.im, -v.re} : cpx{-v.im, v.re};
  } else {
    constexpr float c = ct_round(ct_cos2pi(j, N));
    constexpr float s = SIGN > 0 ? ct_round(ct_sin2pi(j, N)) : -ct_round(ct_sin2pi(j, N));
    constexpr bool eighth = (8 * j) % N == 0 && (8 * j / N) % 2 == 1;  // |c| = |s| = 1 / sqrt 2
    if constexpr (eighth && c == s) {  // w = c (1 + i)
      return {c * (v.re - v.im), c * (v.re + v.im)};
    } else if constexpr (eighth && c == -s) {  // w = c (1 - i)
      return {c * (v.re + v.im), c * (v.im - v.re)};
    } else {
      return {fmaf(v.re, c, -(v.im * s)), fmaf(v.re, s, v.im * c)};
    }
  }
}

constexpr int ct_log2(int n) { return n <= 1 ? 0 : 1 + ct_log2(n / 2); }
constexpr int ct_bitrev(int i, int bits) {
  int r = 0;
  for (int b = 0; b < bits; ++b) r |= ((i >> b) & 1) << (bits - 1 - b);
  return r;
}

// In-place DFT of length N (a power of two) in registers:
//   a[k] <- sum_j a[j] exp(i 2 pi SIGN j k / N),
// natural order in and out (decimation in time: the bit-reversed reordering
// is register renaming), log2 N stages of butterflies.
template <int N, int SIGN>
__host__ __device__ __forceinline__ void fft_reg(cpx (&a)[N]) {
  static_assert((N & (N - 1)) == 0, "radix-2 length");
  constexpr int B = ct_log2(N);
  cpx b[N];
  cfor<0, N>([&](auto I) { b[ct_bitrev(decltype(I)::value, B)] = a[decltype(I)::value]; });
  cfor<1, B + 1>([&](auto S) {
    constexpr int len = 1 << decltype(S)::value, half = len / 2;
    cfor<0, N / len>([&](auto BL) {
      constexpr int base = decltype(BL)::value * len;
      cfor<0, half>([&](auto J) {
        constexpr int j = decltype(J)::value;
        const cpx u = b[base + j];
        const cpx v = twiddle<j, len, SIGN>(b[base + j + half]);
        b[base + j] = cadd(u, v);
        b[base + j + half] = csub(u, v);
      });
    });
  });
  cfor<0, N>([&](auto I) { a[decltype(I)::value] = b[decltype(I)::value]; });
}

// Forward DFT of N real values, twice its outputs m = 0..N/2:
//   X2[m] = 2 sum_k g[k] exp(-i 2 pi m k / N),
// from one complex DFT of length N/2 of the even / odd pairs (z_j = g_2j +
// i g_2j+1): with Z the DFT of z, 2 E[m] = Z[m] + conj Z[N/2 - m] and
// 2 O[m] = -i (Z[m] - conj Z[N/2 - m]) are the DFTs of the even and odd
// samples, and X = E + exp(-i 2 pi m / N) O.
template <int N>
__host__ __device__ __forceinline__ void rfft2_fwd(const float (&g)[N], cpx (&X2)[N / 2 + 1]) {
  constexpr int H = N / 2;
  cpx z[H];
  cfor<0, H>([&](auto J) { z[decltype(J)::value] = {g[2 * decltype(J)::value], g[2 * decltype(J)::value + 1]}; });
  fft_reg<H, -1>(z);
  cfor<0, H + 1>([&](auto M) {
    constexpr int m = decltype(M)::value;
    const cpx zm = z[m % H], zc = cconj(z[(H - m) % H]);
    const cpx e2 = cadd(zm, zc);
    const cpx d = csub(zm, zc);
    const cpx o2 = {d.im, -d.re};
    X2[m] = cadd(e2, twiddle<m, N, -1>(o2));
  });
}

// Powers w^0 .. w^(N-1) of a runtime complex w by a product tree (depth
// log2 N, so the rounding error stays a few units in the last place).
template <int N>
__host__ __device__ __forceinline__ void cpowers(cpx w, cpx (&p)[N]) {
  p[0] = {1.0f, 0.0f};
  if constexpr (N > 1) p[1] = w;
  cfor<2, N>([&](auto K) {
    constexpr int k = decltype(K)::value;
    // k = a + (k - a), a the largest power of two below k (k / 2 for a power
    // of two): both factors are already formed
    constexpr int a = (1 << ct_log2(k)) == k ? k / 2 : (1 << ct_log2(k));
    p[k] = cmul(p[a], p[k - a]);
  });
}

}  // namespace gtp
