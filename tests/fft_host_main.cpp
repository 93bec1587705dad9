// Host build of the register FFT pieces of gtp_fft.hpp (test infrastructure):
// fft_reg, rfft2_fwd and cpowers against plain O(N^2) sums in double
// precision.  Prints the worst relative error of each; exit status 1 if any
// exceeds 1e-6.
#include <cmath>
#include <cstdio>
#include <random>

#include "gtp_fft.hpp"

namespace {

std::mt19937_64 rng(12345);
std::normal_distribution<double> N01(0.0, 1.0);

template <int N, int SIGN>
double check_fft() {
  gtp::cpx a[N];
  double re[N], im[N];
  for (int j = 0; j < N; ++j) {
    re[j] = float(N01(rng));
    im[j] = float(N01(rng));
    a[j] = {float(re[j]), float(im[j])};
  }
  gtp::fft_reg<N, SIGN>(a);
  double worst = 0.0, norm = 0.0;
  for (int k = 0; k < N; ++k) {
    double sr = 0.0, si = 0.0;
    for (int j = 0; j < N; ++j) {
      const double t = 2.0 * M_PI * SIGN * double(j) * double(k) / N;
      sr += re[j] * std::cos(t) - im[j] * std::sin(t);
      si += re[j] * std::sin(t) + im[j] * std::cos(t);
    }
    norm = std::fmax(norm, std::hypot(sr, si));
    worst = std::fmax(worst, std::hypot(a[k].re - sr, a[k].im - si));
  }
  return worst / norm;
}

template <int N>
double check_rfft() {
  float g[N];
  for (int j = 0; j < N; ++j) g[j] = float(N01(rng));
  gtp::cpx X2[N / 2 + 1];
  gtp::rfft2_fwd<N>(g, X2);
  double worst = 0.0, norm = 0.0;
  for (int m = 0; m <= N / 2; ++m) {
    double sr = 0.0, si = 0.0;
    for (int k = 0; k < N; ++k) {
      const double t = -2.0 * M_PI * double(m) * double(k) / N;
      sr += 2.0 * g[k] * std::cos(t);
      si += 2.0 * g[k] * std::sin(t);
    }
    norm = std::fmax(norm, std::hypot(sr, si));
    worst = std::fmax(worst, std::hypot(X2[m].re - sr, X2[m].im - si));
  }
  return worst / norm;
}

template <int N>
double check_powers(int j, int NF) {
  const double t = 2.0 * M_PI * j / NF;
  gtp::cpx p[N];
  gtp::cpowers<N>({float(std::cos(t)), float(std::sin(t))}, p);
  double worst = 0.0;
  for (int k = 0; k < N; ++k)
    worst = std::fmax(worst, std::hypot(p[k].re - std::cos(k * t), p[k].im - std::sin(k * t)));
  return worst;
}

}  // namespace

int main() {
  double e[] = {check_fft<8, 1>(),   check_fft<8, -1>(),  check_fft<16, 1>(), check_fft<16, -1>(),
                check_fft<4, -1>(),  check_fft<32, 1>(),  check_rfft<8>(),    check_rfft<16>(),
                check_powers<8>(3, 128), check_powers<16>(5, 256), check_powers<9>(7, 128), check_powers<9>(127, 128)};
  const char* names[] = {"fft8+", "fft8-", "fft16+", "fft16-", "fft4-", "fft32+", "rfft8", "rfft16",
                         "pow8", "pow16", "pow9", "pow9b"};
  int bad = 0;
  for (int i = 0; i < 12; ++i) {
    std::printf("%s %.3e\n", names[i], e[i]);
    if (!(e[i] <= 1e-6)) bad = 1;
  }
  return bad;
}
