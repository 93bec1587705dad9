// Host-side driver for the sanitizer build of the library's fp64 table
// builders (test infrastructure): builds the tables of a spread of degree
// triples (unequal degrees, truncated and zero-padded outputs, the
// matrix-core kernels' lane-permuted tables at 16, 32, 64, the rotated-frame
// tables at 1..8), runs the host pipeline on seeded inputs and checks that
// every value is finite.  Compiled with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_host_sanitize.py; any report
// aborts the run.
#include <cmath>
#include <cstdio>
#include <random>
#include <vector>

#include "gtp_escn_tables.hpp"
#include "gtp_tables.hpp"

namespace {

bool finite(const std::vector<double>& v) {
  for (double d : v)
    if (!std::isfinite(d)) return false;
  return true;
}

int check(int L1, int L2, int Lout, int n) {
  const gtp::Tables t = gtp::build_tables(L1, L2, Lout);
  if (!finite(t.T1) || !finite(t.Zc) || !finite(t.Zs) || !finite(t.S) || !finite(t.W) || !finite(t.Phi) ||
      !finite(t.TWR) || !finite(t.SMP) || !finite(t.SM0P) || !finite(t.WP)) {
    std::printf("non-finite table entry at (%d, %d, %d)\n", L1, L2, Lout);
    return 1;
  }
  std::mt19937_64 rng(uint64_t(1 + L1 + 100 * L2 + 10000 * Lout));
  std::normal_distribution<double> N(0.0, 1.0);
  std::vector<double> x1(size_t(n) * gtp::nsh(L1)), x2(size_t(n) * gtp::nsh(L2)), y(size_t(n) * gtp::nsh(Lout));
  for (double& v : x1) v = N(rng);
  for (double& v : x2) v = N(rng);
  gtp::host_pipeline(t, x1.data(), x2.data(), n, y.data());
  if (!finite(y)) {
    std::printf("non-finite pipeline output at (%d, %d, %d)\n", L1, L2, Lout);
    return 1;
  }
  if (L1 == L2 && L2 == Lout && L1 >= 1 && L1 <= 8) {
    const gtp::EscnHost e = gtp::build_escn_tables(t);
    if (!finite(e.J) || !finite(e.E)) {
      std::printf("non-finite rotated-frame table at L=%d\n", L1);
      return 1;
    }
  }
  std::printf("ok %d %d %d\n", L1, L2, Lout);
  return 0;
}

}  // namespace

int main() {
  const int triples[][3] = {{0, 0, 0}, {1, 0, 1}, {0, 3, 2}, {2, 2, 2}, {2, 3, 9}, {3, 2, 3}, {4, 6, 5},
                            {6, 6, 2}, {6, 6, 6}, {7, 7, 7}, {8, 8, 8},  {10, 3, 7}, {12, 12, 12}, {16, 16, 16},
                            {20, 9, 30}, {32, 32, 32}, {64, 64, 64}, {64, 0, 64}, {5, 64, 3}};
  int bad = 0;
  for (const auto& t : triples) bad |= check(t[0], t[1], t[2], t[0] >= 32 || t[1] >= 32 ? 1 : 3);
  return bad;
}
