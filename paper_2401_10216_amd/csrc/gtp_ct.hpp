// Compile-time helpers shared by the kernels: a loop whose index is a
// compile-time constant in its body, and cos / sin of 2 pi k / N evaluated at
// compile time (exact integer reduction of the angle, then a Taylor series in
// fp64; rounded once to fp32 where a kernel uses the value).
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>
#include <utility>

namespace gtp {

template <int B, int... Is, typename F>
__host__ __device__ __forceinline__ void cfor_impl(std::integer_sequence<int, Is...>, F& f) {
  (f(std::integral_constant<int, B + Is>{}), ...);
}
// Compile-time loop over [B, E): f(std::integral_constant<int, i>) for each i.
template <int B, int E, typename F>
__host__ __device__ __forceinline__ void cfor(F&& f) {
  if constexpr (E > B) cfor_impl<B>(std::make_integer_sequence<int, E - B>{}, f);
}

constexpr double kPiD = 3.14159265358979323846264338327950288;

constexpr double ct_angle(long long k, long long N) {
  long long r = k % N;
  if (r < 0) r += N;
  double x = 2.0 * kPiD * double(r) / double(N);
  if (x > kPiD) x -= 2.0 * kPiD;
  return x;
}
constexpr double ct_cos2pi(long long k, long long N) {
  const double x = ct_angle(k, N);
  double term = 1.0, sum = 1.0;
  for (int i = 1; i < 40; ++i) {
    term *= -x * x / double((2 * i - 1) * (2 * i));
    sum += term;
  }
  return sum;
}
constexpr double ct_sin2pi(long long k, long long N) {
  const double x = ct_angle(k, N);
  double term = x, sum = x;
  for (int i = 1; i < 40; ++i) {
    term *= -x * x / double((2 * i) * (2 * i + 1));
    sum += term;
  }
  return sum;
}
constexpr float ct_round(double v) {
  // exact zeros and units stay exact; everything else rounds to fp32
  return (v > -1e-15 && v < 1e-15) ? 0.0f : float(v);
}

}  // namespace gtp
