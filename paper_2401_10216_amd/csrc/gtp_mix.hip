// Channel mixing of pair products on the fp32 matrix cores (gfx950).
//
// The channel-mixing combination of the appendix's discussion of channels,
// y[b, co] = sum_{c1, c2} W[co, c1, c2] GTP(x1[b, c1], x2[b, c2]), is linear in
// the pair products T[b, p] = GTP(x1[b, c1], x2[b, c2]) (p = c1 C2 + c2), so
// after the products it is one matrix product per batch entry:
//     y_b (Co x K) = W (Co x P) T_b (P x K),   P = C1 C2.
// One wave computes a 16 x 64 tile of y_b with v_mfma_f32_16x16x4f32: in
// K-step s the A operand of lane 16 g + i is W[co0 + i][4 s + g], the B
// operand of block nb is T_b[4 s + g][n0 + 16 nb + i]; D register r of lane
// 16 g + i is y_b[co0 + 4 g + r][n0 + 16 nb + i].  The operands of the next
// K-step are loaded before the current one's matrix instructions.
#include "gtp_device.hpp"

namespace gtp {
namespace {

typedef float f4v __attribute__((ext_vector_type(4)));

constexpr int kNB = 4;  // 16-column blocks per wave (64 columns)

__global__ __launch_bounds__(64) void k_mix_gemm(const float* __restrict__ W, const float* __restrict__ T,
                                                 float* __restrict__ y, int Co, int64_t P, int K, int ncot,
                                                 int nnt) {
  const int lane = threadIdx.x, g = lane >> 4, i = lane & 15;
  const int64_t b = blockIdx.x / (int64_t(ncot) * nnt);
  const int rem = int(blockIdx.x % (int64_t(ncot) * nnt));
  const int co0 = (rem / nnt) * 16, n0 = (rem % nnt) * (16 * kNB);
  const float* Tb = T + b * P * K;
  const int arow = co0 + i;
  const bool aok = arow < Co;
  const float* Wr = W + int64_t(aok ? arow : 0) * P;
  bool bok[kNB];
  int bcol[kNB];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    bcol[nb] = n0 + 16 * nb + i;
    bok[nb] = bcol[nb] < K;
  }
  f4v acc[kNB];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) acc[nb] = f4v{0.0f, 0.0f, 0.0f, 0.0f};
  // operands of K-step s (rows p = 4 s + g; zero past P, Co or K)
  auto load = [&](int64_t s, float& a, float (&bv)[kNB]) {
    const int64_t p = 4 * s + g;
    const bool pok = p < P;
    a = (aok && pok) ? Wr[p] : 0.0f;
    const float* Tp = Tb + (pok ? p : 0) * K;
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) bv[nb] = (pok && bok[nb]) ? Tp[bcol[nb]] : 0.0f;
  };
  const int64_t steps = (P + 3) / 4;
  float a, bv[kNB];
  load(0, a, bv);
  for (int64_t s = 0; s < steps; ++s) {
    float an = 0.0f, bn[kNB];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) bn[nb] = 0.0f;
    if (s + 1 < steps) load(s + 1, an, bn);
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) acc[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv[nb], acc[nb], 0, 0, 0);
    a = an;
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) bv[nb] = bn[nb];
  }
  float* yb = y + b * int64_t(Co) * K;
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    if (!bok[nb]) continue;
    for (int r = 0; r < 4; ++r) {
      const int row = co0 + 4 * g + r;
      if (row < Co) yb[int64_t(row) * K + bcol[nb]] = acc[nb][r];
    }
  }
}

__global__ __launch_bounds__(256) void k_fill_zero(float* __restrict__ y, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) y[i] = 0.0f;
}

}  // namespace

hipError_t launch_fill_zero(float* y, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t g = (n + 255) / 256;
  if (g > 65536) g = 65536;
  hipLaunchKernelGGL(k_fill_zero, dim3(unsigned(g)), dim3(256), 0, s, y, n);
  return hipGetLastError();
}

hipError_t launch_mix_gemm(const float* W, const float* T, float* y, int Co, int64_t P, int K, int64_t nb,
                           hipStream_t s) {
  if (nb <= 0) return hipSuccess;
  const int ncot = (Co + 15) / 16, nnt = (K + 16 * kNB - 1) / (16 * kNB);
  const int64_t grid = nb * ncot * nnt;
  if (grid > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_mix_gemm, dim3(unsigned(grid)), dim3(64), 0, s, W, T, y, Co, P, K, ncot, nnt);
  return hipGetLastError();
}

}  // namespace gtp
