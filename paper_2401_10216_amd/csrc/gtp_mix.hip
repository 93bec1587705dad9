// Channel mixing of pair products on the fp32 matrix cores (gfx950).
//
// The channel-mixing rule of the appendix (Implementation Details),
// y[b, co] = sum_{c1, c2} W[co, c1, c2] GTP(x1[b, c1], x2[b, c2]), is linear in
// the pair products T[b, p] = GTP(x1[b, c1], x2[b, c2]) (p = c1 C2 + c2), so
// after the products it is one matrix product per batch entry,
//     y_b^T (K x Co) = T_b^T (K x P) W^T (P x Co),   P = C1 C2,
// taken with v_mfma_f32_16x16x4f32 (A[i][k] from lane 16 k + i, B[k][j] from
// lane 16 k + j, D register r of lane 16 g + i = row 4 g + r, column i).
// One wave computes a 16 (k) x 32 (co) tile: in K-step s the A operand of
// lane 16 g + i is T_b[4 s + g][n0 + i] and the B operands are
// W^T[4 s + g][co0 + i] and [co0 + 16 + i], all rows read as contiguous
// 64-byte runs (W^T is a transposed copy made once per call).  The operands
// of the next 8 K-steps are loaded before the current 8 K-steps' matrix
// instructions.
#include "gtp_device.hpp"

namespace gtp {
namespace {

typedef float f4v __attribute__((ext_vector_type(4)));

constexpr int kCB = 2;  // 16-column blocks of output channels per wave
constexpr int kKB = 8;  // K-steps (4 rows of P each) per loaded block

// WT[p][co] = W[co][p], co < CoP (columns past Co are zero)
__global__ __launch_bounds__(256) void k_mix_transpose(const float* __restrict__ W, float* __restrict__ WT, int Co,
                                                       int CoP, int64_t P) {
  const int64_t total = P * CoP;
  for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int64_t p = e / CoP;
    const int co = int(e - p * CoP);
    WT[e] = co < Co ? W[int64_t(co) * P + p] : 0.0f;
  }
}

__global__ __launch_bounds__(64) void k_mix_gemm(const float* __restrict__ WT, const float* __restrict__ T,
                                                 float* __restrict__ y, int Co, int CoP, int64_t P, int K, int nnt,
                                                 int nct) {
  const int lane = threadIdx.x, g = lane >> 4, i = lane & 15;
  const int64_t b = blockIdx.x / (int64_t(nnt) * nct);
  const int rem = int(blockIdx.x % (int64_t(nnt) * nct));
  const int n0 = (rem / nct) * 16, co0 = (rem % nct) * (16 * kCB);
  const float* Tb = T + b * P * K;
  const int acol = n0 + i;  // row of y_b^T (coefficient index)
  const bool aok = acol < K;
  f4v acc[kCB];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) acc[cb] = f4v{0.0f, 0.0f, 0.0f, 0.0f};
  // operands of K-step s (rows p = 4 s + g; zero past P or K; the W^T
  // columns past Co are zero in the copy), a block of kKB K-steps at a time;
  // the next block's loads are issued before this block's matrix instructions
  struct Blk {
    float a[kKB], b[kKB][kCB];
  };
  auto load = [&](int64_t blk, Blk& o) {
#pragma unroll
    for (int t = 0; t < kKB; ++t) {
      const int64_t p = 4 * (blk * kKB + t) + g;
      const bool pok = p < P;
      const int64_t pr = pok ? p : 0;
      o.a[t] = (aok && pok) ? Tb[pr * K + acol] : 0.0f;
#pragma unroll
      for (int cb = 0; cb < kCB; ++cb) o.b[t][cb] = pok ? WT[pr * CoP + co0 + 16 * cb + i] : 0.0f;
    }
  };
  auto mma = [&](const Blk& o) {
#pragma unroll
    for (int t = 0; t < kKB; ++t)
#pragma unroll
      for (int cb = 0; cb < kCB; ++cb) acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a[t], o.b[t][cb], acc[cb], 0, 0, 0);
  };
  const int64_t nblk = (P + 4 * kKB - 1) / (4 * kKB);
  Blk b0, b1;
  load(0, b0);
  for (int64_t blk = 0; blk < nblk; blk += 2) {
    if (blk + 1 < nblk) load(blk + 1, b1);
    mma(b0);
    if (blk + 1 < nblk) {
      if (blk + 2 < nblk) load(blk + 2, b0);
      mma(b1);
    }
  }
  // D[n][co]: lane 16 g + i holds n = n0 + 4 g + r, co = co0 + 16 cb + i
  float* yb = y + b * int64_t(Co) * K;
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
    const int co = co0 + 16 * cb + i;
    if (co >= Co) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int n = n0 + 4 * g + r;
      if (n < K) yb[int64_t(co) * K + n] = acc[cb][r];
    }
  }
}

// WB[q][co][g][s'] = W[co][16 q + 4 s' + g] (zero past P and Co) for
// q < PR / 16, co < CoB: the B operands of four K-steps of the fused mix in
// one 16-byte run per lane.
__global__ __launch_bounds__(256) void k_mix_wt_blocks(const float* __restrict__ W, float* __restrict__ WB, int Co,
                                                       int CoB, int64_t P, int64_t PR) {
  const int64_t total = PR * CoB;
  for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total; e += int64_t(gridDim.x) * 256) {
    const int sp = int(e & 3), g = int((e >> 2) & 3);
    const int64_t qc = e >> 4;
    const int64_t q = qc / CoB;
    const int co = int(qc - q * CoB);
    const int64_t p = 16 * q + 4 * sp + g;
    WB[e] = (co < Co && p < P) ? W[int64_t(co) * P + p] : 0.0f;
  }
}

__global__ __launch_bounds__(256) void k_fill_zero(float* __restrict__ y, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) y[i] = 0.0f;
}

}  // namespace

int mix_cop(int Co) { return (Co + 16 * kCB - 1) / (16 * kCB) * (16 * kCB); }

hipError_t launch_fill_zero(float* y, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t g = (n + 255) / 256;
  if (g > 65536) g = 65536;
  hipLaunchKernelGGL(k_fill_zero, dim3(unsigned(g)), dim3(256), 0, s, y, n);
  return hipGetLastError();
}

hipError_t launch_mix_transpose(const float* W, float* WT, int Co, int64_t P, hipStream_t s) {
  const int CoP = mix_cop(Co);
  int64_t g = (P * CoP + 255) / 256;
  if (g > 65536) g = 65536;
  if (g < 1) return hipSuccess;
  hipLaunchKernelGGL(k_mix_transpose, dim3(unsigned(g)), dim3(256), 0, s, W, WT, Co, CoP, P);
  return hipGetLastError();
}

hipError_t launch_mix_wt_blocks(const float* W, float* WB, int Co, int64_t P, int nct, hipStream_t s) {
  const int CoB = 16 * nct;
  const int64_t PR = (P + 255) / 256 * 256;
  int64_t g = (PR * CoB + 255) / 256;
  if (g > 65536) g = 65536;
  if (g < 1) return hipSuccess;
  hipLaunchKernelGGL(k_mix_wt_blocks, dim3(unsigned(g)), dim3(256), 0, s, W, WB, Co, CoB, P, PR);
  return hipGetLastError();
}

hipError_t launch_mix_gemm(const float* WT, const float* T, float* y, int Co, int64_t P, int K, int64_t nb,
                           hipStream_t s) {
  if (nb <= 0) return hipSuccess;
  const int CoP = mix_cop(Co);
  const int nnt = (K + 15) / 16, nct = CoP / (16 * kCB);
  const int64_t grid = nb * nnt * nct;
  if (grid > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_mix_gemm, dim3(unsigned(grid)), dim3(64), 0, s, WT, T, y, Co, CoP, P, K, nnt, nct);
  return hipGetLastError();
}

}  // namespace gtp
