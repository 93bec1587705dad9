// Device-side declarations shared by the HIP kernels and the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gtp {

// fp32 copies of a plan's tables on one device (see gtp_tables.hpp for the
// definitions).  Row index tri(l, m) = l(l+1)/2 + m.
struct DevTables {
  int L1, L2, Lout, U, Le, Lin, NT, NJ, NP, Mphi, ldT1, ldZ;
  const float* S;     // [tri(l<=Lin)][NJ]   Theta_lm at theta nodes
  const float* W;     // [tri(l<=Le)][NJ]    analysis weights
  const float* WT;    // [NJ][tri(l<=Le)]    transposed W (node-major)
  const float* ST;    // [NJ][tri(l<=Lin)]   transposed S (node-major)
  int ntS, ntW;       // row lengths of ST and WT
  const float* Phi;   // [2 Mphi + 1][NP]    trig(mp, k)
  const float* PhiT;  // [NP][2 Mphi + 1]
  const float* T1;    // [tri(l<=Lt)][ldT1]  theta-Fourier series of Theta_lm
  const float* Zc;    // [tri(l<=Le)][ldZ]
  const float* Zs;    // [tri(l<=Le)][ldZ]
  // Lane-permuted tables of the matrix-core wave kernel (L1 = L2 = Lout =
  // waveL in {16, 32}; null and waveL = 0 otherwise).
  int waveL;
  const float* TWR;   // [lane][24]             seeds of the phi operands (rotation recurrences)
  const float* SMP;   // [pass][s][u2][lane][4] theta synthesis values
  const float* SM0P;  // [pass][lane][v]        m = 0 theta synthesis values (+ pole)
  const float* WP;    // [pass][it][lane][8]    theta analysis weights
  const int* XMAP;    // [lane][k]              LDS slot of input coefficient lane + 64 k
  int XQUADS;
  int phi_fft;        // 1: the matrix-core kernel's phi transforms by radix-2 FFT (GTP_CONV_FFT)
};

enum InType : int { IN_F32 = 0, IN_BF16 = 1 };

// Per-degree weights folded into one product's input loads and output store
// (Sec. 3.1, the weights w_{l1} w_{l2} w_l of a weighted combination): the
// degree-l block of x1 is scaled by w1[row][l], of x2 by w2[row][l], of y by
// wo[row][l], with row = (pbase + p) % C when per_channel, else 0, for the
// launch's product p (pbase: the launch's first product in the caller's
// batch).  A null pointer means all ones; on = false when all three are null.
struct DegWeights {
  const float* w1;
  const float* w2;
  const float* wo;
  int64_t C;
  int64_t pbase;
  int per_channel;
  bool on;
};

// Outer-product indexing of a batch of pair products (channel mixing):
// product p = (b C1 + c1) C2 + c2 takes row b C1 + c1 of x1 and row b C2 + c2
// of x2.  C2 = 0: plain indexing (product p takes row p of both).
struct PairIdx {
  int64_t C1, C2;
};

__device__ __forceinline__ void pair_rows(const PairIdx& q, int64_t p, int64_t& r1, int64_t& r2) {
  const int64_t bc1 = p / q.C2;
  r1 = bc1;
  r2 = (bc1 / q.C1) * q.C2 + (p - bc1 * q.C2);
}

__device__ __forceinline__ int64_t weight_row(const DegWeights& w, int64_t p) {
  return w.per_channel ? (w.pbase + p) % w.C : 0;
}

// degree l of SH coefficient index i = l*l + l + m
__device__ __forceinline__ int degree_of(int i) {
  int l = int(sqrtf(float(i)));
  l += ((l + 1) * (l + 1) <= i) ? 1 : 0;
  l -= (l * l > i) ? 1 : 0;
  return l;
}

// Poisoned-LDS debug build (compiled with -DGTP_POISON_LDS; the library
// then carries the name libgtp_poison.so): every kernel fills its LDS with a
// quiet-NaN pattern before first use, so a read of a location the kernel has
// not written yet (a race, a missing wait, a bad index) turns its results
// into NaN.  All threads of the workgroup call it; it ends with a barrier.
// Compiled to nothing in the regular build.
__device__ __forceinline__ void lds_poison(float* p, int n) {
#ifdef GTP_POISON_LDS
  const int nt = int(blockDim.x * blockDim.y * blockDim.z);
  for (int i = int(threadIdx.x); i < n; i += nt) p[i] = __int_as_float(0x7fc0dead);
  __syncthreads();
#else
  (void)p;
  (void)n;
#endif
}

// Logical index of workgroup w among n: the dispatcher deals workgroups to
// the 8 XCDs round robin (w mod 8), so XCD x takes the x-th contiguous run of
// logical indices (runs of n / 8, the first n mod 8 one longer).  Work items
// with neighbouring indices share cache lines (adjacent rows, one edge's
// rotation matrices); this keeps their readers in one XCD's L2.  A bijection
// of [0, n).
__device__ __forceinline__ int64_t xcd_product(int64_t w, int64_t n) {
  const int64_t q = n >> 3, r = n & 7, x = w & 7;
  return x * q + (x < r ? x : r) + (w >> 3);
}

// Launchers (return the launch's hipError_t).  n = number of products.
// Thread-per-product fused kernel for the degree triples it is instantiated
// for; *supported = false when (L1, L2, Lout, nu) or the pair of input types
// (it1, it2) has no instantiation.
hipError_t launch_full_small(const DevTables& t, const void* x1, int it1, const void* x2, int it2, int64_t n,
                             float* y, int nu, const DegWeights& wt, hipStream_t s, bool* supported);
// Stepwise many-body chain in one kernel (thread per product) for the
// instantiated (L, nu, Lout); t1 = tables of (L, L, Lout), t2 = (Lout, L, Lout).
hipError_t launch_self_stepwise_small(const DevTables& t1, const DevTables& t2, int nu, const void* x,
                                      int in_type, int64_t n, float* y, hipStream_t s, bool* supported);
// Wave-per-product fused kernel with the phi stage on the matrix cores, for
// L1 = L2 = Lout = L in {16, 32, 64}; *supported = false otherwise, or for a
// bf16 x1 with an fp32 x2.
// Degree-padded thread-per-product kernel (padded degree L in 1..8, tables
// compiled in): inputs of k1 / k2 coefficients per row read as degree-L
// vectors (zeros above), ko outputs per row written (zeros above degree L).
hipError_t launch_full_small_padded(int L, const void* x1, int it1, int k1, const void* x2, int it2, int k2,
                                    int64_t n, float* y, int ko, hipStream_t s, bool* supported);
// k1, k2, ko > 0: a plan of lower degrees padded to the tables' degree
// (input rows of k1 / k2 coefficients, output rows of ko; no weights).
hipError_t launch_full_wave(const DevTables& t, const void* x1, int it1, const void* x2, int it2, int64_t n,
                            float* y, const DegWeights& wt, hipStream_t s, bool* supported, int k1 = 0, int k2 = 0,
                            int ko = 0);
// Workgroup-per-product fused kernel, any degrees (nu = 0: x1 * x2;
// nu >= 2: x1^nu with the plan built for U = nu * L).
hipError_t launch_full_generic(const DevTables& t, const void* x1, int type1, const void* x2, int type2,
                               int64_t n, float* y, int nu, const DegWeights& wt, hipStream_t s,
                               const PairIdx& pi = PairIdx{0, 0});
// All pair products T[b, c1, c2] = P_Lout(x1[b, c1] * x2[b, c2]) for n = B C1 C2
// products (outer-product indexing) with the thread-per-product kernel, for
// L1 = L2 = Lout <= 8 and equal input types; *supported = false otherwise.
hipError_t launch_pairs_small(const DevTables& t, const void* x1, int it1, const void* x2, int it2, int64_t n,
                              float* y, const PairIdx& pi, hipStream_t s, bool* supported);
// Channel mixing of pair products: y[b, co, k] = sum_p W[co, p] T[b, p, k],
// p < P, k < K, for nb batch entries (fp32 matrix cores), from the
// transposed copy WT[p][co] (mix_cop(Co) columns, made by
// launch_mix_transpose).
int mix_cop(int Co);
hipError_t launch_mix_transpose(const float* W, float* WT, int Co, int64_t P, hipStream_t s);
hipError_t launch_mix_gemm(const float* WT, const float* T, float* y, int Co, int64_t P, int K, int64_t nb,
                           hipStream_t s);
// y[0 .. n) = 0 with a kernel (safe inside captured graphs).
hipError_t launch_fill_zero(float* y, int64_t n, hipStream_t s);
// Weight gradients of the weighted product (gtp_wgrad.hip): per-chunk
// partial sums of per-degree dot products of a (in_type) and u over the
// products of each weight row (rows = C with per_channel, else 1), optionally
// writing out = w[row, l] u, then (dw != null) the chunks summed into
// dw[row, l].  partial: wgrad_nchunk(B, C, per_channel) * rows * (L + 1) floats.
int64_t wgrad_chunk(int64_t B, int64_t C, int per_channel);
int64_t wgrad_nchunk(int64_t B, int64_t C, int per_channel);
hipError_t launch_wgrad(const void* a, int a_type, const float* u, float* out, const float* w, int64_t B, int64_t C,
                        int L, int per_channel, float* partial, float* dw, hipStream_t s);

// Fused channel mixing for equal degrees 1..8 and Co <= 128 (*supported =
// false otherwise): pair products and the mix in one kernel, one workgroup
// per batch entry.  WB: the weights in the blocked layout made by
// launch_mix_wt_blocks with mix_fused_nct(Co) 16-channel column tiles.
int mix_fused_nct(int Co);
hipError_t launch_mix_wt_blocks(const float* W, float* WB, int Co, int64_t P, int nct, hipStream_t s);
hipError_t launch_mix_fused(const DevTables& t, const void* x1, const void* x2, int it, const float* WB, float* y,
                            int64_t B, int64_t C1, int64_t C2, int Co, hipStream_t s, bool* supported);
// y[p, :(Lout+1)^2] = x[p, :(L+1)^2] truncated or zero-padded.
// Lout = 0 products: y = <x1, x2> / sqrt(4 pi) over the common coefficients.
hipError_t launch_dot0(const void* x1, int it1, int k1, const void* x2, int it2, int k2, int64_t n, float* y,
                       hipStream_t s, bool* supported);
hipError_t launch_pad_copy(const void* x, int in_type, int L, int64_t n, float* y, int Lout, hipStream_t s);
// Direct 2D convolution of the real-form Fourier grids (the paper's eq.
// 2D-conv without the convolution theorem), workgroup per product.
hipError_t launch_full_direct(const DevTables& t, const void* x1, int it1, const void* x2, int it2, int64_t n,
                              float* y, hipStream_t s);
// Unfused stages with the paper's complex grids.
hipError_t launch_sh2fourier(const DevTables& t, int L, const void* x, int in_type, int64_t n, float* grid,
                             hipStream_t s);
hipError_t launch_fourier_conv(int L1, int L2, const float* g1, const float* g2, int64_t n, float* g3,
                               hipStream_t s);
hipError_t launch_fourier2sh(const DevTables& t, const float* g3, int64_t n, float* y, hipStream_t s);
// SH filter out[b,c,lm] = h[b,c,l] Y_lm(r_b).
hipError_t launch_sh_filter(int L, const float* r, const float* h, int64_t B, int64_t C, float* out,
                            hipStream_t s);

}  // namespace gtp
