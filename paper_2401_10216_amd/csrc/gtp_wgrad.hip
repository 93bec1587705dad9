// Gradients of the per-degree weights of the weighted Gaunt tensor product
// (Sec. 3.1, eq. tp-eq-mul-weight, weights w_{l1} w_{l2} w_l): each is a sum,
// over the products that share a weight row, of per-degree dot products
//   dw[r, l] = sum_{p in row r} sum_{m} a[p, (l, m)] u[p, (l, m)]
// (a the unweighted input and u the gradient with respect to the weighted
// input; or a = dy and u the unweighted-output product for the output
// weights).  Two deterministic passes: per-chunk partial sums, then the sum
// of the chunks in a fixed order.  The first pass can also write
// out = w[r, l] u (the input gradient) while it reads u.
#include "gtp_device.hpp"

namespace gtp {
namespace {

constexpr int kWgBlock = 256;
constexpr int kWgMaxSlices = 17;  // ceil((64 + 1)^2 / 256)

__device__ __forceinline__ float wg_ld(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float wg_ld(const uint16_t* p, int64_t i) { return __uint_as_float(uint32_t(p[i]) << 16); }

// Workgroup (chunk, r): the products of chunk `chunk` in row r -- with
// per_channel, p = b C + r for b in the chunk's range of batch entries;
// otherwise the chunk's contiguous range of products (r = 0).  Thread roles:
// for K <= 256, S = 256 / K sub-streams of products, thread (s, i) owns
// coefficient i of every S-th product; for K > 256, every thread owns the
// coefficients i = tid + 256 j of every product.
template <typename TA>
__global__ __launch_bounds__(kWgBlock) void k_wgrad_partial(const TA* __restrict__ a, const float* __restrict__ u,
                                                            float* __restrict__ out, const float* __restrict__ w,
                                                            int64_t B, int64_t C, int L, int per_channel,
                                                            int64_t chunk, float* __restrict__ partial) {
  extern __shared__ float red[];
  const int K = (L + 1) * (L + 1);
  const int tid = threadIdx.x;
  const int64_t ck = blockIdx.x;
  const int64_t r = blockIdx.y;
  const int64_t nprod = per_channel ? B : B * C;  // products in the row's sequence
  const int64_t q0 = ck * chunk, q1 = (q0 + chunk < nprod) ? q0 + chunk : nprod;
  const int S = K <= kWgBlock ? kWgBlock / K : 1;
  lds_poison(red, S * K);
  const int s = K <= kWgBlock ? tid / K : 0;
  const int i0 = K <= kWgBlock ? tid % K : tid;
  const bool active = s < S;
  float acc[kWgMaxSlices];
  int deg[kWgMaxSlices];
#pragma unroll
  for (int j = 0; j < kWgMaxSlices; ++j) {
    acc[j] = 0.0f;
    const int i = i0 + kWgBlock * j;
    deg[j] = i < K ? degree_of(i) : 0;
  }
  if (active) {
    for (int64_t q = q0 + s; q < q1; q += S) {
      const int64_t p = per_channel ? q * C + r : q;
      const int64_t base = p * K;
      const float* wr = w ? w + (per_channel ? r : 0) * (L + 1) : nullptr;
#pragma unroll
      for (int j = 0; j < kWgMaxSlices; ++j) {
        const int i = i0 + kWgBlock * j;
        if (i < K && (K > kWgBlock || j == 0)) {
          const float uv = u[base + i];
          acc[j] = fmaf(wg_ld(a, base + i), uv, acc[j]);
          if (out) out[base + i] = wr ? wr[deg[j]] * uv : uv;
        }
      }
    }
  }
  // per-coefficient partials into LDS, then one thread per degree sums its
  // coefficients (and the sub-streams) in a fixed order
  if (K <= kWgBlock) {
    if (active) red[s * K + i0] = acc[0];
  } else {
#pragma unroll
    for (int j = 0; j < kWgMaxSlices; ++j)
      if (i0 + kWgBlock * j < K) red[i0 + kWgBlock * j] = acc[j];
  }
  __syncthreads();
  if (tid <= L) {
    const int l = tid;
    float v = 0.0f;
    for (int ss = 0; ss < S; ++ss)
      for (int i = l * l; i < (l + 1) * (l + 1); ++i) v += red[ss * K + i];
    partial[(ck * gridDim.y + r) * (L + 1) + l] = v;
  }
}

// dw[r, l] = sum over the chunks of partial[chunk, r, l], chunks in order.
__global__ __launch_bounds__(kWgBlock) void k_wgrad_final(const float* __restrict__ partial, int64_t nchunk,
                                                          int64_t R, int L, float* __restrict__ dw) {
  const int64_t e = int64_t(blockIdx.x) * kWgBlock + threadIdx.x;
  if (e >= R * (L + 1)) return;
  float v = 0.0f;
  for (int64_t c = 0; c < nchunk; ++c) v += partial[c * R * (L + 1) + e];
  dw[e] = v;
}

}  // namespace

int64_t wgrad_chunk(int64_t B, int64_t C, int per_channel) {
  const int64_t nprod = per_channel ? B : B * C;
  // about 8192 workgroups over the rows, at least 64 products each
  const int64_t R = per_channel ? C : 1;
  int64_t want = (8192 + R - 1) / R;
  if (want < 1) want = 1;
  int64_t chunk = (nprod + want - 1) / want;
  if (chunk < 64) chunk = 64;
  return chunk;
}

int64_t wgrad_nchunk(int64_t B, int64_t C, int per_channel) {
  const int64_t nprod = per_channel ? B : B * C;
  const int64_t chunk = wgrad_chunk(B, C, per_channel);
  return (nprod + chunk - 1) / chunk;
}

hipError_t launch_wgrad(const void* a, int a_type, const float* u, float* out, const float* w, int64_t B, int64_t C,
                        int L, int per_channel, float* partial, float* dw, hipStream_t s) {
  const int64_t R = per_channel ? C : 1;
  const int64_t chunk = wgrad_chunk(B, C, per_channel);
  const int64_t nchunk = wgrad_nchunk(B, C, per_channel);
  if (nchunk <= 0 || R <= 0) return hipSuccess;
  if (nchunk > 0x7fffffff || R > 65535) return hipErrorInvalidValue;
  const int K = (L + 1) * (L + 1);
  const int S = K <= kWgBlock ? kWgBlock / K : 1;
  const size_t lds = size_t(S) * K * sizeof(float);
  const dim3 grid{unsigned(nchunk), unsigned(R), 1u}, block{unsigned(kWgBlock), 1u, 1u};
  if (a_type == IN_BF16)
    hipLaunchKernelGGL(k_wgrad_partial<uint16_t>, grid, block, lds, s, static_cast<const uint16_t*>(a), u, out, w, B,
                       C, L, per_channel, chunk, partial);
  else
    hipLaunchKernelGGL(k_wgrad_partial<float>, grid, block, lds, s, static_cast<const float*>(a), u, out, w, B, C, L,
                       per_channel, chunk, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (!dw) return hipSuccess;
  const int64_t tot = R * (L + 1);
  hipLaunchKernelGGL(k_wgrad_final, dim3(unsigned((tot + kWgBlock - 1) / kWgBlock)), dim3(kWgBlock), 0, s, partial,
                     nchunk, R, L, dw);
  return hipGetLastError();
}

}  // namespace gtp
