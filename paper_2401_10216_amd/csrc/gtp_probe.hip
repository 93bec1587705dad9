// Streaming probes of the HBM roof and compute probes of the fp32 VALU and
// matrix-core rates (measurement aids, not part of the product).  Streaming: a read-only sweep, a write-only sweep, a copy and a two-stream
// read with one written stream (the read/write mix of the pair products),
// moving 16 bytes per lane per access (global_load_dwordx4; non-temporal
// global_store_dwordx4, which does not keep the written lines in the caches).
// Each workgroup streams one contiguous chunk, and the chunks are dealt to
// the 8 XCDs in contiguous runs (the dispatcher hands workgroups to the XCDs
// round robin); against grid-stride sweeps this reaches 6.2 against 5.3 TB/s
// for reads and 5.6 against 4.4 TB/s for the copy.  They give the bandwidth
// the chip reaches for each access pattern, against which the HBM-bound
// kernels are read.
#include "gtp_device.hpp"
#include "gtp_probe.hpp"

namespace gtp {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
constexpr int kProbeBlock = 256;
constexpr int kProbeGroups = 16384;  // 64 workgroups of 256 lanes per CU
constexpr int kProbeUnroll = 16;     // independent 16-byte loads in flight per lane

// The chunk of workgroup b of nwg (a multiple of 8): XCD x = b % 8 takes the
// chunks x nwg / 8 .. (x + 1) nwg / 8 - 1.
__device__ __forceinline__ int64_t probe_chunk(int64_t b, int64_t nwg) { return (b % 8) * (nwg / 8) + b / 8; }

// MODE 0: read src (the sum written to sink only if it is NaN, which finite
// data never gives, so the loads cannot be dropped); 1: write dst; 2: copy
// src to dst; 3: dst = src + src2 (two read streams, one written).
template <int MODE>
__global__ __launch_bounds__(kProbeBlock) void k_probe(const v4f* __restrict__ src, const v4f* __restrict__ src2,
                                                       v4f* __restrict__ dst, int64_t n4, int64_t chunk,
                                                       float* __restrict__ sink) {
  const int64_t c0 = probe_chunk(blockIdx.x, gridDim.x) * chunk;
  const int64_t c1 = c0 + chunk < n4 ? c0 + chunk : n4;
  if constexpr (MODE == 1) {
    const v4f v = {1.0f, 2.0f, 3.0f, 4.0f};
    for (int64_t i = c0 + threadIdx.x; i < c1; i += kProbeBlock) __builtin_nontemporal_store(v, dst + i);
  } else {
    float acc = 0.0f;
    for (int64_t i = c0 + threadIdx.x; i < c1; i += kProbeUnroll * kProbeBlock) {
      v4f v[kProbeUnroll];
#pragma unroll
      for (int u = 0; u < kProbeUnroll; ++u) {
        const int64_t j = i + u * kProbeBlock;
        if (j < c1) {
          v[u] = src[j];
          if constexpr (MODE == 3) v[u] += src2[j];
        }
      }
#pragma unroll
      for (int u = 0; u < kProbeUnroll; ++u) {
        const int64_t j = i + u * kProbeBlock;
        if (j < c1) {
          if constexpr (MODE == 0) acc += (v[u][0] + v[u][1]) + (v[u][2] + v[u][3]);
          else __builtin_nontemporal_store(v[u], dst + j);
        }
      }
    }
    if constexpr (MODE == 0) {
      if (acc != acc) sink[0] = acc;
    }
  }
}

// the copy under its own name: the calibration of the traffic counters
__global__ __launch_bounds__(kProbeBlock) void k_probe_copy(const v4f* __restrict__ src, v4f* __restrict__ dst,
                                                            int64_t n4, int64_t chunk) {
  const int64_t c0 = probe_chunk(blockIdx.x, gridDim.x) * chunk;
  const int64_t c1 = c0 + chunk < n4 ? c0 + chunk : n4;
  for (int64_t i = c0 + threadIdx.x; i < c1; i += kProbeUnroll * kProbeBlock) {
    v4f v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) {
      const int64_t j = i + u * kProbeBlock;
      if (j < c1) v[u] = src[j];
    }
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) {
      const int64_t j = i + u * kProbeBlock;
      if (j < c1) __builtin_nontemporal_store(v[u], dst + j);
    }
  }
}

// Compute probes: the fp32 rates the chip delivers under load (the shader
// clock under full load sits below the 2.4 GHz of the published peak).
// VALU: every lane runs kFmaChains independent chains a = a b + c (plain
// fp32 FMA, all operands in vector registers: an operand in a scalar
// register halves the issue rate); MFMA: every wave runs kMfmaChains
// independent accumulations of v_mfma_f32_16x16x4f32.  The results are
// written to sink only if they are NaN (never, for the values used), so the
// chains cannot be dropped.
constexpr int kFmaChains = 8;
constexpr int kMfmaChains = 4;
typedef float f4p __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kProbeBlock) void k_probe_fma(float* __restrict__ sink, int64_t iters) {
  float b = 0.999f, c = 0.001f;
  asm volatile("" : "+v"(b), "+v"(c));  // vector operands
  float a[kFmaChains];
#pragma unroll
  for (int k = 0; k < kFmaChains; ++k) a[k] = 1e-3f * float(threadIdx.x) + float(k);
#pragma unroll 8
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < kFmaChains; ++k) a[k] = fmaf(a[k], b, c);
  }
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < kFmaChains; ++k) s += a[k];
  if (s != s) sink[0] = s;
}

__global__ __launch_bounds__(kProbeBlock) void k_probe_mfma(float* __restrict__ sink, int64_t iters) {
  float a = 1e-3f * float(threadIdx.x & 63), b = 0.5f;
  asm volatile("" : "+v"(a), "+v"(b));
  f4p acc[kMfmaChains];
#pragma unroll
  for (int k = 0; k < kMfmaChains; ++k) acc[k] = f4p{0.0f, 0.0f, 0.0f, 0.0f};
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < kMfmaChains; ++k) acc[k] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[k], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < kMfmaChains; ++k) s += (acc[k][0] + acc[k][1]) + (acc[k][2] + acc[k][3]);
  if (s != s) sink[0] = s;
}

}  // namespace

// 2048 workgroups of 256 lanes: 8 waves per SIMD.  Returns the flops issued.
hipError_t launch_compute_probe(int mode, int64_t iters, float* sink, double* flops, hipStream_t s) {
  constexpr unsigned kGroups = 2048;
  const double waves = double(kGroups) * (kProbeBlock / 64);
  if (mode == 0) {
    *flops = waves * 64.0 * double(iters) * kFmaChains * 2.0;
    hipLaunchKernelGGL(k_probe_fma, dim3(kGroups), dim3(kProbeBlock), 0, s, sink, iters);
  } else {
    *flops = waves * double(iters) * kMfmaChains * (16.0 * 16.0 * 4.0 * 2.0);
    hipLaunchKernelGGL(k_probe_mfma, dim3(kGroups), dim3(kProbeBlock), 0, s, sink, iters);
  }
  return hipGetLastError();
}

hipError_t launch_stream_probe(int mode, const void* src, void* dst, int64_t nbytes, hipStream_t s) {
  // mode 3 reads two streams of nbytes / 2 (the halves of src) and writes one
  const int64_t n4 = mode == 3 ? nbytes / 32 : nbytes / 16;
  if (n4 <= 0) return hipSuccess;
  // workgroups: a multiple of 8, each a chunk of at least one pass of the block
  int64_t g = (n4 + kProbeBlock - 1) / kProbeBlock;
  if (g > kProbeGroups) g = kProbeGroups;
  g = (g + 7) / 8 * 8;
  const int64_t chunk = (n4 + g - 1) / g;
  const v4f* a = static_cast<const v4f*>(src);
  v4f* d = static_cast<v4f*>(dst);
  switch (mode) {
    case 0:
      hipLaunchKernelGGL(k_probe<0>, dim3(unsigned(g)), dim3(kProbeBlock), 0, s, a, a, d, n4, chunk,
                         static_cast<float*>(dst));
      break;
    case 1:
      hipLaunchKernelGGL(k_probe<1>, dim3(unsigned(g)), dim3(kProbeBlock), 0, s, a, a, d, n4, chunk, nullptr);
      break;
    case 2:
      hipLaunchKernelGGL(k_probe_copy, dim3(unsigned(g)), dim3(kProbeBlock), 0, s, a, d, n4, chunk);
      break;
    default:
      hipLaunchKernelGGL(k_probe<3>, dim3(unsigned(g)), dim3(kProbeBlock), 0, s, a, a + n4, d, n4, chunk, nullptr);
      break;
  }
  return hipGetLastError();
}

}  // namespace gtp
