// Streaming probes of the HBM roof (measurement aids, not part of the
// product): a read-only sweep, a write-only sweep and a copy, each moving
// 16 bytes per lane per access with the loads and stores the product kernels
// use (global_load_dwordx4; non-temporal global_store_dwordx4, which does not
// keep the written lines in the caches).  They give the bandwidth the chip
// reaches for each access pattern, against which the HBM-bound kernels are
// read.
#include "gtp_device.hpp"

namespace gtp {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
constexpr int kProbeBlock = 256;
constexpr int kProbeUnroll = 4;  // independent 16-byte accesses in flight per lane

// Sum of the buffer's values; written only if it is NaN (never for the
// finite data the probe reads), so the loads cannot be dropped.
__global__ __launch_bounds__(kProbeBlock) void k_probe_read(const v4f* __restrict__ src, int64_t n4,
                                                            float* __restrict__ sink) {
  const int64_t stride = int64_t(gridDim.x) * kProbeBlock;
  float acc = 0.0f;
  int64_t i = int64_t(blockIdx.x) * kProbeBlock + threadIdx.x;
  for (; i + (kProbeUnroll - 1) * stride < n4; i += kProbeUnroll * stride) {
    v4f v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) acc += (v[u][0] + v[u][1]) + (v[u][2] + v[u][3]);
  }
  for (; i < n4; i += stride) {
    const v4f v = src[i];
    acc += (v[0] + v[1]) + (v[2] + v[3]);
  }
  if (acc != acc) sink[0] = acc;
}

__global__ __launch_bounds__(kProbeBlock) void k_probe_write(v4f* __restrict__ dst, int64_t n4) {
  const int64_t stride = int64_t(gridDim.x) * kProbeBlock;
  const v4f v = {1.0f, 2.0f, 3.0f, 4.0f};
  for (int64_t i = int64_t(blockIdx.x) * kProbeBlock + threadIdx.x; i < n4; i += stride)
    __builtin_nontemporal_store(v, dst + i);
}

__global__ __launch_bounds__(kProbeBlock) void k_probe_copy(const v4f* __restrict__ src, v4f* __restrict__ dst,
                                                            int64_t n4) {
  const int64_t stride = int64_t(gridDim.x) * kProbeBlock;
  int64_t i = int64_t(blockIdx.x) * kProbeBlock + threadIdx.x;
  for (; i + (kProbeUnroll - 1) * stride < n4; i += kProbeUnroll * stride) {
    v4f v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) __builtin_nontemporal_store(v[u], dst + i + u * stride);
  }
  for (; i < n4; i += stride) __builtin_nontemporal_store(src[i], dst + i);
}

}  // namespace

hipError_t launch_stream_probe(int mode, const void* src, void* dst, int64_t nbytes, hipStream_t s) {
  const int64_t n4 = nbytes / 16;
  if (n4 <= 0) return hipSuccess;
  // 16 workgroups of 256 lanes per CU (256 CUs), or fewer for small buffers
  int64_t g = (n4 + kProbeBlock - 1) / kProbeBlock;
  if (g > 4096) g = 4096;
  if (mode == 0)
    hipLaunchKernelGGL(k_probe_read, dim3(unsigned(g)), dim3(kProbeBlock), 0, s, static_cast<const v4f*>(src), n4,
                       static_cast<float*>(dst));
  else if (mode == 1)
    hipLaunchKernelGGL(k_probe_write, dim3(unsigned(g)), dim3(kProbeBlock), 0, s, static_cast<v4f*>(dst), n4);
  else
    hipLaunchKernelGGL(k_probe_copy, dim3(unsigned(g)), dim3(kProbeBlock), 0, s, static_cast<const v4f*>(src),
                       static_cast<v4f*>(dst), n4);
  return hipGetLastError();
}

}  // namespace gtp
