// Streaming probes of the HBM roof (measurement aids, not part of the
// product): a read-only sweep, a write-only sweep, a copy and a two-stream
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

}  // namespace

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
