// Launchers of the measurement probes (HBM streaming and fp32 compute rates;
// not part of the product path).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gtp {

// HBM streaming probes: mode 0 reads nbytes of src (dst receives at most one
// float), 1 writes nbytes to dst, 2 copies src to dst, 3 writes the sum of
// src's halves to dst; 16-byte accesses.
hipError_t launch_stream_probe(int mode, const void* src, void* dst, int64_t nbytes, hipStream_t s);
// Compute probes: mode 0 fp32 VALU FMA chains, 1 fp32 16x16x4 MFMA chains,
// iters steps each; *flops receives the flops issued (sink: one device float,
// written only on NaN).
hipError_t launch_compute_probe(int mode, int64_t iters, float* sink, double* flops, hipStream_t s);

}  // namespace gtp
