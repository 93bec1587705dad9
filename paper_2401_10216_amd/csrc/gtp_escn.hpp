// Rotated-frame equivariant convolution (Sec. 3.3 "Equivariant Convolutions";
// Appendix, eq. sh2fs-escn): the Gaunt product of x with the SH filter
// h_l Y_l(r / |r|) of an edge, computed in the frame where the edge points
// at the pole.  There the filter has only m = 0 coefficients, its 2D Fourier
// grid only v = 0, and the product is a theta-only operation per m.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "gtp_escn_tables.hpp"

namespace gtp {

// fp32 device copies.
struct EscnDev {
  const float* J;
  const float* E;
  int LM, NPAIR, ERL;
  const float* A;  // operand images of the matrix-core kernel (LM = kEscnWaveL)
  const float* Z;
  const float* JI;
};

// Floats of one edge's rotation matrices in the workspace (0 when no
// rotated-frame kernel exists for degree L, or when its kernel needs none).
int64_t escn_rot_floats(int L);

// Launches the rotated-frame kernels for L1 = L2 = Lout = L in 1..8 (one
// product per lane) and L = 16 (matrix cores; launch_conv_escn_wave)
// (*supported = false otherwise).  x: [B, C, (L+1)^2] (in_type), r: [B, 3],
// h: [B, C, L+1], y: [B, C, (L+1)^2]; dws: device workspace of
// B * escn_rot_floats(L) floats (the per-edge rotation matrices).
hipError_t launch_conv_escn(const EscnDev& e, int L1, int L2, int Lout, const void* x, int in_type, const float* r,
                            const float* h, int64_t B, int64_t C, float* y, float* dws, hipStream_t s,
                            bool* supported);

// The matrix-core kernel of degree kEscnWaveL = 16 (tables of a 16-plan):
// rows of k1 = (L1+1)^2 input coefficients, h rows of kh = L2 + 1 weights and
// output rows of ko = (Lout+1)^2 floats, each at most that of degree 16 (rows
// read zero-padded to degree 16, outputs truncated).  It applies each edge's
// rotation factor by factor from its angles and needs no workspace.
hipError_t launch_conv_escn_wave(const EscnDev& e, const void* x, int in_type, const float* r, const float* h,
                                 int64_t B, int64_t C, float* y, int k1, int kh, int ko, hipStream_t s);

}  // namespace gtp
