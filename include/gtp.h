/*
 * gtp.h -- C ABI of the MI355X (gfx950) Gaunt Tensor Product library.
 *
 * The Gaunt Tensor Product (Luo, Chen, He, "Enabling efficient equivariant
 * operations in the Fourier basis via Gaunt Tensor Products", ICLR 2024) of
 * two real spherical-harmonic (SH) coefficient vectors x1 (degrees <= L1) and
 * x2 (degrees <= L2) is the SH expansion, truncated to degree Lout, of the
 * product of the two spherical functions they define (Sec. 3.1, eq.
 * tp-eq-mul):
 *
 *   y_l^m = sum G^{(l,m)}_{(l1,m1)(l2,m2)} x1_{l1}^{m1} x2_{l2}^{m2},
 *   G     = int_{S^2} Y_{l1}^{m1} Y_{l2}^{m2} Y_l^m dOmega   (real Gaunt coefficients).
 *
 * The library computes it the paper's way (Sec. 3.2): change of basis SH ->
 * 2D Fourier, product of the two functions as a 2D convolution of their Fourier
 * grids, projection back to SH.
 *
 * Conventions shared by every entry point
 *   - Real SH, z polar axis, no Condon-Shortley phase:
 *       Y_l^0 = Q_l^0(cos t), Y_l^{+m} = sqrt2 Q_l^m(cos t) cos(m p),
 *       Y_l^{-m} = sqrt2 Q_l^m(cos t) sin(m p),  Q_l^m = N_lm P_l^m,
 *     so Y_1 = sqrt(3/(4 pi)) (y, z, x).
 *   - Coefficient vectors are contiguous, index i = l*l + l + m, (L+1)^2 long.
 *     Batched tensors are row-major [B, C, (L+1)^2] (channel-wise products:
 *     product (b,c) uses channel c of both inputs, Appendix "Implementation
 *     Details", channel-wise combination).
 *   - Every data pointer is a DEVICE pointer on the current HIP device, owned
 *     by the caller; the library only reads inputs and writes outputs, never
 *     allocates or frees caller memory.  Pointers must be 4-byte aligned
 *     (2-byte for bf16 inputs).
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls are
 *     asynchronous on that stream; a launch failure returns GTP_ERR_HIP.
 *   - Every argument is validated on the host BEFORE any HIP call; invalid
 *     arguments return GTP_ERR_INVALID_ARG and touch nothing.
 *   - Functions never throw.  gtp_last_error() gives a thread-local message.
 *   - Floating point: tables are built in fp64 on the host and rounded once to
 *     fp32; arithmetic and outputs are fp32; bf16 applies to inputs only.
 *   - Limits: 0 <= L1, L2, Lout <= 64.  Output degrees above L1 + L2 are
 *     written as zeros.
 */
#ifndef GTP_H
#define GTP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GTP_OK = 0,
  GTP_ERR_INVALID_ARG = 1, /* bad sizes, null pointers, overlap, bad enum */
  GTP_ERR_UNSUPPORTED = 2, /* valid request the library does not implement  */
  GTP_ERR_NO_DEVICE = 3,   /* no HIP device visible                          */
  GTP_ERR_HIP = 4,         /* a HIP runtime call or kernel launch failed      */
  GTP_ERR_ALLOC = 5        /* host or device allocation failed                */
} gtp_status;

typedef enum { GTP_F32 = 0, GTP_BF16 = 1 } gtp_dtype;

/* Plan flags (bitwise or).  The two low bits pick step 2 (eq. 2D-conv). */
#define GTP_CONV_AUTO 0u      /* the algorithm the measured crossover picks for the degrees */
#define GTP_CONV_DIRECT 1u    /* direct 2D convolution of the Fourier grids */
#define GTP_CONV_FFT 2u       /* convolution theorem, phi transforms by radix-2 FFTs where the library has such a
                                 kernel (L1 = L2 = Lout in {16, 32}), by the direct DFTs below otherwise */
#define GTP_CONV_DFT 3u       /* convolution theorem, phi transforms as direct DFTs over the 4-fold symmetric
                                 sample grid (unrolled at small degree, matrix-core contractions from 16 on) */
#define GTP_PLAN_HOST_ONLY 16u /* build the fp64 tables only; no HIP call (host-side checks) */

/* Many-body modes for gtp_selfproduct. */
#define GTP_SELF_STEPWISE 0u /* B_1 = A, B_{k+1} = P_Lout(B_k * A): truncate after every product */
#define GTP_SELF_FUSED 1u    /* P_Lout(A^nu): one multi-convolution, projected once */

/* Opaque plan: the SH <-> Fourier change-of-basis tables for one
 * (L1, L2, Lout), built in fp64 and uploaded once to the device that is
 * current at creation.  Use a plan only while that device is current. */
typedef struct gtp_plan_ *gtp_plan;

/* Create a plan (Sec. 3.2: the coefficients y^{l,m,*}_{u,v} of eq. sh-fs and
 * z^{l,m,*}_{u,v} of eq. fs-sh, plus the grids of the convolution).
 * out: receives the plan.  Returns GTP_ERR_NO_DEVICE without a device unless
 * GTP_PLAN_HOST_ONLY is set.  The plan owns its host and device tables.  A
 * triple whose product or rotated-frame convolution runs on an equal-degree
 * kernel of higher degree (16, 32 or 64; rows zero-padded) also gets that
 * degree's plan here, kept by the library until the process ends, so that
 * no later call needs to allocate. */
gtp_status gtp_plan_create(gtp_plan *out, int L1, int L2, int Lout, unsigned flags);

/* Destroy a plan and free its tables (NULL is a no-op).  Not stream-ordered:
 * the caller must make sure no launch using the plan is still pending. */
gtp_status gtp_plan_destroy(gtp_plan p);

/* Fused Gaunt tensor product (Sec. 3.1 eq. tp-eq-mul computed by Sec. 3.2):
 *   y[b,c,:] = GTP(x1[b,c,:], x2[b,c,:]) truncated to degree Lout.
 * x1: [B, C, (L1+1)^2], x2: [B, C, (L2+1)^2] of type in_dtype;
 * y: [B, C, (Lout+1)^2] fp32.  B*C == 0 is a successful no-op.  y must not
 * overlap x1 or x2.  The Fourier grids never leave the chip.  The plan's
 * GTP_CONV_* flag picks step 2 (eq. 2D-conv): the convolution theorem with
 * radix-2 FFTs (GTP_CONV_FFT) or direct DFTs (GTP_CONV_DFT) for the phi
 * transforms, or the direct real-form convolution (GTP_CONV_DIRECT;
 * GTP_ERR_UNSUPPORTED when its per-product working set exceeds 64 KB of LDS,
 * about L1 = L2 = 40); GTP_CONV_AUTO takes the measured fastest. */
gtp_status gtp_full(gtp_plan p, const void *x1, const void *x2, gtp_dtype in_dtype,
                    int64_t B, int64_t C, float *y, void *stream);

/* Channel mixing (Appendix, combination rules of features in different
 * channels, channel-mixing case):
 *   y[b, co] = sum_{c1 < C1, c2 < C2} W[co, c1, c2] GTP(x1[b, c1], x2[b, c2]),
 * O(C1 C2) full products per batch entry.  The pair products are taken by the
 * fused product kernels (outer-product indexing) into a stream-ordered
 * workspace (hipMallocAsync, at most 256 MiB, chunked over b) and combined as
 * y_b = W T_b (Co x C1C2 times C1C2 x (Lout+1)^2) on the fp32 matrix cores.
 * x1: [B, C1, (L1+1)^2], x2: [B, C2, (L2+1)^2] (in_dtype); W: [Co, C1, C2]
 * fp32; y: [B, Co, (Lout+1)^2] fp32, not overlapping the inputs or W.
 * C1 C2 == 0 writes zeros (x1, x2 and W may then be NULL); B Co == 0 is a
 * no-op.  The thread-per-product
 * kernel serves L1 = L2 = Lout <= 8; other degrees take the workgroup kernel. */
gtp_status gtp_channel_mix(gtp_plan p, const void *x1, const void *x2, gtp_dtype in_dtype, const float *W,
                           int64_t B, int64_t C1, int64_t C2, int64_t Co, float *y, void *stream);

/* Equivariant convolution with the SH filter of an edge (Sec. 3.3
 * "Equivariant Convolutions"; Appendix, eq. sh2fs-escn):
 *   y[b,c] = GTP(x[b,c], F[b,c]),  F[b,c,(l,m)] = h[b,c,l] Y_l^m(r_b / |r_b|),
 * the result of gtp_full(x, gtp_sh_filter(r, h)), computed in the frame in
 * which the edge points at the pole: x is rotated by the real-SH matrix D_b of
 * a rotation taking r_b / |r_b| to (0, 0, 1); there the filter has only the
 * m = 0 coefficients h_l Y_l^0(pole) (2D Fourier coefficients only at v = 0),
 * the product with it needs theta transforms only, and the result is rotated
 * back by D_b^T.  (The z pole is this library's polar axis; the paper uses
 * (0, 1, 0) in its y-up convention.)
 * x: [B, C, (L1+1)^2] (in_dtype); r: [B, 3] fp32 edge vectors (need not be
 * unit; a zero vector is taken as (0, 0, 1)); h: [B, C, L2+1] fp32 radial
 * weights; y: [B, C, (Lout+1)^2] fp32, not overlapping the inputs.  The
 * rotated-frame kernels cover L1 = L2 = Lout in 1..8 (one product per lane;
 * the per-edge rotation matrices go to a stream-ordered workspace,
 * hipMallocAsync) and 16 (the matrix cores, 16 channels per wave, the
 * rotation applied from the edge angles: no workspace), which also serves
 * every other triple whose highest degree is 9..16 (rows read zero-padded
 * to degree 16, outputs truncated: exact); both take one workgroup per edge
 * and 64 channels, so C >= 64 fills it.  Other degrees, and plans built with
 * GTP_CONV_DIRECT, build the filter in a stream-ordered workspace and take
 * gtp_full. */
gtp_status gtp_conv_escn(gtp_plan p, const void *x, gtp_dtype in_dtype, const float *r, const float *h, int64_t B,
                         int64_t C, float *y, void *stream);

/* gtp_conv_escn without any device allocation, for callers that cannot
 * allocate: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, result and errors as gtp_conv_escn; no
 * hipMalloc / hipMallocAsync / hipFree / allocating library call is made.
 * The per-edge rotation matrices of L = 1..8 (or, for degrees without a
 * rotated-frame kernel, the filter rows; L = 16 needs none) go to a static
 * device scratch array of
 * GTP_NOALLOC_SCRATCH_BYTES (64 MiB) per device, which exists from the
 * library's load on that device until the process ends; the edges are
 * processed in chunks that fit it.  Returns GTP_ERR_UNSUPPORTED (before any
 * HIP call) when one edge alone needs more: C (L2+1)^2 4 bytes above 64 MiB
 * on the filter route.  Every call on a device shares that device's array
 * and leaves it holding the last chunk's values (each launch writes what it
 * reads, nothing has to start at zero): calls that may overlap on one device
 * (different streams, different host threads) race and must be serialised
 * by the caller.  The plan must have been created on the current device. */
#define GTP_NOALLOC_SCRATCH_BYTES (64ll << 20)
gtp_status gtp_conv_escn_noalloc(gtp_plan p, const void *x, gtp_dtype in_dtype, const float *r, const float *h,
                                 int64_t B, int64_t C, float *y, void *stream);

/* Weighted Gaunt tensor product (Sec. 3.1, eq. tp-eq-mul-weight; Appendix
 * "Feature Interaction" weights w^l_{l1,l2} reparameterized as
 * w_{l1} w_{l2} w_l):
 *   y[b,c,(l,m)] = wout[r,l] * sum_{l1,l2} w1[r,l1] w2[r,l2] (x1^(l1) (x) x2^(l2))^(l)_m,
 * computed as gtp_full of the degree-scaled inputs, scaled per output degree
 * (the weights are applied as the inputs are loaded and the output stored).
 * A degree mask (weights 0 / 1) gives the partial products x^(l1) (x) x^(l2).
 * r = c when per_channel = 1 (one weight row per channel), r = 0 when
 * per_channel = 0 (one row shared by every channel).
 * w1: [R, L1+1], w2: [R, L2+1], wout: [R, Lout+1] fp32 device arrays with
 * R = C or 1; any of them may be NULL (all ones).  Other arguments as in
 * gtp_full; y must not overlap the inputs or the weights.  Plans built with
 * GTP_CONV_DIRECT return GTP_ERR_UNSUPPORTED. */
gtp_status gtp_full_weighted(gtp_plan p, const void *x1, const void *x2, gtp_dtype in_dtype, const float *w1,
                             const float *w2, const float *wout, int per_channel, int64_t B, int64_t C, float *y,
                             void *stream);

/* Backward pass of gtp_full_weighted, weight gradients included (Sec. 3.1,
 * eq. tp-eq-mul-weight; the learnable weights of the feature-interaction
 * layers).  With y = wout GTP(w1 x1, w2 x2) and a loss gradient dy, writes
 *   dx1   = w1 P_L1 GTP(wout dy, w2 x2)                 [B, C, (L1+1)^2],
 *   dx2   = w2 P_L2 GTP(wout dy, w1 x1)                 [B, C, (L2+1)^2],
 *   dw1[r, l1] = sum over the products of weight row r of
 *                <x1, P_L1 GTP(wout dy, w2 x2)> on degree l1     [R, L1+1],
 *   dw2 likewise                                                 [R, L2+1],
 *   dwout[r, l] = sum over row r of <dy, GTP(w1 x1, w2 x2)> on degree l
 *                                                                [R, Lout+1],
 * R = C with per_channel = 1 (row c holds channel c's products), else 1.
 * Weights as in gtp_full_weighted (NULL = ones; the gradient is still that
 * of a weight of ones).  Any of dx1, dx2, dw1, dw2, dwout may be NULL (not
 * computed); the rest are written, not accumulated, and must not overlap an
 * input or each other.  The sums over the products are deterministic (fixed
 * order, no atomics).  Uses a stream-ordered workspace (hipMallocAsync) for
 * the partial sums and the products that are not outputs.  B*C == 0 writes
 * zero weight gradients.  GTP_ERR_UNSUPPORTED for GTP_CONV_DIRECT plans and
 * more than 65535 weight rows. */
gtp_status gtp_full_weighted_backward(gtp_plan p, const void *x1, const void *x2, gtp_dtype in_dtype,
                                      const float *w1, const float *w2, const float *wout, int per_channel,
                                      const float *dy, int64_t B, int64_t C, float *dx1, float *dx2, float *dw1,
                                      float *dw2, float *dwout, void *stream);

/* Backward pass (vector-Jacobian product) of gtp_full: given the gradient dy
 * of a scalar loss with respect to y = gtp_full(x1, x2), the gradients
 *   dx1[b,c,i] = sum_{j,k} G_{i j k} x2[b,c,j] dy[b,c,k]   (i over degrees <= L1),
 *   dx2[b,c,j] = sum_{i,k} G_{i j k} x1[b,c,i] dy[b,c,k]   (j over degrees <= L2),
 * with G the real Gaunt coefficients of Sec. 3.1 (eq. tp-eq-mul).  G is the
 * integral of a product of three real SH, symmetric in its three (l, m)
 * pairs, so dx1 is the Gaunt tensor product of dy and x2 truncated to degree
 * L1 (and dx2 that of dy and x1 truncated to L2); both are computed that way
 * (Sec. 3.2), with the plan's GTP_CONV_* choice.
 * x1, x2: the forward inputs (in_dtype); dy: [B, C, (Lout+1)^2] fp32;
 * dx1: [B, C, (L1+1)^2] fp32 or NULL (not computed); dx2: [B, C, (L2+1)^2]
 * fp32 or NULL.  x1 may be NULL when dx2 is, x2 when dx1 is.  The gradients
 * are written, not accumulated.  Neither may overlap an input or the other.
 * B*C == 0, or dx1 == dx2 == NULL, is a successful no-op.  Tables for
 * (Lout, L2, L1) and (Lout, L1, L2) are built on first use and cached per
 * device (that first call is synchronous); equal degrees reuse the plan's.
 * With L1 = L2 = Lout <= 7 and both gradients asked for, both come from one
 * launch that reads dy once (results equal bit for bit to asking for each
 * gradient alone). */
gtp_status gtp_full_backward(gtp_plan p, const void *x1, const void *x2, gtp_dtype in_dtype, const float *dy,
                             int64_t B, int64_t C, float *dx1, float *dx2, void *stream);

/* Step 1 (Sec. 3.2, eq. sh-fs): SH coefficients -> 2D Fourier coefficients
 * x*_{u,v}, |u|,|v| <= L, for L = L1 (which = 1) or L2 (which = 2).
 * The function is extended to theta in [-pi, pi) by F(-t, p) = F(t, p + pi).
 * x: [n, (L+1)^2] (in_dtype); grid: [n, 2L+1, 2L+1] complex64 interleaved
 * (re, im), element (u, v) at [(u+L)*(2L+1) + (v+L)]. */
gtp_status gtp_sh2fourier(gtp_plan p, int which, const void *x, gtp_dtype in_dtype, int64_t n,
                          float *grid, void *stream);

/* Step 2 (Sec. 3.2, eq. 2D-conv): f3_{u,v} = sum_{u1+u2=u, v1+v2=v} f1_{u1,v1} f2_{u2,v2}.
 * g1: [n, 2L1+1, 2L1+1], g2: [n, 2L2+1, 2L2+1], g3: [n, 2U+1, 2U+1] with
 * U = L1 + L2, all complex64 interleaved and centred as above.  Computed as a
 * direct convolution (the grids are the public, paper-layout grids). */
gtp_status gtp_fourier_conv(gtp_plan p, const float *g1, const float *g2, int64_t n, float *g3,
                            void *stream);

/* Step 3 (Sec. 3.2, eq. fs-sh): y_l^m = Re sum_{u,v} g3_{u,v} z^{l,m}_{u,v},
 * z^{l,m}_{u,v} = int_{S^2} exp(i(u t + v p)) Y_l^m dOmega (the projection of
 * the grid's function onto the SH basis), l <= Lout.
 * g3: [n, 2U+1, 2U+1] complex64; y: [n, (Lout+1)^2] fp32.  For grids of real
 * functions (anything made by gtp_sh2fourier and gtp_fourier_conv) the
 * discarded imaginary part is zero. */
gtp_status gtp_fourier2sh(gtp_plan p, const float *g3, int64_t n, float *y, void *stream);

/* Many-body self product (Sec. 3.3 "Equivariant Many-body Interactions";
 * Appendix "Implementation Details", generalized Gaunt coefficients and the
 * divide-and-conquer multi-convolution): the nu-fold product of A = x with
 * itself, nu >= 1.
 *   mode GTP_SELF_STEPWISE: B_1 = P_Lout(A), B_{k+1} = P_Lout(B_k * A).
 *   mode GTP_SELF_FUSED   : P_Lout(A^nu) with no intermediate truncation.
 * x: [B, C, (L+1)^2] (in_dtype); y: [B, C, (Lout+1)^2] fp32.  Plans for the
 * needed degrees are built and cached internally (per device).  The fused
 * mode needs nu * L <= 64 (GTP_ERR_UNSUPPORTED otherwise).  The stepwise
 * mode may take a stream-ordered device workspace (hipMallocAsync) when no
 * single-kernel path exists for (L, nu, Lout). */
gtp_status gtp_selfproduct(int L, int nu, int Lout, unsigned mode, const void *x,
                           gtp_dtype in_dtype, int64_t B, int64_t C, float *y, void *stream);

/* Spherical-harmonic filter of an equivariant convolution (Sec. 3.3
 * "Equivariant Convolutions"): out[b,c,(l,m)] = h[b,c,l] * Y_l^m(r_b / |r_b|).
 * r: [B, 3] fp32 edge vectors (need not be unit; zero vectors give the
 * direction (0,0,1)); h: [B, C, L+1] fp32 per-degree radial weights, or NULL
 * for h = 1 (then C must be 1); out: [B, C, (L+1)^2] fp32.  0 <= L <= 64. */
gtp_status gtp_sh_filter(int L, const float *r, const float *h, int64_t B, int64_t C, float *out,
                         void *stream);

/* HBM streaming probe (measurement aid: the roof the HBM-bound kernels are
 * read against; each workgroup streams one contiguous chunk, the chunks
 * dealt to the XCDs in contiguous runs).  mode 0: read nbytes of src (dst: a
 * device float written only if the data holds a NaN); 1: write nbytes to dst
 * (non-temporal stores); 2: copy nbytes from src to dst (non-overlapping);
 * 3: dst = first half of src + second half (two read streams of nbytes / 2,
 * one written stream of nbytes / 2: the read/write mix of the pair
 * products; dst must not overlap src).  Device pointers 16-byte aligned,
 * nbytes >= 0 a multiple of 16 (32 for mode 3). */
gtp_status gtp_stream_probe(int mode, const void *src, void *dst, int64_t nbytes, void *stream);

/* Compute probe (measurement aid: the fp32 rates the chip delivers under
 * load, beside the published peak).  mode 0: fp32 VALU FMA chains (8
 * independent chains per lane); 1: fp32 v_mfma_f32_16x16x4f32 chains (4
 * independent accumulators per wave); 2048 workgroups of 256 lanes, iters
 * steps (1..2^30).  sink: one device float (4-byte aligned), written only if
 * a result is NaN; *flops (host) receives the flops the launch issues, for
 * the caller to divide by its own timing of the launch on stream. */
gtp_status gtp_compute_probe(int mode, int64_t iters, float *sink, double *flops, void *stream);

/* Number of floats of one per-product public grid: which = 1 or 2 gives the
 * input grids (2 * (2L+1)^2), which = 3 the product grid (2 * (2U+1)^2).
 * Returns -1 on a bad argument. */
int64_t gtp_grid_floats(gtp_plan p, int which);

/* Plan geometry: out[0..7] = {L1, L2, Lout, U = L1+L2, Le = min(Lout, U),
 * NT (theta intervals of the sampling grid on [0, pi]), NP (phi samples),
 * step-2 algorithm gtp_full actually runs: GTP_CONV_DIRECT, GTP_CONV_FFT or GTP_CONV_DFT}. */
gtp_status gtp_plan_info(gtp_plan p, int64_t *out8);

/* Copy one of the plan's fp64 host tables (test aid, host memory):
 *   which 0: T1   [tri(l,m)][u], u in [0, Lin]      theta-Fourier series of Q_l^m (step 1)
 *   which 1: Zc   [tri(l,m)][u], u in [0, U]        int cos(u t) Q sin t dt (step 3)
 *   which 2: Zs   [tri(l,m)][u], u in [0, U]        int sin(u t) Q sin t dt (step 3)
 *   which 3: S    [tri(l,m)][j], j in [0, NT]       synthesis at the theta nodes
 *   which 4: W    [tri(l,m)][j], j in [0, NT]       analysis weights at the theta nodes
 *   which 5: TWR  [lane][24]            phi-operand seeds of the matrix-core kernel
 *   which 6: SMP  [pass][s][u2][lane][4]  its lane-permuted theta synthesis values
 *   which 7: SM0P [pass][lane][v]         its m = 0 theta synthesis values (+ pole)
 *   which 8: WP   [pass][it][lane][8]     its lane-permuted theta analysis weights
 *   which 9: XMAP [lane][k]               its LDS slot of input coefficient lane + 64k
 *   which 10: J   per degree l, (2l+1)^2    real-SH matrix of the rotation R_x(90 deg)
 *   which 11: E   [pair][row]               theta-node rows of the rotated-frame convolution
 *   which 12: A   [m][lane][step]           its matrix-core operand images (theta tables)
 *   which 13: Z   [group][pair][l] + poles  its zonal-filter table
 *   which 14: JI  [l][tile][lane][step]     its operand images of J and J^T
 * with tri(l,m) = l(l+1)/2 + m, m >= 0.  Tables 5..9 exist only for
 * L1 = L2 = Lout = L in {16, 32, 64}, tables 10..11 for L1 = L2 = Lout in
 * 1..8 and 16, tables 12..14 for L1 = L2 = Lout = 16 (length 0 otherwise);
 * their layouts are internal to those kernels.  Pass buf = NULL to
 * get the length in *count; otherwise *count is the capacity in doubles. */
gtp_status gtp_plan_table(gtp_plan p, int which, double *buf, int64_t *count);

/* fp64 host evaluation of the plan's three-step transform pipeline on host
 * arrays (x1[n,(L1+1)^2], x2[n,(L2+1)^2] -> y[n,(Lout+1)^2]).  A CPU check of
 * the tables only; gtp_full never calls it and it is not a fallback. */
gtp_status gtp_debug_host_pipeline(gtp_plan p, const double *x1, const double *x2, int64_t n,
                                   double *y);

const char *gtp_status_str(gtp_status s);
const char *gtp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GTP_H */
