// Wave-per-product fused Gaunt tensor product for L1 = L2 = Lout = L with
// 2L <= 64 (gfx950).
//
// Same sampled pipeline as the small-degree kernel (Sec. 3.2 with the
// convolution theorem): theta nodes t_j = j pi / (2L+1), mirror pairs
// (j, 2L+1-j), j = 1..L, plus the two poles; phi samples p_k = 2 pi k / NP.
// Work is spread over the 2L lanes of a product:
//   1. theta synthesis: lane (h, j) sums the m-parts with m = h (mod 2) for
//      both mirror nodes (table column S[., j], coalesced; x as broadcast
//      quads from LDS), then a lane-pair exchange leaves each lane holding
//      every m-part of ONE node;
//   2. phi transforms per node in registers (4-fold symmetric direct DFT,
//      twiddles uniform per quarter angle, i.e. scalar registers), pointwise
//      product, moments of the product;
//   3. mirror combination (lane-pair exchange) into LDS;
//   4. theta analysis: lanes own output coefficients and sum the weights
//      W[., j] times the combined moments over the pairs.
#include <type_traits>
#include <utility>

#include "gtp_device.hpp"

namespace gtp {
namespace {

template <int B, int... Is, typename F>
__device__ __forceinline__ void lfor_impl(std::integer_sequence<int, Is...>, F& f) {
  (f(std::integral_constant<int, B + Is>{}), ...);
}
template <int B, int E, typename F>
__device__ __forceinline__ void lfor(F&& f) {
  if constexpr (E > B) lfor_impl<B>(std::make_integer_sequence<int, E - B>{}, f);
}

__device__ __forceinline__ int ltri(int l, int m) { return l * (l + 1) / 2 + m; }

// Table reads go through buffer resources: 32-bit byte offsets stepped
// incrementally (no 64-bit address arithmetic), and reads past the table
// return zero.
constexpr int kBufDword3 = 0x00020000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t table_rsrc(const float* p, int nfloats) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p), (short)0, nfloats * 4, kBufDword3);
}
__device__ __forceinline__ float tload(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0));  // raw bits -> float
}
// same with a wave-uniform part of the offset in a scalar register
__device__ __forceinline__ float tload_s(__amdgpu_buffer_rsrc_t r, int byte_off, int uniform_off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, byte_off, uniform_off, 0));
}
// 16-byte table read (byte_off a multiple of 16)
__device__ __forceinline__ float4 tload4_s(__amdgpu_buffer_rsrc_t r, int byte_off, int uniform_off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, uniform_off, 0);
  return make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]), __uint_as_float(v[3]));
}

__device__ __forceinline__ float ld_in_any(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld_in_any(const uint16_t* p, int64_t i) {
  return __uint_as_float(uint32_t(p[i]) << 16);
}

template <int L>
struct LGeo {
  static constexpr int NT = 2 * L + 1;          // theta intervals; nodes 0..NT
  static constexpr int NJ = NT + 1;
  static constexpr int NP = (3 * L + 1 + 3) / 4 * 4;  // same rule as the host tables (U = 2L, Le = L)
  static constexpr int Q = NP / 4;
  static constexpr int LPP = 2 * L;             // lanes per product
  static constexpr int PPW = 64 / LPP;          // products per wave
  static constexpr int K = (L + 1) * (L + 1);
  static constexpr int NQ = (L + 1) * (L + 2) / 2;  // (m, l >= m) quads per product
  static constexpr int ME = L / 2 + 1;          // even m: 0, 2, .., L (L even)
  static constexpr int MO = L / 2;              // odd m: 1, 3, .., L - 1
  static constexpr int NMP = 2 * L + 1;         // m-parts
  static constexpr int EO_STRIDE = NMP;         // floats per (parity, pair) row of moments
};

// x quad offset of (m, l): quads for m are stored for l = m..L.
__device__ __forceinline__ int qoff(int L, int m) { return m * (L + 1) - m * (m - 1) / 2; }

template <int L, typename TIn>
__global__ __launch_bounds__(64) void k_full_large(const TIn* __restrict__ x1, const TIn* __restrict__ x2,
                                                   float* __restrict__ y, int64_t n, DevTables t) {
  using G = LGeo<L>;
  static_assert(L % 2 == 0 && 2 * L <= 64 && (L & (L - 1)) == 0, "L must be a power of two <= 32");
  constexpr int NJ = G::NJ, NP = G::NP, Q = G::Q, LPP = G::LPP, PPW = G::PPW, K = G::K, NQ = G::NQ;
  constexpr int ME = G::ME, MO = G::MO, NMP = G::NMP;
  // LDS: x quads during theta synthesis, then (aliased) the mirror-combined
  // moments, plus the pole products.
  constexpr int XQ_FLOATS = PPW * NQ * 4;
  constexpr int EO_FLOATS = PPW * 2 * L * NMP;
  constexpr int BUF = XQ_FLOATS > EO_FLOATS ? XQ_FLOATS : EO_FLOATS;
  __shared__ __align__(16) float buf[BUF];
  __shared__ float poles[PPW * 2];

  const int lane = threadIdx.x;
  const int p = lane / LPP;           // product within the wave
  const int r = lane % LPP;           // lane within the product
  const int h = r / L;                // m parity handled in theta synthesis
  const int jp = r % L + 1;           // mirror pair (jp, NT - jp)
  const int64_t P = int64_t(blockIdx.x) * PPW + p;
  const bool live = P < n;

  // ---- 0. x into LDS as quads (x1 cos, x1 sin, x2 cos, x2 sin) per (m, l)
  for (int i = lane; i < PPW * 2 * K; i += 64) {
    const int pp = i / (2 * K), rem = i % (2 * K), which = rem / K, idx = rem % K;
    const int64_t PP = int64_t(blockIdx.x) * PPW + pp;
    float v = 0.0f;
    if (PP < n) v = which == 0 ? ld_in_any(x1, PP * K + idx) : ld_in_any(x2, PP * K + idx);
    int l = int(sqrtf(float(idx)));
    while (l * l > idx) --l;
    while ((l + 1) * (l + 1) <= idx) ++l;
    const int ms = idx - l * l - l, m = ms < 0 ? -ms : ms;
    buf[(pp * NQ + qoff(L, m) + (l - m)) * 4 + 2 * which + (ms < 0 ? 1 : 0)] = v;
  }
  // sine slots of m = 0 hold zeros
  for (int i = lane; i < PPW * (L + 1); i += 64) {
    const int pp = i / (L + 1), l = i % (L + 1);
    buf[(pp * NQ + l) * 4 + 1] = 0.0f;
    buf[(pp * NQ + l) * 4 + 3] = 0.0f;
  }
  __syncthreads();

  // ---- 1. theta synthesis for the m-parts with m = h (mod 2) at both mirror nodes
  const float4* xq = reinterpret_cast<const float4*>(buf) + p * NQ;
  const float sgn = h == 0 ? 1.0f : -1.0f;
  const __amdgpu_buffer_rsrc_t Sr = table_rsrc(t.S, t.ntS * NJ);
  float keep[4 * ME], send[4 * ME];
  float pole1n = 0.0f, pole1s = 0.0f, pole2n = 0.0f, pole2s = 0.0f;
  lfor<0, ME>([&](auto MI) {
    constexpr int mi = decltype(MI)::value;
    const int m = 2 * mi + h;
    float e[4] = {0.0f, 0.0f, 0.0f, 0.0f}, o[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    const float4* xm = xq + qoff(L, m);
    const int dmax = L - m;  // -1 when this lane has no m-part in this slot
    // byte offset of S[tri(m + d, m)][jp]; consecutive d are (m + d + 1) rows apart
    int off = (ltri(m, m) * NJ + jp) * 4;
    int step = (m + 1) * NJ * 4;
    for (int d = 0; d <= dmax; d += 2) {
      // even d = l - m: (l + m) even, feeds the even partial sums
      const float4 q = xm[d];
      const float s = tload(Sr, off);
      off += step;
      step += NJ * 4;
      e[0] = fmaf(s, q.x, e[0]);
      e[1] = fmaf(s, q.y, e[1]);
      e[2] = fmaf(s, q.z, e[2]);
      e[3] = fmaf(s, q.w, e[3]);
      if (d + 1 <= dmax) {
        const float4 q1 = xm[d + 1];
        const float s1 = tload(Sr, off);
        o[0] = fmaf(s1, q1.x, o[0]);
        o[1] = fmaf(s1, q1.y, o[1]);
        o[2] = fmaf(s1, q1.z, o[2]);
        o[3] = fmaf(s1, q1.w, o[3]);
      }
      off += step;
      step += NJ * 4;
    }
    lfor<0, 4>([&](auto C) {
      constexpr int c = decltype(C)::value;
      keep[4 * mi + c] = fmaf(sgn, o[c], e[c]);
      send[4 * mi + c] = fmaf(-sgn, o[c], e[c]);
    });
    // bound the table loads in flight to one m-part's column
    __builtin_amdgcn_sched_barrier(0);
  });
  // poles (only m = 0 is non-zero there); lanes with h = 0 compute them
  if (h == 0 && jp == 1) {
    for (int l = 0; l <= L; ++l) {
      const float4 q = xq[l];
      const float sn = t.S[ltri(l, 0) * NJ];
      const float ss = (l & 1) ? -sn : sn;
      pole1n = fmaf(sn, q.x, pole1n);
      pole1s = fmaf(ss, q.x, pole1s);
      pole2n = fmaf(sn, q.z, pole2n);
      pole2s = fmaf(ss, q.z, pole2s);
    }
  }
  __syncthreads();  // x quads are dead from here on (the buffer is reused)
  if (h == 0 && jp == 1) {
    poles[2 * p] = pole1n * pole2n;
    poles[2 * p + 1] = pole1s * pole2s;
  }

  // ---- exchange: lane h = 0 keeps node jp, lane h = 1 keeps node NT - jp;
  // in place: keep[] becomes the even-m values, send[] the odd-m values
  lfor<0, 4 * ME>([&](auto I) {
    constexpr int i = decltype(I)::value;
    const float a = keep[i];
    const float rv = __shfl_xor(send[i], L);
    keep[i] = h ? rv : a;
    send[i] = h ? a : rv;
  });
  float (&Ev)[4 * ME] = keep;
  float (&Ov)[4 * ME] = send;

  // ---- 2. phi transforms at this lane's node: Cc[m] = sum_k H cos, Cs[m] = sum_k H sin
  float Cc[L + 1], Cs[L + 1];
  lfor<0, L + 1>([&](auto I) {
    Cc[decltype(I)::value] = 0.0f;
    Cs[decltype(I)::value] = 0.0f;
  });
  const int nmp_all = 2 * t.Mphi + 1;
  for (int k = 0; k <= Q; ++k) {
    const float* tw = t.PhiT + k * nmp_all;  // tw[2m-1] = cos(m p_k), tw[2m] = sin(m p_k)
    float pe1 = Ev[0], po1 = 0.0f, qe1 = 0.0f, qo1 = 0.0f;
    float pe2 = Ev[2], po2 = 0.0f, qe2 = 0.0f, qo2 = 0.0f;
    lfor<1, L + 1>([&](auto MM) {
      constexpr int m = decltype(MM)::value;
      const float c = tw[2 * m - 1], s = tw[2 * m];
      constexpr int b = 4 * (m / 2);
      if constexpr (m % 2 == 0) {
        pe1 = fmaf(Ev[b + 0], c, pe1);
        qe1 = fmaf(Ev[b + 1], s, qe1);
        pe2 = fmaf(Ev[b + 2], c, pe2);
        qe2 = fmaf(Ev[b + 3], s, qe2);
      } else {
        po1 = fmaf(Ov[b + 0], c, po1);
        qo1 = fmaf(Ov[b + 1], s, qo1);
        po2 = fmaf(Ov[b + 2], c, po2);
        qo2 = fmaf(Ov[b + 3], s, qo2);
      }
    });
    float ce, co, se, so;
    if (k == 0) {
      const float h0 = (pe1 + po1) * (pe2 + po2), h2 = (pe1 - po1) * (pe2 - po2);
      ce = h0 + h2;
      co = h0 - h2;
      se = 0.0f;
      so = 0.0f;
    } else if (k == Q) {
      const float hq = (pe1 + qo1) * (pe2 + qo2), h3 = (pe1 - qo1) * (pe2 - qo2);
      ce = hq + h3;
      so = hq - h3;
      co = 0.0f;
      se = 0.0f;
    } else {
      const float s1 = pe1 + po1, d1 = pe1 - po1, s2 = qe1 + qo1, d2 = qe1 - qo1;
      const float t1 = pe2 + po2, u1 = pe2 - po2, t2 = qe2 + qo2, u2 = qe2 - qo2;
      const float hk = (s1 + s2) * (t1 + t2), hmk = (s1 - s2) * (t1 - t2);
      const float hpk = (d1 + d2) * (u1 + u2), hpmk = (d1 - d2) * (u1 - u2);
      const float a = hk + hmk, b = hpk + hpmk, dd = hk - hmk, ee = hpk - hpmk;
      ce = a + b;
      co = a - b;
      se = dd + ee;
      so = dd - ee;
    }
    Cc[0] += ce;
    lfor<1, L + 1>([&](auto MM) {
      constexpr int m = decltype(MM)::value;
      const float c = tw[2 * m - 1], s = tw[2 * m];
      Cc[m] = fmaf((m % 2 == 0) ? ce : co, c, Cc[m]);
      Cs[m] = fmaf((m % 2 == 0) ? se : so, s, Cs[m]);
    });
  }

  // ---- 3. mirror combination: h = 0 lanes form C(j) + C(NT - j), h = 1 lanes C(j) - C(NT - j)
  float* eo = buf + ((p * 2 + h) * L + (jp - 1)) * NMP;
  lfor<0, L + 1>([&](auto MM) {
    constexpr int m = decltype(MM)::value;
    const float pc = __shfl_xor(Cc[m], L);
    eo[m == 0 ? 0 : 2 * m - 1] = fmaf(sgn, Cc[m], pc);
    if constexpr (m > 0) {
      const float ps = __shfl_xor(Cs[m], L);
      eo[2 * m] = fmaf(sgn, Cs[m], ps);
    }
  });
  __syncthreads();

  // ---- 4. theta analysis: lane r of the product owns rows tri(l, m) = r, r + 2L, ...
  // (both the cos and the sin coefficient of each row), so the weight loads
  // W[j][row] are contiguous across lanes.
  const float fN = poles[2 * p] * float(NP), fS = poles[2 * p + 1] * float(NP);
  const float* eop = buf + p * 2 * L * NMP;
  const int ntW = t.ntW;
  const __amdgpu_buffer_rsrc_t Wr = table_rsrc(t.WT, NJ * ntW);
  constexpr int NTRI = (L + 1) * (L + 2) / 2;
  // rows with m = 0: only the cos coefficient, plus the pole terms
  for (int l = r; l <= L; l += LPP) {
    const int tr = l * (l + 1) / 2;
    const float* src = eop + (l & 1) * L * NMP;
    float acc = tload(Wr, tr * 4) * (fN + ((l & 1) ? -fS : fS));
    int off = (ntW + tr) * 4;
#pragma unroll 8
    for (int j = 1; j <= L; ++j, off += ntW * 4) acc = fmaf(tload(Wr, off), src[(j - 1) * NMP], acc);
    if (live) y[P * K + l * l + l] = acc;
  }
  // rows with m > 0: lane r takes the r-th, (r + 2L)-th, ... of them
  constexpr int NROW = NTRI - (L + 1);
  for (int q = r; q < NROW; q += LPP) {
    // q-th row with m > 0 in tri order: l >= 1, rows of degree l are l in number
    // degree l with l(l-1)/2 <= q < l(l+1)/2 (one correction step each way)
    int l = int((sqrtf(8.0f * float(q) + 1.0f) + 1.0f) * 0.5f);
    l -= (l * (l - 1) / 2 > q) ? 1 : 0;
    l += ((l + 1) * l / 2 <= q) ? 1 : 0;
    const int m = q - l * (l - 1) / 2 + 1;
    const int tr = l * (l + 1) / 2 + m;
    const float* src = eop + ((l + m) & 1) * L * NMP + 2 * m - 1;
    float accc = 0.0f, accs = 0.0f;
    int off = (ntW + tr) * 4;
#pragma unroll 8
    for (int j = 1; j <= L; ++j, off += ntW * 4) {
      const float w = tload(Wr, off);
      accc = fmaf(w, src[(j - 1) * NMP], accc);
      accs = fmaf(w, src[(j - 1) * NMP + 1], accs);
    }
    if (live) {
      y[P * K + l * l + l + m] = accc;
      y[P * K + l * l + l - m] = accs;
    }
  }
}

template <int L>
hipError_t launch_large_one(const DevTables& t, const void* x1, const void* x2, int in_type, int64_t n, float* y,
                            hipStream_t s) {
  using G = LGeo<L>;
  const int64_t blocks = (n + G::PPW - 1) / G::PPW;
  if (in_type == IN_BF16)
    hipLaunchKernelGGL((k_full_large<L, uint16_t>), dim3(unsigned(blocks)), dim3(64), 0, s,
                       static_cast<const uint16_t*>(x1), static_cast<const uint16_t*>(x2), y, n, t);
  else
    hipLaunchKernelGGL((k_full_large<L, float>), dim3(unsigned(blocks)), dim3(64), 0, s,
                       static_cast<const float*>(x1), static_cast<const float*>(x2), y, n, t);
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// Matrix-core variant (L in {16, 32}).  One 64-lane wave per product, lane =
// 16 g + i, i = 8 h + pi.  The phi stage at every theta node is a set of small
// dense contractions whose operands are shared by all nodes and products, so
// it runs on the fp32 MFMA units (16x16x4: A = phi operand table, B = theta
// synthesis values; the 16 columns are the 8 mirror pairs of a pass, column
// pi = node jp, column 8 + pi = node NT - jp):
//   synthesis  pe/po/qe/qo[k][node] = sum over the even/odd-m cos/sin parts
//              of trig(m phi_k) * value[m][node], k = 0..Q (4-fold phi
//              symmetry as in the direct kernel: points k, -k, 2Q - k, 2Q + k);
//   product    the four sample products folded into ce/co/se/so[k][node];
//   analysis   C[m][node] = sum_k w_k trig(m phi_k) * {ce, co, se, so}[k][node]
//              (w_k = 1/2 at k = 0, Q, where the 4-point sets repeat points).
// The accumulator layout of one contraction is the B layout of the next
// (register r of lane (g, i) holds row 4 g + r, column i), so nothing moves
// between them.  Theta synthesis (VALU) produces the B operands in place: in
// K-step s lane (g, 8h + pi) sums the m-parts m = 8s + 2g + 1 and + 2 at node
// jp over the l with l - m = h (mod 2); one exchange between lanes i and i ^ 8
// then gives node jp (even + odd) and its mirror (even - odd).  Theta analysis
// (VALU) accumulates per pass.
typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

template <int L>
struct WGeo {
  static constexpr int NT = 2 * L + 1;
  static constexpr int NJ = NT + 1;
  static constexpr int NP = (3 * L + 1 + 3) / 4 * 4;  // host rule with U = 2L, Le = L
  static constexpr int Q = NP / 4;
  static constexpr int PASSES = L / 8;               // 8 mirror pairs per pass
  static constexpr int NKS = L / 8;                  // K-steps per class of m-parts
  static constexpr int NMB = (Q + 1 + 15) / 16;      // 16-sample blocks of k = 0..Q
  static constexpr int RS = L + 2;                   // SM row length
  static constexpr int NC = L + 1;                   // SM columns (nodes 0..L)
  static constexpr int NMP = 2 * L + 1;
  static constexpr int K = (L + 1) * (L + 1);
  static constexpr int NMP2 = 2 * L + 2;             // moment row: [m=0, -, cos 1, sin 1, .., cos L, sin L]
  static constexpr int EOP = 2 * 8 * NMP2;           // floats of one pass's combined moments
  static constexpr int NROW = (L + 1) * (L + 2) / 2 - (L + 1);  // output rows with m > 0
  static constexpr int NIT = (NROW + 63) / 64;
  // u-steps (two degrees each) of K-step s
  __host__ __device__ static constexpr int nu(int s) { return L / 2 - 4 * s; }
  // quad offset of the x block of m-pair c = 4 s + g (m = 2c + 1, 2c + 2): the
  // m = 0 block (L + 1 quads) first, then 4 nu(s) quads + 1 pad per pair
  __host__ __device__ static constexpr int xb(int c) {
    return (L + 1) + c + 4 * (4 * ((c / 4) * (L / 2) - 2 * (c / 4) * (c / 4 - 1)) + (c % 4) * nu(c / 4));
  }
  static constexpr int XQ = xb(L / 2);
  // u-step pairs before K-step s, and in all K-steps
  __host__ __device__ static constexpr int u2off(int s) { return s * (L / 4) - s * (s - 1); }
  static constexpr int TU2 = u2off(NKS);
  static constexpr int NV0 = (L + 1 + 7) / 8;          // m = 0 steps of 8 degrees
  static constexpr int NV0P = (NV0 + 3) / 4 * 4;
};

// m = 0 theta synthesis reduction: lane (g, 8h + pi) holds the partial sum
// over l = g + 4h (mod 8); returns the value at the lane's column node (the
// node itself for h = 0, its mirror, odd l negated, for h = 1).
__device__ __forceinline__ float m0_reduce(float a, int g, int h) {
  a += __shfl_xor(a, 8);
  const float t = __shfl_xor(a, 16);
  const float sum = a + t, dif = (g & 1) ? t - a : a - t;
  const float node = sum + __shfl_xor(sum, 32), mirror = dif + __shfl_xor(dif, 32);
  return h ? mirror : node;
}

template <int L, typename TIn>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(3))) void k_full_wave(
    const TIn* __restrict__ x1, const TIn* __restrict__ x2, float* __restrict__ y, int64_t n, DevTables t) {
  using G = WGeo<L>;
  static_assert(L % 16 == 0 && L <= 32, "L must be 16 or 32");
  constexpr int NJ = G::NJ, NP = G::NP, NMB = G::NMB, NKS = G::NKS, RS = G::RS, NC = G::NC;
  constexpr int NMP2 = G::NMP2, K = G::K, PASSES = G::PASSES, NROW = G::NROW, NIT = G::NIT;
  __shared__ __align__(16) float xs[G::XQ * 4];
  __shared__ __align__(16) float eo[G::EOP];
  const float4* const xq = reinterpret_cast<const float4*>(xs);

  const int lane = threadIdx.x, g = lane >> 4, i = lane & 15, h = i >> 3, pi = i & 7;
  const int64_t P = blockIdx.x;
  if (P >= n) return;  // whole-wave exit (one product per workgroup)

  // ---- 0. x into the LDS image (quads x1 cos, x1 sin, x2 cos, x2 sin): every
  // load is issued before the first wait
  {
    constexpr int NXK = (K + 63) / 64, NXKP = (NXK + 3) / 4 * 4;
    int slot[NXKP];
    lfor<0, NXKP / 4>([&](auto K4) {
      constexpr int k4 = decltype(K4)::value;
      const int4 v = reinterpret_cast<const int4*>(t.XMAP + lane * NXKP)[k4];
      slot[4 * k4] = v.x;
      slot[4 * k4 + 1] = v.y;
      slot[4 * k4 + 2] = v.z;
      slot[4 * k4 + 3] = v.w;
    });
    float v1[NXK], v2[NXK];
    lfor<0, NXK>([&](auto KK) {
      constexpr int k = decltype(KK)::value;
      const int e = lane + 64 * k;
      if (64 * k + 63 < K || e < K) {
        v1[k] = ld_in_any(x1, P * K + e);
        v2[k] = ld_in_any(x2, P * K + e);
      }
    });
    lfor<0, G::XQ / 64>([&](auto Z) {
      reinterpret_cast<float4*>(xs)[lane + 64 * decltype(Z)::value] = make_float4(0.f, 0.f, 0.f, 0.f);
    });
    if (lane < G::XQ % 64) reinterpret_cast<float4*>(xs)[lane + 64 * (G::XQ / 64)] = make_float4(0.f, 0.f, 0.f, 0.f);
    __syncthreads();
    lfor<0, NXK>([&](auto KK) {
      constexpr int k = decltype(KK)::value;
      if (64 * k + 63 < K || lane + 64 * k < K) {
        xs[slot[k]] = v1[k];
        xs[slot[k] + 2] = v2[k];
      }
    });
  }
  __syncthreads();

  const __amdgpu_buffer_rsrc_t SPr = table_rsrc(t.SMP, PASSES * G::TU2 * 64 * 4);
  const __amdgpu_buffer_rsrc_t S0r = table_rsrc(t.SM0P, (PASSES + 1) * 64 * G::NV0P);
  const __amdgpu_buffer_rsrc_t WPr = table_rsrc(t.WP, PASSES * (NIT + 1) * 64 * 8);
  const __amdgpu_buffer_rsrc_t Wr = table_rsrc(t.WT, NJ * t.ntW);
  // m = 0 theta synthesis at the lane's column node (x1 and x2 cos parts);
  // pass = PASSES gives the poles.  Split into the table read and the sums so
  // that other loads can be issued in between.
  auto m0_load = [&](int pass, float (&sv)[G::NV0P]) {
    lfor<0, G::NV0P / 4>([&](auto V4) {
      constexpr int v4 = decltype(V4)::value;
      const float4 w = tload4_s(S0r, lane * G::NV0P * 4 + 16 * v4, pass * 64 * G::NV0P * 4);
      sv[4 * v4] = w.x;
      sv[4 * v4 + 1] = w.y;
      sv[4 * v4 + 2] = w.z;
      sv[4 * v4 + 3] = w.w;
    });
  };
  auto m0_finish = [&](const float (&sv)[G::NV0P], float& a1, float& a2) {
    float s1 = 0.0f, s2 = 0.0f;
    lfor<0, G::NV0>([&](auto V) {
      constexpr int v = decltype(V)::value;
      const int l = 8 * v + g + 4 * h;
      if (8 * v + 7 <= L || l <= L) {
        const float4 q = xq[l];
        s1 = fmaf(sv[v], q.x, s1);
        s2 = fmaf(sv[v], q.z, s2);
      }
    });
    a1 = m0_reduce(s1, g, h);
    a2 = m0_reduce(s2, g, h);
  };
  // phi-stage operands from per-lane seeds: cos/sin of m phi advance by
  // rotations (angle addition) instead of table reads
  auto rot = [](float& c, float& s, float cr, float sr) {
    const float cn = c * cr - s * sr;
    s = fmaf(s, cr, c * sr);
    c = cn;
  };

  // theta-analysis rows: tri(l, 0) with l = lane (l <= L), and the rows with
  // m > 0 numbered q = lane + 64 it; per row the byte offset of its weight
  // column and the LDS offset of its moment (parity of l + m, m-part)
  float y0 = 0.0f, yc[NIT], ys[NIT];
  int er[NIT];
  const int wr0 = (lane * (lane + 1) / 2) * 4, er0 = (lane & 1) * 8 * NMP2;
  lfor<0, NIT>([&](auto IT) {
    constexpr int it = decltype(IT)::value;
    yc[it] = 0.0f;
    ys[it] = 0.0f;
    const int q = lane + 64 * it;
    int l = int((sqrtf(8.0f * float(q) + 1.0f) + 1.0f) * 0.5f);
    l -= (l * (l - 1) / 2 > q) ? 1 : 0;
    l += ((l + 1) * l / 2 <= q) ? 1 : 0;
    const int m = q - l * (l - 1) / 2 + 1;
    er[it] = ((l + m) & 1) * 8 * NMP2 + 2 * m;
  });

  for (int pass = 0; pass < PASSES; ++pass) {
    const int pu = __builtin_amdgcn_readfirstlane(pass);  // uniform: keep it scalar
    // loads first (m = 0 part, the first theta-table steps, the first phi
    // operands), then the m = 0 sums
    constexpr int D = 5;  // theta-table steps in flight
    const int sbase = pu * G::TU2 * 64 * 16;
    float s0v[G::NV0P];
    m0_load(pu, s0v);
    float4 sring[D];
    lfor<0, D>([&](auto T) {
      constexpr int tt = decltype(T)::value;
      if constexpr (tt < G::TU2) sring[tt] = tload4_s(SPr, lane * 16, sbase + tt * 64 * 16);
    });
    // synthesis operands twc[type][mb] of K-step 0 and the rotation by 8 phi_k
    float twc[4][NMB], r8c[NMB], r8s[NMB];
    {
      const f4* src = reinterpret_cast<const f4*>(t.TWR + lane * 24);
      const f4 a = src[0], b = src[1], c = src[2];
      const float sd[12] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w, c.x, c.y, c.z, c.w};
      lfor<0, NMB>([&](auto MB) {
        constexpr int mb = decltype(MB)::value;
        twc[0][mb] = sd[6 * mb + 0];  // cos, even m
        twc[2][mb] = sd[6 * mb + 1];  // sin, even m
        twc[1][mb] = sd[6 * mb + 2];  // cos, odd m
        twc[3][mb] = sd[6 * mb + 3];  // sin, odd m
        r8c[mb] = sd[6 * mb + 4];
        r8s[mb] = sd[6 * mb + 5];
      });
    }
    float c1, c2;
    m0_finish(s0v, c1, c2);

    // ---- 1 + 2a. theta synthesis feeding the phi-synthesis contractions
    f4 acc[2][NMB][4];  // [input][k block][type]
    lfor<0, NMB>([&](auto MB) {
      constexpr int mb = decltype(MB)::value;
      acc[0][mb][0] = f4{c1, c1, c1, c1};  // m = 0 enters every pe sample
      acc[1][mb][0] = f4{c2, c2, c2, c2};
      lfor<1, 4>([&](auto TY) {
        acc[0][mb][decltype(TY)::value] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        acc[1][mb][decltype(TY)::value] = f4{0.0f, 0.0f, 0.0f, 0.0f};
      });
    });
    float twa[5][NMB][4];
    lfor<0, NKS>([&](auto SS) {
      constexpr int s = decltype(SS)::value;
      const int c = 4 * s + g;
      // this lane's parity: h = 0 takes (mo, l_a) and (mo+1, l_b), h = 1 (mo, l_b) and (mo+1, l_a)
      const float4* xa = xq + G::xb(c) + h;
      const float4* xe = xq + G::xb(c) + 3 - h;
      f4 Vo = {0.0f, 0.0f, 0.0f, 0.0f}, Ve = Vo;
      lfor<0, G::nu(s) / 2>([&](auto U2) {
        constexpr int u2 = decltype(U2)::value, tt = G::u2off(s) + u2;
        const float4 sv = sring[tt % D];
        if constexpr (tt + D < G::TU2) sring[tt % D] = tload4_s(SPr, lane * 16, sbase + (tt + D) * 64 * 16);
        lfor<0, 2>([&](auto E) {
          constexpr int u = 2 * u2 + decltype(E)::value;
          const float so = E == 0 ? sv.x : sv.z, se = E == 0 ? sv.y : sv.w;
          const float4 qa = xa[4 * u], qe = xe[4 * u];
          Vo += so * f4{qa.x, qa.y, qa.z, qa.w};
          Ve += se * f4{qe.x, qe.y, qe.z, qe.w};
        });
        __builtin_amdgcn_sched_barrier(0);  // keep the prefetch distance
      });
      if constexpr (s == NKS - 1) {
        // phi-analysis operands twa[type][mb][r] = w_k trig(m phi_k), k = 16 mb + 4 g + r,
        // m = 2i + 2 (even types) or 2i + 1 (odd types); type 4 = w_k
        const f4* src = reinterpret_cast<const f4*>(t.TWR + lane * 24);
        const f4 a = src[3], b = src[4], st = src[5];
        const float sd[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
        lfor<0, NMB>([&](auto MB) {
          constexpr int mb = decltype(MB)::value;
          float ce = sd[4 * mb + 0], se = sd[4 * mb + 1], co = sd[4 * mb + 2], so = sd[4 * mb + 3];
          lfor<0, 4>([&](auto R) {
            constexpr int r = decltype(R)::value;
            if constexpr (r > 0) {
              rot(ce, se, st.x, st.y);
              rot(co, so, st.z, st.w);
            }
            const int k = 16 * mb + 4 * g + r;
            const float w = k > G::Q ? 0.0f : (k == 0 || k == G::Q) ? 0.5f : 1.0f;
            twa[0][mb][r] = w * ce;
            twa[1][mb][r] = w * co;
            twa[2][mb][r] = w * se;
            twa[3][mb][r] = w * so;
            twa[4][mb][r] = w;
          });
        });
      }
      // column value: node jp (h = 0: own even + partner odd) or its mirror (h = 1: partner even - own odd)
      f4 Bo, Be;
      lfor<0, 4>([&](auto C) {
        constexpr int cc = decltype(C)::value;
        const float po = __shfl_xor(Vo[cc], 8), pe = __shfl_xor(Ve[cc], 8);
        Bo[cc] = h ? po - Vo[cc] : po + Vo[cc];
        Be[cc] = h ? pe - Ve[cc] : pe + Ve[cc];
      });
      lfor<0, NMB>([&](auto MB) {
        constexpr int mb = decltype(MB)::value;
        lfor<0, 2>([&](auto TI) {
          constexpr int ti = decltype(TI)::value;
          acc[ti][mb][0] = mfma4(twc[0][mb], Be[2 * ti], acc[ti][mb][0]);
          acc[ti][mb][1] = mfma4(twc[1][mb], Bo[2 * ti], acc[ti][mb][1]);
          acc[ti][mb][2] = mfma4(twc[2][mb], Be[2 * ti + 1], acc[ti][mb][2]);
          acc[ti][mb][3] = mfma4(twc[3][mb], Bo[2 * ti + 1], acc[ti][mb][3]);
        });
      });
      if constexpr (s + 1 < NKS) {
        // next K-step: m -> m + 8
        lfor<0, NMB>([&](auto MB) {
          constexpr int mb = decltype(MB)::value;
          rot(twc[0][mb], twc[2][mb], r8c[mb], r8s[mb]);
          rot(twc[1][mb], twc[3][mb], r8c[mb], r8s[mb]);
        });
      }
    });

    // ---- 2b. sample products, folded over the 4-point sets
    lfor<0, NMB>([&](auto MB) {
      constexpr int mb = decltype(MB)::value;
      const f4 pe1 = acc[0][mb][0], po1 = acc[0][mb][1], qe1 = acc[0][mb][2], qo1 = acc[0][mb][3];
      const f4 pe2 = acc[1][mb][0], po2 = acc[1][mb][1], qe2 = acc[1][mb][2], qo2 = acc[1][mb][3];
      const f4 s1 = pe1 + po1, d1 = pe1 - po1, s2 = qe1 + qo1, d2 = qe1 - qo1;
      const f4 t1 = pe2 + po2, u1 = pe2 - po2, t2 = qe2 + qo2, u2 = qe2 - qo2;
      const f4 hk = (s1 + s2) * (t1 + t2), hmk = (s1 - s2) * (t1 - t2);
      const f4 hpk = (d1 + d2) * (u1 + u2), hpmk = (d1 - d2) * (u1 - u2);
      const f4 a = hk + hmk, b = hpk + hpmk, dd = hk - hmk, ee = hpk - hpmk;
      acc[0][mb][0] = a + b;
      acc[0][mb][1] = a - b;
      acc[0][mb][2] = dd + ee;
      acc[0][mb][3] = dd - ee;
    });

    // ---- 2c. phi analysis contractions, then 3. mirror combination into LDS
    // eo[parity][pi][slot]: parity 0 = C(jp) + C(NT - jp), 1 = C(jp) - C(NT - jp);
    // slot 0 = m 0, 2m = cos m, 2m + 1 = sin m
    float* const eoh = eo + (h * 8 + pi) * NMP2;
    f4 o[4];
    lfor<0, 4>([&](auto TY) {
      constexpr int ty = decltype(TY)::value;
      f4 a = {0.0f, 0.0f, 0.0f, 0.0f};
      lfor<0, NMB>([&](auto MB) {
        constexpr int mb = decltype(MB)::value;
        lfor<0, 4>([&](auto R) {
          constexpr int r = decltype(R)::value;
          a = mfma4(twa[ty][mb][r], acc[0][mb][ty][r], a);
        });
      });
      o[ty] = a;
    });
    lfor<0, 2>([&](auto PAR) {
      constexpr int odd = decltype(PAR)::value;  // types odd (cos), odd + 2 (sin)
      lfor<0, 4>([&](auto R) {
        constexpr int r = decltype(R)::value;
        const int m = 2 * (4 * g + r) + (odd ? 1 : 2);
        const float pc = __shfl_xor(o[odd][r], 8), ps = __shfl_xor(o[odd + 2][r], 8);
        const float vc = h ? pc - o[odd][r] : pc + o[odd][r];
        const float vs = h ? ps - o[odd + 2][r] : ps + o[odd + 2][r];
        if (L == 32 || m <= L) *reinterpret_cast<float2*>(eoh + 2 * m) = make_float2(vc, vs);
      });
    });
    {
      float zz = 0.0f;
      lfor<0, NMB>([&](auto MB) {
        constexpr int mb = decltype(MB)::value;
        lfor<0, 4>([&](auto R) {
          constexpr int r = decltype(R)::value;
          zz = fmaf(twa[4][mb][r], acc[0][mb][0][r], zz);
        });
      });
      zz += __shfl_xor(zz, 16);
      zz += __shfl_xor(zz, 32);
      const float pz = __shfl_xor(zz, 8);
      if (g == 0) eoh[0] = h ? pz - zz : pz + zz;
    }
    __syncthreads();

    // ---- 4. theta analysis over this pass's pairs (lane-permuted weights)
    const int wbase = pu * (NIT + 1) * 64 * 32;
    if (lane <= L) {
      const float4 w0 = tload4_s(WPr, lane * 32, wbase + NIT * 64 * 32);
      const float4 w1 = tload4_s(WPr, lane * 32 + 16, wbase + NIT * 64 * 32);
      const float w[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
      lfor<0, 8>([&](auto JJ) {
        constexpr int jj = decltype(JJ)::value;
        y0 = fmaf(w[jj], eo[er0 + jj * NMP2], y0);
      });
    }
    lfor<0, NIT>([&](auto IT) {
      constexpr int it = decltype(IT)::value;
      if (lane + 64 * it < NROW) {
        const float4 w0 = tload4_s(WPr, lane * 32, wbase + it * 64 * 32);
        const float4 w1 = tload4_s(WPr, lane * 32 + 16, wbase + it * 64 * 32);
        const float w[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
        lfor<0, 8>([&](auto JJ) {
          constexpr int jj = decltype(JJ)::value;
          const float2 cs = *reinterpret_cast<const float2*>(eo + er[it] + jj * NMP2);
          yc[it] = fmaf(w[jj], cs.x, yc[it]);
          ys[it] = fmaf(w[jj], cs.y, ys[it]);
        });
      }
      if constexpr (it % 3 == 2) __builtin_amdgcn_sched_barrier(0);  // bound the loads in flight
    });
    __syncthreads();  // eo is rewritten by the next pass
  }

  // poles (only the m = 0 parts are non-zero there) and the stores
  float p1, p2;
  {
    float sv[G::NV0P];
    m0_load(PASSES, sv);
    m0_finish(sv, p1, p2);  // h = 0 lanes: north pole, h = 1 lanes: south pole
  }
  const float f = p1 * p2 * float(NP);
  const float fN = __shfl(f, 0), fS = __shfl(f, 8);
  if (lane <= L) {
    const int l = lane;
    y0 = fmaf(tload(Wr, wr0), fN + ((l & 1) ? -fS : fS), y0);
    y[P * K + l * l + l] = y0;
  }
  lfor<0, NIT>([&](auto IT) {
    constexpr int it = decltype(IT)::value;
    const int q = lane + 64 * it;
    if (q < NROW) {
      int l = int((sqrtf(8.0f * float(q) + 1.0f) + 1.0f) * 0.5f);
      l -= (l * (l - 1) / 2 > q) ? 1 : 0;
      l += ((l + 1) * l / 2 <= q) ? 1 : 0;
      const int m = q - l * (l - 1) / 2 + 1;
      y[P * K + l * l + l + m] = yc[it];
      y[P * K + l * l + l - m] = ys[it];
    }
  });
}

template <int L>
hipError_t launch_wave_one(const DevTables& t, const void* x1, const void* x2, int in_type, int64_t n, float* y,
                           hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (in_type == IN_BF16)
    hipLaunchKernelGGL((k_full_wave<L, uint16_t>), dim3(unsigned(n)), dim3(64), 0, s,
                       static_cast<const uint16_t*>(x1), static_cast<const uint16_t*>(x2), y, n, t);
  else
    hipLaunchKernelGGL((k_full_wave<L, float>), dim3(unsigned(n)), dim3(64), 0, s, static_cast<const float*>(x1),
                       static_cast<const float*>(x2), y, n, t);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_full_large(const DevTables& t, const void* x1, const void* x2, int in_type, int64_t n, float* y,
                             hipStream_t s, bool* supported) {
  *supported = true;
  if (t.waveL == 16 && t.SM) return launch_wave_one<16>(t, x1, x2, in_type, n, y, s);
  if (t.waveL == 32 && t.SM) return launch_wave_one<32>(t, x1, x2, in_type, n, y, s);
  if (t.L1 == t.L2 && t.L1 == t.Lout) {
    if (t.L1 == 16) return launch_large_one<16>(t, x1, x2, in_type, n, y, s);
    if (t.L1 == 32) return launch_large_one<32>(t, x1, x2, in_type, n, y, s);
  }
  *supported = false;
  return hipSuccess;
}

}  // namespace gtp
