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

}  // namespace

hipError_t launch_full_large(const DevTables& t, const void* x1, const void* x2, int in_type, int64_t n, float* y,
                             hipStream_t s, bool* supported) {
  *supported = true;
  if (t.L1 == t.L2 && t.L1 == t.Lout) {
    if (t.L1 == 16) return launch_large_one<16>(t, x1, x2, in_type, n, y, s);
    if (t.L1 == 32) return launch_large_one<32>(t, x1, x2, in_type, n, y, s);
  }
  *supported = false;
  return hipSuccess;
}

}  // namespace gtp
