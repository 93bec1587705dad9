// Wave-per-product fused Gaunt tensor product on the matrix cores, for
// L1 = L2 = Lout = L in {16, 32} (gfx950).
//
// Same sampled pipeline as the small-degree kernel (Sec. 3.2 with the
// convolution theorem): theta nodes t_j = j pi / (2L+1), taken as mirror
// pairs (j, 2L+1-j), j = 1..L, plus the two poles; phi samples
// p_k = 2 pi k / NP.
#include <type_traits>
#include <utility>

#include "gtp_ct.hpp"
#include "gtp_device.hpp"
#include "gtp_fft.hpp"

namespace gtp {
namespace {

// Table reads go through buffer resources: 32-bit offsets (the wave-uniform
// part in a scalar register), and reads past the table return zero.
constexpr int kBufDword3 = 0x00020000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t table_rsrc(const float* p, int nfloats) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p), (short)0, nfloats * 4, kBufDword3);
}
__device__ __forceinline__ float tload(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0));  // raw bits -> float
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
// Element i of a product's row that starts at the wave-uniform pointer r:
// the byte offset stays a 32-bit unsigned value, so the access is a scalar
// base plus one offset register (no 64-bit address arithmetic per lane).
__device__ __forceinline__ float ld_row(const float* r, unsigned i) {
  return *reinterpret_cast<const float*>(reinterpret_cast<const char*>(r) + i * 4u);
}
__device__ __forceinline__ float ld_row(const uint16_t* r, unsigned i) {
  return __uint_as_float(uint32_t(*reinterpret_cast<const uint16_t*>(reinterpret_cast<const char*>(r) + i * 2u)) << 16);
}
__device__ __forceinline__ void st_row_bytes(float* r, unsigned byte_off, float v) {
  *reinterpret_cast<float*>(reinterpret_cast<char*>(r) + byte_off) = v;
}

// One 64-lane wave per product, lane = 16 g + i, i = 8 h + pi.  The phi stage
// at every theta node is a set of small dense contractions whose operands are
// shared by all nodes and products, so it runs on the fp32 MFMA units
// (16x16x4; A = phi operands, B = theta-synthesis values; the 16 columns are
// the 8 mirror pairs of a pass: column pi = node jp, column 8 + pi = node
// NT - jp):
//   synthesis  pe/po/qe/qo[k][node] = sum over the even/odd-m cos/sin parts of
//              trig(m phi_k) * value[m][node], k = 0..Q, Q = NP / 4 (the 4-fold
//              phi symmetry of the small-degree kernel: the sample sets
//              {k, -k, 2Q - k, 2Q + k} share these four sums);
//   product    the four sample products folded into ce/co/se/so[k][node];
//   analysis   C[m][node] = sum_k w_k trig(m phi_k) * {ce, co, se, so}[k][node]
//              (w_k = 1/2 at k = 0, Q, where a 4-point set repeats points).
// The accumulator layout of one contraction is the B layout of the next
// (register r of lane (g, i) holds row 4 g + r, column i), so nothing moves
// between them; synthesis row 4 g + r computes sample k = 16 mb + 4 r + g, so
// that each analysis contraction (fixed r, K index g) takes four consecutive
// samples and those past Q drop out whole.  The A operands are generated in
// registers from per-lane seeds by angle-addition rotations.  Theta synthesis (VALU) produces the B
// operands in place: in K-step s lane (g, 8h + pi) sums the m-parts
// m = 8s + 2g + 1 and + 2 at node jp over the l with l - m = h (mod 2); one
// exchange between lanes i and i ^ 8 then gives node jp (even + odd) and its
// mirror (even - odd).  Theta analysis (VALU) accumulates over the passes.
// All table reads are lane-permuted copies read as one 16-byte load per lane
// (the texture-address unit, not the bytes, bounds the table traffic).
typedef float f4 __attribute__((ext_vector_type(4)));
// an 8-byte-aligned (cos, sin) moment pair, read from LDS as one 64-bit load
// whose immediate offset reaches the whole moment block
typedef float f2 __attribute__((ext_vector_type(2)));

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
  static constexpr int NW = L > 32 ? 4 : 1;          // waves per product
  static constexpr int NTH = 64 * NW;
  static constexpr int K = (L + 1) * (L + 1);
  static constexpr int NMP2 = 2 * L + 2;             // moment row: [m=0, -, cos 1, sin 1, .., cos L, sin L]
  static constexpr int EOP = 2 * 8 * NMP2;           // floats of one pass's combined moments
  static constexpr int NROW = (L + 1) * (L + 2) / 2 - (L + 1);  // output rows with m > 0
  static constexpr int NIT = (NROW + NTH - 1) / NTH;
  static constexpr int NMBP = (NMB + 1) / 2 * 2;     // phi blocks in the seed layout (even)
  static constexpr int NMR = L > 32 ? L / 32 : 1;    // 16-row blocks of analysis m-rows per class
  static constexpr int ASD = 6 * NMBP;               // seed offsets: analysis seeds,
  static constexpr int AST = ASD + 4 * NMR * NMBP;   //   analysis rotation steps,
  static constexpr int TWRN = AST + 4 * NMR;         //   total per lane
  // u-steps (two degrees each) of K-step s
  __host__ __device__ static constexpr int nu(int s) { return L / 2 - 4 * s; }
  // quad offset of the x block of m-pair c = 4 s + g (m = 2c + 1, 2c + 2): the
  // m = 0 block (L + 1 quads) first, then per pair 4 quads for each of the
  // nu(s) - g u-steps that hold a coefficient, + 1 pad.  Group g still runs
  // all nu(s) u-steps of its K-step: the last g of them read the next blocks
  // (finite values, whose theta-table entries are zero: l > L there), the
  // last blocks' a zero tail.
  __host__ __device__ static constexpr int xb(int c) {
    int q = L + 1;
    for (int i = 0; i < c; ++i) q += 4 * (nu(i / 4) - i % 4) + 1;
    return q;
  }
  // quads the image spans: the blocks and the reach of every group's reads
  __host__ __device__ static constexpr int x_quads() {
    int e = xb(L / 2);
    for (int c = 0; c < L / 2; ++c) e = e > xb(c) + 4 * nu(c / 4) ? e : xb(c) + 4 * nu(c / 4);
    return e;
  }
  static constexpr int XQ = x_quads();
  // u-step pairs before K-step s, and in all K-steps
  __host__ __device__ static constexpr int u2off(int s) { return s * (L / 4) - s * (s - 1); }
  static constexpr int TU2 = u2off(NKS);
  static constexpr int NV0 = (L + 1 + 7) / 8;          // m = 0 steps of 8 degrees
  static constexpr int NV0P = (NV0 + 3) / 4 * 4;
  static constexpr int NXK = (K + NTH - 1) / NTH;      // staged coefficients per thread
  static constexpr int NXKP = (NXK + 3) / 4 * 4;
};

// Sizes of the FFT variant (radix-2 phi transforms of length NF = N1 N2,
// NF >= 3L + 1: alias-free for the output moments |m| <= L of a product of
// phi-degree 2L).  Per pass, in LDS: the packed spectra of the 16 column
// nodes (NS = 2L + 1 entries each), the column-stage output T and the
// row-stage output T2 (which reuses the spectra's space); the row strides
// are padded by one complex entry against bank conflicts.
template <int L>
struct FGeo {
  static constexpr int NF = L <= 16 ? 64 : (L <= 32 ? 128 : 256);
  static constexpr int N1 = L <= 32 ? 8 : 16;  // column DFTs (over m1 / k1)
  static constexpr int N2 = NF / N1;           // row DFTs (over m2 / k2)
  static constexpr int NS = 2 * L + 1;         // packed spectrum of one node: m = 0..L, then -L..-1
  static constexpr int H2 = N2 / 2 + 1;        // forward row outputs of a real row
  static constexpr int TS = NF + 1;            // T column-node stride (complex entries)
  static constexpr int T2S = H2 * N1 + 1;      // T2 column-node stride
  static constexpr int AC = (16 * NS > 16 * T2S) ? 16 * NS : 16 * T2S;  // complex entries of A (spectra / T2)
  static constexpr int TC = 16 * TS;                                    // complex entries of T
  static_assert(NF >= 3 * L + 1 && NF == N1 * N2, "FFT length");
};

// exp(i 2 pi j / NF), j < NF (fp32 from fp64 compile-time values)
template <int NF>
struct TwTab {
  cpx v[NF];
};
template <int NF>
constexpr TwTab<NF> make_tw() {
  TwTab<NF> t{};
  for (int j = 0; j < NF; ++j) t.v[j] = cpx{ct_round(ct_cos2pi(j, NF)), ct_round(ct_sin2pi(j, NF))};
  return t;
}
__device__ const TwTab<64> kTw64 = make_tw<64>();
__device__ const TwTab<128> kTw128 = make_tw<128>();
__device__ const TwTab<256> kTw256 = make_tw<256>();
template <int NF>
__device__ __forceinline__ cpx tw_root(int j) {
  if constexpr (NF == 64) return kTw64.v[j];
  else if constexpr (NF == 128) return kTw128.v[j];
  else return kTw256.v[j];
}

// The value of lane i ^ 8: a DPP rotate by 8 within each 16-lane row (a
// plain VALU move, no LDS round trip as with a lane permute).  These
// exchanges run with all 64 lanes active (no divergent branch around them).
__device__ __forceinline__ float xor8(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x128 /* row_ror:8 */, 0xf, 0xf, true));
}

// The two rows of each 16-lane row pair (2k, 2k + 1), in every lane of the
// pair: gfx950's permlane16 swap of a value with itself leaves row 2k's
// value in the first result and row 2k + 1's in the second.  Likewise the
// two 32-lane halves (permlane32 swap).
__device__ __forceinline__ void row_pair(float v, float& even, float& odd) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  even = __uint_as_float(r[0]);
  odd = __uint_as_float(r[1]);
}
__device__ __forceinline__ float half_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// m = 0 theta synthesis reduction: lane (g, 8h + pi) holds the partial sum
// over l = g + 4h (mod 8); returns the value at the lane's column node (the
// node itself for h = 0, its mirror, odd l negated, for h = 1).
__device__ __forceinline__ float m0_reduce(float a, int h) {
  a += xor8(a);
  float e, o;  // rows g = 0, 2 (l = 0, 2 mod 4) and g = 1, 3 (l = 1, 3 mod 4)
  row_pair(a, e, o);
  const float node = half_sum(e + o), mirror = half_sum(e - o);
  return h ? mirror : node;
}

// cos/sin of m phi advanced by angle addition
__device__ __forceinline__ void rot(float& c, float& s, float cr, float sr) {
  const float cn = c * cr - s * sr;
  s = fmaf(s, cr, c * sr);
  c = cn;
}

// The per-wave view of one product: lane roles, the x image in LDS, the
// theta tables.
template <int L>
struct WaveCtx {
  using G = WGeo<L>;
  int lane, g, h, pi;
  float sg;  // +1 for h = 0 (node), -1 for h = 1 (mirror)
  const float4* xq;
  __amdgpu_buffer_rsrc_t SPr, S0r;
  const float* TWR;

  __device__ __forceinline__ WaveCtx(int lane_, const float4* xq_, const DevTables& t)
      : lane(lane_), g(lane_ >> 4), h((lane_ >> 3) & 1), pi(lane_ & 7), sg(h ? -1.0f : 1.0f), xq(xq_), TWR(t.TWR) {
    SPr = table_rsrc(t.SMP, G::PASSES * G::TU2 * 64 * 4);
    S0r = table_rsrc(t.SM0P, (G::PASSES + 1) * 64 * G::NV0P);
  }

  // m = 0 theta synthesis at the lane's column node (x1 and x2 cos parts);
  // pass = PASSES gives the poles.  Split into the table read and the sums so
  // that other loads can be issued in between.
  __device__ __forceinline__ void m0_load(int pass, float (&sv)[G::NV0P]) const {
    cfor<0, G::NV0P / 4>([&](auto V4) {
      constexpr int v4 = decltype(V4)::value;
      const float4 w = tload4_s(S0r, lane * G::NV0P * 4 + 16 * v4, pass * 64 * G::NV0P * 4);
      sv[4 * v4] = w.x;
      sv[4 * v4 + 1] = w.y;
      sv[4 * v4 + 2] = w.z;
      sv[4 * v4 + 3] = w.w;
    });
  }
  __device__ __forceinline__ void m0_finish(const float (&sv)[G::NV0P], float& a1, float& a2) const {
    float s1 = 0.0f, s2 = 0.0f;
    cfor<0, G::NV0>([&](auto V) {
      constexpr int v = decltype(V)::value;
      const int l = 8 * v + g + 4 * h;
      if (8 * v + 7 <= L || l <= L) {
        const float4 q = xq[l];
        s1 = fmaf(sv[v], q.x, s1);
        s2 = fmaf(sv[v], q.z, s2);
      }
    });
    a1 = m0_reduce(s1, h);
    a2 = m0_reduce(s2, h);
  }

  // One pass (8 mirror pairs, jp = 8 pu + pi + 1): theta synthesis, phi
  // synthesis contractions, sample products, phi analysis contractions.
  // Returns the analysis accumulators o[mr][type] (row 4g + r of m-row block
  // mr, column i) and zz, the m = 0 moment of the lane's column node.
  // FFT = true (the radix-FFT variant) runs the theta synthesis only and
  // writes each column node's packed phi spectrum to spec (phi_fft takes it
  // from there); o and zz are then not written.  K-steps S0..S1-1 only (the
  // m-parts 8 S0 + 1 .. 8 S1; the m = 0 part with S0 = 0): the four waves of
  // the L = 64 FFT kernel split one pass's synthesis this way.
  template <bool FFT = false, int S0 = 0, int S1 = G::NKS>
  __device__ __forceinline__ void pass(int pu, f4 (&o)[G::NMR][4], float& zz, float2* spec = nullptr) const {
    constexpr int NMB = G::NMB, NMBP = G::NMBP, NKS = G::NKS, TWRN = G::TWRN, NMR = G::NMR;
    static_assert(FFT || (S0 == 0 && S1 == NKS), "a K-step window only in the FFT variant");
    // loads first (m = 0 part, the first theta-table steps, the first phi
    // operands), then the m = 0 sums
    constexpr int D = 5;  // theta-table steps in flight
    constexpr int T0 = G::u2off(S0), T1 = G::u2off(S1);  // the window's table steps
    const int sbase = pu * G::TU2 * 64 * 16;
    float s0v[G::NV0P];
    if constexpr (S0 == 0) m0_load(pu, s0v);
    float4 sring[D];
    cfor<0, D>([&](auto T) {
      constexpr int tt = T0 + decltype(T)::value;
      if constexpr (tt < T1) sring[tt - T0] = tload4_s(SPr, lane * 16, sbase + tt * 64 * 16);
    });
    // synthesis operands twc[type][mb] of K-step 0 and the rotation by 8 phi_k
    const f4* seeds = reinterpret_cast<const f4*>(TWR + lane * TWRN);
    float twc[4][NMB], r8c[NMB], r8s[NMB];
    if constexpr (!FFT) {
      float sd[6 * NMBP];
      cfor<0, 6 * NMBP / 4>([&](auto Q4) {
        constexpr int q4 = decltype(Q4)::value;
        const f4 v = seeds[q4];
        cfor<0, 4>([&](auto E) { sd[4 * q4 + decltype(E)::value] = v[decltype(E)::value]; });
      });
      cfor<0, NMB>([&](auto MB) {
        constexpr int mb = decltype(MB)::value;
        twc[0][mb] = sd[6 * mb + 0];  // cos, even m
        twc[2][mb] = sd[6 * mb + 1];  // sin, even m
        twc[1][mb] = sd[6 * mb + 2];  // cos, odd m
        twc[3][mb] = sd[6 * mb + 3];  // sin, odd m
        r8c[mb] = sd[6 * mb + 4];
        r8s[mb] = sd[6 * mb + 5];
      });
    }
    float c1 = 0.0f, c2 = 0.0f;
    if constexpr (S0 == 0) m0_finish(s0v, c1, c2);

    // ---- 1 + 2a. theta synthesis feeding the phi-synthesis contractions
    f4 acc[2][NMB][4];  // [input][k block][type]
    // the FFT variant's packed spectrum of the lane's column node (see phi_fft)
    float2* const sc = spec + (8 * h + pi) * FGeo<L>::NS;
    if constexpr (FFT && S0 == 0) {
      if (g == 0) sc[0] = make_float2(2.0f * c1, 2.0f * c2);
    }
    if constexpr (!FFT) cfor<0, NMB>([&](auto MB) {
      constexpr int mb = decltype(MB)::value;
      acc[0][mb][0] = f4{c1, c1, c1, c1};  // m = 0 enters every pe sample
      acc[1][mb][0] = f4{c2, c2, c2, c2};
      cfor<1, 4>([&](auto TY) {
        acc[0][mb][decltype(TY)::value] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        acc[1][mb][decltype(TY)::value] = f4{0.0f, 0.0f, 0.0f, 0.0f};
      });
    });
    float asd[NMR][4 * NMB];  // analysis seeds, read during the last K-step
    f4 ast[NMR];
    cfor<S0, S1>([&](auto SS) {
      constexpr int s = decltype(SS)::value;
      // the x block of m-pair c = 4 s + g: xb(4 s + g) = xb(4 s) + g (4 nu(s) + 1)
      // - 2 g (g - 1), written so that only the g terms are left to run time
      const int xo = G::xb(4 * s) + g * (4 * G::nu(s) + 1) - 2 * g * (g - 1);
      // this lane's parity: h = 0 takes (mo, l_a) and (mo+1, l_b), h = 1 (mo, l_b) and (mo+1, l_a)
      const float4* xa = xq + xo + h;
      const float4* xe = xq + xo + 3 - h;
      f4 Vo = {0.0f, 0.0f, 0.0f, 0.0f}, Ve = Vo;
      cfor<0, G::nu(s) / 2>([&](auto U2) {
        constexpr int u2 = decltype(U2)::value, tt = G::u2off(s) + u2;
        const float4 sv = sring[(tt - T0) % D];
        if constexpr (tt + D < T1) sring[(tt - T0) % D] = tload4_s(SPr, lane * 16, sbase + (tt + D) * 64 * 16);
        cfor<0, 2>([&](auto E) {
          constexpr int u = 2 * u2 + decltype(E)::value;
          const float so = E == 0 ? sv.x : sv.z, se = E == 0 ? sv.y : sv.w;
          const float4 qa = xa[4 * u], qe = xe[4 * u];
          Vo += so * f4{qa.x, qa.y, qa.z, qa.w};
          Ve += se * f4{qe.x, qe.y, qe.z, qe.w};
        });
        __builtin_amdgcn_sched_barrier(0);  // keep the prefetch distance
      });
      if constexpr (s == NKS - 1 && !FFT) {
        cfor<0, NMR>([&](auto MR) {
          constexpr int mr = decltype(MR)::value;
          cfor<0, NMB>([&](auto Q4) {
            constexpr int q4 = decltype(Q4)::value;
            const f4 v = seeds[(G::ASD + 4 * (mr * NMBP + q4)) / 4];
            cfor<0, 4>([&](auto E) { asd[mr][4 * q4 + decltype(E)::value] = v[decltype(E)::value]; });
          });
          ast[mr] = seeds[(G::AST + 4 * mr) / 4];
        });
      }
      // column value: node jp (h = 0: own even + partner odd) or its mirror
      // (h = 1: partner even - own odd); sg * v + partner is exact for sg = +-1
      f4 Bo, Be;
      cfor<0, 4>([&](auto C) {
        constexpr int cc = decltype(C)::value;
        Bo[cc] = fmaf(sg, Vo[cc], xor8(Vo[cc]));
        Be[cc] = fmaf(sg, Ve[cc], xor8(Ve[cc]));
      });
      if constexpr (FFT) {
        // B = (x1 cos, x1 sin, x2 cos, x2 sin) of m-parts mo = 8 s + 2 g + 1
        // (Bo) and mo + 1 (Be): twice the packed coefficients
        // d_{+m} = (a1 + b2, a2 - b1), d_{-m} = (a1 - b2, a2 + b1)
        constexpr int NS = FGeo<L>::NS;
        const int mo = 8 * s + 2 * g + 1;
        sc[mo] = make_float2(Bo[0] + Bo[3], Bo[2] - Bo[1]);
        sc[NS - mo] = make_float2(Bo[0] - Bo[3], Bo[2] + Bo[1]);
        sc[mo + 1] = make_float2(Be[0] + Be[3], Be[2] - Be[1]);
        sc[NS - mo - 1] = make_float2(Be[0] - Be[3], Be[2] + Be[1]);
      } else {
        cfor<0, NMB>([&](auto MB) {
          constexpr int mb = decltype(MB)::value;
          cfor<0, 2>([&](auto TI) {
            constexpr int ti = decltype(TI)::value;
            acc[ti][mb][0] = mfma4(twc[0][mb], Be[2 * ti], acc[ti][mb][0]);
            acc[ti][mb][1] = mfma4(twc[1][mb], Bo[2 * ti], acc[ti][mb][1]);
            acc[ti][mb][2] = mfma4(twc[2][mb], Be[2 * ti + 1], acc[ti][mb][2]);
            acc[ti][mb][3] = mfma4(twc[3][mb], Bo[2 * ti + 1], acc[ti][mb][3]);
          });
        });
      }
      if constexpr (s + 1 < NKS && !FFT) {
        // next K-step: m -> m + 8
        cfor<0, NMB>([&](auto MB) {
          constexpr int mb = decltype(MB)::value;
          rot(twc[0][mb], twc[2][mb], r8c[mb], r8s[mb]);
          rot(twc[1][mb], twc[3][mb], r8c[mb], r8s[mb]);
        });
      }
    });

    if constexpr (FFT) return;
    // ---- 2b. sample products, folded over the 4-point sets.  The samples at
    // k, -k, 2Q + k, 2Q - k are pe + po +- (qe + qo) and pe - po +- (qe - qo);
    // summed over the four points the product folds to 4 (pe pe' + po po' +
    // qe qe' + qo qo') (even-m cos), 4 (pe po' + po pe' + qe qo' + qo qe')
    // (odd-m cos), 4 (pe qe' + po qo' + qe pe' + qo po') (even-m sin) and
    // 4 (pe qo' + po qe' + qe po' + qo pe') (odd-m sin), so no sample is
    // formed; the 4 goes into the analysis weight (coinciding points at k = 0
    // and Q are counted twice there and weighted 1/2).  At L = 64 (256
    // registers) the samples are formed and folded instead (weights 1/2 and
    // 1), which keeps fewer values live; the result is the same.
    cfor<0, NMB>([&](auto MB) {
      constexpr int mb = decltype(MB)::value;
      const f4 pe1 = acc[0][mb][0], po1 = acc[0][mb][1], qe1 = acc[0][mb][2], qo1 = acc[0][mb][3];
      const f4 pe2 = acc[1][mb][0], po2 = acc[1][mb][1], qe2 = acc[1][mb][2], qo2 = acc[1][mb][3];
      if constexpr (L < 64) {
        acc[0][mb][0] = pe1 * pe2 + po1 * po2 + qe1 * qe2 + qo1 * qo2;
        acc[0][mb][1] = pe1 * po2 + po1 * pe2 + qe1 * qo2 + qo1 * qe2;
        acc[0][mb][2] = pe1 * qe2 + po1 * qo2 + qe1 * pe2 + qo1 * po2;
        acc[0][mb][3] = pe1 * qo2 + po1 * qe2 + qe1 * po2 + qo1 * pe2;
      } else {
        const f4 s1 = pe1 + po1, d1 = pe1 - po1, s2 = qe1 + qo1, d2 = qe1 - qo1;
        const f4 t1 = pe2 + po2, u1 = pe2 - po2, t2 = qe2 + qo2, u2 = qe2 - qo2;
        const f4 hk = (s1 + s2) * (t1 + t2), hmk = (s1 - s2) * (t1 - t2);
        const f4 hpk = (d1 + d2) * (u1 + u2), hpmk = (d1 - d2) * (u1 - u2);
        const f4 a = hk + hmk, b = hpk + hpmk, dd = hk - hmk, ee = hpk - hpmk;
        acc[0][mb][0] = a + b;
        acc[0][mb][1] = a - b;
        acc[0][mb][2] = dd + ee;
        acc[0][mb][3] = dd - ee;
      }
    });

    // ---- 2c. phi analysis contractions; operands per k block from the seeds:
    // w_k trig(m phi_k) (the seeds hold fold * trig), k = 16 mb + 4 r + g
    // (the synthesis rows are ordered so that register r of lane group g
    // holds that sample), m = 2(16 mr + i) + 2 (even types) or + 1 (odd
    // types).  A contraction whose four samples all lie past Q (weight zero)
    // is skipped.
    cfor<0, NMR>([&](auto MR) {
      cfor<0, 4>([&](auto TY) { o[decltype(MR)::value][decltype(TY)::value] = f4{0.0f, 0.0f, 0.0f, 0.0f}; });
    });
    zz = 0.0f;
    cfor<0, NMB>([&](auto MB) {
      constexpr int mb = decltype(MB)::value;
      cfor<0, NMR>([&](auto MR) {
        constexpr int mr = decltype(MR)::value;
        float ce = asd[mr][4 * mb + 0], se = asd[mr][4 * mb + 1], co = asd[mr][4 * mb + 2], so = asd[mr][4 * mb + 3];
        cfor<0, 4>([&](auto R) {
          constexpr int r = decltype(R)::value;
          if constexpr (16 * mb + 4 * r <= G::Q) {
            if constexpr (r > 0) {
              rot(ce, se, ast[mr].x, ast[mr].y);
              rot(co, so, ast[mr].z, ast[mr].w);
            }
            // the seeds carry the weight shared by all samples (fold: see the
            // sample products); only a contraction holding k = 0, Q or samples
            // past Q scales its operands by 1/2 or 0 per lane
            constexpr float fold = L < 64 ? 4.0f : 1.0f;
            if constexpr (16 * mb + 4 * r > 0 && 16 * mb + 4 * r + 3 < G::Q) {
              o[mr][0] = mfma4(ce, acc[0][mb][0][r], o[mr][0]);
              o[mr][1] = mfma4(co, acc[0][mb][1][r], o[mr][1]);
              o[mr][2] = mfma4(se, acc[0][mb][2][r], o[mr][2]);
              o[mr][3] = mfma4(so, acc[0][mb][3][r], o[mr][3]);
              if constexpr (mr == 0) zz = fmaf(fold, acc[0][mb][0][r], zz);
            } else {
              const int k = 16 * mb + 4 * r + g;
              const float wr = k > G::Q ? 0.0f : (k == 0 || k == G::Q) ? 0.5f : 1.0f;
              o[mr][0] = mfma4(wr * ce, acc[0][mb][0][r], o[mr][0]);
              o[mr][1] = mfma4(wr * co, acc[0][mb][1][r], o[mr][1]);
              o[mr][2] = mfma4(wr * se, acc[0][mb][2][r], o[mr][2]);
              o[mr][3] = mfma4(wr * so, acc[0][mb][3][r], o[mr][3]);
              if constexpr (mr == 0) zz = fmaf(wr * fold, acc[0][mb][0][r], zz);
            }
          }
        });
      });
    });
    {
      float ze, zo;
      row_pair(zz, ze, zo);
      zz = half_sum(ze + zo);
    }
  }

  // ---- 3. mirror combination into LDS, eo[parity][pi][slot]: parity 0 =
  // C(jp) + C(NT - jp), 1 = C(jp) - C(NT - jp); slot 0 = m 0, 2m = cos m,
  // 2m + 1 = sin m
  __device__ __forceinline__ void store_moments(float* eo, const f4 (&o)[G::NMR][4], float zz) const {
    float* const eoh = eo + (h * 8 + pi) * G::NMP2;
    cfor<0, G::NMR>([&](auto MR) {
      constexpr int mr = decltype(MR)::value;
      cfor<0, 2>([&](auto PAR) {
        constexpr int odd = decltype(PAR)::value;  // types odd (cos), odd + 2 (sin)
        cfor<0, 4>([&](auto R) {
          constexpr int r = decltype(R)::value;
          const int m = 2 * (16 * mr + 4 * g + r) + (odd ? 1 : 2);
          const float vc = fmaf(sg, o[mr][odd][r], xor8(o[mr][odd][r]));
          const float vs = fmaf(sg, o[mr][odd + 2][r], xor8(o[mr][odd + 2][r]));
          // m-rows past L exist only at L = 16 (16 rows per class)
          if (L != 16 || m <= L) *reinterpret_cast<float2*>(eoh + 2 * m) = make_float2(vc, vs);
        });
      });
    });
    const float vz = fmaf(sg, zz, xor8(zz));
    if (g == 0) eoh[0] = vz;
  }

  // ---- 2 (FFT variant). The phi transforms of one pass by radix-2 FFTs of
  // length NF = N1 N2 (four-step split, index n = N2 n1 + n2 on the
  // spectrum side, k = k1 + N1 k2 on the sample side).  A holds, for each of
  // the 16 column nodes, twice the packed spectrum d_m = c1_m + i c2_m of the
  // two inputs (c_m the complex Fourier coefficients of the node's phi
  // function, |m| <= L), so that one inverse transform gives 2 (f1 + i f2) at
  // the NF samples and the product is Re * Im.  Then:
  //   1. columns (node, n2): inverse DFT over n1 of d[N2 n1 + n2], times
  //      exp(+i 2 pi n2 k1 / NF)                                    -> T[node][k1][n2]
  //   2. rows (node, k1): inverse DFT over n2 (the samples k1 + N1 k2), the
  //      product g, forward DFT over k2 of the real g (outputs m2 <= N2/2),
  //      times exp(-i 2 pi m2 k1 / NF)                              -> T2[node][m2][k1]
  //   3. columns (pair, m2): forward DFT over k1 of the node's and the
  //      mirror's column; the outputs with |m| <= L are the moments
  //      sum_k g cos(m p_k) and sum_k g sin(m p_k), combined into the sum and
  //      difference of the mirror nodes (the layout store_moments writes).
  // The moments are rescaled to the plan's NP-point convention (NP / NF,
  // and 1/8 for the factors 2 of the packing and of the real transform).
  __device__ __forceinline__ void phi_fft(float* eo, float2* A, float2* T) const {
    using F = FGeo<L>;
    constexpr int NF = F::NF, N1 = F::N1, N2 = F::N2, NS = F::NS, H2 = F::H2, TS = F::TS, T2S = F::T2S;
    const int ci = lane & 15, q = lane >> 4;
    // 1. columns n2 = q + 4 t of node ci
    cfor<0, N2 / 4>([&](auto TT) {
      const int n2 = q + 4 * decltype(TT)::value;
      const float2* sp = A + ci * NS;
      cpx a[N1];
      cfor<0, N1>([&](auto M1) {
        constexpr int lo = N2 * decltype(M1)::value, hi = lo + N2 - 1;
        // spectrum index n = lo + n2 holds m = n (n <= L) or m = n - NF (n >= NF - L)
        if constexpr (hi <= L) {
          const float2 v = sp[lo + n2];
          a[decltype(M1)::value] = {v.x, v.y};
        } else if constexpr (lo >= NF - L) {
          const float2 v = sp[NS - NF + lo + n2];
          a[decltype(M1)::value] = {v.x, v.y};
        } else if constexpr (lo <= L) {
          const int n = lo + n2;
          const float2 v = sp[n <= L ? n : 0];
          a[decltype(M1)::value] = n <= L ? cpx{v.x, v.y} : cpx{0.0f, 0.0f};
        } else if constexpr (hi >= NF - L) {
          const int n = lo + n2;
          const float2 v = sp[n >= NF - L ? NS - NF + n : 0];
          a[decltype(M1)::value] = n >= NF - L ? cpx{v.x, v.y} : cpx{0.0f, 0.0f};
        } else {
          a[decltype(M1)::value] = {0.0f, 0.0f};
        }
      });
      fft_reg<N1, +1>(a);
      cpx w[N1];
      cpowers<N1>(tw_root<NF>(n2), w);
      float2* tp = T + ci * TS + n2;
      cfor<0, N1>([&](auto K1) {
        constexpr int k1 = decltype(K1)::value;
        const cpx v = k1 == 0 ? a[0] : cmul(a[k1], w[k1]);
        tp[k1 * N2] = make_float2(v.re, v.im);
      });
    });
    __syncthreads();
    // 2. rows k1 = q + 4 t of node ci
    cfor<0, N1 / 4>([&](auto TT) {
      const int k1 = q + 4 * decltype(TT)::value;
      const float2* tp = T + ci * TS + k1 * N2;
      cpx a[N2];
      cfor<0, N2>([&](auto M2) {
        const float2 v = tp[decltype(M2)::value];
        a[decltype(M2)::value] = {v.x, v.y};
      });
      fft_reg<N2, +1>(a);
      float gv[N2];
      cfor<0, N2>([&](auto K2) { gv[decltype(K2)::value] = a[decltype(K2)::value].re * a[decltype(K2)::value].im; });
      cpx X2[H2];
      rfft2_fwd<N2>(gv, X2);
      cpx w[H2];
      cpowers<H2>(cconj(tw_root<NF>(k1)), w);
      float2* t2 = A + ci * T2S + k1;
      cfor<0, H2>([&](auto M2) {
        constexpr int m2 = decltype(M2)::value;
        const cpx v = m2 == 0 ? X2[0] : cmul(X2[m2], w[m2]);
        t2[m2 * N1] = make_float2(v.re, v.im);
      });
    });
    __syncthreads();
    // 3. columns m2 of pair pp (node column pp, mirror column 8 + pp); lanes
    // with m2 = 0 also take the column N2 / 2
    const int pp = lane & 7, cm = lane >> 3;
    constexpr float scale = float(G::NP) / (8.0f * float(NF));
    auto column = [&](int m2) {
      cpx bn[N1], bm[N1];
      const float2* t2n = A + pp * T2S + m2 * N1;
      const float2* t2m = A + (8 + pp) * T2S + m2 * N1;
      cfor<0, N1>([&](auto K1) {
        constexpr int k1 = decltype(K1)::value;
        const float2 u = t2n[k1], v = t2m[k1];
        bn[k1] = {u.x, u.y};
        bm[k1] = {v.x, v.y};
      });
      fft_reg<N1, -1>(bn);
      fft_reg<N1, -1>(bm);
      float* es = eo + pp * G::NMP2;          // sum of the mirror nodes
      float* ed = eo + (8 + pp) * G::NMP2;    // difference
      // moment m from X = sum_k g exp(-i m p_k): cos part Re X, sin part -Im X
      auto emit = [&](int m, cpx xn, cpx xm) {
        es[2 * m] = (xn.re + xm.re) * scale;
        ed[2 * m] = (xn.re - xm.re) * scale;
        if (m > 0) {
          es[2 * m + 1] = -(xn.im + xm.im) * scale;
          ed[2 * m + 1] = -(xn.im - xm.im) * scale;
        }
      };
      // m = N2 m1 + m2 <= L from output m1; m = N2 a - m2 <= L (0 < m2 < N2 / 2)
      // from output N1 - a, conjugated (the transform of a real g)
      cfor<0, N1>([&](auto M1) {
        constexpr int m1 = decltype(M1)::value;
        if constexpr (N2 * m1 <= L) {
          const int m = N2 * m1 + m2;
          if (m <= L) emit(m, bn[m1], bm[m1]);
        }
      });
      if (m2 != 0 && 2 * m2 != N2) {
        cfor<1, N1>([&](auto AA) {
          constexpr int aa = decltype(AA)::value;
          if constexpr (N2 * aa - N2 / 2 < L + 1) {
            const int m = N2 * aa - m2;
            if (m <= L) emit(m, cconj(bn[N1 - aa]), cconj(bm[N1 - aa]));
          }
        });
      }
    };
    if (cm < N2 / 2) column(cm);
    if (cm == 0) column(N2 / 2);
  }
};

// The phi transforms of one pass by radix-2 FFTs, shared by the NTH threads
// of a multi-wave workgroup (the L = 64 FFT kernel), one half pass at a time
// (half h: the mirror pairs 4 h .. 4 h + 3, i.e. the columns 4 h + j and
// 8 + 4 h + j, j < 4).  The steps of WaveCtx::phi_fft with 8 nodes: (1)
// column tasks (node, n2), (2) row tasks (node, k1), their results first held
// in registers so that T2 can take T's place, (3) forward column tasks
// (pair, m2).  A holds the 16 columns' packed spectra; T the half's column
// outputs, then its T2.  All NTH threads call it (it has barriers).
template <int L>
__device__ __forceinline__ void phi_fft_half(int tid, int half, float* eo, const float2* A, float2* T) {
  using F = FGeo<L>;
  using G = WGeo<L>;
  constexpr int NF = F::NF, N1 = F::N1, N2 = F::N2, NS = F::NS, H2 = F::H2, TS = F::TS, T2S = F::T2S;
  static_assert(8 * N2 <= G::NTH && 8 * N1 <= G::NTH, "one column or row task per thread");
  auto col_of = [&](int nh) { return nh < 4 ? 4 * half + nh : 8 + 4 * half + (nh - 4); };
  // 1. columns: node nh, n2
  if (tid < 8 * N2) {
    const int nh = tid & 7, n2 = tid >> 3;
    const float2* sp = A + col_of(nh) * NS;
    cpx a[N1];
    cfor<0, N1>([&](auto M1) {
      constexpr int lo = N2 * decltype(M1)::value, hi = lo + N2 - 1;
      if constexpr (hi <= L) {
        const float2 v = sp[lo + n2];
        a[decltype(M1)::value] = {v.x, v.y};
      } else if constexpr (lo >= NF - L) {
        const float2 v = sp[NS - NF + lo + n2];
        a[decltype(M1)::value] = {v.x, v.y};
      } else if constexpr (lo <= L) {
        const int n = lo + n2;
        const float2 v = sp[n <= L ? n : 0];
        a[decltype(M1)::value] = n <= L ? cpx{v.x, v.y} : cpx{0.0f, 0.0f};
      } else if constexpr (hi >= NF - L) {
        const int n = lo + n2;
        const float2 v = sp[n >= NF - L ? NS - NF + n : 0];
        a[decltype(M1)::value] = n >= NF - L ? cpx{v.x, v.y} : cpx{0.0f, 0.0f};
      } else {
        a[decltype(M1)::value] = {0.0f, 0.0f};
      }
    });
    fft_reg<N1, +1>(a);
    cpx w[N1];
    cpowers<N1>(tw_root<NF>(n2), w);
    float2* tp = T + nh * TS + n2;
    cfor<0, N1>([&](auto K1) {
      constexpr int k1 = decltype(K1)::value;
      const cpx v = k1 == 0 ? a[0] : cmul(a[k1], w[k1]);
      tp[k1 * N2] = make_float2(v.re, v.im);
    });
  }
  __syncthreads();
  // 2. rows: node nh, k1 -> forward outputs m2 <= N2 / 2 in registers
  cpx X2[H2];
  const int rnh = tid & 7, rk1 = tid >> 3;
  if (tid < 8 * N1) {
    const float2* tp = T + rnh * TS + rk1 * N2;
    cpx a[N2];
    cfor<0, N2>([&](auto M2) {
      const float2 v = tp[decltype(M2)::value];
      a[decltype(M2)::value] = {v.x, v.y};
    });
    fft_reg<N2, +1>(a);
    float gv[N2];
    cfor<0, N2>([&](auto K2) { gv[decltype(K2)::value] = a[decltype(K2)::value].re * a[decltype(K2)::value].im; });
    rfft2_fwd<N2>(gv, X2);
    cpx w[H2];
    cpowers<H2>(cconj(tw_root<NF>(rk1)), w);
    cfor<1, H2>([&](auto M2) { X2[decltype(M2)::value] = cmul(X2[decltype(M2)::value], w[decltype(M2)::value]); });
  }
  __syncthreads();  // every row of T is read: T2 takes its place
  if (tid < 8 * N1) {
    float2* t2 = T + rnh * T2S + rk1;
    cfor<0, H2>([&](auto M2) { t2[decltype(M2)::value * N1] = make_float2(X2[decltype(M2)::value].re,
                                                                           X2[decltype(M2)::value].im); });
  }
  __syncthreads();
  // 3. forward columns: pair j (node j, mirror 4 + j), m2; threads 4 * H2
  if (tid < 4 * H2) {
    const int j = tid & 3, m2 = tid >> 2;
    const int pp = 4 * half + j;
    constexpr float scale = float(G::NP) / (8.0f * float(NF));
    cpx bn[N1], bm[N1];
    const float2* t2n = T + j * T2S + m2 * N1;
    const float2* t2m = T + (4 + j) * T2S + m2 * N1;
    cfor<0, N1>([&](auto K1) {
      constexpr int k1 = decltype(K1)::value;
      const float2 u = t2n[k1], v = t2m[k1];
      bn[k1] = {u.x, u.y};
      bm[k1] = {v.x, v.y};
    });
    fft_reg<N1, -1>(bn);
    fft_reg<N1, -1>(bm);
    float* es = eo + pp * G::NMP2;        // sum of the mirror nodes
    float* ed = eo + (8 + pp) * G::NMP2;  // difference
    auto emit = [&](int m, cpx xn, cpx xm) {
      es[2 * m] = (xn.re + xm.re) * scale;
      ed[2 * m] = (xn.re - xm.re) * scale;
      if (m > 0) {
        es[2 * m + 1] = -(xn.im + xm.im) * scale;
        ed[2 * m + 1] = -(xn.im - xm.im) * scale;
      }
    };
    cfor<0, N1>([&](auto M1) {
      constexpr int m1 = decltype(M1)::value;
      if constexpr (N2 * m1 <= L) {
        const int m = N2 * m1 + m2;
        if (m <= L) emit(m, bn[m1], bm[m1]);
      }
    });
    if (m2 != 0 && 2 * m2 != N2) {
      cfor<1, N1>([&](auto AA) {
        constexpr int aa = decltype(AA)::value;
        if constexpr (N2 * aa - N2 / 2 < L + 1) {
          const int m = N2 * aa - m2;
          if (m <= L) emit(m, cconj(bn[N1 - aa]), cconj(bm[N1 - aa]));
        }
      });
    }
  }
  __syncthreads();
}

// x into the LDS image (quads x1 cos, x1 sin, x2 cos, x2 sin) by the NTH
// threads of the workgroup: every load is issued before the first wait
// PAD: the rows hold k1 / k2 <= K coefficients (inputs of lower degree read
// as degree-L vectors with zeros above their own degrees).
template <int L, bool WGT, bool PAD = false, typename T1, typename T2>
__device__ __forceinline__ void stage_x(float* xs, const T1* x1, const T2* x2, int64_t P, int tid,
                                        const int* xmap, const DegWeights& wt, int k1 = 0, int k2 = 0) {
  using G = WGeo<L>;
  constexpr int K = G::K, NTH = G::NTH, NXK = G::NXK, NXKP = G::NXKP;
  int slot[NXKP];
  cfor<0, NXKP / 4>([&](auto K4) {
    constexpr int k4 = decltype(K4)::value;
    const int4 v = reinterpret_cast<const int4*>(xmap + tid * NXKP)[k4];
    slot[4 * k4] = v.x;
    slot[4 * k4 + 1] = v.y;
    slot[4 * k4 + 2] = v.z;
    slot[4 * k4 + 3] = v.w;
  });
  float v1[NXK], v2[NXK];
  const T1* const r1 = x1 + P * (PAD ? k1 : K);  // this product's rows (wave-uniform)
  const T2* const r2 = x2 + P * (PAD ? k2 : K);
  cfor<0, NXK>([&](auto KK) {
    constexpr int k = decltype(KK)::value;
    const int e = tid + NTH * k;
    if (NTH * k + NTH - 1 < K || e < K) {
      if constexpr (PAD) {
        // in-bounds index first, then the select: no load past a row's end
        const float a = ld_row(r1, unsigned(e < k1 ? e : 0));
        const float b = ld_row(r2, unsigned(e < k2 ? e : 0));
        v1[k] = e < k1 ? a : 0.0f;
        v2[k] = e < k2 ? b : 0.0f;
      } else {
        v1[k] = ld_row(r1, unsigned(e));
        v2[k] = ld_row(r2, unsigned(e));
      }
    }
  });
  if constexpr (WGT) {
    // per-degree weights of this product (Sec. 3.1), gathered per coefficient
    const int64_t row = weight_row(wt, P) * (L + 1);
    cfor<0, NXK>([&](auto KK) {
      constexpr int k = decltype(KK)::value;
      const int e = tid + NTH * k;
      if (NTH * k + NTH - 1 < K || e < K) {
        const int l = degree_of(e);
        if (wt.w1) v1[k] *= wt.w1[row + l];
        if (wt.w2) v2[k] *= wt.w2[row + l];
      }
    });
  }
  cfor<0, G::XQ / NTH>([&](auto Z) {
    reinterpret_cast<float4*>(xs)[tid + NTH * decltype(Z)::value] = make_float4(0.f, 0.f, 0.f, 0.f);
  });
  if (tid < G::XQ % NTH) reinterpret_cast<float4*>(xs)[tid + NTH * (G::XQ / NTH)] = make_float4(0.f, 0.f, 0.f, 0.f);
  __syncthreads();
  cfor<0, NXK>([&](auto KK) {
    constexpr int k = decltype(KK)::value;
    if (NTH * k + NTH - 1 < K || tid + NTH * k < K) {
      xs[slot[k]] = v1[k];
      xs[slot[k] + 2] = v2[k];
    }
  });
  __syncthreads();
}

// Output coefficient i of product P: rows of K (unpadded) or of ko values,
// of which those past ko (degrees above the plan's Lout) are not written.
template <bool PAD, int K>
__device__ __forceinline__ void store_out(float* y, int64_t P, int ko, int i, float v) {
  if constexpr (PAD) {
    if (i < ko) y[P * ko + i] = v;
  } else {
    y[P * K + i] = v;
  }
}
// The same from the product's own output row yr (wave-uniform) and the
// coefficient's byte offset in it.
template <bool PAD>
__device__ __forceinline__ void store_row(float* yr, int ko, unsigned byte_off, float v) {
  if constexpr (PAD) {
    if (byte_off < 4u * unsigned(ko)) st_row_bytes(yr, byte_off, v);
  } else {
    st_row_bytes(yr, byte_off, v);
  }
}
// A padded plan's outputs above degree L (when its Lout > L) are zeros.
template <int K>
__device__ __forceinline__ void zero_tail(float* y, int64_t P, int ko, int tid, int nth) {
  for (int i = K + tid; i < ko; i += nth) y[P * ko + i] = 0.0f;
}

// degree l and order m > 0 of the q-th output row with m > 0 in tri order
__device__ __forceinline__ void row_lm(int q, int& l, int& m) {
  l = int((sqrtf(8.0f * float(q) + 1.0f) + 1.0f) * 0.5f);
  l -= (l * (l - 1) / 2 > q) ? 1 : 0;
  l += ((l + 1) * l / 2 <= q) ? 1 : 0;
  m = q - l * (l - 1) / 2 + 1;
}

// LDS offset, within one pass's combined moments, of every theta-analysis
// row q = lane + 64 it (rows with m > 0 in tri order; parity of l + m picks
// the sum or the difference of the mirror nodes, 2 m the m-part): a
// compile-time table, read once per pass, instead of inverting the
// triangular index in every pass.
template <int L>
struct RowErTab {
  int v[WGeo<L>::NIT * 64];
};
template <int L>
constexpr RowErTab<L> make_row_er() {
  using G = WGeo<L>;
  RowErTab<L> t{};
  int q = 0;
  for (int l = 1; l <= L; ++l)
    for (int m = 1; m <= l; ++m, ++q) t.v[q] = ((l + m) & 1) * 8 * G::NMP2 + 2 * m;
  return t;
}
__device__ const RowErTab<16> kRowEr16 = make_row_er<16>();
__device__ const RowErTab<32> kRowEr32 = make_row_er<32>();
template <int L>
__device__ __forceinline__ const int* row_er_table() {
  if constexpr (L == 16) {
    return kRowEr16.v;
  } else {
    return kRowEr32.v;
  }
}
// Output byte offsets of the same rows: the (l, m) coefficient in the low
// half, the (l, -m) one in the high half (4 (l^2 + l +- m) < 2^16 for
// L <= 32); zero past the last row.
template <int L>
struct RowOutTab {
  unsigned v[WGeo<L>::NIT * 64];
};
template <int L>
constexpr RowOutTab<L> make_row_out() {
  RowOutTab<L> t{};
  int q = 0;
  for (int l = 1; l <= L; ++l)
    for (int m = 1; m <= l; ++m, ++q)
      t.v[q] = unsigned(4 * (l * l + l + m)) | (unsigned(4 * (l * l + l - m)) << 16);
  return t;
}
__device__ const RowOutTab<16> kRowOut16 = make_row_out<16>();
__device__ const RowOutTab<32> kRowOut32 = make_row_out<32>();
template <int L>
__device__ __forceinline__ const unsigned* row_out_table() {
  static_assert(4 * ((L + 1) * (L + 1)) <= 65536, "byte offsets must fit 16 bits");
  if constexpr (L == 16) {
    return kRowOut16.v;
  } else {
    return kRowOut32.v;
  }
}

// L in {16, 32}: one wave per product; theta analysis accumulates in
// registers after every pass.  FFT: the phi transforms by radix-2 FFTs
// (phi_fft) instead of the direct-DFT contractions on the matrix cores.
// PAD: a plan of lower degrees padded to L (rows of k1, k2 inputs, ko outputs;
// see stage_x and store_row).
template <int L, typename T1, typename T2, bool WGT, bool FFT, bool PAD = false>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(FFT ? 1 : 3))) void k_full_wave(
    const T1* __restrict__ x1, const T2* __restrict__ x2, float* __restrict__ y, int64_t n, DevTables t,
    DegWeights wt, int k1, int k2, int ko) {
  using G = WGeo<L>;
  static_assert(L % 16 == 0 && L <= 32, "L must be 16 or 32");
  constexpr int NJ = G::NJ, NP = G::NP;
  constexpr int NMP2 = G::NMP2, K = G::K, PASSES = G::PASSES, NROW = G::NROW, NIT = G::NIT;
  // the moments first: their reads then carry small immediate offsets
  constexpr int FFTF = FFT ? 2 * (FGeo<L>::AC + FGeo<L>::TC) : 0;  // the FFT variant's spectra and T
  __shared__ __align__(16) float lds[G::EOP + G::XQ * 4 + FFTF];
  lds_poison(lds, G::EOP + G::XQ * 4 + FFTF);
  float* const eo = lds;
  float* const xs = lds + G::EOP;
  float2* const fa = reinterpret_cast<float2*>(lds + G::EOP + G::XQ * 4);
  float2* const ft = fa + (FFT ? FGeo<L>::AC : 0);

  const int lane = threadIdx.x;
  if (int64_t(blockIdx.x) >= n) return;  // whole-wave exit (one product per workgroup)
  const int64_t P = xcd_product(blockIdx.x, n);
  stage_x<L, WGT, PAD>(xs, x1, x2, P, lane, t.XMAP, wt, k1, k2);

  const __amdgpu_buffer_rsrc_t WPr = table_rsrc(t.WP, PASSES * (NIT + 1) * 64 * 8);
  const __amdgpu_buffer_rsrc_t Wr = table_rsrc(t.WT, NJ * t.ntW);
  // theta-analysis rows: tri(l, 0) with l = lane (l <= L), and the rows with
  // m > 0 numbered q = lane + 64 it
  float y0 = 0.0f, yc[NIT], ys[NIT];
  const int wr0 = (lane * (lane + 1) / 2) * 4;
  cfor<0, NIT>([&](auto IT) {
    yc[decltype(IT)::value] = 0.0f;
    ys[decltype(IT)::value] = 0.0f;
  });
  const int* const er_tab = row_er_table<L>();

  for (int pass = 0; pass < PASSES; ++pass) {
    const int pu = __builtin_amdgcn_readfirstlane(pass);  // uniform: keep it scalar
    // the pass context from an opaque copy of the lane id: its lane-derived
    // offsets are recomputed each pass instead of being held (or spilled)
    // across the passes
    int lnp = lane;
    asm volatile("" : "+v"(lnp));
    const WaveCtx<L> w(lnp, reinterpret_cast<const float4*>(xs), t);
    f4 o[1][4];
    float zz;
    w.template pass<FFT>(pu, o, zz, fa);
    // this pass's row offsets (loaded here, not held across the passes:
    // that would keep NIT more registers live through the contractions)
    int er[NIT];
    cfor<0, NIT>([&](auto IT) {
      constexpr int it = decltype(IT)::value;
      er[it] = (lane + 64 * it < NROW) ? er_tab[64 * it + lane] : 0;
    });
    // ---- 4. theta analysis over this pass's pairs (lane-permuted weights):
    // the weights of the pole rows and of the first WQ row blocks are read
    // before the moments are stored (the table is read-only), the later
    // blocks WQ blocks ahead of their use (every lane reads: the table holds
    // all 64 lanes of every block)
    constexpr int WQ = 3;
    const int wbase = pu * (NIT + 1) * 64 * 32;
    float4 wq[WQ][2];
    cfor<0, (WQ < NIT ? WQ : NIT)>([&](auto IT) {
      constexpr int it = decltype(IT)::value;
      wq[it][0] = tload4_s(WPr, lane * 32, wbase + it * 64 * 32);
      wq[it][1] = tload4_s(WPr, lane * 32 + 16, wbase + it * 64 * 32);
    });
    const float4 wz0 = tload4_s(WPr, lane * 32, wbase + NIT * 64 * 32);
    const float4 wz1 = tload4_s(WPr, lane * 32 + 16, wbase + NIT * 64 * 32);
    if constexpr (FFT) {
      __syncthreads();  // the spectra of all 16 column nodes are in LDS
      w.phi_fft(eo, fa, ft);
    } else {
      w.store_moments(eo, o, zz);
    }
    __syncthreads();

    if (lane <= L) {
      const float wv[8] = {wz0.x, wz0.y, wz0.z, wz0.w, wz1.x, wz1.y, wz1.z, wz1.w};
      cfor<0, 8>([&](auto JJ) {
        constexpr int jj = decltype(JJ)::value;
        y0 = fmaf(wv[jj], eo[(lnp & 1) * 8 * NMP2 + jj * NMP2], y0);  // row tri(lane, 0)
      });
    }
    cfor<0, NIT>([&](auto IT) {
      constexpr int it = decltype(IT)::value;
      const float4 w0 = wq[it % WQ][0], w1 = wq[it % WQ][1];
      if constexpr (it + WQ < NIT) {
        wq[it % WQ][0] = tload4_s(WPr, lane * 32, wbase + (it + WQ) * 64 * 32);
        wq[it % WQ][1] = tload4_s(WPr, lane * 32 + 16, wbase + (it + WQ) * 64 * 32);
      }
      if (lane + 64 * it < NROW) {
        const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
        cfor<0, 8>([&](auto JJ) {
          constexpr int jj = decltype(JJ)::value;
          const f2 cs = *reinterpret_cast<const f2*>(eo + er[it] + jj * NMP2);
          yc[it] = fmaf(wv[jj], cs.x, yc[it]);
          ys[it] = fmaf(wv[jj], cs.y, ys[it]);
        });
      }
      __builtin_amdgcn_sched_barrier(0);  // keep the ring's distance
    });
    __syncthreads();  // eo is rewritten by the next pass
  }

  // poles (only the m = 0 parts are non-zero there) and the stores
  float p1, p2;
  {
    int lnp = lane;
    asm volatile("" : "+v"(lnp));
    const WaveCtx<L> w(lnp, reinterpret_cast<const float4*>(xs), t);
    float sv[G::NV0P];
    w.m0_load(PASSES, sv);
    w.m0_finish(sv, p1, p2);  // h = 0 lanes: north pole, h = 1 lanes: south pole
  }
  const float f = p1 * p2 * float(NP);
  const float fN = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), 0));  // wave-uniform
  const float fS = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), 8));
  float* const yr = y + P * (PAD ? ko : K);  // this product's output row (wave-uniform)
  if (lane <= L) {
    const int l = lane;
    y0 = fmaf(tload(Wr, wr0), fN + ((l & 1) ? -fS : fS), y0);
    if constexpr (WGT) {
      if (wt.wo) y0 *= wt.wo[weight_row(wt, P) * (L + 1) + l];
    }
    store_row<PAD>(yr, ko, unsigned(4 * (l * l + l)), y0);
  }
  int ln = lane;
  asm volatile("" : "+v"(ln));
  const unsigned* const ro_tab = row_out_table<L>();
  cfor<0, NIT>([&](auto IT) {
    constexpr int it = decltype(IT)::value;
    const int q = ln + 64 * it;
    if (q < NROW) {
      const unsigned ro = ro_tab[q];
      float wl = 1.0f;
      if constexpr (WGT) {
        int l, m;
        row_lm(q, l, m);
        if (wt.wo) wl = wt.wo[weight_row(wt, P) * (L + 1) + l];
      }
      store_row<PAD>(yr, ko, ro & 0xffffu, yc[it] * wl);
      store_row<PAD>(yr, ko, ro >> 16, ys[it] * wl);
    }
  });
  if constexpr (PAD) zero_tail<K>(y, P, ko, lane, 64);
}

// L = 64: four waves per product (256 threads), wave v runs passes 2v and
// 2v + 1.  The moments of the first pass go to LDS at once; those of the
// second stay in registers until every wave is done with the x image, then
// go into its place.  The 256 threads then do the theta analysis, each over
// all 64 mirror pairs of its output rows.
template <int L, typename T1, typename T2, bool WGT, bool PAD = false>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_full_wave4(
    const T1* __restrict__ x1, const T2* __restrict__ x2, float* __restrict__ y, int64_t n, DevTables t,
    DegWeights wt, int k1, int k2, int ko) {
  using G = WGeo<L>;
  static_assert(G::NW == 4 && G::PASSES == 8, "four waves, two passes each");
  constexpr int NJ = G::NJ, NP = G::NP, NMP2 = G::NMP2, K = G::K, PASSES = G::PASSES, NROW = G::NROW,
                NIT = G::NIT, EOP = G::EOP, NTH = G::NTH;
  constexpr int XF = (G::XQ * 4 > 4 * EOP) ? G::XQ * 4 : 4 * EOP;  // x image, later the odd passes' moments
  __shared__ __align__(16) float lds[XF + 4 * EOP];               // + the even passes' moments
  lds_poison(lds, XF + 4 * EOP);
  float* const eo_odd = lds;
  float* const eo_even = lds + XF;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (int64_t(blockIdx.x) >= n) return;  // whole-workgroup exit (one product per workgroup)
  const int64_t P = xcd_product(blockIdx.x, n);
  stage_x<L, WGT, PAD>(lds, x1, x2, P, tid, t.XMAP, wt, k1, k2);
  const WaveCtx<L> w(lane, reinterpret_cast<const float4*>(lds), t);

  f4 o[G::NMR][4];
  float zz;
  w.pass(__builtin_amdgcn_readfirstlane(2 * wave), o, zz);
  w.store_moments(eo_even + wave * EOP, o, zz);
  w.pass(__builtin_amdgcn_readfirstlane(2 * wave + 1), o, zz);
  // poles (only the m = 0 parts are non-zero there), before the x image goes
  float p1, p2;
  {
    float sv[G::NV0P];
    w.m0_load(PASSES, sv);
    w.m0_finish(sv, p1, p2);  // h = 0 lanes: north pole, h = 1 lanes: south pole
  }
  const float f = p1 * p2 * float(NP);
  const float fN = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), 0));  // wave-uniform
  const float fS = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), 8));
  __syncthreads();  // the x image is dead
  w.store_moments(eo_odd + wave * EOP, o, zz);
  __syncthreads();

  // ---- 4. theta analysis: thread tid owns row tri(tid, 0) (tid <= L) and
  // the m > 0 rows q = tid + 256 it; weights WP[it][tid][j - 1], j = 1..L
  const __amdgpu_buffer_rsrc_t WPr = table_rsrc(t.WP, (NIT + 1) * NTH * L);
  auto row_sum = [&](int it, int er, float& ac, float& as, bool with_sin) {
    cfor<0, PASSES>([&](auto PP) {
      constexpr int pp = decltype(PP)::value;  // pass: pairs 8 pp + 1 .. 8 pp + 8
      const float* eop = (pp % 2 == 0 ? eo_even : eo_odd) + (pp / 2) * EOP;
      const float4 w0 = tload4_s(WPr, tid * L * 4 + pp * 32, it * NTH * L * 4);
      const float4 w1 = tload4_s(WPr, tid * L * 4 + pp * 32 + 16, it * NTH * L * 4);
      const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
      cfor<0, 8>([&](auto JJ) {
        constexpr int jj = decltype(JJ)::value;
        const f2 cs = *reinterpret_cast<const f2*>(eop + er + jj * NMP2);
        ac = fmaf(wv[jj], cs.x, ac);
        if (with_sin) as = fmaf(wv[jj], cs.y, as);
      });
      if constexpr (pp % 4 == 3) __builtin_amdgcn_sched_barrier(0);  // bound the loads in flight
    });
  };
  if (tid <= L) {
    const int l = tid;
    float a0 = 0.0f, unused = 0.0f;
    row_sum(NIT, (l & 1) * 8 * NMP2, a0, unused, false);
    const __amdgpu_buffer_rsrc_t Wr = table_rsrc(t.WT, NJ * t.ntW);
    a0 = fmaf(tload(Wr, (l * (l + 1) / 2) * 4), fN + ((l & 1) ? -fS : fS), a0);
    if constexpr (WGT) {
      if (wt.wo) a0 *= wt.wo[weight_row(wt, P) * (L + 1) + l];
    }
    store_out<PAD, K>(y, P, ko, l * l + l, a0);
  }
  for (int it = 0; it < NIT; ++it) {
    const int q = tid + NTH * it;
    if (q < NROW) {
      int l, m;
      row_lm(q, l, m);
      float ac = 0.0f, as = 0.0f;
      row_sum(it, ((l + m) & 1) * 8 * NMP2 + 2 * m, ac, as, true);
      if constexpr (WGT) {
        if (wt.wo) {
          const float wl = wt.wo[weight_row(wt, P) * (L + 1) + l];
          ac *= wl;
          as *= wl;
        }
      }
      store_out<PAD, K>(y, P, ko, l * l + l + m, ac);
      store_out<PAD, K>(y, P, ko, l * l + l - m, as);
    }
  }
  if constexpr (PAD) zero_tail<K>(y, P, ko, tid, NTH);
}

// L = 64 with the phi transforms by radix-2 FFT: four waves per product
// working on one pass at a time -- wave v synthesises the m-parts of K-steps
// v and 7 - v of the pass's 16 columns into the shared spectra, the 256
// threads run the FFT stages in two half passes (phi_fft_half) and
// accumulate the theta analysis of the pass's 8 mirror pairs in registers
// (thread tid owns the rows tri(tid, 0) and q = tid + 256 it, as in
// k_full_wave4).  LDS: the x image, one pass's moments, the spectra and one
// half pass's transposes (76.6 KB: two products per CU).
template <int L, typename T1, typename T2, bool WGT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_full_wave4_fft(
    const T1* __restrict__ x1, const T2* __restrict__ x2, float* __restrict__ y, int64_t n, DevTables t,
    DegWeights wt) {
  using G = WGeo<L>;
  using F = FGeo<L>;
  static_assert(G::NW == 4 && G::NKS == 8, "four waves, two K-steps each");
  constexpr int NJ = G::NJ, NP = G::NP, NMP2 = G::NMP2, K = G::K, PASSES = G::PASSES, NROW = G::NROW,
                NIT = G::NIT, EOP = G::EOP, NTH = G::NTH;
  __shared__ __align__(16) float lds[G::XQ * 4 + EOP + 2 * (16 * F::NS + 8 * F::TS)];
  lds_poison(lds, G::XQ * 4 + EOP + 2 * (16 * F::NS + 8 * F::TS));
  float* const xs = lds;
  float* const eo = lds + G::XQ * 4;
  float2* const fa = reinterpret_cast<float2*>(eo + EOP);
  float2* const ft = fa + 16 * F::NS;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (int64_t(blockIdx.x) >= n) return;  // whole-workgroup exit (one product per workgroup)
  const int64_t P = xcd_product(blockIdx.x, n);
  stage_x<L, WGT>(xs, x1, x2, P, tid, t.XMAP, wt);
  const __amdgpu_buffer_rsrc_t WPr = table_rsrc(t.WP, (NIT + 1) * NTH * L);
  float a0 = 0.0f, ac[NIT], as[NIT];
  int er[NIT];
  cfor<0, NIT>([&](auto IT) {
    constexpr int it = decltype(IT)::value;
    ac[it] = as[it] = 0.0f;
    er[it] = 0;
    const int q = tid + NTH * it;
    if (q < NROW) {
      int l, m;
      row_lm(q, l, m);
      er[it] = ((l + m) & 1) * 8 * NMP2 + 2 * m;
    }
  });
  for (int pass = 0; pass < PASSES; ++pass) {
    const int pu = __builtin_amdgcn_readfirstlane(pass);
    {
      int lnp = lane;
      asm volatile("" : "+v"(lnp));
      const WaveCtx<L> w(lnp, reinterpret_cast<const float4*>(xs), t);
      f4 o[G::NMR][4];
      float zz;
      // K-step s has L / 2 - 4 s u-steps: wave v takes K-steps v and 7 - v,
      // the same work for every wave
      if (wave == 0) {
        w.template pass<true, 0, 1>(pu, o, zz, fa);
        w.template pass<true, 7, 8>(pu, o, zz, fa);
      } else if (wave == 1) {
        w.template pass<true, 1, 2>(pu, o, zz, fa);
        w.template pass<true, 6, 7>(pu, o, zz, fa);
      } else if (wave == 2) {
        w.template pass<true, 2, 3>(pu, o, zz, fa);
        w.template pass<true, 5, 6>(pu, o, zz, fa);
      } else {
        w.template pass<true, 3, 4>(pu, o, zz, fa);
        w.template pass<true, 4, 5>(pu, o, zz, fa);
      }
    }
    __syncthreads();  // the 16 spectra are complete
    phi_fft_half<L>(tid, 0, eo, fa, ft);
    phi_fft_half<L>(tid, 1, eo, fa, ft);
    // theta analysis over this pass's pairs 8 pu + 1 .. 8 pu + 8
    if (tid <= L) {
      const float4 w0 = tload4_s(WPr, tid * L * 4 + pu * 32, NIT * NTH * L * 4);
      const float4 w1 = tload4_s(WPr, tid * L * 4 + pu * 32 + 16, NIT * NTH * L * 4);
      const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
      cfor<0, 8>([&](auto JJ) {
        constexpr int jj = decltype(JJ)::value;
        a0 = fmaf(wv[jj], eo[(tid & 1) * 8 * NMP2 + jj * NMP2], a0);
      });
    }
    cfor<0, NIT>([&](auto IT) {
      constexpr int it = decltype(IT)::value;
      if (tid + NTH * it < NROW) {
        const float4 w0 = tload4_s(WPr, tid * L * 4 + pu * 32, it * NTH * L * 4);
        const float4 w1 = tload4_s(WPr, tid * L * 4 + pu * 32 + 16, it * NTH * L * 4);
        const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
        cfor<0, 8>([&](auto JJ) {
          constexpr int jj = decltype(JJ)::value;
          const f2 cs = *reinterpret_cast<const f2*>(eo + er[it] + jj * NMP2);
          ac[it] = fmaf(wv[jj], cs.x, ac[it]);
          as[it] = fmaf(wv[jj], cs.y, as[it]);
        });
      }
    });
    __syncthreads();  // the next pass rewrites the spectra and the moments
  }
  // poles (only the m = 0 parts are non-zero there) and the stores
  float p1, p2;
  {
    const WaveCtx<L> w(lane, reinterpret_cast<const float4*>(xs), t);
    float sv[G::NV0P];
    w.m0_load(PASSES, sv);
    w.m0_finish(sv, p1, p2);  // h = 0 lanes: north pole, h = 1 lanes: south pole
  }
  const float f = p1 * p2 * float(NP);
  const float fN = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), 0));
  const float fS = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), 8));
  if (tid <= L) {
    const int l = tid;
    const __amdgpu_buffer_rsrc_t Wr = table_rsrc(t.WT, NJ * t.ntW);
    a0 = fmaf(tload(Wr, (l * (l + 1) / 2) * 4), fN + ((l & 1) ? -fS : fS), a0);
    if constexpr (WGT) {
      if (wt.wo) a0 *= wt.wo[weight_row(wt, P) * (L + 1) + l];
    }
    y[P * K + l * l + l] = a0;
  }
  cfor<0, NIT>([&](auto IT) {
    constexpr int it = decltype(IT)::value;
    const int q = tid + NTH * it;
    if (q < NROW) {
      int l, m;
      row_lm(q, l, m);
      float wl = 1.0f;
      if constexpr (WGT) {
        if (wt.wo) wl = wt.wo[weight_row(wt, P) * (L + 1) + l];
      }
      y[P * K + l * l + l + m] = ac[it] * wl;
      y[P * K + l * l + l - m] = as[it] * wl;
    }
  });
}

template <int L, typename T1, typename T2, bool WGT, bool PAD = false>
hipError_t launch_wave_typed(const void* x1, const void* x2, int64_t n, float* y, const DevTables& t,
                             const DegWeights& wt, hipStream_t s, int k1 = WGeo<L>::K, int k2 = WGeo<L>::K,
                             int ko = WGeo<L>::K) {
  // the radix-FFT phi transforms where the plan asks for them and a
  // one-wave kernel exists (L = 16, 32)
  const bool fft = t.phi_fft != 0;
  using G = WGeo<L>;
  // at most 2^30 workgroups per launch
  for (int64_t p0 = 0; p0 < n; p0 += (int64_t(1) << 30)) {
    const int64_t nn = n - p0 < (int64_t(1) << 30) ? n - p0 : (int64_t(1) << 30);
    const T1* a = static_cast<const T1*>(x1) + size_t(p0) * k1;
    const T2* b = static_cast<const T2*>(x2) + size_t(p0) * k2;
    float* yy = y + size_t(p0) * ko;
    DegWeights w = wt;
    w.pbase += p0;  // the chunk's products start at p0
    if constexpr (G::NW == 1) {
      if (fft && !PAD)
        hipLaunchKernelGGL((k_full_wave<L, T1, T2, WGT, true>), dim3(unsigned(nn)), dim3(64), 0, s, a, b, yy, nn, t, w,
                           k1, k2, ko);
      else
        hipLaunchKernelGGL((k_full_wave<L, T1, T2, WGT, false, PAD>), dim3(unsigned(nn)), dim3(64), 0, s, a, b, yy, nn,
                           t, w, k1, k2, ko);
    } else if (fft && !PAD) {
      hipLaunchKernelGGL((k_full_wave4_fft<L, T1, T2, WGT>), dim3(unsigned(nn)), dim3(G::NTH), 0, s, a, b, yy, nn, t,
                         w);
    } else {
      hipLaunchKernelGGL((k_full_wave4<L, T1, T2, WGT, PAD>), dim3(unsigned(nn)), dim3(G::NTH), 0, s, a, b, yy, nn, t,
                         w, k1, k2, ko);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Input types: both fp32, both bf16, or fp32 x1 with bf16 x2 (a backward
// pass: fp32 output gradient times a bf16 input); *supported = false for
// bf16 x1 with fp32 x2, and for per-degree weights with mixed types.  k1,
// k2, ko > 0: a padded plan (no weights).
template <int L>
hipError_t launch_wave_one(const DevTables& t, const void* x1, int it1, const void* x2, int it2, int64_t n,
                           float* y, const DegWeights& wt, hipStream_t s, bool* supported, int k1, int k2, int ko) {
  // the scatter map's slots must fit the kernel's LDS image
  if (t.XQUADS != WGeo<L>::XQ) return hipErrorInvalidValue;
  if (ko > 0) {
    if (wt.on || k1 > WGeo<L>::K || k2 > WGeo<L>::K) {
      *supported = false;
      return hipSuccess;
    }
    if (it1 == IN_F32 && it2 == IN_F32)
      return launch_wave_typed<L, float, float, false, true>(x1, x2, n, y, t, wt, s, k1, k2, ko);
    if (it1 == IN_BF16 && it2 == IN_BF16)
      return launch_wave_typed<L, uint16_t, uint16_t, false, true>(x1, x2, n, y, t, wt, s, k1, k2, ko);
    if (it1 == IN_F32 && it2 == IN_BF16)
      return launch_wave_typed<L, float, uint16_t, false, true>(x1, x2, n, y, t, wt, s, k1, k2, ko);
    *supported = false;
    return hipSuccess;
  }
  if (wt.on) {
    if (it1 == IN_F32 && it2 == IN_F32) return launch_wave_typed<L, float, float, true>(x1, x2, n, y, t, wt, s);
    if (it1 == IN_BF16 && it2 == IN_BF16)
      return launch_wave_typed<L, uint16_t, uint16_t, true>(x1, x2, n, y, t, wt, s);
    *supported = false;
    return hipSuccess;
  }
  if (it1 == IN_F32 && it2 == IN_F32) return launch_wave_typed<L, float, float, false>(x1, x2, n, y, t, wt, s);
  if (it1 == IN_BF16 && it2 == IN_BF16)
    return launch_wave_typed<L, uint16_t, uint16_t, false>(x1, x2, n, y, t, wt, s);
  if (it1 == IN_F32 && it2 == IN_BF16) return launch_wave_typed<L, float, uint16_t, false>(x1, x2, n, y, t, wt, s);
  *supported = false;
  return hipSuccess;
}

}  // namespace

hipError_t launch_full_wave(const DevTables& t, const void* x1, int it1, const void* x2, int it2, int64_t n,
                            float* y, const DegWeights& wt, hipStream_t s, bool* supported, int k1, int k2, int ko) {
  *supported = true;
  if (t.waveL == 16 && t.SMP) return launch_wave_one<16>(t, x1, it1, x2, it2, n, y, wt, s, supported, k1, k2, ko);
  if (t.waveL == 32 && t.SMP) return launch_wave_one<32>(t, x1, it1, x2, it2, n, y, wt, s, supported, k1, k2, ko);
  if (t.waveL == 64 && t.SMP) return launch_wave_one<64>(t, x1, it1, x2, it2, n, y, wt, s, supported, k1, k2, ko);
  *supported = false;
  return hipSuccess;
}

}  // namespace gtp
