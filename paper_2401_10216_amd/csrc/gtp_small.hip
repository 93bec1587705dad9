// Thread-per-product fused Gaunt tensor product for small degrees (gfx950).
//
// One lane owns one (b, c) product.  The three steps of Sec. 3.2 run with the
// convolution theorem: the 2D Fourier series of each input is sampled on a
// uniform (theta, phi) torus grid (the inverse transforms, with step 1 folded
// into the theta part: table S), the samples are multiplied pointwise, and the
// forward transforms followed by step 3 (table W) give the SH coefficients.
// The theta transforms use the grid's mirror symmetry t <-> pi - t (Theta_lm
// has parity (-1)^(l+m)), the phi transforms use p <-> -p and pi -+ p: they
// are unrolled direct DFTs with compile-time twiddles, and the pointwise
// product is taken, already folded over each quarter angle's four points,
// from the two inputs' quarter-angle class sums.  For equal degrees the S
// and W rows are compile-time constants too.  Nothing but x and y touches
// HBM.
#include <type_traits>
#include <utility>

#include "gtp_ct.hpp"
#include "gtp_device.hpp"
#include "gtp_small.hpp"

// Scheduling fence between the per-node stages: keeps the two mirror nodes
// from being interleaved (which costs registers) and keeps the table
// prefetch behind the LDS reads it would otherwise make wait.
#define GTP_SCHED_FENCE() __builtin_amdgcn_sched_barrier(0)

namespace gtp {
namespace {

constexpr int ctri(int l, int m) { return l * (l + 1) / 2 + m; }
// degree of coefficient index i = l*l + l + m
constexpr int cdeg(int i) {
  int l = 0;
  while ((l + 1) * (l + 1) <= i) ++l;
  return l;
}
constexpr int csh(int L) { return (L + 1) * (L + 1); }
constexpr int cmin(int a, int b) { return a < b ? a : b; }
constexpr int cmax(int a, int b) { return a > b ? a : b; }
// LDS row stride of K-float rows that each lane reads or writes as its own
// row: odd, so that one column of the 64 lanes' rows falls in 64 distinct
// banks.  K = (L + 1)^2 is even (a multiple of 4) for odd L, where a stride
// of K put every lane's element i in one bank.
constexpr int lds_stride(int k) { return k | 1; }

// Coefficient accessors of one lane's input vector: in registers, or a row of
// the workgroup's LDS tile.  touch() makes the LDS row offset opaque so the
// reads stay inside the node loop instead of being hoisted into registers.
template <int K>
struct RegX {
  float (&a)[K];
  template <class I>
  __device__ __forceinline__ float operator()(I) const { return a[I::value]; }
  __device__ __forceinline__ void touch() {}
};
struct LdsX {
  const float* tile;
  int off;
  template <class I>
  __device__ __forceinline__ float operator()(I) const { return tile[off + I::value]; }
  __device__ __forceinline__ void touch() { asm volatile("" : "+v"(off)); }
};

__device__ __forceinline__ float ld_in(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld_in(const uint16_t* p, int64_t i) {
  return __uint_as_float(uint32_t(p[i]) << 16);
}

// phi grid p_k = 2 pi k / NP with NP = 4Q.  The points k, -k, 2Q + k, 2Q - k
// share |cos(m p)| and |sin(m p)|, with signs set by the parity of m, so both
// transforms work on the quarter 0 <= k <= Q and fan out.

// a += s x, or a = s x for the first term of a sum: a multiply-add onto a
// zero cannot drop the addend (signed zeros), and its three-operand form
// cannot carry a literal constant.  The first product is kept out of
// multiply-add fusion for the same reason (x s - y needs that form too).
template <bool FIRST>
__device__ __forceinline__ void mac(float& a, float s, float x) {
  if constexpr (FIRST) {
#pragma clang fp contract(off)
    a = s * x;
  } else {
    a = fmaf(s, x, a);
  }
}

// Whether m is the first degree of its parity (m >= 1) with a non-zero
// cos (S = false) or sin (S = true) twiddle at sample k: the first term of a
// phi-synthesis partial sum.
constexpr bool first_m(int m, long long k, int NP, bool S) {
  for (int mm = (m % 2 == 0) ? 2 : 1; mm < m; mm += 2) {
    const float v = S ? ct_round(ct_sin2pi(mm * k, NP)) : ct_round(ct_cos2pi(mm * k, NP));
    if (v != 0.0f) return false;
  }
  return true;
}
// Whether k is the first sample with a non-zero cos / sin twiddle of degree
// m: the first term of a phi-analysis sum.
constexpr bool first_k(int m, int k, int NP, bool S) {
  for (int kk = 0; kk < k; ++kk) {
    const float v = S ? ct_round(ct_sin2pi((long long)m * kk, NP)) : ct_round(ct_cos2pi((long long)m * kk, NP));
    if (v != 0.0f) return false;
  }
  return true;
}

// F[k] = A0 + sum_m A[2m-1] cos(m p_k) + A[2m] sin(m p_k), k < NP, for a
// function of phi-degree <= M.
template <int M, int NP>
__device__ __forceinline__ void phi_synth(const float (&A)[2 * M + 1], float (&F)[NP]) {
  static_assert(NP % 4 == 0, "phi grid size must be a multiple of 4");
  constexpr int Q = NP / 4;
  cfor<0, Q + 1>([&](auto KK) {
    constexpr int k = decltype(KK)::value;
    // partial sums over even / odd m of the cos and sin parts
    float pe = A[0], po = 0.0f, qe = 0.0f, qo = 0.0f;
    cfor<1, M + 1>([&](auto MM) {
      constexpr int m = decltype(MM)::value;
      constexpr float c = ct_round(ct_cos2pi((long long)m * k, NP));
      constexpr float sn = ct_round(ct_sin2pi((long long)m * k, NP));
      if constexpr (m % 2 == 0) {
        if constexpr (c != 0.0f) pe = fmaf(A[2 * m - 1], c, pe);
        if constexpr (sn != 0.0f) mac<first_m(m, k, NP, true)>(qe, sn, A[2 * m]);
      } else {
        if constexpr (c != 0.0f) mac<first_m(m, k, NP, false)>(po, c, A[2 * m - 1]);
        if constexpr (sn != 0.0f) mac<first_m(m, k, NP, true)>(qo, sn, A[2 * m]);
      }
    });
    if constexpr (k == 0) {
      F[0] = pe + po;
      F[2 * Q] = pe - po;
    } else if constexpr (k == Q) {
      F[Q] = pe + qo;  // cos(odd m pi/2) = sin(even m pi/2) = 0
      F[3 * Q] = pe - qo;
    } else {
      const float s1 = pe + po, d1 = pe - po, s2 = qe + qo, d2 = qe - qo;
      F[k] = s1 + s2;
      F[NP - k] = s1 - s2;
      F[2 * Q + k] = d1 + d2;
      F[2 * Q - k] = d1 - d2;
    }
  });
}

// C[0] = sum_k F_k, C[2m-1] = sum_k F_k cos(m p_k), C[2m] = sum_k F_k sin(m p_k), m <= MO.
template <int MO, int NP>
__device__ __forceinline__ void phi_analysis(const float (&F)[NP], float (&C)[2 * MO + 1]) {
  static_assert(NP % 4 == 0, "phi grid size must be a multiple of 4");
  constexpr int Q = NP / 4;
  cfor<0, 2 * MO + 1>([&](auto I) { C[decltype(I)::value] = 0.0f; });
  cfor<0, Q + 1>([&](auto KK) {
    constexpr int k = decltype(KK)::value;
    // even-m / odd-m folds of the four points sharing this quarter angle
    float ce, co, se = 0.0f, so = 0.0f;
    if constexpr (k == 0) {
      ce = F[0] + F[2 * Q];
      co = F[0] - F[2 * Q];
    } else if constexpr (k == Q) {
      ce = F[Q] + F[3 * Q];
      co = 0.0f;
      so = F[Q] - F[3 * Q];
    } else {
      const float a = F[k] + F[NP - k], b = F[2 * Q + k] + F[2 * Q - k];
      const float d = F[k] - F[NP - k], e = F[2 * Q + k] - F[2 * Q - k];
      ce = a + b;
      co = a - b;
      se = d + e;
      so = d - e;
    }
    cfor<0, MO + 1>([&](auto MM) {
      constexpr int m = decltype(MM)::value;
      constexpr float c = ct_round(ct_cos2pi((long long)m * k, NP));
      constexpr float sn = ct_round(ct_sin2pi((long long)m * k, NP));
      constexpr int ic = m == 0 ? 0 : 2 * m - 1;
      if constexpr (c != 0.0f) mac<first_k(m, k, NP, false)>(C[ic], c, (m % 2 == 0) ? ce : co);
      if constexpr (m > 0 && sn != 0.0f) mac<first_k(m, k, NP, true)>(C[2 * m], sn, (m % 2 == 0) ? se : so);
    });
  });
}

// Theta synthesis at the mirror pair (t_j, t_{NT-j}) of one input of degree
// L: even-parity and odd-parity (l + m) partial sums give both nodes.  x(I)
// returns coefficient I; ST row j holds Theta_lm(t_j) for all (l, m).
template <int L, typename X, typename T>
__device__ __forceinline__ void theta_synth_pair(X x, const T& Sj, float (&Aj)[2 * L + 1],
                                                 float (&Ajp)[2 * L + 1]) {
  cfor<0, L + 1>([&](auto MM) {
    constexpr int m = decltype(MM)::value;
    float ec = 0.0f, oc = 0.0f, es = 0.0f, os = 0.0f;
    cfor<m, L + 1>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      const float sv = Sj[ctri(l, m)];
      if constexpr ((l + m) % 2 == 0) {
        mac<l == m>(ec, sv, x(std::integral_constant<int, l * l + l + m>{}));
        if constexpr (m > 0) mac<l == m>(es, sv, x(std::integral_constant<int, l * l + l - m>{}));
      } else {
        mac<l == m + 1>(oc, sv, x(std::integral_constant<int, l * l + l + m>{}));
        if constexpr (m > 0) mac<l == m + 1>(os, sv, x(std::integral_constant<int, l * l + l - m>{}));
      }
    });
    if constexpr (m == 0) {
      Aj[0] = ec + oc;
      Ajp[0] = ec - oc;
    } else {
      Aj[2 * m - 1] = ec + oc;
      Ajp[2 * m - 1] = ec - oc;
      Aj[2 * m] = es + os;
      Ajp[2 * m] = es - os;
    }
  });
}

// Theta synthesis at one node of the mirror pair: MIRROR = false gives t_j,
// MIRROR = true gives t_{NT-j} (Theta_lm picks up (-1)^(l+m)).
template <int L, bool MIRROR, typename X, typename T>
__device__ __forceinline__ void theta_synth_node(X x, const T& Sj, float (&A)[2 * L + 1]) {
  cfor<0, L + 1>([&](auto MM) {
    constexpr int m = decltype(MM)::value;
    float ec = 0.0f, es = 0.0f;
    cfor<m, L + 1>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      const float sv = (MIRROR && (l + m) % 2) ? -Sj[ctri(l, m)] : Sj[ctri(l, m)];
      mac<l == m>(ec, sv, x(std::integral_constant<int, l * l + l + m>{}));
      if constexpr (m > 0) mac<l == m>(es, sv, x(std::integral_constant<int, l * l + l - m>{}));
    });
    if constexpr (m == 0) {
      A[0] = ec;
    } else {
      A[2 * m - 1] = ec;
      A[2 * m] = es;
    }
  });
}

// acc += W(t_j) * C for the moments C of one node; MIRROR uses the weights of
// t_{NT-j}, which are (-1)^(l+m) times those of t_j.  FIRST: the first node
// with m > 0 terms (acc holds only the poles' m = 0 terms).
template <int LE, bool MIRROR, typename T, bool FIRST = false>
__device__ __forceinline__ void theta_analysis_node(const T& Wj, const float (&C)[2 * LE + 1],
                                                    float (&acc)[(LE + 1) * (LE + 1)]) {
  cfor<0, LE + 1>([&](auto MM) {
    constexpr int m = decltype(MM)::value;
    cfor<m, LE + 1>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      const float w = (MIRROR && (l + m) % 2) ? -Wj[ctri(l, m)] : Wj[ctri(l, m)];
      mac<(FIRST && m > 0)>(acc[l * l + l + m], w, C[m == 0 ? 0 : 2 * m - 1]);
      if constexpr (m > 0) mac<FIRST>(acc[l * l + l - m], w, C[2 * m]);
    });
  });
}

// Theta synthesis at the equator (only even l + m survive).
template <int L, typename X>
__device__ __forceinline__ void theta_synth_eq(X x, const float* __restrict__ Sj, float (&A)[2 * L + 1]) {
  cfor<0, L + 1>([&](auto MM) {
    constexpr int m = decltype(MM)::value;
    float ec = 0.0f, es = 0.0f;
    cfor<m, L + 1>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      if constexpr ((l + m) % 2 == 0) {
        const float sv = Sj[ctri(l, m)];
        ec = fmaf(sv, x(std::integral_constant<int, l * l + l + m>{}), ec);
        if constexpr (m > 0) es = fmaf(sv, x(std::integral_constant<int, l * l + l - m>{}), es);
      }
    });
    if constexpr (m == 0) {
      A[0] = ec;
    } else {
      A[2 * m - 1] = ec;
      A[2 * m] = es;
    }
  });
}

template <int NU>
__device__ __forceinline__ float ipow(float v) {
  if constexpr (NU == 1) {
    return v;
  } else if constexpr (NU % 2 == 0) {
    const float h = ipow<NU / 2>(v);
    return h * h;
  } else {
    return v * ipow<NU - 1>(v);
  }
}

// Quarter-angle class sums of a function of phi-degree <= M at sample k:
// pe / po = sum over even / odd m of A_cos(m) cos(m p_k) (pe with A0), qe / qo
// the same for the sin parts.  The samples at k, NP - k, 2Q + k, 2Q - k are
// pe + po +- (qe + qo) and pe - po +- (qe - qo).
template <int M, int NP, int k>
__device__ __forceinline__ void phi_classes(const float (&A)[2 * M + 1], float& pe, float& po, float& qe,
                                            float& qo) {
  pe = A[0];
  po = qe = qo = 0.0f;
  cfor<1, M + 1>([&](auto MM) {
    constexpr int m = decltype(MM)::value;
    constexpr float c = ct_round(ct_cos2pi((long long)m * k, NP));
    constexpr float sn = ct_round(ct_sin2pi((long long)m * k, NP));
    if constexpr (m % 2 == 0) {
      if constexpr (c != 0.0f) pe = fmaf(A[2 * m - 1], c, pe);
      if constexpr (sn != 0.0f) mac<first_m(m, k, NP, true)>(qe, sn, A[2 * m]);
    } else {
      if constexpr (c != 0.0f) mac<first_m(m, k, NP, false)>(po, c, A[2 * m - 1]);
      if constexpr (sn != 0.0f) mac<first_m(m, k, NP, true)>(qo, sn, A[2 * m]);
    }
  });
}

// One node, product of two functions: the phi moments m <= LE of f g from
// the class sums of f and g.  Summed over the four points of a quarter angle
// (the grid's p -> -p, pi -+ p symmetry), f g folds to
//   even-m cos: 4 (pe pe' + po po' + qe qe' + qo qo'),
//   odd-m cos:  4 (pe po' + po pe' + qe qo' + qo qe'),
//   even-m sin: 4 (pe qe' + po qo' + qe pe' + qo po'),
//   odd-m sin:  4 (pe qo' + po qe' + qe po' + qo pe')
// (2 and two points at k = 0 and k = Q), so no sample is formed; the factor
// goes into the analysis twiddles.
template <int L1, int L2, int LE, int NP>
__device__ __forceinline__ void node_product_cls(const float (&A)[2 * L1 + 1], const float (&B)[2 * L2 + 1],
                                                 float (&C)[2 * LE + 1]) {
  static_assert(NP % 4 == 0, "phi grid size must be a multiple of 4");
  constexpr int Q = NP / 4;
  cfor<0, 2 * LE + 1>([&](auto I) { C[decltype(I)::value] = 0.0f; });
  cfor<0, Q + 1>([&](auto KK) {
    constexpr int k = decltype(KK)::value;
    float pe, po, qe, qo, pf, pg, qf, qg;  // f: pe po qe qo; g: pf pg qf qg
    phi_classes<L1, NP, k>(A, pe, po, qe, qo);
    phi_classes<L2, NP, k>(B, pf, pg, qf, qg);
    float ce, co = 0.0f, se = 0.0f, so = 0.0f;
    constexpr float fac = (k == 0 || k == Q) ? 2.0f : 4.0f;
    if constexpr (k == 0) {
      ce = fmaf(po, pg, pe * pf);
      co = fmaf(po, pf, pe * pg);
    } else if constexpr (k == Q) {
      ce = fmaf(qo, qg, pe * pf);
      so = fmaf(qo, pf, pe * qg);
    } else {
      ce = fmaf(qo, qg, fmaf(qe, qf, fmaf(po, pg, pe * pf)));
      co = fmaf(qo, qf, fmaf(qe, qg, fmaf(po, pf, pe * pg)));
      se = fmaf(qo, pg, fmaf(qe, pf, fmaf(po, qg, pe * qf)));
      so = fmaf(qo, pf, fmaf(qe, pg, fmaf(po, qf, pe * qg)));
    }
    cfor<0, LE + 1>([&](auto MM) {
      constexpr int m = decltype(MM)::value;
      constexpr float c = ct_round(ct_cos2pi((long long)m * k, NP));
      constexpr float sn = ct_round(ct_sin2pi((long long)m * k, NP));
      constexpr int ic = m == 0 ? 0 : 2 * m - 1;
      if constexpr (c != 0.0f) mac<first_k(m, k, NP, false)>(C[ic], fac * c, (m % 2 == 0) ? ce : co);
      if constexpr (m > 0 && sn != 0.0f) mac<first_k(m, k, NP, true)>(C[2 * m], fac * sn, (m % 2 == 0) ? se : so);
    });
  });
}

// One node: the phi moments m <= LE of the product of two functions (from
// their class sums), or of a power of one function (through its samples).
template <int L1, int L2, int LE, int NP, int NU>
__device__ __forceinline__ void node_product(const float (&A)[2 * L1 + 1], const float (&B)[2 * L2 + 1],
                                             float (&C)[2 * LE + 1]) {
  if constexpr (NU == 0) {
    node_product_cls<L1, L2, LE, NP>(A, B, C);
  } else {
    float F[NP];
    phi_synth<L1, NP>(A, F);
    cfor<0, NP>([&](auto KK) { F[decltype(KK)::value] = ipow<NU>(F[decltype(KK)::value]); });
    phi_analysis<LE, NP>(F, C);
  }
}

// Degree bookkeeping of one product stage.  NU = 0: x1 (deg L1) times x2
// (deg L2); NU >= 2: x1^NU (L2 unused).
template <int L1, int L2, int LO, int NU>
struct Geo {
  static constexpr int U = NU == 0 ? L1 + L2 : NU * L1;
  static constexpr int LE = cmin(LO, U);
  static constexpr int NT = U + 1;
  static constexpr int NJ = NT + 1;
  static constexpr int NP = (U + LE + 1 + 3) / 4 * 4;  // same rule as the host tables
  static constexpr int KE = csh(LE);
};

// Compile-time copies of the node-major S and W rows of the equal-degree
// triples L1 = L2 = Lout = 1..8 (SmallConsts<L>::S[j][tri(l, m)], ::W[j][..]),
// generated at build time from the same fp64 builder and fp32 rounding as a
// plan's device tables.  Read with constant indices they become instruction
// literals: a VALU instruction with a literal operand issues at the rate of
// an all-VGPR one, one with a scalar-register operand at about half of it.
#include "gtp_small_consts.inc"

template <int L, int J, bool IS_W>
struct LitRow {
  __device__ __forceinline__ constexpr float operator[](int i) const {
    return IS_W ? SmallConsts<L>::W[J][i] : SmallConsts<L>::S[J][i];
  }
};

template <int L1, int L2, int LO, int NU>
constexpr bool lit_tables() {
  return NU == 0 && L1 == L2 && L2 == LO && L1 >= 1 && L1 <= 8;
}

// gtp_core for L1 = L2 = Lout = L with the tables as literals: the node-pair
// loop is unrolled at compile time (NT = 2 L + 1 is odd: no equator node).
template <int L, typename XA, typename XB>
__device__ __forceinline__ void gtp_core_lit(XA xa, XB xb, float (&acc)[(L + 1) * (L + 1)]) {
  using G = Geo<L, L, L, 0>;
  constexpr int NT = G::NT, NP = G::NP;
  static_assert(NT % 2 == 1, "equal degrees give an odd node count");
  cfor<0, G::KE>([&](auto I) { acc[decltype(I)::value] = 0.0f; });
  {
    // poles: only m = 0 is non-zero and all phi samples are equal
    constexpr LitRow<L, 0, false> S0{};
    constexpr LitRow<L, 0, true> W0{};
    float ae = 0.0f, ao = 0.0f, be = 0.0f, bo = 0.0f;
    cfor<0, L + 1>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      if constexpr (l % 2 == 0) {
        mac<l == 0>(ae, S0[ctri(l, 0)], xa(std::integral_constant<int, l * l + l>{}));
        mac<l == 0>(be, S0[ctri(l, 0)], xb(std::integral_constant<int, l * l + l>{}));
      } else {
        mac<l == 1>(ao, S0[ctri(l, 0)], xa(std::integral_constant<int, l * l + l>{}));
        mac<l == 1>(bo, S0[ctri(l, 0)], xb(std::integral_constant<int, l * l + l>{}));
      }
    });
    const float fn = (ae + ao) * (be + bo), fs = (ae - ao) * (be - bo);
    const float ce = float(NP) * (fn + fs), co = float(NP) * (fn - fs);
    cfor<0, L + 1>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      acc[l * l + l] = W0[ctri(l, 0)] * ((l % 2 == 0) ? ce : co);
    });
  }
  cfor<1, (NT + 1) / 2>([&](auto JJ) {
    constexpr int j = decltype(JJ)::value;
    constexpr LitRow<L, j, false> Sj{};
    constexpr LitRow<L, j, true> Wj{};
    xa.touch();
    xb.touch();
    float Aj[2 * L + 1], Ajp[2 * L + 1], Bj[2 * L + 1];
    theta_synth_pair<L>(xa, Sj, Aj, Ajp);
    theta_synth_node<L, false>(xb, Sj, Bj);
    GTP_SCHED_FENCE();
    {
      float C[2 * L + 1];
      node_product<L, L, L, NP, 0>(Aj, Bj, C);
      theta_analysis_node<L, false, LitRow<L, j, true>, j == 1>(Wj, C, acc);
    }
    GTP_SCHED_FENCE();
    {
      theta_synth_node<L, true>(xb, Sj, Bj);
      float C[2 * L + 1];
      node_product<L, L, L, NP, 0>(Ajp, Bj, C);
      theta_analysis_node<L, true>(Wj, C, acc);
    }
    GTP_SCHED_FENCE();
  });
}

// acc (degree <= LE) = product of xa and xb (or xa^NU) for one lane.
// xa(I), xb(I) return input coefficient I; ST / WT are the node-major
// synthesis and analysis tables with row lengths ntS / ntW (for equal degrees
// 1..8 the compile-time copies are used instead).
template <int L1, int L2, int LO, int NU, typename XA, typename XB>
__device__ __forceinline__ void gtp_core(XA xa, XB xb, float (&acc)[Geo<L1, L2, LO, NU>::KE],
                                         const float* __restrict__ ST, int ntS, const float* __restrict__ WT,
                                         int ntW) {
  if constexpr (lit_tables<L1, L2, LO, NU>()) {
    gtp_core_lit<L1>(xa, xb, acc);
    return;
  }
  using G = Geo<L1, L2, LO, NU>;
  constexpr int LE = G::LE, NT = G::NT, NP = G::NP;
  cfor<0, G::KE>([&](auto I) { acc[decltype(I)::value] = 0.0f; });

  // Poles (t = 0 and t = pi): only m = 0 is non-zero; the phi samples are all
  // equal, so the m = 0 moment is NP times the product value.
  {
    float ae = 0.0f, ao = 0.0f, be = 0.0f, bo = 0.0f;
    cfor<0, L1 + 1>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      const float sv = ST[ctri(l, 0)];
      if constexpr (l % 2 == 0) ae = fmaf(sv, xa(std::integral_constant<int, l * l + l>{}), ae);
      else ao = fmaf(sv, xa(std::integral_constant<int, l * l + l>{}), ao);
    });
    float fn, fs;
    if constexpr (NU == 0) {
      cfor<0, L2 + 1>([&](auto LL) {
        constexpr int l = decltype(LL)::value;
        const float sv = ST[ctri(l, 0)];
        if constexpr (l % 2 == 0) be = fmaf(sv, xb(std::integral_constant<int, l * l + l>{}), be);
        else bo = fmaf(sv, xb(std::integral_constant<int, l * l + l>{}), bo);
      });
      fn = (ae + ao) * (be + bo);
      fs = (ae - ao) * (be - bo);
    } else {
      fn = ipow<NU>(ae + ao);
      fs = ipow<NU>(ae - ao);
    }
    const float ce = float(NP) * (fn + fs), co = float(NP) * (fn - fs);
    cfor<0, LE + 1>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      const float w = WT[ctri(l, 0)];
      acc[l * l + l] = fmaf(w, (l % 2 == 0) ? ce : co, acc[l * l + l]);
    });
  }

  // Interior mirror pairs (j, NT - j), 1 <= j < NT / 2 (runtime tables:
  // degree triples without compile-time constants).
  // The node-pair tables are software-pipelined through scalar registers:
  // S of pair j + 1 and W of pair j are requested after the first LDS reads
  // of pair j (LDS reads share the scalar loads' wait counter) and arrive
  // while the phi transforms of pair j run.
  constexpr int NS = ctri(cmax(L1, L2), cmax(L1, L2)) + 1;
  constexpr int NW = ctri(LE, LE) + 1;
  float scur[NS];
  cfor<0, NS>([&](auto I) { scur[decltype(I)::value] = ST[ntS + decltype(I)::value]; });
  for (int j = 1; 2 * j < NT; ++j) {
    xa.touch();
    xb.touch();
    // x1 at both mirror nodes from shared even / odd partial sums; x2 node by
    // node (fewer live registers), its first node before the table prefetch
    float Aj[2 * L1 + 1], Ajp[2 * L1 + 1];
    float Bj[2 * L2 + 1];
    theta_synth_pair<L1>(xa, scur, Aj, Ajp);
    if constexpr (NU == 0) theta_synth_node<L2, false>(xb, scur, Bj);
    GTP_SCHED_FENCE();
    float sb[NS];
    cfor<0, NS>([&](auto I) { sb[decltype(I)::value] = scur[decltype(I)::value]; });
    // row j + 1 always exists (j + 1 <= NT), even when it is not used
    const float* Sn = ST + (j + 1) * ntS;
    cfor<0, NS>([&](auto I) { scur[decltype(I)::value] = Sn[decltype(I)::value]; });
    const float* Wj = WT + j * ntW;
    float wcur[NW];
    cfor<0, NW>([&](auto I) { wcur[decltype(I)::value] = Wj[decltype(I)::value]; });
    GTP_SCHED_FENCE();
    {
      float C[2 * LE + 1];
      node_product<L1, L2, LE, NP, NU>(Aj, Bj, C);
      theta_analysis_node<LE, false>(wcur, C, acc);
    }
    GTP_SCHED_FENCE();
    {
      if constexpr (NU == 0) theta_synth_node<L2, true>(xb, sb, Bj);
      float C[2 * LE + 1];
      node_product<L1, L2, LE, NP, NU>(Ajp, Bj, C);
      theta_analysis_node<LE, true>(wcur, C, acc);
    }
    GTP_SCHED_FENCE();
  }

  // Equator node when NT is even.
  if constexpr (NT % 2 == 0) {
    constexpr int j = NT / 2;
    const float* Sj = ST + j * ntS;
    const float* Wj = WT + j * ntW;
    float A[2 * L1 + 1], B[2 * L2 + 1];
    theta_synth_eq<L1>(xa, Sj, A);
    if constexpr (NU == 0) theta_synth_eq<L2>(xb, Sj, B);
    float Cq[2 * LE + 1];
    node_product<L1, L2, LE, NP, NU>(A, B, Cq);
    cfor<0, LE + 1>([&](auto MM) {
      constexpr int m = decltype(MM)::value;
      cfor<m, LE + 1>([&](auto LL) {
        constexpr int l = decltype(LL)::value;
        if constexpr ((l + m) % 2 == 0) {
          const float w = Wj[ctri(l, m)];
          acc[l * l + l + m] = fmaf(w, Cq[m == 0 ? 0 : 2 * m - 1], acc[l * l + l + m]);
          if constexpr (m > 0) acc[l * l + l - m] = fmaf(w, Cq[2 * m], acc[l * l + l - m]);
        }
      });
    });
  }
}

constexpr int kTile = 64;  // products per workgroup (one wave)
// Waves per SIMD the register budget is sized for: x1 and the accumulators
// stay in registers, so the budget shrinks with the degree.
constexpr int small_waves(int L1, int L2, int LO) { return (L1 > 6 || L2 > 6 || LO > 6) ? 2 : 3; }

// Row tid (product p0 + tid, the last one for lanes past the end) of x into
// registers, each lane loading its own row.
template <int K, typename TIn>
__device__ __forceinline__ void load_rows(const TIn* __restrict__ x, int64_t p0, int cnt, float (&r)[K]) {
  const int tid = threadIdx.x;
  const TIn* const xr = x + (p0 + (tid < cnt ? tid : cnt - 1)) * K;
  cfor<0, K>([&](auto I) { r[decltype(I)::value] = ld_in(xr, decltype(I)::value); });
}

template <int KO, int KE>
__device__ __forceinline__ void store_rows(float* __restrict__ y, int64_t p0, int cnt, float* tile,
                                           const float (&acc)[KE], int tid = threadIdx.x) {
  constexpr int SO = lds_stride(KO);
  cfor<0, KO>([&](auto I) {
    constexpr int i = decltype(I)::value;
    tile[tid * SO + i] = (i < KE) ? acc[i < KE ? i : 0] : 0.0f;
  });
  __syncthreads();
  float* out = y + p0 * KO;
  typedef float sv4 __attribute__((ext_vector_type(4)));
  if (cnt == kTile && (reinterpret_cast<uintptr_t>(out) & 15) == 0) {
    // a full workgroup's rows are 64 KO floats, a whole number of 16-byte
    // runs: 16-byte non-temporal stores (the outputs are not read again:
    // 1.6 % faster at L = 6 than plain stores; non-temporal loads of the
    // input rows, by contrast, measured 1.5x slower)
    constexpr int N4 = kTile * KO / 4;
    if constexpr (SO == KO) {
      // compact rows: the tile (16-byte aligned) is the output's layout
      for (int i = tid; i < N4; i += kTile)
        __builtin_nontemporal_store(reinterpret_cast<const sv4*>(tile)[i], reinterpret_cast<sv4*>(out) + i);
    } else {
      // padded rows; KO is a multiple of 4, so no 16-byte run crosses a row
      static_assert(KO % 4 == 0, "even row lengths are (2m)^2");
      for (int i = tid; i < N4; i += kTile) {
        const int r = (4 * i) / KO, c = 4 * i - r * KO;
        const float* const t = tile + r * SO + c;
        __builtin_nontemporal_store(sv4{t[0], t[1], t[2], t[3]}, reinterpret_cast<sv4*>(out) + i);
      }
    }
  } else {
    for (int i = tid; i < cnt * KO; i += kTile) {
      const int r = i / KO;
      out[i] = tile[r * SO + (i - r * KO)];
    }
  }
}

// Per-degree weights of one lane's product (WGT = true): scale the K values
// at(I) (degrees <= L) by wrow[degree].
template <int L, int K, typename V>
__device__ __forceinline__ void scale_by_degree(const float* __restrict__ wrow, V&& at) {
  float wl[L + 1];
  cfor<0, L + 1>([&](auto LL) { wl[decltype(LL)::value] = wrow[decltype(LL)::value]; });
  cfor<0, K>([&](auto I) { at(I) *= wl[cdeg(decltype(I)::value)]; });
}

// Row tid of a workgroup's products (xr: this lane's row, the last product's
// for lanes past the end) into the LDS tile, row stride lds_stride(K); each
// lane later reads only its own row.  fp32 rows of degree 5..7 with a compact
// tile: when the workgroup is full and the slab is 16-byte aligned (dma), the
// whole slab x + p0 K by coalesced 16-byte loads straight into LDS (lane
// q 64 + tid carries floats 4 (q 64 + tid) .. + 3, no registers on the way;
// the slab is a whole number of 16-byte runs, 64 K floats).  (Measured: 2.4 %
// faster at L = 6; at L = 4 4 % and at L = 8 1 % slower than the per-lane
// loads, so degrees 5..7 only.  Staging x1 the same way, through the tile
// before x2, measured 1 % slower at L = 6.)
template <int L, bool ALLOW_DMA, typename T>
__device__ __forceinline__ void stage_tile_rows(float* tile, const T* __restrict__ x, const T* __restrict__ xr,
                                                int64_t p0, int cnt, int tid, int dma) {
  constexpr int K = csh(L), S = lds_stride(K);
  bool staged = false;
  if constexpr (std::is_same<T, float>::value && ALLOW_DMA && L >= 5 && L <= 7 && S == K) {
    if (dma && cnt == kTile) {
      typedef __attribute__((address_space(3))) void lds_void;
      typedef const __attribute__((address_space(1))) void glb_void;
      constexpr int NF = kTile * K, NQ = (NF + 255) / 256;
      const float* const slab = x + p0 * K;
      cfor<0, NQ>([&](auto Q) {
        constexpr int q = decltype(Q)::value;
        const int e = (q * 64 + tid) * 4;
        if (q + 1 < NQ || e < NF)
          __builtin_amdgcn_global_load_lds((glb_void*)(slab + e), (lds_void*)(tile + q * 256), 16, 0, 0);
      });
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the whole wave's rows are in LDS
      staged = true;
    }
  }
  if (!staged) cfor<0, K>([&](auto I) { tile[tid * S + decltype(I)::value] = ld_in(xr, decltype(I)::value); });
}

template <int L1, int L2, int LO, int NU, typename T1, typename T2, bool WGT, bool OUT>
__global__ __launch_bounds__(kTile) __attribute__((amdgpu_waves_per_eu(small_waves(L1, L2, LO)))) void k_full_small(const T1* __restrict__ x1, const T2* __restrict__ x2,
                                                      float* __restrict__ y, int64_t n,
                                                      const float* __restrict__ ST, int ntS,
                                                      const float* __restrict__ WT, int ntW, DegWeights wt,
                                                      PairIdx pi, int dma) {
  using G = Geo<L1, L2, LO, NU>;
  constexpr int K1 = csh(L1), K2 = NU == 0 ? csh(L2) : 1, KO = csh(LO);
  constexpr int S2 = lds_stride(K2);
  constexpr int KT = cmax(S2, lds_stride(KO));
  __shared__ __align__(16) float tile[kTile * KT];
  lds_poison(tile, kTile * KT);
  const int tid = threadIdx.x;
  const int64_t p0 = int64_t(blockIdx.x) * kTile;
  const int cnt = int((n - p0) < kTile ? (n - p0) : kTile);
  float xa[K1];
  float acc[G::KE];
  if constexpr (NU == 0) {
    // each lane loads its own two rows, x1 into registers and x2 into its
    // tile row (row-major, odd row stride: conflict-free reads); a wave's
    // rows are contiguous, so every cache line still comes from HBM once.
    // Lanes past the end repeat the last product.  Outer-product indexing
    // (pair products of channel mixing) takes rows b C1 + c1 and b C2 + c2.
    const int64_t p = p0 + (tid < cnt ? tid : cnt - 1);
    int64_t r1 = p, r2 = p;
    if constexpr (OUT) pair_rows(pi, p, r1, r2);
    const T1* const xr1 = x1 + r1 * K1;
    const T2* const xr2 = x2 + r2 * K2;
    cfor<0, K1>([&](auto I) { xa[decltype(I)::value] = ld_in(xr1, decltype(I)::value); });
    // x2 into its tile rows (the pair products' rows are not one slab)
    stage_tile_rows<L2, !OUT>(tile, x2, xr2, p0, cnt, tid, dma);
    if constexpr (WGT) {
      // each lane scales its own product: x1 in registers, x2 in its tile row
      const int64_t row = weight_row(wt, p0 + tid);
      if (wt.w1)
        scale_by_degree<L1, K1>(wt.w1 + row * (L1 + 1), [&](auto I) -> float& { return xa[decltype(I)::value]; });
      if (wt.w2)
        scale_by_degree<L2, K2>(wt.w2 + row * (L2 + 1),
                                [&](auto I) -> float& { return tile[tid * S2 + decltype(I)::value]; });
    }
    RegX<K1> A{xa};
    LdsX B{tile, tid * S2};
    gtp_core<L1, L2, LO, NU>(A, B, acc, ST, ntS, WT, ntW);
    if constexpr (WGT) {
      // outputs above degree LE are zeros and stay zeros
      if (wt.wo) {
        // the row index from an opaque copy of the lane id (not held across the core)
        int tq = threadIdx.x;
        asm volatile("" : "+v"(tq));
        scale_by_degree<G::LE, G::KE>(wt.wo + weight_row(wt, p0 + tq) * (LO + 1),
                                      [&](auto I) -> float& { return acc[decltype(I)::value]; });
      }
    }
    __syncthreads();
  } else {
    load_rows<K1>(x1, p0, cnt, xa);
    RegX<K1> A{xa};
    gtp_core<L1, L2, LO, NU>(A, A, acc, ST, ntS, WT, ntW);
  }
  store_rows<KO, G::KE>(y, p0, cnt, tile, acc);
}

// Both input gradients of an equal-degree product (the backward of Sec. 3.1's
// product, L1 = L2 = Lout = L <= 8): dx1 = P_L(GTP(dy, x2)) and then
// dx2 = P_L(GTP(dy, x1)), each the forward product on the compile-time
// tables of (L, L, L).  Each lane's dy row is read once and stays in
// registers for both products; x2, then x1, pass through the one LDS tile,
// and each gradient leaves through it as the forward's output does.  Against
// two forward launches this saves dy's second read: five rows move per
// product instead of six.  The two products run as a loop that is not
// unrolled, so the core's code is not duplicated.
template <int L, typename TX>
__global__ __launch_bounds__(kTile) __attribute__((amdgpu_waves_per_eu(small_waves(L, L, L)))) void k_bwd_small(
    const float* __restrict__ dy, const TX* __restrict__ x1, const TX* __restrict__ x2, float* __restrict__ dx1,
    float* __restrict__ dx2, int64_t n, int dma) {
  constexpr int K = csh(L), S = lds_stride(K);
  __shared__ __align__(16) float tile[kTile * S];
  lds_poison(tile, kTile * S);
  const int64_t p0 = int64_t(blockIdx.x) * kTile;
  const int cnt = int((n - p0) < kTile ? (n - p0) : kTile);
  float xd[K], acc[K];
  {
    const int tid = threadIdx.x;
    const float* const dr = dy + (p0 + (tid < cnt ? tid : cnt - 1)) * K;
    cfor<0, K>([&](auto I) { xd[decltype(I)::value] = dr[decltype(I)::value]; });
  }
#pragma unroll 1
  for (int g = 0; g < 2; ++g) {
    // dy's values opaque to the compiler in each product (its node
    // syntheses, the same in both, are not hoisted out of the loop and held:
    // that would take more registers than the core has), and the lane's row
    // addresses rebuilt from an opaque copy of the lane id in each product
    // rather than held across it
#pragma unroll
    for (int i = 0; i < K; ++i) asm volatile("" : "+v"(xd[i]));
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int64_t p = p0 + (tid < cnt ? tid : cnt - 1);
    const TX* const x = g == 0 ? x2 : x1;  // dx1 pairs dy with x2, dx2 with x1
    float* const out = g == 0 ? dx1 : dx2;
    stage_tile_rows<L, true>(tile, x, x + p * K, p0, cnt, tid, dma);
    gtp_core_lit<L>(RegX<K>{xd}, LdsX{tile, tid * S}, acc);
    __syncthreads();
    store_rows<K, K>(out, p0, cnt, tile, acc, tid);
    __syncthreads();  // the stores' tile reads are done before the next rows land there
  }
}

// Degree-padded product: a plan of degrees (a, b, c) whose padded degree
// L = max(a, b, min(c, a + b)) is at most 8 runs on the equal-degree core of
// degree L (compile-time tables).  The inputs are read as degree-L vectors
// whose coefficients above their own degrees are zero (rows of k1 = (a+1)^2
// and k2 = (b+1)^2 values), and the first ko = (c+1)^2 outputs are written
// (zeros above degree L when c > L).  Exact: the degree-L sampling grid
// integrates the product of any two degree-L functions exactly, and
// zero-padding or truncating the coefficient vectors changes nothing else.
template <int L, typename T1, typename T2>
__global__ __launch_bounds__(kTile) __attribute__((amdgpu_waves_per_eu(small_waves(L, L, L)))) void k_full_small_pad(
    const T1* __restrict__ x1, const T2* __restrict__ x2, float* __restrict__ y, int64_t n, int k1, int k2, int ko) {
  constexpr int K = csh(L), S = lds_stride(K);
  __shared__ __align__(16) float tile[kTile * S];
  lds_poison(tile, kTile * S);
  const int tid = threadIdx.x;
  const int64_t p0 = int64_t(blockIdx.x) * kTile;
  const int cnt = int((n - p0) < kTile ? (n - p0) : kTile);
  const int64_t p = p0 + (tid < cnt ? tid : cnt - 1);
  const int row = tid < cnt ? tid : cnt - 1;
  // The workgroup's rows of each input are one contiguous slab: coalesced
  // loads of the slab into the tile (compact rows of k floats), then each
  // lane takes its own row out of LDS, zero-padded to degree L.
  auto slab_to_tile = [&](auto src, int k) {
    const int tot = cnt * k;
    int e = tid;
    for (; e + 3 * kTile < tot; e += 4 * kTile) {
      const float v0 = ld_in(src, e), v1 = ld_in(src, e + kTile), v2 = ld_in(src, e + 2 * kTile),
                  v3 = ld_in(src, e + 3 * kTile);
      tile[e] = v0;
      tile[e + kTile] = v1;
      tile[e + 2 * kTile] = v2;
      tile[e + 3 * kTile] = v3;
    }
    for (; e < tot; e += kTile) tile[e] = ld_in(src, e);
    __syncthreads();
  };
  float xa[K];
  slab_to_tile(x1 + p0 * k1, k1);
  cfor<0, K>([&](auto I) {
    constexpr int i = decltype(I)::value;
    const float v = tile[row * k1 + (i < k1 ? i : 0)];  // in-bounds index, then the select
    xa[i] = i < k1 ? v : 0.0f;
  });
  __syncthreads();
  {
    float xb[K];
    slab_to_tile(x2 + p0 * k2, k2);
    cfor<0, K>([&](auto I) {
      constexpr int i = decltype(I)::value;
      const float v = tile[row * k2 + (i < k2 ? i : 0)];
      xb[i] = i < k2 ? v : 0.0f;
    });
    __syncthreads();
    cfor<0, K>([&](auto I) { tile[tid * S + decltype(I)::value] = xb[decltype(I)::value]; });
  }
  float acc[K];
  RegX<K> A{xa};
  LdsX B{tile, tid * S};
  gtp_core<L, L, L, 0>(A, B, acc, nullptr, 0, nullptr, 0);
  __syncthreads();
  if (ko <= K) {
    cfor<0, K>([&](auto I) {
      constexpr int i = decltype(I)::value;
      if (i < ko) tile[tid * ko + i] = acc[i];
    });
    __syncthreads();
    float* const out = y + p0 * ko;
    for (int i = tid; i < cnt * ko; i += kTile) out[i] = tile[i];
  } else if (tid < cnt) {
    float* const out = y + p * ko;
    cfor<0, K>([&](auto I) { out[decltype(I)::value] = acc[decltype(I)::value]; });
    for (int i = K; i < ko; ++i) out[i] = 0.0f;
  }
}

// Stepwise many-body chain: B_2 = P_LO(A A), B_{k+1} = P_LO(B_k A).
template <int L, int LO, typename TIn>
__global__ __launch_bounds__(kTile) void k_self_stepwise_small(const TIn* __restrict__ x, float* __restrict__ y,
                                                               int64_t n, int nu, DevTables t1, DevTables t2) {
  constexpr int K = csh(L), KO = csh(LO);
  using G1 = Geo<L, L, LO, 0>;
  using G2 = Geo<LO, L, LO, 0>;
  constexpr int KT = lds_stride(KO);  // the output rows (store_rows)
  __shared__ __align__(16) float tile[kTile * KT];
  lds_poison(tile, kTile * KT);
  const int64_t p0 = int64_t(blockIdx.x) * kTile;
  const int cnt = int((n - p0) < kTile ? (n - p0) : kTile);
  float a[K];
  load_rows<K>(x, p0, cnt, a);
  float b[KO];
  {
    float acc[G1::KE];
    RegX<K> A{a};
    gtp_core<L, L, LO, 0>(A, A, acc, t1.ST, t1.ntS, t1.WT, t1.ntW);
    cfor<0, KO>([&](auto I) {
      constexpr int i = decltype(I)::value;
      b[i] = i < G1::KE ? acc[i < G1::KE ? i : 0] : 0.0f;
    });
  }
  for (int step = 2; step < nu; ++step) {
    float acc[G2::KE];
    RegX<K> A{a};
    RegX<KO> Bv{b};
    gtp_core<LO, L, LO, 0>(Bv, A, acc, t2.ST, t2.ntS, t2.WT, t2.ntW);
    cfor<0, KO>([&](auto I) {
      constexpr int i = decltype(I)::value;
      b[i] = i < G2::KE ? acc[i < G2::KE ? i : 0] : 0.0f;
    });
  }
  store_rows<KO, KO>(y, p0, cnt, tile, b);
}

template <int L1, int L2, int LO, int NU, typename T1, typename T2, bool WGT, bool OUT = false>
hipError_t launch_typed(const DevTables& t, const void* x1, const void* x2, int64_t n, float* y,
                        const DegWeights& wt, hipStream_t s, const PairIdx& pi = PairIdx{0, 0}) {
  const dim3 grid(unsigned((n + kTile - 1) / kTile)), block(kTile);
  const int dma = (reinterpret_cast<uintptr_t>(x2) % 16) == 0;  // 16-byte runs straight into LDS
  hipLaunchKernelGGL((k_full_small<L1, L2, LO, NU, T1, T2, WGT, OUT>), grid, block, 0, s, static_cast<const T1*>(x1),
                     static_cast<const T2*>(x2), y, n, t.ST, t.ntS, t.WT, t.ntW, wt, pi, dma);
  return hipGetLastError();
}

// Input types: both fp32, both bf16, or (equal degrees only) fp32 x1 with
// bf16 x2, the pairing of a backward pass (fp32 output gradient times a bf16
// input).  Per-degree weights: equal degrees, equal input types.  Other
// combinations are not instantiated (*supported = false).
template <int L1, int L2, int LO, int NU>
hipError_t launch_one(const DevTables& t, const void* x1, int it1, const void* x2, int it2, int64_t n, float* y,
                      const DegWeights& wt, hipStream_t s, bool* supported) {
  constexpr bool equal = L1 == L2 && L2 == LO && NU == 0;
  if (wt.on) {
    if constexpr (equal) {
      if (it1 == IN_BF16 && it2 == IN_BF16)
        return launch_typed<L1, L2, LO, NU, uint16_t, uint16_t, true>(t, x1, x2, n, y, wt, s);
      if (it1 == IN_F32 && it2 == IN_F32) return launch_typed<L1, L2, LO, NU, float, float, true>(t, x1, x2, n, y, wt, s);
    }
    *supported = false;
    return hipSuccess;
  }
  if (it1 == IN_BF16 && it2 == IN_BF16)
    return launch_typed<L1, L2, LO, NU, uint16_t, uint16_t, false>(t, x1, x2, n, y, wt, s);
  if (it1 == IN_F32 && it2 == IN_F32) return launch_typed<L1, L2, LO, NU, float, float, false>(t, x1, x2, n, y, wt, s);
  if constexpr (equal) {
    if (it1 == IN_F32 && it2 == IN_BF16)
      return launch_typed<L1, L2, LO, NU, float, uint16_t, false>(t, x1, x2, n, y, wt, s);
  }
  *supported = false;
  return hipSuccess;
}

// Outer-product pair products (channel mixing), equal degrees, equal types.
template <int L>
hipError_t launch_pairs_one(const DevTables& t, const void* x1, int it1, const void* x2, int it2, int64_t n,
                            float* y, const PairIdx& pi, hipStream_t s, bool* supported) {
  const DegWeights nw{nullptr, nullptr, nullptr, 1, 0, 0, false};
  if (it1 == IN_F32 && it2 == IN_F32) return launch_typed<L, L, L, 0, float, float, false, true>(t, x1, x2, n, y, nw, s, pi);
  if (it1 == IN_BF16 && it2 == IN_BF16)
    return launch_typed<L, L, L, 0, uint16_t, uint16_t, false, true>(t, x1, x2, n, y, nw, s, pi);
  *supported = false;
  return hipSuccess;
}

// Fused channel mixing (the channel-mixing rule of the appendix, Implementation
// Details; equal degrees L, Kd = (L+1)^2):
//   y[b, co] = sum_p W[co, p] T[b, p],  T[b, p] = GTP(x1[b, c1], x2[b, c2]),
// p = c1 C2 + c2.  One workgroup (four waves) per batch entry, in rounds of
// 256 pairs: each lane takes one pair product with the thread-per-product
// core (x2 row in its LDS row), writes the product over that row, and after
// a barrier the waves mix the round's 256 products on the matrix cores,
//   y_b^T (Kd x Co) += T_round^T (Kd x 256) W^T_round (256 x Co),
// wave w taking the 16-coefficient row tiles w, w + 4, ... and every
// 16-channel column tile (v_mfma_f32_16x16x4f32: A[i][k] from lane 16 k + i,
// B[k][j] from lane 16 k + j, D register r of lane 16 g + i = row 4 g + r,
// column i).  K-step s of a round covers the pair slots 4 s + g; the weights
// come in the blocked layout WB[p / 16][co][g][s'] (p = 16 (p / 16) + 4 s' +
// g, zero past P and Co), so one 16-byte load gives a lane its B operands of
// four K-steps.  The partial y_b of each wave's tiles passes from one round
// to the next through y itself (each lane reads back what it wrote; the
// lines stay in L2), so no accumulator is live during the products.  Only
// x1, x2, W and y touch HBM.
typedef float mixv4 __attribute__((ext_vector_type(4)));
constexpr int kMixThreads = 256;
// waves per SIMD of the fused mix: the thread-per-product core's budget,
// except at L = 8 where the 81 KB tile admits one workgroup per CU anyway
constexpr int mix_waves(int L) { return L == 8 ? 1 : small_waves(L, L, L); }

template <int L, typename TIn, int NCT>
__global__ __launch_bounds__(kMixThreads) __attribute__((amdgpu_waves_per_eu(mix_waves(L)))) void k_mix_fused(
    const TIn* __restrict__ x1, const TIn* __restrict__ x2, const float* __restrict__ WB, float* __restrict__ y,
    int64_t C1, int64_t C2, int Co, int64_t P, const float* __restrict__ ST, int ntS, const float* __restrict__ WT,
    int ntW) {
  constexpr int Kd = csh(L);
  constexpr int NKT = (Kd + 15) / 16, KTW = (NKT + 3) / 4, CoB = 16 * NCT, KS = lds_stride(Kd);
  __shared__ float tile[kMixThreads * KS];
  lds_poison(tile, kMixThreads * KS);
  const int64_t b = blockIdx.x;
  const int64_t nround = (P + kMixThreads - 1) / kMixThreads;
  for (int64_t r = 0; r < nround; ++r) {
    // thread-derived indices from an opaque copy of the thread id each round
    // (recomputed, not held across the product)
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, wv = tid >> 6, g = lane >> 4, i = lane & 15;
    {
      // pair index split in 32 bits (the launcher takes C1 C2 < 2^31)
      const unsigned pl = unsigned(r) * kMixThreads + unsigned(tid);
      const unsigned pc = pl < unsigned(P) ? pl : unsigned(P) - 1u;
      const unsigned c1 = pc / unsigned(C2), c2 = pc - c1 * unsigned(C2);
      const TIn* const xr1 = x1 + (b * C1 + c1) * Kd;
      const TIn* const xr2 = x2 + (b * C2 + c2) * Kd;
      float xa[Kd], acc[Kd];
      cfor<0, Kd>([&](auto I) { xa[decltype(I)::value] = ld_in(xr1, decltype(I)::value); });
      cfor<0, Kd>([&](auto I) { tile[tid * KS + decltype(I)::value] = ld_in(xr2, decltype(I)::value); });
      RegX<Kd> A{xa};
      LdsX Bx{tile, tid * KS};
      gtp_core<L, L, L, 0>(A, Bx, acc, ST, ntS, WT, ntW);
      // over the lane's own row (its x2 reads are done).  Slots past P hold
      // a copy of the last pair's product; their weight rows are zero.
      cfor<0, Kd>([&](auto I) { tile[tid * KS + decltype(I)::value] = acc[decltype(I)::value]; });
    }
    // this wave's partial sums of the previous rounds (output rows k0 + 4 g +
    // rr of channel 16 ct + i) and its first weight block, requested before
    // the barrier so that they arrive while the other waves finish
    mixv4 macc[KTW][NCT], bw[KTW][NCT];
    const float* const wb = WB + ((r * 16) * CoB + i) * 16 + g * 4;
    cfor<0, KTW>([&](auto TT) {
      constexpr int t = decltype(TT)::value;
      const int k0 = (wv + 4 * t) * 16;
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) {
        const int co = ct * 16 + i;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int k = k0 + 4 * g + rr;
          macc[t][ct][rr] = (r > 0 && co < Co && k < Kd) ? y[(b * Co + co) * Kd + k] : 0.0f;
        }
        bw[t][ct] = *reinterpret_cast<const mixv4*>(wb + ct * 256);
      }
    });
    __syncthreads();
    cfor<0, KTW>([&](auto TT) {
      constexpr int t = decltype(TT)::value;
      const int k0 = (wv + 4 * t) * 16;
      if (k0 < Kd) {  // wave-uniform
        const int ka = k0 + i < Kd ? k0 + i : Kd - 1;
        const bool kok = k0 + i < Kd;
        mixv4 bn[NCT];
#pragma unroll 2
        for (int q = 0; q < 16; ++q) {
          float a[4];
#pragma unroll
          for (int sp = 0; sp < 4; ++sp) {
            const float v = tile[(16 * q + 4 * sp + g) * KS + ka];
            a[sp] = kok ? v : 0.0f;
          }
          const int qn = q + 1 < 16 ? q + 1 : q;
#pragma unroll
          for (int ct = 0; ct < NCT; ++ct)
            bn[ct] = *reinterpret_cast<const mixv4*>(wb + int64_t(qn) * CoB * 16 + ct * 256);
#pragma unroll
          for (int sp = 0; sp < 4; ++sp)
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct)
              macc[t][ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[sp], bw[t][ct][sp], macc[t][ct], 0, 0, 0);
#pragma unroll
          for (int ct = 0; ct < NCT; ++ct) bw[t][ct] = bn[ct];
        }
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) {
          const int co = ct * 16 + i;
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const int k = k0 + 4 * g + rr;
            if (co < Co && k < Kd) y[(b * Co + co) * Kd + k] = macc[t][ct][rr];
          }
        }
      }
    });
    __syncthreads();
  }
}

template <int L, typename TIn>
hipError_t launch_mix_fused_typed(const DevTables& t, const void* x1, const void* x2, const float* WB, float* y,
                                  int64_t B, int64_t C1, int64_t C2, int Co, int nct, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(B)), block(kMixThreads);
  const int64_t P = C1 * C2;
  const TIn* a = static_cast<const TIn*>(x1);
  const TIn* c = static_cast<const TIn*>(x2);
  switch (nct) {
    case 1:
      hipLaunchKernelGGL((k_mix_fused<L, TIn, 1>), grid, block, 0, s, a, c, WB, y, C1, C2, Co, P, t.ST, t.ntS, t.WT, t.ntW);
      break;
    case 2:
      hipLaunchKernelGGL((k_mix_fused<L, TIn, 2>), grid, block, 0, s, a, c, WB, y, C1, C2, Co, P, t.ST, t.ntS, t.WT, t.ntW);
      break;
    case 4:
      hipLaunchKernelGGL((k_mix_fused<L, TIn, 4>), grid, block, 0, s, a, c, WB, y, C1, C2, Co, P, t.ST, t.ntS, t.WT, t.ntW);
      break;
    case 8:
      hipLaunchKernelGGL((k_mix_fused<L, TIn, 8>), grid, block, 0, s, a, c, WB, y, C1, C2, Co, P, t.ST, t.ntS, t.WT, t.ntW);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int L>
hipError_t launch_mix_fused_one(const DevTables& t, const void* x1, const void* x2, int it, const float* WB, float* y,
                                int64_t B, int64_t C1, int64_t C2, int Co, int nct, hipStream_t s) {
  if (it == IN_BF16) return launch_mix_fused_typed<L, uint16_t>(t, x1, x2, WB, y, B, C1, C2, Co, nct, s);
  return launch_mix_fused_typed<L, float>(t, x1, x2, WB, y, B, C1, C2, Co, nct, s);
}

template <int L, int LO>
hipError_t launch_chain(const DevTables& t1, const DevTables& t2, int nu, const void* x, int in_type, int64_t n,
                        float* y, hipStream_t s) {
  const dim3 grid(unsigned((n + kTile - 1) / kTile)), block(kTile);
  if (in_type == IN_BF16)
    hipLaunchKernelGGL((k_self_stepwise_small<L, LO, uint16_t>), grid, block, 0, s,
                       static_cast<const uint16_t*>(x), y, n, nu, t1, t2);
  else
    hipLaunchKernelGGL((k_self_stepwise_small<L, LO, float>), grid, block, 0, s, static_cast<const float*>(x), y,
                       n, nu, t1, t2);
  return hipGetLastError();
}

}  // namespace

// (L1, L2, Lout) pair products and (L, nu, Lout) fused powers with a
// thread-per-product instantiation.  Everything else takes the generic path.
#define GTP_SMALL_PAIRS(X) \
  X(1, 1, 1) X(2, 2, 2) X(3, 3, 3) X(4, 4, 4) X(5, 5, 5) X(6, 6, 6) X(7, 7, 7) X(8, 8, 8) X(2, 2, 3) X(3, 2, 3) X(1, 2, 2) \
      X(2, 1, 3)
#define GTP_SMALL_POWERS(X) X(2, 2, 3) X(2, 3, 3) X(2, 4, 3) X(1, 3, 2) X(3, 3, 3)
#define GTP_SMALL_CHAINS(X) X(2, 3) X(1, 2) X(3, 3) X(2, 2)

hipError_t launch_full_small(const DevTables& t, const void* x1, int it1, const void* x2, int it2, int64_t n,
                             float* y, int nu, const DegWeights& wt, hipStream_t s, bool* supported) {
  *supported = true;
  if (nu == 0) {
#define GTP_CASE(a, b, c) \
  if (t.L1 == a && t.L2 == b && t.Lout == c) return launch_one<a, b, c, 0>(t, x1, it1, x2, it2, n, y, wt, s, supported);
    GTP_SMALL_PAIRS(GTP_CASE)
#undef GTP_CASE
  } else {
    // power plans are built as (L, (nu - 1) L, Lout)
#define GTP_CASE(a, v, c) \
  if (nu == v && t.L1 == a && t.L2 == (v - 1) * a && t.Lout == c) \
    return launch_one<a, 0, c, v>(t, x1, it1, x1, it1, n, y, wt, s, supported);
    GTP_SMALL_POWERS(GTP_CASE)
#undef GTP_CASE
  }
  *supported = false;
  return hipSuccess;
}

template <int L>
hipError_t launch_pad_one(const void* x1, int it1, const void* x2, int it2, int64_t n, float* y, int k1, int k2,
                          int ko, hipStream_t s, bool* supported) {
  const dim3 grid(unsigned((n + kTile - 1) / kTile)), block(kTile);
  if (it1 == IN_F32 && it2 == IN_F32)
    hipLaunchKernelGGL((k_full_small_pad<L, float, float>), grid, block, 0, s, static_cast<const float*>(x1),
                       static_cast<const float*>(x2), y, n, k1, k2, ko);
  else if (it1 == IN_BF16 && it2 == IN_BF16)
    hipLaunchKernelGGL((k_full_small_pad<L, uint16_t, uint16_t>), grid, block, 0, s, static_cast<const uint16_t*>(x1),
                       static_cast<const uint16_t*>(x2), y, n, k1, k2, ko);
  else if (it1 == IN_F32 && it2 == IN_BF16)
    hipLaunchKernelGGL((k_full_small_pad<L, float, uint16_t>), grid, block, 0, s, static_cast<const float*>(x1),
                       static_cast<const uint16_t*>(x2), y, n, k1, k2, ko);
  else {
    *supported = false;
    return hipSuccess;
  }
  return hipGetLastError();
}

template <int L>
hipError_t launch_bwd_one(const float* dy, const void* x1, const void* x2, int it, int64_t n, float* dx1, float* dx2,
                          hipStream_t s, bool* supported) {
  const dim3 grid(unsigned((n + kTile - 1) / kTile)), block(kTile);
  // 16-byte runs straight into LDS when both input slabs are aligned
  const int dma = ((reinterpret_cast<uintptr_t>(x1) | reinterpret_cast<uintptr_t>(x2)) % 16) == 0;
  if (it == IN_F32)
    hipLaunchKernelGGL((k_bwd_small<L, float>), grid, block, 0, s, dy, static_cast<const float*>(x1),
                       static_cast<const float*>(x2), dx1, dx2, n, dma);
  else if (it == IN_BF16)
    hipLaunchKernelGGL((k_bwd_small<L, uint16_t>), grid, block, 0, s, dy, static_cast<const uint16_t*>(x1),
                       static_cast<const uint16_t*>(x2), dx1, dx2, n, dma);
  else {
    *supported = false;
    return hipSuccess;
  }
  return hipGetLastError();
}

hipError_t launch_bwd_small(int L, const float* dy, const void* x1, const void* x2, int it, int64_t n, float* dx1,
                            float* dx2, hipStream_t s, bool* supported) {
  *supported = true;
  switch (L) {
    case 1: return launch_bwd_one<1>(dy, x1, x2, it, n, dx1, dx2, s, supported);
    case 2: return launch_bwd_one<2>(dy, x1, x2, it, n, dx1, dx2, s, supported);
    case 3: return launch_bwd_one<3>(dy, x1, x2, it, n, dx1, dx2, s, supported);
    case 4: return launch_bwd_one<4>(dy, x1, x2, it, n, dx1, dx2, s, supported);
    case 5: return launch_bwd_one<5>(dy, x1, x2, it, n, dx1, dx2, s, supported);
    case 6: return launch_bwd_one<6>(dy, x1, x2, it, n, dx1, dx2, s, supported);
    case 7: return launch_bwd_one<7>(dy, x1, x2, it, n, dx1, dx2, s, supported);
    default: break;  // L = 8: the forward's registers are already all in use; two launches
  }
  *supported = false;
  return hipSuccess;
}

hipError_t launch_full_small_padded(int L, const void* x1, int it1, int k1, const void* x2, int it2, int k2,
                                    int64_t n, float* y, int ko, hipStream_t s, bool* supported) {
  *supported = true;
  switch (L) {
    case 1: return launch_pad_one<1>(x1, it1, x2, it2, n, y, k1, k2, ko, s, supported);
    case 2: return launch_pad_one<2>(x1, it1, x2, it2, n, y, k1, k2, ko, s, supported);
    case 3: return launch_pad_one<3>(x1, it1, x2, it2, n, y, k1, k2, ko, s, supported);
    case 4: return launch_pad_one<4>(x1, it1, x2, it2, n, y, k1, k2, ko, s, supported);
    case 5: return launch_pad_one<5>(x1, it1, x2, it2, n, y, k1, k2, ko, s, supported);
    case 6: return launch_pad_one<6>(x1, it1, x2, it2, n, y, k1, k2, ko, s, supported);
    case 7: return launch_pad_one<7>(x1, it1, x2, it2, n, y, k1, k2, ko, s, supported);
    case 8: return launch_pad_one<8>(x1, it1, x2, it2, n, y, k1, k2, ko, s, supported);
    default: break;
  }
  *supported = false;
  return hipSuccess;
}

hipError_t launch_pairs_small(const DevTables& t, const void* x1, int it1, const void* x2, int it2, int64_t n,
                              float* y, const PairIdx& pi, hipStream_t s, bool* supported) {
  *supported = true;
  if (t.L1 == t.L2 && t.L2 == t.Lout) {
    switch (t.L1) {
      case 1: return launch_pairs_one<1>(t, x1, it1, x2, it2, n, y, pi, s, supported);
      case 2: return launch_pairs_one<2>(t, x1, it1, x2, it2, n, y, pi, s, supported);
      case 3: return launch_pairs_one<3>(t, x1, it1, x2, it2, n, y, pi, s, supported);
      case 4: return launch_pairs_one<4>(t, x1, it1, x2, it2, n, y, pi, s, supported);
      case 5: return launch_pairs_one<5>(t, x1, it1, x2, it2, n, y, pi, s, supported);
      case 6: return launch_pairs_one<6>(t, x1, it1, x2, it2, n, y, pi, s, supported);
      case 7: return launch_pairs_one<7>(t, x1, it1, x2, it2, n, y, pi, s, supported);
      case 8: return launch_pairs_one<8>(t, x1, it1, x2, it2, n, y, pi, s, supported);
      default: break;
    }
  }
  *supported = false;
  return hipSuccess;
}

int mix_fused_nct(int Co) {
  const int n = (Co + 15) / 16;
  if (n <= 1) return 1;
  if (n <= 2) return 2;
  if (n <= 4) return 4;
  if (n <= 8) return 8;
  return 0;
}

hipError_t launch_mix_fused(const DevTables& t, const void* x1, const void* x2, int it, const float* WB, float* y,
                            int64_t B, int64_t C1, int64_t C2, int Co, hipStream_t s, bool* supported) {
  *supported = false;
  const int nct = mix_fused_nct(Co);
  if (nct == 0 || t.L1 != t.L2 || t.L2 != t.Lout || B <= 0 || B > 0x7fffffff || C1 <= 0 || C2 <= 0 ||
      C1 * C2 > 0x7fffffff - kMixThreads)
    return hipSuccess;
  if (it != IN_F32 && it != IN_BF16) return hipSuccess;
  *supported = true;
  switch (t.L1) {
    case 1: return launch_mix_fused_one<1>(t, x1, x2, it, WB, y, B, C1, C2, Co, nct, s);
    case 2: return launch_mix_fused_one<2>(t, x1, x2, it, WB, y, B, C1, C2, Co, nct, s);
    case 3: return launch_mix_fused_one<3>(t, x1, x2, it, WB, y, B, C1, C2, Co, nct, s);
    case 4: return launch_mix_fused_one<4>(t, x1, x2, it, WB, y, B, C1, C2, Co, nct, s);
    case 5: return launch_mix_fused_one<5>(t, x1, x2, it, WB, y, B, C1, C2, Co, nct, s);
    case 6: return launch_mix_fused_one<6>(t, x1, x2, it, WB, y, B, C1, C2, Co, nct, s);
    case 7: return launch_mix_fused_one<7>(t, x1, x2, it, WB, y, B, C1, C2, Co, nct, s);
    case 8: return launch_mix_fused_one<8>(t, x1, x2, it, WB, y, B, C1, C2, Co, nct, s);
    default: break;
  }
  *supported = false;
  return hipSuccess;
}

hipError_t launch_self_stepwise_small(const DevTables& t1, const DevTables& t2, int nu, const void* x, int in_type,
                                      int64_t n, float* y, hipStream_t s, bool* supported) {
  *supported = true;
#define GTP_CASE(a, c) \
  if (t1.L1 == a && t1.L2 == a && t1.Lout == c && t2.L1 == c && t2.L2 == a && t2.Lout == c) \
    return launch_chain<a, c>(t1, t2, nu, x, in_type, n, y, s);
  GTP_SMALL_CHAINS(GTP_CASE)
#undef GTP_CASE
  *supported = false;
  return hipSuccess;
}

}  // namespace gtp
