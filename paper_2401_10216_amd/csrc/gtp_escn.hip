// Rotated-frame equivariant convolution (Sec. 3.3 "Equivariant Convolutions";
// Appendix, eq. sh2fs-escn) for L1 = L2 = Lout = L <= 8.
//
// y[b,c] = GTP(x[b,c], F_b) with the SH filter F_b = sum_l h[b,c,l] Y_l(r_b /
// |r_b|).  GTP commutes with rotations, so with a rotation R_b taking the
// edge direction to the pole and D_b its real-SH matrix,
//     y = D_b^T GTP(D_b x, D_b F_b),
// and D_b F_b has only m = 0 coefficients, h_l Theta_l0(0): the filter's 2D
// Fourier grid has only v = 0, so the product needs no phi transform at all.
// Per m-part the rotated x is synthesised at the theta nodes (mirror pairs),
// multiplied by the zonal filter and analysed back (the plan's S and W tables,
// with the phi-moment factor NP or NP / 2 folded into W).
//
// Two kernels.  k_escn_rot builds every edge's D_b = J^T Z(-beta) J Z(-alpha)
// once (Z: rotation about z; J: the fixed matrix of R_x(90 deg), J^T Z(t) J a
// rotation about y) into a workspace; k_conv_escn takes one workgroup per
// (edge, 64 channels), one product per lane: it loads D_b with its x slab,
// applies it to each lane's x, takes the zonal product and applies D_b^T.
// Its LDS holds the x tile, then D_b and the node-pair table, then the y
// tile: 12.5 KB at L = 6.
#include <type_traits>
#include <utility>

#include "gtp_ct.hpp"
#include "gtp_device.hpp"
#include "gtp_escn.hpp"

namespace gtp {
namespace {

constexpr int kEW = 64;

// Scheduling fence: bounds the loads the scheduler hoists ahead (each row of
// D read early holds registers until it is used).
#define GTP_ESCN_FENCE() __builtin_amdgcn_sched_barrier(0)

constexpr int ensh(int L) { return (L + 1) * (L + 1); }
// padded row length of the degree-l block of D in LDS (16-byte rows)
constexpr int erow(int l) { return (2 * l + 1 + 3) / 4 * 4; }
constexpr int dofs(int l) {
  int s = 0;
  for (int k = 0; k < l; ++k) s += (2 * k + 1) * erow(k);
  return s;
}
// offset of the degree-l block of J (and T) without padding
constexpr int jofs(int l) {
  int s = 0;
  for (int k = 0; k < l; ++k) s += (2 * k + 1) * (2 * k + 1);
  return s;
}

__device__ __forceinline__ float ld_x(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld_x(const uint16_t* p, int64_t i) { return __uint_as_float(uint32_t(p[i]) << 16); }

// node-pair table row (m-major, chunks padded to 4 floats): the unit zonal
// filter at t_j (L + 1 values), then per m Theta_lm(t_j) for l = m..L, then
// per m c_m W for l = m..L
constexpr int pad4(int n) { return (n + 3) / 4 * 4; }
template <int L>
struct EGeo {
  static constexpr int PZ = pad4(L + 1);
  static constexpr int OS(int m) {
    int o = PZ;
    for (int k = 0; k < m; ++k) o += pad4(L + 1 - k);
    return o;
  }
  static constexpr int OW(int m) { return OS(L + 1) + OS(m) - PZ; }
  static constexpr int ERL = OW(L + 1), NPAIR = L + 1;
};

// The node-pair rows as compile-time constants (EscnConsts<L>::E[j][..], the
// same fp64 builder and fp32 rounding as a plan's device copy): read with
// constant indices they are instruction literals, and the product loop needs
// neither loads nor LDS for them.
#include "gtp_escn_consts.inc"

// a += s x, or a = s x for the first term of a sum (a multiply-add onto zero
// would need the three-operand form, which cannot carry a literal)
template <bool FIRST>
__device__ __forceinline__ void emac(float& a, float s, float x) {
  if constexpr (FIRST) {
#pragma clang fp contract(off)
    a = s * x;
  } else {
    a = fmaf(s, x, a);
  }
}
// first degree l (l >= l0, step 2) with a non-zero entry E[j][off + l - base]
template <int L>
constexpr int first_nz(int j, int off, int base, int l0) {
  for (int l = l0; l <= L; l += 2)
    if (EscnConsts<L>::E[j][off + l - base] != 0.0f) return l;
  return -1;
}
// first node pair with a non-zero entry E[j][i]
template <int L>
constexpr int first_pair_nz(int i) {
  for (int j = 0; j < EscnConsts<L>::NPAIR; ++j)
    if (EscnConsts<L>::E[j][i] != 0.0f) return j;
  return -1;
}

// ---------------------------------------------------------------------------
// Per-edge rotation matrices: one wave per edge, four edges per workgroup.
// D_b = J^T Z(-beta) J Z(-alpha) for every degree l <= L, written in the
// padded row layout the product kernel reads (block l at dofs(l), rows of
// erow(l) floats, padding zero).
constexpr int kRotEdges = 4;

template <int L>
__global__ __launch_bounds__(64 * kRotEdges) void k_escn_rot(const float* __restrict__ r, int64_t B,
                                                             float* __restrict__ Dout, EscnDev t) {
  constexpr int H = L + 1, JS = jofs(L + 1), DS = dofs(L + 1);
  __shared__ float Jl[JS];
  __shared__ __align__(16) float Tw[kRotEdges][DS];  // T in D's padded row layout
  __shared__ float4 tw[kRotEdges][H];               // (cos m a, sin m a, cos m b, sin m b)
  lds_poison(Jl, JS);
  lds_poison(&Tw[0][0], kRotEdges * DS);
  lds_poison(reinterpret_cast<float*>(&tw[0][0]), kRotEdges * H * 4);
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int64_t b = int64_t(blockIdx.x) * kRotEdges + w;
  const bool valid = b < B;
  float* const Tl = Tw[w];
  float4* const trig = tw[w];
  for (int e = tid; e < JS; e += 64 * kRotEdges) Jl[e] = t.J[e];
  for (int e = lane; e < DS; e += 64) Tl[e] = 0.0f;  // row padding stays zero
  if (valid && lane <= L) {
    // the edge's angles (beta from the pole, alpha in the xy plane); a zero
    // vector takes the direction (0, 0, 1)
    const float rx = r[3 * b], ry = r[3 * b + 1], rz = r[3 * b + 2];
    const float rho = sqrtf(rx * rx + ry * ry);
    const float al = rho > 0.0f ? atan2f(ry, rx) : 0.0f;
    const float be = (rho > 0.0f || rz != 0.0f) ? atan2f(rho, rz) : 0.0f;
    float sa, ca, sb, cb;
    sincosf(float(lane) * al, &sa, &ca);
    sincosf(float(lane) * be, &sb, &cb);
    trig[lane] = make_float4(ca, sa, cb, sb);
  }
  __syncthreads();
  // T = Z(-beta) J Z(-alpha), block by block, in 2 x 2 mirror groups: rows
  // l +- p and columns l +- q (p, q >= 0) share four entries of J and the
  // trig values of orders p and q.  Z(-g) on a coefficient pair (c, s) of
  // order m > 0: c' = c cos mg + s sin mg, s' = -c sin mg + s cos mg.
  if (valid) {
    cfor<0, L + 1>([&](auto LL) {
      constexpr int l = decltype(LL)::value, d = 2 * l + 1, jo = jofs(l), ew = erow(l);
      for (int e = lane; e < (l + 1) * (l + 1); e += 64) {
        const int p = e / (l + 1), q = e - p * (l + 1);
        const float4 tq = trig[q], tp = trig[p];
        const float* Jr = Jl + jo + (l + p) * d;  // row l + p
        const float* Jm = Jl + jo + (l - p) * d;  // row l - p
        // (J Z(-alpha)) at rows l +- p, columns l + q (c) and l - q (s)
        float uc, us, vc, vs;
        if (q > 0) {
          uc = Jr[l + q] * tq.x - Jr[l - q] * tq.y;
          us = Jr[l - q] * tq.x + Jr[l + q] * tq.y;
          vc = Jm[l + q] * tq.x - Jm[l - q] * tq.y;
          vs = Jm[l - q] * tq.x + Jm[l + q] * tq.y;
        } else {
          uc = us = Jr[l];
          vc = vs = Jm[l];
        }
        float* Tr = Tl + dofs(l) + (l + p) * ew;
        float* Tm = Tl + dofs(l) + (l - p) * ew;
        if (p > 0) {
          Tr[l + q] = tp.z * uc + tp.w * vc;
          Tm[l + q] = -tp.w * uc + tp.z * vc;
          if (q > 0) {
            Tr[l - q] = tp.z * us + tp.w * vs;
            Tm[l - q] = -tp.w * us + tp.z * vs;
          }
        } else {
          Tr[l + q] = uc;
          if (q > 0) Tr[l - q] = us;
        }
      }
    });
  }
  __syncthreads();
  if (!valid) return;
  // D = J^T T: each item is four consecutive entries of one row (one J value
  // and one 16-byte quad of T per k), stored as one 16-byte write
  float* const Db = Dout + b * DS;
  cfor<0, L + 1>([&](auto LL) {
    constexpr int l = decltype(LL)::value, d = 2 * l + 1, jo = jofs(l), nq = erow(l) / 4;
    for (int e = lane; e < d * nq; e += 64) {
      const int a = e / nq, q = e - a * nq;
      float4 s = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      cfor<0, d>([&](auto KK) {
        constexpr int k = decltype(KK)::value;
        const float jv = Jl[jo + k * d + a];
        const float4 tv = reinterpret_cast<const float4*>(Tl + dofs(l) + k * erow(l))[q];
        s.x = fmaf(jv, tv.x, s.x);
        s.y = fmaf(jv, tv.y, s.y);
        s.z = fmaf(jv, tv.z, s.z);
        s.w = fmaf(jv, tv.w, s.w);
      });
      reinterpret_cast<float4*>(Db + dofs(l) + a * erow(l))[q] = s;
    }
  });
}

// ---------------------------------------------------------------------------
// The product: one workgroup (one wave) per (edge, 64 channels).

// degree of row R = l*l + a of the rotation blocks
constexpr int rdeg(int R) {
  int l = 0;
  while ((l + 1) * (l + 1) <= R) ++l;
  return l;
}
template <int E>
__device__ __forceinline__ float f4at(const float4& v) {
  if constexpr (E == 0) return v.x;
  else if constexpr (E == 1) return v.y;
  else if constexpr (E == 2) return v.z;
  else return v.w;
}
// the 16-byte chunks of row R of D (LDS)
template <int R, int NQ>
__device__ __forceinline__ void load_drow(const float* Dl, float4 (&buf)[NQ]) {
  constexpr int l = rdeg(R), a = R - l * l;
  const float4* row = reinterpret_cast<const float4*>(Dl + dofs(l) + a * erow(l));
  cfor<0, erow(l) / 4>([&](auto QQ) { buf[decltype(QQ)::value] = row[decltype(QQ)::value]; });
}

// register budget per lane: 3 waves per SIMD up to L = 6, 2 above
constexpr int escn_waves(int L) { return L <= 6 ? 3 : 2; }
// LDS stride of the x / y rows each lane reads or writes as its own: odd, so
// that one column of the 64 rows lies in 64 distinct banks (K = (L + 1)^2 is
// a multiple of 4 for odd L)
constexpr int escn_stride(int k) { return k | 1; }

template <int L, typename TIn>
__global__ __launch_bounds__(kEW) __attribute__((amdgpu_waves_per_eu(escn_waves(L)))) void k_conv_escn(
    const TIn* __restrict__ x, const float* __restrict__ Dall, const float* __restrict__ h, float* __restrict__ y,
    int64_t C, int ncb, int dma) {
  using EG = EGeo<L>;
  constexpr int K = ensh(L), H = L + 1, NPAIR = EG::NPAIR;
  static_assert(EscnConsts<L>::NPAIR == NPAIR && EscnConsts<L>::ERL == EG::ERL, "node-pair table layout");
  constexpr int DS = dofs(L + 1);
  constexpr int S = escn_stride(K);
  constexpr int XT = kEW * S;  // x / y tile
  // once the x rows are in registers the tile's space holds D (16-byte rows)
  static_assert(DS % 4 == 0 && DS <= XT, "LDS layout");
  constexpr int ND4 = DS / 4, RD = (ND4 + kEW - 1) / kEW;
  __shared__ __align__(16) float lds[XT];
  lds_poison(lds, XT);
  float* const tile = lds;
  float* const Dl = lds;

  const int tid = threadIdx.x;
  // XCD-aware: the ncb workgroups of an edge (which read its rotation
  // matrices) run on one XCD
  const int64_t wg = xcd_product(blockIdx.x, gridDim.x);
  const int64_t b = wg / ncb;
  const int64_t c0 = (wg % ncb) * kEW;
  const int cnt = int(C - c0 < kEW ? C - c0 : kEW);
  const int64_t p0 = b * C + c0;

  // ---- 1. every load issued before the first wait: this workgroup's x slab
  // (coalesced), the edge's rotation matrix (16-byte loads), the lane's
  // radial weights
  // (uniform base pointers, 32-bit lane offsets)
  const TIn* const xb = x + p0 * K;
  const unsigned nx = unsigned(cnt * K);
  float v[K];
  bool staged = false;
  if constexpr (std::is_same<TIn, float>::value) {
    if (S == K && dma && cnt == kEW && ((p0 * K) & 3) == 0) {
      // (odd K) the slab is laid out as the tile: coalesced 16-byte loads straight
      // into LDS (lane q 64 + tid carries floats 4 (q 64 + tid) .. + 3); a
      // whole number of 16-byte runs (64 K floats) from a 16-byte aligned
      // start (base checked by the host, offset here)
      typedef __attribute__((address_space(3))) void lds_void;
      typedef const __attribute__((address_space(1))) void glb_void;
      constexpr int NF = kEW * K, NQ = (NF + 255) / 256;
      cfor<0, NQ>([&](auto Q) {
        constexpr int q = decltype(Q)::value;
        const int e = (q * 64 + tid) * 4;
        if (q + 1 < NQ || e < NF)
          __builtin_amdgcn_global_load_lds((glb_void*)(xb + e), (lds_void*)(tile + q * 256), 16, 0, 0);
      });
      staged = true;
    }
  }
  if (!staged) {
    cfor<0, K>([&](auto I) {
      constexpr int k = decltype(I)::value;
      const unsigned i = unsigned(tid + k * kEW);
      v[k] = ld_x(xb, i < nx ? i : nx - 1);
    });
  }
  // (16-byte loads kept as plain floats; indices clamped into range: every
  // lane loads, so the values stay in registers; the out-of-range copies are
  // never stored)
  float dv[4 * RD];
  const float4* Dg = reinterpret_cast<const float4*>(Dall + b * DS);
  cfor<0, RD>([&](auto I) {
    constexpr int q = decltype(I)::value;
    const int i = tid + q * kEW;
    const float4 w = Dg[i < ND4 ? i : ND4 - 1];
    dv[4 * q] = w.x;
    dv[4 * q + 1] = w.y;
    dv[4 * q + 2] = w.z;
    dv[4 * q + 3] = w.w;
  });
  float hv[H];
  const float* const hb = h + p0 * H;
  const unsigned hl = unsigned(tid < cnt ? tid : cnt - 1);  // lanes past the last channel read a valid row
  cfor<0, H>([&](auto I) { hv[decltype(I)::value] = hb[hl * H + decltype(I)::value]; });

  // ---- 2. x rows into registers through the tile, then D into the tile's
  // space
  if (staged) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the slab is in LDS
  } else {
    cfor<0, K>([&](auto I) {
      // slab element i is row i / K, column i % K of the tile
      const int i = tid + decltype(I)::value * kEW;
      const int r = i / K;
      tile[r * S + (i - r * K)] = v[decltype(I)::value];
    });
  }
  __syncthreads();
  float xr[K];
  cfor<0, K>([&](auto I) { xr[decltype(I)::value] = tile[tid * S + decltype(I)::value]; });
  __syncthreads();
  cfor<0, RD>([&](auto I) {
    constexpr int q = decltype(I)::value;
    const int i = tid + q * kEW;
    if (i < ND4) reinterpret_cast<float4*>(Dl)[i] = make_float4(dv[4 * q], dv[4 * q + 1], dv[4 * q + 2], dv[4 * q + 3]);
  });
  __syncthreads();
  // ---- 3. x' = D x, row by row over all degrees (row R = l*l + a); each
  // row's 16-byte LDS reads (the same address in every lane) are issued
  // before the previous row is consumed
  constexpr int NQM = erow(L) / 4;
  float xp[K];
  {
    float4 cur[NQM], nxt[NQM];
    load_drow<0>(Dl, cur);
    cfor<0, K>([&](auto RR) {
      constexpr int R = decltype(RR)::value, l = rdeg(R), d = 2 * l + 1;
      if constexpr (R + 1 < K) load_drow<R + 1>(Dl, nxt);
      GTP_ESCN_FENCE();
      float s = 0.0f;
      cfor<0, erow(l) / 4>([&](auto QQ) {
        constexpr int q = decltype(QQ)::value;
        cfor<0, 4>([&](auto EE) {
          constexpr int bb = 4 * q + decltype(EE)::value;
          if constexpr (bb < d) s = fmaf(f4at<decltype(EE)::value>(cur[q]), xr[l * l + bb], s);
        });
      });
      xp[R] = s;
      GTP_ESCN_FENCE();
      if constexpr (R + 1 < K) cfor<0, NQM>([&](auto QQ) { cur[decltype(QQ)::value] = nxt[decltype(QQ)::value]; });
    });
  }

  // ---- 4. product with the zonal filter, mirror pair by mirror pair (the
  // pair loop unrolled: table values are literals, zero entries dropped)
  float acc[K];
  cfor<0, K>([&](auto I) { acc[decltype(I)::value] = 0.0f; });
  cfor<0, NPAIR>([&](auto JJ) {
    constexpr int j = decltype(JJ)::value;
    GTP_ESCN_FENCE();
    // filter at t_j and its mirror (Theta_l0(pi - t) = (-1)^l Theta_l0(t))
    float fe = 0.0f, fo = 0.0f;
    cfor<0, H>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      constexpr float z = EscnConsts<L>::E[j][l];
      if constexpr (z != 0.0f) {
        if constexpr (l % 2 == 0) emac<l == first_nz<L>(j, 0, 0, 0)>(fe, z, hv[l]);
        else emac<l == first_nz<L>(j, 0, 0, 1)>(fo, z, hv[l]);
      }
    });
    const float fj = fe + fo, fm = fe - fo;
    cfor<0, L + 1>([&](auto MM) {
      constexpr int m = decltype(MM)::value;
      cfor<0, (m == 0 ? 1 : 2)>([&](auto SS) {
        constexpr int sg = decltype(SS)::value;  // 0: cos part (+m), 1: sin part (-m)
        float ae = 0.0f, ao = 0.0f;
        cfor<m, L + 1>([&](auto LL) {
          constexpr int l = decltype(LL)::value, i = l * l + l + (sg ? -m : m);
          constexpr float sv = EscnConsts<L>::E[j][EG::OS(m) + l - m];
          if constexpr (sv != 0.0f) {
            if constexpr ((l + m) % 2 == 0) emac<l == first_nz<L>(j, EG::OS(m), m, m)>(ae, sv, xp[i]);
            else emac<l == first_nz<L>(j, EG::OS(m), m, m + 1)>(ao, sv, xp[i]);
          }
        });
        const float pj = fj * (ae + ao), pm = fm * (ae - ao);
        const float pe = pj + pm, po = pj - pm;
        cfor<m, L + 1>([&](auto LL) {
          constexpr int l = decltype(LL)::value, i = l * l + l + (sg ? -m : m);
          constexpr int wi = EG::OW(m) + l - m;
          constexpr float wv = EscnConsts<L>::E[j][wi];
          if constexpr (wv != 0.0f) emac<j == first_pair_nz<L>(wi)>(acc[i], wv, (l + m) % 2 == 0 ? pe : po);
        });
      });
      GTP_ESCN_FENCE();
    });
  });
  GTP_ESCN_FENCE();

  // ---- 5. y = D^T y', row by row with the same prefetch
  float yv[K];
  cfor<0, K>([&](auto I) { yv[decltype(I)::value] = 0.0f; });
  {
    float4 cur[NQM], nxt[NQM];
    load_drow<0>(Dl, cur);
    cfor<0, K>([&](auto RR) {
      constexpr int R = decltype(RR)::value, l = rdeg(R), d = 2 * l + 1;
      if constexpr (R + 1 < K) load_drow<R + 1>(Dl, nxt);
      GTP_ESCN_FENCE();
      cfor<0, erow(l) / 4>([&](auto QQ) {
        constexpr int q = decltype(QQ)::value;
        cfor<0, 4>([&](auto EE) {
          constexpr int bb = 4 * q + decltype(EE)::value;
          if constexpr (bb < d) yv[l * l + bb] = fmaf(f4at<decltype(EE)::value>(cur[q]), acc[R], yv[l * l + bb]);
        });
      });
      GTP_ESCN_FENCE();
      if constexpr (R + 1 < K) cfor<0, NQM>([&](auto QQ) { cur[decltype(QQ)::value] = nxt[decltype(QQ)::value]; });
    });
  }

  // ---- 6. store through the tile (coalesced)
  __syncthreads();  // every lane is done with D and the table
  cfor<0, K>([&](auto I) { tile[tid * S + decltype(I)::value] = yv[decltype(I)::value]; });
  __syncthreads();
  // store indices from an opaque copy of the lane id: not kept alive from the
  // loads' index arithmetic
  int ln = tid;
  asm volatile("" : "+v"(ln));
  float* const yb = y + p0 * K;
  if (cnt == kEW && (reinterpret_cast<uintptr_t>(yb) & 15) == 0) {
    // a full workgroup's rows (64 K floats, a whole number of 16-byte runs)
    // in 16-byte stores from the 16-byte aligned tile
    typedef float sv4 __attribute__((ext_vector_type(4)));
    constexpr int N4 = kEW * K / 4, NQ = (N4 + kEW - 1) / kEW;
    cfor<0, NQ>([&](auto Q) {
      const int i4 = ln + decltype(Q)::value * kEW;
      if (i4 < N4) {
        if constexpr (S == K) {
          __builtin_nontemporal_store(reinterpret_cast<const sv4*>(tile)[i4], reinterpret_cast<sv4*>(yb) + i4);
        } else {
          // padded rows; K is a multiple of 4, so no 16-byte run crosses a row
          const int r = (4 * i4) / K;
          const float* const t = tile + r * S + (4 * i4 - r * K);
          __builtin_nontemporal_store(sv4{t[0], t[1], t[2], t[3]}, reinterpret_cast<sv4*>(yb) + i4);
        }
      }
    });
  } else {
    cfor<0, K>([&](auto I) {
      const unsigned i = unsigned(ln + decltype(I)::value * kEW);
      const unsigned r = i / unsigned(K);
      if (i < nx) yb[i] = tile[r * S + (i - r * K)];
    });
  }
}

template <int L>
hipError_t launch_l(const EscnDev& e, const void* x, int in_type, const float* r, const float* h, int64_t B,
                    int64_t C, float* y, float* dws, hipStream_t s) {
  if (e.ERL != EGeo<L>::ERL) return hipErrorInvalidValue;  // table layout and kernel disagree
  const int64_t ncb = (C + kEW - 1) / kEW;
  if (B * ncb > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((k_escn_rot<L>), dim3(unsigned((B + kRotEdges - 1) / kRotEdges)), dim3(64 * kRotEdges), 0, s, r,
                     B, dws, e);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const dim3 grid(unsigned(B * ncb)), block(kEW);
  if (in_type == IN_BF16)
    hipLaunchKernelGGL((k_conv_escn<L, uint16_t>), grid, block, 0, s, static_cast<const uint16_t*>(x), dws, h, y, C,
                       int(ncb), 0);
  else
    hipLaunchKernelGGL((k_conv_escn<L, float>), grid, block, 0, s, static_cast<const float*>(x), dws, h, y, C,
                       int(ncb), int(reinterpret_cast<uintptr_t>(x) % 16 == 0));
  return hipGetLastError();
}

}  // namespace

int64_t escn_rot_floats(int L) {
  return (L >= 1 && L <= 8) ? dofs(L + 1) : 0;
}

hipError_t launch_conv_escn(const EscnDev& e, int L1, int L2, int Lout, const void* x, int in_type, const float* r,
                            const float* h, int64_t B, int64_t C, float* y, float* dws, hipStream_t s,
                            bool* supported) {
  *supported = true;
  if (L1 == L2 && L2 == Lout && e.E && e.LM == L1 && e.NPAIR == L1 + 1) {
    switch (L1) {
      case 1: return launch_l<1>(e, x, in_type, r, h, B, C, y, dws, s);
      case 2: return launch_l<2>(e, x, in_type, r, h, B, C, y, dws, s);
      case 3: return launch_l<3>(e, x, in_type, r, h, B, C, y, dws, s);
      case 4: return launch_l<4>(e, x, in_type, r, h, B, C, y, dws, s);
      case 5: return launch_l<5>(e, x, in_type, r, h, B, C, y, dws, s);
      case 6: return launch_l<6>(e, x, in_type, r, h, B, C, y, dws, s);
      case 7: return launch_l<7>(e, x, in_type, r, h, B, C, y, dws, s);
      case 8: return launch_l<8>(e, x, in_type, r, h, B, C, y, dws, s);
      default: break;
    }
  }
  if (L1 == L2 && L2 == Lout && L1 == kEscnWaveL && e.A && e.JI && e.LM == kEscnWaveL)
    return launch_conv_escn_wave(e, x, in_type, r, h, B, C, y, ensh(L1), L2 + 1, ensh(Lout), s);
  *supported = false;
  return hipSuccess;
}

}  // namespace gtp
