// Rotated-frame equivariant convolution (Sec. 3.3 "Equivariant Convolutions";
// Appendix, eq. sh2fs-escn) at degree 16 on the fp32 matrix cores.
//
// Same computation as the small-degree kernel (y = D_b^T Z(D_b x, h), Z the
// product with a zonal filter taken per order m at the theta nodes), but the
// per-product state (289 coefficients) does not fit one lane's registers, so
// the work is laid out across the channels of an edge, which share D_b and
// every table: each stage is a small dense contraction with the 16 channels
// of a wave as the N index of v_mfma_f32_16x16x4f32 (A[i][k] from lane 16 k +
// i, B[k][j] from lane 16 k + j, register r of lane 16 g + i = row 4 g + r,
// column i):
//   rotate in    x'_l (rows 2l+1) = D_l x_l, per degree block, in place;
//   synthesis    per m-part (m, cos / sin) and degree parity (l - m even /
//                odd): the partial sums at the 16 interior node pairs,
//                G[pair][c] = sum_l Theta_lm(t_pair) x'[(l, m)][c] (row 4 g + r
//                of the tile is node pair 4 r + g + 1);
//   product      with the zonal filter at the pair's node and its mirror
//                (f = fe +- fo, g = ge +- go), folded to even and odd parts;
//   analysis     y'[(l, m)][c] = sum_pair c_m W_lm(t_pair) P[pair][c]: K-step
//                r takes register r of every lane (node pairs 4 r + g + 1, as
//                the synthesis left them), so nothing moves between the two;
//   poles        (only m = 0 is non-zero there) on the VALU;
//   rotate out   y_l = D_l^T y'_l.
// One workgroup per (edge, 64 channels), one wave per 16 channels; LDS holds
// the edge's D_b (compact rows of odd length 2l+1, as the rotation kernel
// writes them above L = 8: conflict-free column and row reads) and each
// wave's coefficient tile [k][16 channels], which the stages rewrite in place
// (100 KB: one workgroup per CU, so the kernel keeps every load of a stage in
// flight at once and prefetches the next order's operands).
#include <type_traits>

#include "gtp_ct.hpp"
#include "gtp_device.hpp"
#include "gtp_escn.hpp"

namespace gtp {
namespace {

constexpr int kWL = kEscnWaveL;            // 16
constexpr int kWK = (kWL + 1) * (kWL + 1);  // 289 coefficients
constexpr int kWH = kWL + 1;                // 17 radial weights
constexpr int kWaves = 4;                   // 16-channel tiles per workgroup
// floats of one wave's tile: rows 0..288, row 289 takes the writes of
// padding rows, rows up to 291 the reads past the last block (whose values
// are then dropped)
constexpr int kTileF = (kWK + 3) * 16;

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f4 mfma(float a, float b, f4 c) { return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0); }

// compact D: block l at cofs(l), rows of 2l+1 floats
constexpr int cofs(int l) {
  int s = 0;
  for (int k = 0; k < l; ++k) s += (2 * k + 1) * (2 * k + 1);
  return s;
}
constexpr int kDC = cofs(kWL + 1);  // 6545
// D in LDS with room for the reads past its last block (row 47, column 35 of
// the 33 x 33 block: values dropped)
constexpr int kDCL = cofs(kWL) + 47 * (2 * kWL + 1) + 36;

// The stages rewrite the tile in place: lanes read rows that other lanes then
// overwrite, and read rows that other lanes wrote.  The wave issues its LDS
// operations in program order and the LDS performs them in that order; this
// fence keeps the compiler from moving a lane's LDS reads and writes across
// it (it only sees the lane's own addresses).
#define GTP_TILE_ORDER() asm volatile("" ::: "memory")

__device__ __forceinline__ float ldx(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ldx(const uint16_t* p, int64_t i) { return __uint_as_float(uint32_t(p[i]) << 16); }

template <typename TIn>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_conv_escn_wave(
    const TIn* __restrict__ x, const float* __restrict__ Dall, const float* __restrict__ h, float* __restrict__ y,
    int64_t C, int ncb, const float* __restrict__ At, const float* __restrict__ Zt, int k1, int kh, int ko) {
  __shared__ __align__(16) float Dl[kDCL];
  __shared__ __align__(16) float tiles[kWaves * kTileF];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, g = lane >> 4, i = lane & 15;
  // XCD-aware: the ncb workgroups of an edge (which read its rotation
  // matrices) run on one XCD
  const int64_t wg = xcd_product(blockIdx.x, gridDim.x);
  const int64_t b = wg / ncb;
  const int64_t c0 = (wg % ncb) * (16 * kWaves) + 16 * w;  // first channel of this wave
  const int cnt = C - c0 <= 0 ? 0 : (C - c0 < 16 ? int(C - c0) : 16);
  float* const X = tiles + w * kTileF;  // rows 0..288; row 289 takes the writes of padding rows

  // ---- 1. every load in flight before the first use: the wave's x tile
  // (lane (g, c) takes rows g, g + 4, ..: 16 B of each of 16 rows per load),
  // its share of D_b, the radial weights of channel i, the operands of m = 0
  constexpr int NXL = (kWK + 3) / 4;  // 73 rows per lane group
  float xv[NXL];
  {
    // unconditional loads from clamped addresses (a valid row of the edge,
    // a valid column), then the select: no divergent branches
    const int c = lane & 15;
    const int64_t ch = c0 + c < C ? c0 + c : C - 1;
    const TIn* const xr = x + (b * C + ch) * int64_t(k1);
    cfor<0, NXL>([&](auto Q) {
      constexpr int q = decltype(Q)::value;
      const int k = g + 4 * q;
      const float v = ldx(xr, k < k1 ? k : k1 - 1);
      xv[q] = (c < cnt && k < k1) ? v : 0.0f;
    });
  }
  constexpr int NDL = (kDC + 64 * kWaves - 1) / (64 * kWaves);  // 26 entries of D per thread
  float dv[NDL];
  {
    const float* const Db = Dall + b * kDC;  // compact rows (the rotation kernel's layout above L = 8)
    cfor<0, NDL>([&](auto Q) {
      const int e = tid + decltype(Q)::value * 64 * kWaves;
      dv[decltype(Q)::value] = Db[e < kDC ? e : 0];
    });
  }
  float hv[kWH];
  {
    const int64_t ch = c0 + i < C ? c0 + i : C - 1;
    const float* const hb = h + (b * C + ch) * int64_t(kh);
    cfor<0, kWH>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      const float v = hb[l < kh ? l : kh - 1];
      hv[l] = (i < cnt && l < kh) ? v : 0.0f;
    });
  }
  f4 avq[2][4];  // the operands of order m (and m + 1, prefetched), four quads
  auto load_ops = [&](auto MM, f4(&dst)[4]) {
    constexpr int m = decltype(MM)::value, NL = escn_wave_lane_floats(kWL, m);
    const f4* const src = reinterpret_cast<const f4*>(At + escn_wave_moff(kWL, m) + lane * NL);
    cfor<0, NL / 4>([&](auto Q) { dst[decltype(Q)::value] = src[decltype(Q)::value]; });
  };
  load_ops(std::integral_constant<int, 0>{}, avq[0]);
  cfor<0, NXL>([&](auto Q) {
    constexpr int q = decltype(Q)::value;
    const int k = g + 4 * q;
    X[(k < kWK ? k : kWK) * 16 + i] = xv[q];
  });
  cfor<0, NDL>([&](auto Q) {
    constexpr int q = decltype(Q)::value;
    const int e = tid + q * 64 * kWaves;
    if (q + 1 < NDL || e < kDC) Dl[e < kDC ? e : 0] = dv[q];
  });
  // the zonal filter at the lane's node pairs 4 r + g + 1 (even and odd
  // degrees apart) and at the poles
  f4 FE, FO;
  float fe0 = 0.0f, fo0 = 0.0f;
  {
    const float* const zg = Zt + g * 4 * kWH;
    cfor<0, 4>([&](auto RR) {
      constexpr int r = decltype(RR)::value;
      float e = 0.0f, o = 0.0f;
      cfor<0, kWH>([&](auto LL) {
        constexpr int l = decltype(LL)::value;
        if constexpr (l % 2 == 0) e = fmaf(zg[r * kWH + l], hv[l], e);
        else o = fmaf(zg[r * kWH + l], hv[l], o);
      });
      FE[r] = e;
      FO[r] = o;
    });
    const float* const zp = Zt + 16 * kWH;
    cfor<0, kWH>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      if constexpr (l % 2 == 0) fe0 = fmaf(zp[l], hv[l], fe0);
      else fo0 = fmaf(zp[l], hv[l], fo0);
    });
  }
  __syncthreads();

  // LDS reads are unconditional (clamped addresses; the value then selected),
  // writes of padding rows go to the spare row kWK: no divergent branches.
  auto xrd = [&](int row, bool ok) {
    const float v = X[(ok ? row : 0) * 16 + i];
    return ok ? v : 0.0f;
  };
  // the same for rows past a degree block, which stay inside the tile
  auto xrd_block = [&](int row, bool ok) {
    const float v = X[row * 16 + i];
    return ok ? v : 0.0f;
  };
  // ---- 2. rotate in (M = rows of D_l, K = its columns), two degree blocks
  // at a time: the MFMAs of both, then their writes (blocks touch disjoint
  // rows; a block's reads precede its writes)
  auto rot_in_mma = [&](auto LL, auto& acc) {
    constexpr int l = decltype(LL)::value, d = 2 * l + 1, NM = (d + 15) / 16, NK = (d + 3) / 4, R0 = l * l;
    cfor<0, NM>([&](auto M) { acc[decltype(M)::value] = f4{0.0f, 0.0f, 0.0f, 0.0f}; });
    cfor<0, NK>([&](auto KS) {
      constexpr int ks = decltype(KS)::value;
      const int a = 4 * ks + g;
      const float bv = xrd_block(R0 + a, a < d);
      cfor<0, NM>([&](auto M) {
        constexpr int mt = decltype(M)::value;
        const int row = 16 * mt + i;
        const bool ok = row < d && a < d;
        const float t = Dl[cofs(l) + row * d + a];
        acc[mt] = mfma(ok ? t : 0.0f, bv, acc[mt]);
      });
    });
  };
  auto rot_in_store = [&](auto LL, const auto& acc) {
    constexpr int l = decltype(LL)::value, d = 2 * l + 1, NM = (d + 15) / 16, R0 = l * l;
    cfor<0, NM>([&](auto M) {
      constexpr int mt = decltype(M)::value;
      cfor<0, 4>([&](auto RR) {
        constexpr int r = decltype(RR)::value;
        const int row = 16 * mt + 4 * g + r;
        X[(row < d ? R0 + row : kWK) * 16 + i] = acc[mt][r];
      });
    });
  };
  cfor<0, (kWL + 2) / 2>([&](auto PP) {
    constexpr int l0 = 2 * decltype(PP)::value, l1 = l0 + 1 <= kWL ? l0 + 1 : l0;
    constexpr int NM0 = (2 * l0 + 1 + 15) / 16, NM1 = (2 * l1 + 1 + 15) / 16;
    f4 a0[NM0], a1[NM1];
    rot_in_mma(std::integral_constant<int, l0>{}, a0);
    if constexpr (l1 != l0) rot_in_mma(std::integral_constant<int, l1>{}, a1);
    GTP_TILE_ORDER();
    rot_in_store(std::integral_constant<int, l0>{}, a0);
    if constexpr (l1 != l0) rot_in_store(std::integral_constant<int, l1>{}, a1);
  });
  GTP_TILE_ORDER();

  // ---- 3. the zonal product per order m, its cos and sin parts together
  // (m-parts touch disjoint rows)
  const float* const zp = Zt + 16 * kWH;
  cfor<0, kWL + 1>([&](auto MM) {
    constexpr int m = decltype(MM)::value, n = kWL + 1 - m, NE = (n + 1) / 2, NO = n / 2;
    constexpr int KE = (NE + 3) / 4, KO = (NO + 3) / 4, NSG = m == 0 ? 1 : 2;
    f4(&cur)[4] = avq[m & 1];
    if constexpr (m + 1 <= kWL) load_ops(std::integral_constant<int, m + 1>{}, avq[(m + 1) & 1]);
    auto av = [&](int t) { return cur[t >> 2][t & 3]; };
    auto row_of = [](int l, int sg) { return l * l + l + (sg ? -m : m); };
    f4 GE[NSG], GO[NSG];
    cfor<0, NSG>([&](auto SG) {
      constexpr int sg = decltype(SG)::value;  // 0: cos part (+m), 1: sin part (-m)
      GE[sg] = f4{0.0f, 0.0f, 0.0f, 0.0f};
      GO[sg] = GE[sg];
    });
    cfor<0, KE>([&](auto KS) {
      constexpr int ks = decltype(KS)::value;
      const int l = m + 2 * (4 * ks + g);
      cfor<0, NSG>([&](auto SG) {
        constexpr int sg = decltype(SG)::value;
        GE[sg] = mfma(av(ks), xrd(row_of(l, sg), l <= kWL), GE[sg]);
      });
    });
    cfor<0, KO>([&](auto KS) {
      constexpr int ks = decltype(KS)::value;
      const int l = m + 1 + 2 * (4 * ks + g);
      cfor<0, NSG>([&](auto SG) {
        constexpr int sg = decltype(SG)::value;
        GO[sg] = mfma(av(KE + ks), xrd(row_of(l, sg), l <= kWL), GO[sg]);
      });
    });
    // pole pair (m = 0 only): the lane's channel, every lane group alike
    float pe0 = 0.0f, po0 = 0.0f;
    if constexpr (m == 0) {
      float ae = 0.0f, ao = 0.0f;
      cfor<0, kWH>([&](auto LL) {
        constexpr int l = decltype(LL)::value;
        const float v = zp[kWH + l] * X[(l * l + l) * 16 + i];
        if constexpr (l % 2 == 0) ae += v;
        else ao += v;
      });
      const float pj = (fe0 + fo0) * (ae + ao), pm = (fe0 - fo0) * (ae - ao);
      pe0 = pj + pm;
      po0 = pj - pm;
    }
    f4 YE[NSG], YO[NSG];
    cfor<0, NSG>([&](auto SG) {
      constexpr int sg = decltype(SG)::value;
      // products at the node (f, g = even + odd) and its mirror (even - odd)
      const f4 pj = (FE + FO) * (GE[sg] + GO[sg]), pm = (FE - FO) * (GE[sg] - GO[sg]);
      const f4 PE = pj + pm, PO = pj - pm;
      YE[sg] = f4{0.0f, 0.0f, 0.0f, 0.0f};
      YO[sg] = YE[sg];
      cfor<0, 4>([&](auto RR) {
        constexpr int r = decltype(RR)::value;
        YE[sg] = mfma(av(KE + KO + r), PE[r], YE[sg]);
        if constexpr (NO > 0) YO[sg] = mfma(av(KE + KO + 4 + r), PO[r], YO[sg]);
      });
    });
    // rows 4 g + r of the tiles: degrees m + 2 (4 g + r) (even set) and
    // m + 1 + 2 (4 g + r) (odd set), over the x' rows of this order
    GTP_TILE_ORDER();
    cfor<0, NSG>([&](auto SG) {
      constexpr int sg = decltype(SG)::value;
      cfor<0, 4>([&](auto RR) {
        constexpr int r = decltype(RR)::value;
        const int ie = 4 * g + r;
        {
          const int l = m + 2 * ie;
          float v = YE[sg][r];
          if constexpr (m == 0) v = fmaf(zp[2 * kWH + (ie < NE ? l : 0)], pe0, v);
          X[(ie < NE ? row_of(l, sg) : kWK) * 16 + i] = v;
        }
        if constexpr (NO > 0) {
          const int l = m + 1 + 2 * ie;
          float v = YO[sg][r];
          if constexpr (m == 0) v = fmaf(zp[2 * kWH + (ie < NO ? l : 0)], po0, v);
          X[(ie < NO ? row_of(l, sg) : kWK) * 16 + i] = v;
        }
      });
    });
  });
  GTP_TILE_ORDER();

  // ---- 4. rotate out (M = columns of D_l, K = its rows), two blocks at a
  // time; blocks past Lout are skipped
  auto rot_out_mma = [&](auto LL, auto& acc) {
    constexpr int l = decltype(LL)::value, d = 2 * l + 1, NM = (d + 15) / 16, NK = (d + 3) / 4, R0 = l * l;
    cfor<0, NM>([&](auto M) { acc[decltype(M)::value] = f4{0.0f, 0.0f, 0.0f, 0.0f}; });
    cfor<0, NK>([&](auto KS) {
      constexpr int ks = decltype(KS)::value;
      const int rr = 4 * ks + g;
      const float bv = xrd_block(R0 + rr, rr < d);
      cfor<0, NM>([&](auto M) {
        constexpr int mt = decltype(M)::value;
        const int a = 16 * mt + i;
        const bool ok = a < d && rr < d;
        const float t = Dl[cofs(l) + rr * d + a];
        acc[mt] = mfma(ok ? t : 0.0f, bv, acc[mt]);
      });
    });
  };
  auto rot_out_store = [&](auto LL, const auto& acc) {
    constexpr int l = decltype(LL)::value, d = 2 * l + 1, NM = (d + 15) / 16, R0 = l * l;
    cfor<0, NM>([&](auto M) {
      constexpr int mt = decltype(M)::value;
      cfor<0, 4>([&](auto RR) {
        constexpr int r = decltype(RR)::value;
        const int a = 16 * mt + 4 * g + r;
        X[(a < d ? R0 + a : kWK) * 16 + i] = acc[mt][r];
      });
    });
  };
  cfor<0, (kWL + 2) / 2>([&](auto PP) {
    constexpr int l0 = 2 * decltype(PP)::value, l1 = l0 + 1 <= kWL ? l0 + 1 : l0;
    constexpr int NM0 = (2 * l0 + 1 + 15) / 16, NM1 = (2 * l1 + 1 + 15) / 16;
    if (l0 * l0 < ko) {  // wave-uniform
      f4 a0[NM0], a1[NM1];
      rot_out_mma(std::integral_constant<int, l0>{}, a0);
      if constexpr (l1 != l0) rot_out_mma(std::integral_constant<int, l1>{}, a1);
      GTP_TILE_ORDER();
      rot_out_store(std::integral_constant<int, l0>{}, a0);
      if constexpr (l1 != l0) rot_out_store(std::integral_constant<int, l1>{}, a1);
    }
  });
  GTP_TILE_ORDER();

  // ---- 5. store: rows of ko floats of the wave's channels
  {
    float* const yb = y + (b * C + c0) * int64_t(ko);
    const int c = lane & 15;
    if (c < cnt)
      cfor<0, NXL>([&](auto Q) {
        const int k = g + 4 * decltype(Q)::value;
        if (k < ko) yb[int64_t(c) * ko + k] = X[k * 16 + c];
      });
  }
}

}  // namespace

hipError_t launch_conv_escn_wave(const EscnDev& e, const void* x, int in_type, const float* r, const float* h,
                                 int64_t B, int64_t C, float* y, float* dws, int k1, int kh, int ko, hipStream_t s) {
  if (!e.A || !e.Z || e.LM != kWL || k1 > kWK || kh > kWH || ko > kWK || k1 < 1 || kh < 1 || ko < 1)
    return hipErrorInvalidValue;
  if (B <= 0 || C <= 0) return hipSuccess;
  const int64_t ncb = (C + 16 * kWaves - 1) / (16 * kWaves);
  if (B * ncb > 0x7fffffff) return hipErrorInvalidValue;
  hipError_t err = launch_escn_rot(e, kWL, r, B, dws, s);
  if (err != hipSuccess) return err;
  const dim3 grid(unsigned(B * ncb)), block(64 * kWaves);
  if (in_type == IN_BF16)
    hipLaunchKernelGGL((k_conv_escn_wave<uint16_t>), grid, block, 0, s, static_cast<const uint16_t*>(x), dws, h, y,
                       C, int(ncb), e.A, e.Z, k1, kh, ko);
  else
    hipLaunchKernelGGL((k_conv_escn_wave<float>), grid, block, 0, s, static_cast<const float*>(x), dws, h, y, C,
                       int(ncb), e.A, e.Z, k1, kh, ko);
  return hipGetLastError();
}

}  // namespace gtp
