// Rotated-frame equivariant convolution (Sec. 3.3 "Equivariant Convolutions";
// Appendix, eq. sh2fs-escn) at degree 16 on the fp32 matrix cores.
//
// Same computation as the small-degree kernel (y = D_b^T Z(D_b x, h), Z the
// product with a zonal filter taken per order m at the theta nodes), but the
// per-product state (289 coefficients) does not fit one lane's registers, so
// the work is laid out across the channels of an edge, which share the edge's
// rotation and every table: each dense stage is a small contraction with the
// 16 channels of a wave as the N index of v_mfma_f32_16x16x4f32 (A[i][k] from
// lane 16 k + i, B[k][j] from lane 16 k + j, register r of lane 16 g + i = row
// 4 g + r, column i).  The rotation D_b = J^T Z(-beta) J Z(-alpha) is applied
// factor by factor: Z, a rotation about the pole, turns each (cos m, sin m)
// coefficient pair by m times the edge angle (VALU), and J, the fixed real-SH
// matrix of R_x(90 deg), is a per-degree-block contraction whose operands are
// the same for every edge.  The stages, all in place on the wave's tile:
//   rotate in    x' = J^T Z(-beta) J Z(-alpha) x;
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
//   rotate out   y = Z(alpha) J^T Z(beta) J y'.
// One workgroup per (edge, 64 channels), one wave per 16 channels; LDS holds
// each wave's coefficient tile (16 channels x 289 coefficients, channel-major:
// 74.5 KB per workgroup, two workgroups per CU) and the edge's trig values.
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
// One wave's tile, channel-major: coefficient k of channel c at c kTS + k,
// the layout of the wave's 16 rows in memory (contiguous copies in and out).
// Rows 0..288, row 289 takes the writes of padding rows; reads past the last
// block reach rows 290 and 291, the next channel's first rows (past the last
// tile: kTilePad), whose values are then dropped.  The LDS serves a wave's
// access a half-wave (lane groups 0 and 1, or 2 and 3) at a time over 32
// banks; with the stride = 2 (mod 32) the 16 channels of one row take the
// even or the odd banks, so two lane groups whose rows are one apart (the
// rotation stages' reads and writes) are conflict-free.
constexpr int kTS = kWK + 1;   // 290
constexpr int kSpare = kWK;    // 289
constexpr int kTileF = 16 * kTS;
constexpr int kTilePad = 4;
static_assert(kTS % 32 == 2, "bank layout");

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f4 mfma(float a, float b, f4 c) { return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0); }


// The stages rewrite the tile in place: lanes read rows that other lanes then
// overwrite, and read rows that other lanes wrote.  The wave issues its LDS
// operations in program order and the LDS performs them in that order; this
// fence keeps the compiler from moving a lane's LDS reads and writes across
// it (it only sees the lane's own addresses).
#define GTP_TILE_ORDER() asm volatile("" ::: "memory")

// A copy of v the compiler cannot see through: addresses derived from it are
// computed in the stage that uses them, not once and kept live across stages.
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

__device__ __forceinline__ float ldx(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ldx(const uint16_t* p, int64_t i) { return __uint_as_float(uint32_t(p[i]) << 16); }

template <typename TIn>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_conv_escn_wave(
    const TIn* __restrict__ x, const float* __restrict__ rv, const float* __restrict__ h, float* __restrict__ y,
    int64_t C, int ncb, const float* __restrict__ At, const float* __restrict__ Zt, const float* __restrict__ JI,
    int k1, int kh, int ko) {
  __shared__ __align__(16) float tiles[kWaves * kTileF + kTilePad];
  __shared__ float4 tw[kWH];  // (cos m alpha, sin m alpha, cos m beta, sin m beta)
  lds_poison(tiles, kWaves * kTileF + kTilePad);
  lds_poison(reinterpret_cast<float*>(tw), kWH * 4);
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, g = lane >> 4, i = lane & 15;
  const int64_t wg = xcd_product(blockIdx.x, gridDim.x);
  const int64_t b = wg / ncb;
  const int64_t c0 = (wg % ncb) * (16 * kWaves) + 16 * w;  // first channel of this wave
  const int cnt = C - c0 <= 0 ? 0 : (C - c0 < 16 ? int(C - c0) : 16);
  float* const X = tiles + w * kTileF;  // rows 0..288, row 289 takes the writes of padding rows

  // ---- 1. every load in flight before the first use: the wave's x tile
  // (lane (g, c) takes rows g, g + 4, ..), the radial weights of channel i,
  // the operands of m = 0; the edge's angles (beta from the pole, alpha in
  // the xy plane; a zero vector is taken as (0, 0, 1))
  // the wave's 16 rows as one block of 16 k1 floats: element e = lane + 64 q
  // (64 consecutive floats per load), channel e / k1, coefficient e % k1
  constexpr int NXL = (16 * kWK + 63) / 64;  // 73 loads per lane
  float xv[NXL];
  const bool full = k1 == kWK && cnt == 16;  // wave-uniform
  if (full) {
    // one base per lane, constant offsets (the last load: lanes 0..15)
    const TIn* const xl = x + (b * C + c0) * int64_t(kWK) + lane;
    cfor<0, NXL>([&](auto Q) {
      constexpr int q = decltype(Q)::value;
      if constexpr (64 * q + 63 < 16 * kWK) {
        xv[q] = ldx(xl, 64 * q);
      } else {
        const float v = ldx(xl, lane < 16 * kWK - 64 * q ? 64 * q : 0);
        xv[q] = lane < 16 * kWK - 64 * q ? v : 0.0f;
      }
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
  if (tid < kWH) {
    const float rx = rv[3 * b], ry = rv[3 * b + 1], rz = rv[3 * b + 2];
    const float rho = sqrtf(rx * rx + ry * ry);
    const float al = rho > 0.0f ? atan2f(ry, rx) : 0.0f;
    const float be = (rho > 0.0f || rz != 0.0f) ? atan2f(rho, rz) : 0.0f;
    float sa, ca, sb, cb;
    sincosf(float(tid) * al, &sa, &ca);
    sincosf(float(tid) * be, &sb, &cb);
    tw[tid] = make_float4(ca, sa, cb, sb);
  }
  f4 avq[2][4];  // the operands of order m (and m + 1, prefetched), four quads
  auto load_ops = [&](auto MM, f4(&dst)[4]) {
    constexpr int m = decltype(MM)::value, NL = escn_wave_lane_floats(kWL, m);
    const f4* const src = reinterpret_cast<const f4*>(At + escn_wave_moff(kWL, m) + lane * NL);
    cfor<0, NL / 4>([&](auto Q) { dst[decltype(Q)::value] = src[decltype(Q)::value]; });
  };
  load_ops(std::integral_constant<int, 0>{}, avq[0]);
  if (full) {
    cfor<0, NXL>([&](auto Q) {
      const int e = lane + 64 * decltype(Q)::value;
      const int c = e / kWK, k = e - c * kWK;
      if (e < 16 * kWK) X[c * kTS + k] = xv[decltype(Q)::value];
    });
  } else {
    // padded rows or a partial tile: zeros first, then the wave's cnt rows
    // of k1 floats (a plain loop: the uncommon shapes)
    for (int e = lane; e < kTileF; e += 64) X[e] = 0.0f;
    GTP_TILE_ORDER();
    const TIn* const xb = x + (b * C + c0) * int64_t(k1);
    const int tot = cnt * k1;
    for (int e = lane; e < tot; e += 64) {
      const int c = e / k1, k = e - c * k1;
      X[c * kTS + k] = ldx(xb, e);
    }
  }
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
  __syncthreads();  // the trig values (and each wave's own tile)

  // LDS reads of the tile are unconditional (past a degree block they stay
  // inside the tile; the value is then selected), writes of padding rows go
  // to the spare row kWK: no divergent branches.
  auto xrd = [&](int row, bool ok) {
    const float v = X[i * kTS + (ok ? row : 0)];
    return ok ? v : 0.0f;
  };
  auto xrd_block = [&](int row, bool ok) {
    const float v = X[i * kTS + row];
    return ok ? v : 0.0f;
  };

  // ---- rotations about the pole: each (cos m, sin m) pair of the tile turned
  // by m times the edge angle, AB = 0 alpha, 1 beta, SGN = -1 for Z(-angle):
  //   c' = c cos + s sin, s' = -c sin + s cos   (Z(-angle); the transpose for +)
  // Degree by degree, lane group g turning order m = 4 q + g + 1 in step q:
  // rows l^2 + l + m and l^2 + l - m and the trig entry m are the lane
  // group's base plus a constant.  A lane past the degree (m > l, in the
  // last step of a degree, l >= 2) reads rows of blocks l + 1 and l - 1 and
  // writes the spare row, so every row of the tile is written once, by the
  // lane that read it in the same step, and the steps may run in any order.
  // Degree 1 (one pair) is turned by every lane group alike.
  auto zrot = [&](auto AB, auto SGN) {
    constexpr int ab = decltype(AB)::value, sgn = decltype(SGN)::value;
    const int gz = opaque(g);
    float* const Xp = X + i * kTS + gz;      // rows r + g
    float* const Xn = X + i * kTS + 3 - gz;  // rows r + 3 - g
    auto turn = [&](float& c, float& sv, float cm, float sm) {
      const float c0 = c, s0 = sv;
      if constexpr (sgn < 0) {
        c = fmaf(c0, cm, s0 * sm);
        sv = fmaf(s0, cm, -c0 * sm);
      } else {
        c = fmaf(c0, cm, -s0 * sm);
        sv = fmaf(s0, cm, c0 * sm);
      }
    };
    {
      const float4 t = tw[1];
      float c = X[i * kTS + 3], sv = X[i * kTS + 1];
      turn(c, sv, ab ? t.z : t.x, ab ? t.w : t.y);
      X[i * kTS + 3] = c;
      X[i * kTS + 1] = sv;
    }
    cfor<2, kWL + 1>([&](auto LL) {
      constexpr int l = decltype(LL)::value;
      cfor<0, (l + 3) / 4>([&](auto Q) {
        constexpr int m0 = 4 * decltype(Q)::value + 1;
        constexpr int rc = l * l + l + m0, rs = l * l + l - m0 - 3;  // rs >= 1 (l >= 2)
        const float4 t = tw[m0 + gz];  // m0 + g <= 16
        float c = Xp[rc], sv = Xn[rs];
        turn(c, sv, ab ? t.z : t.x, ab ? t.w : t.y);
        if constexpr (m0 + 3 > l) {  // lane groups past the degree write the spare row
          const bool ok = m0 + gz <= l;
          X[i * kTS + (ok ? rc + gz : kSpare)] = c;
          X[i * kTS + (ok ? rs + 3 - gz : kSpare)] = sv;
        } else {
          Xp[rc] = c;
          Xn[rs] = sv;
        }
      });
    });
    GTP_TILE_ORDER();
  };
  // ---- the fixed matrix J (TR = 0) or J^T (TR = 1) on every degree block
  // (M = rows, K = columns), in the output tiles of the operand images
  // (escn_wave_jtile: below degree 8 the whole block; from degree 8 on the
  // four class sub-blocks, two per tile), two blocks at a time: the MFMAs of
  // both, then their writes (blocks touch disjoint rows; a block's reads
  // precede its writes).  Operand images: lane-permuted, four K-steps per
  // 16-byte load.
  auto jpass = [&](auto TR) {
    constexpr int tr = decltype(TR)::value;
    const int gj = opaque(g);
    const int gp = gj & 1, gh = gj >> 1;  // lane-group parity and half
    const float* const img = JI + (tr ? escn_wave_jtoff() : 0);
    constexpr int NPR = (kWL + 2) / 2;  // block pairs (2 p, 2 p + 1); the last holds degree 16 alone
    // class tiles: the block-local first index of a half's classes (rows and
    // the columns they map to); a half without rows takes the other's
    auto rstart = [](int l, int t, int par) {
      const int c = escn_wave_jtcls(l, t, par) < 0 ? escn_wave_jtcls(l, t, 0) : escn_wave_jtcls(l, t, par);
      return escn_cls_start(l, c) + 2 * escn_wave_jtfirst(t);
    };
    auto cstart = [](int l, int t, int par) {
      const int c = escn_wave_jtcls(l, t, par) < 0 ? escn_wave_jtcls(l, t, 0) : escn_wave_jtcls(l, t, par);
      return escn_cls_start(l, escn_cls_map(l, c));
    };
    const int ib2 = i * kTS + 2 * gh, ib8 = i * kTS + 8 * gh;
    // a block's operands (arrays sized for the largest block): per tile the
    // A images and the B values of its K-steps (channel i)
    auto load = [&](auto LL, f4(&a)[3][2], float(&bv)[3][5]) {
      constexpr int l = decltype(LL)::value, d = 2 * l + 1, R0 = l * l;
      cfor<0, escn_wave_jtiles(l)>([&](auto TT) {
        constexpr int t = decltype(TT)::value, NK4 = escn_wave_jnk4(l, t), NS = escn_wave_jsteps(l, t);
        const f4* const src = reinterpret_cast<const f4*>(img + escn_wave_joff(l, t) + lane * NK4);
        cfor<0, NK4 / 4>([&](auto Q) { a[t][decltype(Q)::value] = src[decltype(Q)::value]; });
        if constexpr (l < kEscnClassL) {
          cfor<0, NS>([&](auto KS) {
            constexpr int ks = decltype(KS)::value;
            const int c = 4 * ks + g;
            bv[t][ks] = xrd_block(R0 + c, c < d);
          });
        } else {
          // column element q = 2 ks + g / 2 of the half's class: block index
          // first + 2 q (past the class: a value of the tile, dropped)
          constexpr int C0 = escn_wave_jtcols(l, t, 0), C1 = escn_wave_jtcols(l, t, 1);
          const int cb = ib2 + (gp ? cstart(l, t, 1) : cstart(l, t, 0));
          cfor<0, NS>([&](auto KS) {
            constexpr int ks = decltype(KS)::value;
            const float v = X[cb + R0 + 4 * ks];
            if constexpr (2 * ks + 1 < (C0 < C1 ? C0 : C1)) {
              bv[t][ks] = v;
            } else {
              bv[t][ks] = 2 * ks + gh < (gp ? C1 : C0) ? v : 0.0f;
            }
          });
        }
      });
    };
    auto mma = [&](auto LL, const f4(&a)[3][2], const float(&bv)[3][5], f4(&acc)[3]) {
      constexpr int l = decltype(LL)::value;
      cfor<0, escn_wave_jtiles(l)>([&](auto TT) {
        constexpr int t = decltype(TT)::value;
        acc[t] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        cfor<0, escn_wave_jsteps(l, t)>([&](auto KS) {
          constexpr int ks = decltype(KS)::value;
          acc[t] = mfma(a[t][ks / 4][ks % 4], bv[t][ks], acc[t]);
        });
      });
    };
    // Whole-block tiles (degrees below 8): rows past the block (A rows there
    // are zero) are written unconditionally, into blocks l + 1 .. that the
    // pass has read already and writes later (blocks up to l0 + 3 for the
    // pair (l0, l1): checked for every l by the host replay), except for
    // degree 1, whose padding reaches block 4: it goes to the spare row, as
    // do the padding rows of the class tiles.
    const int jb = i * kTS + escn_wave_jrow(4 * gj);  // + 2 r + l^2
    auto store = [&](auto LL, const f4(&acc)[3]) {
      constexpr int l = decltype(LL)::value, d = 2 * l + 1, R0 = l * l;
      if constexpr (l < kEscnClassL) {
        cfor<0, 4>([&](auto RR) {
          constexpr int r = decltype(RR)::value;
          if constexpr (l == 1) {
            const int row = escn_wave_jrow(4 * gj + r);
            X[i * kTS + (row < d ? R0 + row : kSpare)] = acc[0][r];
          } else {
            X[jb + R0 + 2 * r] = acc[0][r];
          }
        });
      } else {
        cfor<0, escn_wave_jtiles(l)>([&](auto TT) {
          constexpr int t = decltype(TT)::value;
          // row element p = 4 (g / 2) + r of the half's class: block index
          // first + 2 p; past the class: the spare row
          constexpr int N0 = escn_wave_jtrows(l, t, 0), N1 = escn_wave_jtrows(l, t, 1);
          const int rb = ib8 + (gp ? rstart(l, t, 1) : rstart(l, t, 0));
          cfor<0, 4>([&](auto RR) {
            constexpr int r = decltype(RR)::value;
            if constexpr (4 + r < (N0 < N1 ? N0 : N1)) {
              X[rb + R0 + 2 * r] = acc[t][r];
            } else {
              const bool ok = 4 * gh + r < (gp ? N1 : N0);
              X[ok ? rb + R0 + 2 * r : i * kTS + kSpare] = acc[t][r];
            }
          });
        });
      }
    };
    // blocks touch disjoint rows and each is read before it is written: the
    // operands of pair p + 1 are read before the writes of pair p
    f4 a0[3][2], a1[3][2];
    float b0[3][5], b1[3][5];
    load(std::integral_constant<int, 0>{}, a0, b0);
    load(std::integral_constant<int, 1>{}, a1, b1);
    cfor<0, NPR>([&](auto PP) {
      constexpr int p = decltype(PP)::value, l0 = 2 * p, l1 = l0 + 1 <= kWL ? l0 + 1 : l0;
      f4 c0[3], c1[3];
      mma(std::integral_constant<int, l0>{}, a0, b0, c0);
      if constexpr (l1 != l0) mma(std::integral_constant<int, l1>{}, a1, b1, c1);
      if constexpr (p + 1 < NPR) {
        constexpr int n0 = l0 + 2, n1 = n0 + 1 <= kWL ? n0 + 1 : n0;
        load(std::integral_constant<int, n0>{}, a0, b0);
        if constexpr (n1 != n0) load(std::integral_constant<int, n1>{}, a1, b1);
      }
      GTP_TILE_ORDER();
      store(std::integral_constant<int, l0>{}, c0);
      GTP_TILE_ORDER();  // block l1's rows after block l0's padding rows
      if constexpr (l1 != l0) store(std::integral_constant<int, l1>{}, c1);
    });
    GTP_TILE_ORDER();
  };

  // ---- 2. rotate in: x' = J^T Z(-beta) J Z(-alpha) x
  GTP_TILE_ORDER();
  zrot(std::integral_constant<int, 0>{}, std::integral_constant<int, -1>{});
  jpass(std::integral_constant<int, 0>{});
  zrot(std::integral_constant<int, 1>{}, std::integral_constant<int, -1>{});
  jpass(std::integral_constant<int, 1>{});

  // ---- 3. the zonal product per order m, its cos and sin parts together
  // (m-parts touch disjoint rows)
  const float* const zp = Zt + 16 * kWH;
  // the synthesis B values of order m, xz[sg][t]: degree m + 2 (4 t + g) for
  // t < KE (even set), m + 1 + 2 (4 (t - KE) + g) after; order m + 1's are
  // read before order m's writes (disjoint rows)
  auto zrd = [&](auto MM, float(&xz)[2][5]) {
    constexpr int m = decltype(MM)::value, n = kWL + 1 - m, NE = (n + 1) / 2, NO = n / 2;
    constexpr int KE = (NE + 3) / 4, KO = (NO + 3) / 4, NSG = m == 0 ? 1 : 2;
    cfor<0, NSG>([&](auto SG) {
      constexpr int sg = decltype(SG)::value;
      cfor<0, KE + KO>([&](auto T) {
        constexpr int t = decltype(T)::value;
        const int l = t < KE ? m + 2 * (4 * t + g) : m + 1 + 2 * (4 * (t - KE) + g);
        xz[sg][t] = xrd(l * l + l + (sg ? -m : m), l <= kWL);
      });
    });
  };
  float xz[2][5];
  zrd(std::integral_constant<int, 0>{}, xz);
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
        GE[sg] = mfma(av(ks), xz[sg][ks], GE[sg]);
      });
    });
    cfor<0, KO>([&](auto KS) {
      constexpr int ks = decltype(KS)::value;
      const int l = m + 1 + 2 * (4 * ks + g);
      cfor<0, NSG>([&](auto SG) {
        constexpr int sg = decltype(SG)::value;
        GO[sg] = mfma(av(KE + ks), xz[sg][KE + ks], GO[sg]);
      });
    });
    if constexpr (m + 1 <= kWL) zrd(std::integral_constant<int, m + 1>{}, xz);
    // pole pair (m = 0 only): the lane's channel, every lane group alike
    float pe0 = 0.0f, po0 = 0.0f;
    if constexpr (m == 0) {
      float ae = 0.0f, ao = 0.0f;
      cfor<0, kWH>([&](auto LL) {
        constexpr int l = decltype(LL)::value;
        const float v = zp[kWH + l] * X[i * kTS + l * l + l];
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
          X[i * kTS + (ie < NE ? row_of(l, sg) : kSpare)] = v;
        }
        if constexpr (NO > 0) {
          const int l = m + 1 + 2 * ie;
          float v = YO[sg][r];
          if constexpr (m == 0) v = fmaf(zp[2 * kWH + (ie < NO ? l : 0)], po0, v);
          X[i * kTS + (ie < NO ? row_of(l, sg) : kSpare)] = v;
        }
      });
    });
  });
  GTP_TILE_ORDER();

  // ---- 4. rotate out: y = Z(alpha) J^T Z(beta) J y'
  jpass(std::integral_constant<int, 0>{});
  zrot(std::integral_constant<int, 1>{}, std::integral_constant<int, 1>{});
  jpass(std::integral_constant<int, 1>{});
  zrot(std::integral_constant<int, 0>{}, std::integral_constant<int, 1>{});

  // ---- 5. store: the wave's rows of ko floats as one block (64 consecutive
  // floats per store, non-temporal)
  {
    float* const yb = y + (b * C + c0) * int64_t(ko);
    const int tot = cnt * ko;
    if (full && ko == kWK) {
      cfor<0, NXL>([&](auto Q) {
        const int e = lane + 64 * decltype(Q)::value;
        const int c = e / kWK, k = e - c * kWK;
        if (e < 16 * kWK) __builtin_nontemporal_store(X[c * kTS + k], yb + e);
      });
    } else {
      for (int e = lane; e < tot; e += 64) {
        const int c = e / ko, k = e - c * ko;
        __builtin_nontemporal_store(X[c * kTS + k], yb + e);
      }
    }
  }
}

}  // namespace

hipError_t launch_conv_escn_wave(const EscnDev& e, const void* x, int in_type, const float* r, const float* h,
                                 int64_t B, int64_t C, float* y, int k1, int kh, int ko, hipStream_t s) {
  if (!e.A || !e.Z || !e.JI || e.LM != kWL || k1 > kWK || kh > kWH || ko > kWK || k1 < 1 || kh < 1 || ko < 1)
    return hipErrorInvalidValue;
  if (B <= 0 || C <= 0) return hipSuccess;
  const int64_t ncb = (C + 16 * kWaves - 1) / (16 * kWaves);
  if (B * ncb > 0x7fffffff) return hipErrorInvalidValue;
  const dim3 grid(unsigned(B * ncb)), block(64 * kWaves);
  if (in_type == IN_BF16)
    hipLaunchKernelGGL((k_conv_escn_wave<uint16_t>), grid, block, 0, s, static_cast<const uint16_t*>(x), r, h, y, C,
                       int(ncb), e.A, e.Z, e.JI, k1, kh, ko);
  else
    hipLaunchKernelGGL((k_conv_escn_wave<float>), grid, block, 0, s, static_cast<const float*>(x), r, h, y, C,
                       int(ncb), e.A, e.Z, e.JI, k1, kh, ko);
  return hipGetLastError();
}

}  // namespace gtp
