// Workgroup-per-product kernels for any degree (gfx950), the unfused stage
// kernels with the paper's complex grid layout, and the SH filter kernel.
#include "gtp_device.hpp"

namespace gtp {
namespace {

constexpr int kBlock = 256;
constexpr int kMaxOut = 17;  // ceil((64 + 1)^2 / 256) outputs per thread at Le <= 64

__device__ __forceinline__ float ld_in(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld_in(const uint16_t* p, int64_t i) {
  return __uint_as_float(uint32_t(p[i]) << 16);
}
__device__ __forceinline__ int dtri(int l, int m) { return l * (l + 1) / 2 + m; }
// (degree, m-part) of a coefficient index i = l*l + l + m.  mp = 0 for m = 0,
// 2m - 1 for the cos function (m > 0), 2m for the sin function (m < 0).
__device__ __forceinline__ void split_index(int i, int& l, int& m, int& mp) {
  l = int(sqrtf(float(i)));
  while (l * l > i) --l;
  while ((l + 1) * (l + 1) <= i) ++l;
  const int ms = i - l * l - l;
  m = ms < 0 ? -ms : ms;
  mp = ms == 0 ? 0 : (ms > 0 ? 2 * ms - 1 : 2 * m);
}
__device__ __forceinline__ int coef_index(int l, int mp) {
  const int m = (mp + 1) >> 1;
  return (mp == 0 || (mp & 1)) ? l * l + l + m : l * l + l - m;
}

// LDS plan of the generic fused kernel for a node chunk of JC theta nodes.
struct GenericLayout {
  int K1, K2, n1, n2, no, JC;
  int off_x2, off_A1, off_A2, off_F3, off_C, total;
};

__host__ __device__ inline GenericLayout generic_layout(const DevTables& t, int nu, int JC) {
  GenericLayout g;
  g.K1 = (t.L1 + 1) * (t.L1 + 1);
  g.K2 = nu == 0 ? (t.L2 + 1) * (t.L2 + 1) : 0;
  g.n1 = 2 * t.L1 + 1;
  g.n2 = nu == 0 ? 2 * t.L2 + 1 : 0;
  g.no = 2 * t.Le + 1;
  g.JC = JC;
  g.off_x2 = g.K1;
  g.off_A1 = g.off_x2 + g.K2;
  g.off_A2 = g.off_A1 + JC * g.n1;
  g.off_F3 = g.off_A2 + JC * g.n2;
  g.off_C = g.off_F3 + JC * t.NP;
  g.total = g.off_C + JC * g.no;
  return g;
}

// Fused product on the (theta, phi) sampling grid, one product per
// workgroup: theta synthesis (table S), phi synthesis (table Phi), pointwise
// product, phi analysis, theta analysis into per-thread output registers
// (table WT), in chunks of JC theta nodes held in LDS.
template <typename T1, typename T2>
__global__ __launch_bounds__(kBlock) void k_full_generic(DevTables t, const T1* __restrict__ x1,
                                                         const T2* __restrict__ x2, float* __restrict__ y,
                                                         int64_t n, int nu, int JC, DegWeights wt, PairIdx pi) {
  extern __shared__ float smem[];
  const GenericLayout g = generic_layout(t, nu, JC);
  lds_poison(smem, g.total);
  const int tid = threadIdx.x;
  const int KO = (t.Lout + 1) * (t.Lout + 1);
  const int KE = (t.Le + 1) * (t.Le + 1);
  const int nmp = 2 * t.Mphi + 1;
  const int ntE = (t.Le + 1) * (t.Le + 2) / 2;
  float* xs1 = smem;
  float* xs2 = smem + g.off_x2;
  float* A1 = smem + g.off_A1;
  float* A2 = smem + g.off_A2;
  float* F3 = smem + g.off_F3;
  float* Cm = smem + g.off_C;

  for (int64_t p = blockIdx.x; p < n; p += gridDim.x) {
    const int64_t wrow = weight_row(wt, p);
    int64_t r1 = p, r2 = p;
    if (pi.C2) pair_rows(pi, p, r1, r2);
    for (int i = tid; i < g.K1; i += kBlock)
      xs1[i] = ld_in(x1, r1 * g.K1 + i) * (wt.w1 ? wt.w1[wrow * (t.L1 + 1) + degree_of(i)] : 1.0f);
    for (int i = tid; i < g.K2; i += kBlock)
      xs2[i] = ld_in(x2, r2 * g.K2 + i) * (wt.w2 ? wt.w2[wrow * (t.L2 + 1) + degree_of(i)] : 1.0f);
    float acc[kMaxOut];
#pragma unroll
    for (int q = 0; q < kMaxOut; ++q) acc[q] = 0.0f;
    __syncthreads();

    for (int j0 = 0; j0 < t.NJ; j0 += JC) {
      const int jn = min(JC, t.NJ - j0);
      // (1) theta synthesis A[jj][mp] = sum_l S[tri(l, m)][j] x[l, +-m]
      for (int w = tid; w < jn * (g.n1 + g.n2); w += kBlock) {
        const bool second = w >= jn * g.n1;
        const int ww = second ? w - jn * g.n1 : w;
        const int jj = ww % jn, mp = ww / jn;
        const int m = (mp + 1) >> 1;
        const int L = second ? t.L2 : t.L1;
        const float* xs = second ? xs2 : xs1;
        float s = 0.0f;
        for (int l = m; l <= L; ++l) s = fmaf(t.S[dtri(l, m) * t.NJ + j0 + jj], xs[coef_index(l, mp)], s);
        (second ? A2 : A1)[jj * (second ? g.n2 : g.n1) + mp] = s;
      }
      __syncthreads();
      // (2) phi synthesis and pointwise product F3[jj][k]
      for (int w = tid; w < jn * t.NP; w += kBlock) {
        const int jj = w / t.NP, k = w % t.NP;
        float f1 = 0.0f;
        for (int mp = 0; mp < g.n1; ++mp) f1 = fmaf(A1[jj * g.n1 + mp], t.Phi[mp * t.NP + k], f1);
        float f3;
        if (nu == 0) {
          float f2 = 0.0f;
          for (int mp = 0; mp < g.n2; ++mp) f2 = fmaf(A2[jj * g.n2 + mp], t.Phi[mp * t.NP + k], f2);
          f3 = f1 * f2;
        } else {
          f3 = f1;
          for (int e = 1; e < nu; ++e) f3 *= f1;
        }
        F3[jj * t.NP + k] = f3;
      }
      __syncthreads();
      // (3) phi analysis C[jj][mp] = sum_k F3[jj][k] trig(mp, k)
      for (int w = tid; w < jn * g.no; w += kBlock) {
        const int jj = w / g.no, mp = w % g.no;
        float s = 0.0f;
        for (int k = 0; k < t.NP; ++k) s = fmaf(F3[jj * t.NP + k], t.PhiT[k * nmp + mp], s);
        Cm[jj * g.no + mp] = s;
      }
      __syncthreads();
      // (4) theta analysis into this thread's outputs
#pragma unroll
      for (int q = 0; q < kMaxOut; ++q) {
        const int o = tid + q * kBlock;
        if (o < KE) {
          int l, m, mp;
          split_index(o, l, m, mp);
          const int r = dtri(l, m);
          float s = acc[q];
          for (int jj = 0; jj < jn; ++jj) s = fmaf(t.WT[(j0 + jj) * ntE + r], Cm[jj * g.no + mp], s);
          acc[q] = s;
        }
      }
      __syncthreads();
    }
#pragma unroll
    for (int q = 0; q < kMaxOut; ++q) {
      const int o = tid + q * kBlock;
      if (o < KO)
        y[p * KO + o] = (o < KE) ? acc[q] * (wt.wo ? wt.wo[wrow * (t.Lout + 1) + degree_of(o)] : 1.0f) : 0.0f;
    }
  }
}

// Step 1 with the paper's complex grid: grid[p][u+L][v+L] = x*_{u,v}.
template <typename TIn>
__global__ __launch_bounds__(kBlock) void k_sh2fourier(DevTables t, int L, const TIn* __restrict__ x,
                                                       float* __restrict__ grid, int64_t n) {
  const int D = 2 * L + 1;
  const int K = (L + 1) * (L + 1);
  const int64_t total = n * D * D;
  for (int64_t e = int64_t(blockIdx.x) * kBlock + threadIdx.x; e < total; e += int64_t(gridDim.x) * kBlock) {
    const int64_t p = e / (D * D);
    const int r = int(e % (D * D));
    const int u = r / D - L, v = r % D - L;
    const int m = v < 0 ? -v : v, au = u < 0 ? -u : u;
    const TIn* xp = x + p * K;
    float re = 0.0f, im = 0.0f;
    const int l0 = m > au ? m : au;
    for (int l = l0; l <= L; ++l) {
      if ((l + au) & 1) continue;
      const float c = t.T1[dtri(l, m) * t.ldT1 + au];
      // phi factor of the cos / sin functions at v = +-m
      float qr, qi;
      if (m == 0) {
        qr = ld_in(x, p * K + l * l + l);
        qi = 0.0f;
      } else {
        qr = 0.5f * ld_in(xp, l * l + l + m);
        qi = (v > 0 ? -0.5f : 0.5f) * ld_in(xp, l * l + l - m);
      }
      if ((m & 1) == 0) {
        // cos series: coefficient c_0 at u = 0, c_|u| / 2 otherwise
        const float th = au == 0 ? c : 0.5f * c;
        re = fmaf(th, qr, re);
        im = fmaf(th, qi, im);
      } else {
        // sine series: -i sgn(u) c_|u| / 2
        const float th = (u > 0 ? -0.5f : 0.5f) * c;  // multiplies i
        re = fmaf(-th, qi, re);
        im = fmaf(th, qr, im);
      }
    }
    grid[2 * e] = re;
    grid[2 * e + 1] = im;
  }
}

// Step 2: direct complex 2D convolution, workgroup per product; the input
// grids sit in LDS when they fit.
__global__ __launch_bounds__(kBlock) void k_fourier_conv(int L1, int L2, const float* __restrict__ g1,
                                                         const float* __restrict__ g2, float* __restrict__ g3,
                                                         int64_t n, int use_lds) {
  extern __shared__ float smem[];
  const int D1 = 2 * L1 + 1, D2 = 2 * L2 + 1, U = L1 + L2, D3 = 2 * U + 1;
  lds_poison(smem, use_lds ? 2 * D1 * D1 + 2 * D2 * D2 : 0);
  for (int64_t p = blockIdx.x; p < n; p += gridDim.x) {
    const float* a = g1 + p * 2 * D1 * D1;
    const float* b = g2 + p * 2 * D2 * D2;
    if (use_lds) {
      for (int i = threadIdx.x; i < 2 * D1 * D1; i += kBlock) smem[i] = a[i];
      for (int i = threadIdx.x; i < 2 * D2 * D2; i += kBlock) smem[2 * D1 * D1 + i] = b[i];
      __syncthreads();
      a = smem;
      b = smem + 2 * D1 * D1;
    }
    for (int e = threadIdx.x; e < D3 * D3; e += kBlock) {
      const int u3 = e / D3 - U, v3 = e % D3 - U;
      const int ulo = max(-L1, u3 - L2), uhi = min(L1, u3 + L2);
      const int vlo = max(-L1, v3 - L2), vhi = min(L1, v3 + L2);
      float re = 0.0f, im = 0.0f;
      for (int u1 = ulo; u1 <= uhi; ++u1) {
        const int u2 = u3 - u1;
        for (int v1 = vlo; v1 <= vhi; ++v1) {
          const int v2 = v3 - v1;
          const int ia = 2 * ((u1 + L1) * D1 + (v1 + L1));
          const int ib = 2 * ((u2 + L2) * D2 + (v2 + L2));
          const float ar = a[ia], ai = a[ia + 1], br = b[ib], bi = b[ib + 1];
          re = fmaf(ar, br, re);
          re = fmaf(-ai, bi, re);
          im = fmaf(ar, bi, im);
          im = fmaf(ai, br, im);
        }
      }
      g3[(p * D3 * D3 + e) * 2] = re;
      g3[(p * D3 * D3 + e) * 2 + 1] = im;
    }
    if (use_lds) __syncthreads();
  }
}

// Step 3: y_l^m = Re sum_{u, v = +-m} g3[u, v] z^{l,m}_{u,v} with
// z = (phi integral) * (Zc(|u|) + i sgn(u) Zs(|u|)).
__global__ __launch_bounds__(kBlock) void k_fourier2sh(DevTables t, const float* __restrict__ g3,
                                                       float* __restrict__ y, int64_t n) {
  const int U = t.U, D = 2 * U + 1;
  const int KO = (t.Lout + 1) * (t.Lout + 1);
  const int KE = (t.Le + 1) * (t.Le + 1);
  const float kPiF = 3.14159265358979323846f;
  const int64_t total = n * KO;
  for (int64_t e = int64_t(blockIdx.x) * kBlock + threadIdx.x; e < total; e += int64_t(gridDim.x) * kBlock) {
    const int64_t p = e / KO;
    const int o = int(e % KO);
    if (o >= KE) {
      y[e] = 0.0f;
      continue;
    }
    int l, m, mp;
    split_index(o, l, m, mp);
    const float* g = g3 + p * 2 * D * D;
    const float* zc = t.Zc + dtri(l, m) * t.ldZ;
    const float* zs = t.Zs + dtri(l, m) * t.ldZ;
    float acc = 0.0f;
    for (int u = -U; u <= U; ++u) {
      const int au = u < 0 ? -u : u;
      const float cr = zc[au], ci = (u > 0 ? 1.0f : (u < 0 ? -1.0f : 0.0f)) * zs[au];
      const int ip = 2 * ((u + U) * D + (m + U));
      const int in = 2 * ((u + U) * D + (-m + U));
      float sr, si;
      if (m == 0) {
        sr = 2.0f * g[ip];
        si = 2.0f * g[ip + 1];
      } else if (mp & 1) {  // cos(m phi): pi at v = +-m
        sr = g[ip] + g[in];
        si = g[ip + 1] + g[in + 1];
      } else {  // sin(m phi): i pi sgn(v) at v = +-m, folded as i * (g+ - g-)
        const float dr = g[ip] - g[in], di = g[ip + 1] - g[in + 1];
        sr = -di;
        si = dr;
      }
      acc = fmaf(sr, cr, acc);
      acc = fmaf(-si, ci, acc);
    }
    y[e] = kPiF * acc;
  }
}

// SH filter out[b, c, lm] = h[b, c, l] * Y_l^m(r_b) with an fp64 recurrence.
__global__ __launch_bounds__(kBlock) void k_sh_filter(int L, const float* __restrict__ r,
                                                      const float* __restrict__ h, int64_t B, int64_t C,
                                                      float* __restrict__ out) {
  const int K = (L + 1) * (L + 1);
  const double kPi = 3.14159265358979323846;
  for (int64_t b = blockIdx.x; b < B; b += gridDim.x) {
    double rx = r[3 * b], ry = r[3 * b + 1], rz = r[3 * b + 2];
    const double nr = sqrt(rx * rx + ry * ry + rz * rz);
    if (nr > 0.0) {
      rx /= nr;
      ry /= nr;
      rz /= nr;
    } else {
      rx = 0.0;
      ry = 0.0;
      rz = 1.0;
    }
    const double st = sqrt(fmax(0.0, 1.0 - rz * rz));
    const double phi = atan2(ry, rx);
    for (int o = threadIdx.x; o < K; o += kBlock) {
      int l, m, mp;
      split_index(o, l, m, mp);
      double pmm = sqrt(1.0 / (4.0 * kPi));
      for (int k = 1; k <= m; ++k) pmm *= sqrt((2.0 * k + 1.0) / (2.0 * k)) * st;
      double q = pmm;
      if (l > m) {
        double p2 = pmm, p1 = sqrt(2.0 * m + 3.0) * rz * pmm;
        for (int ll = m + 2; ll <= l; ++ll) {
          const double a = sqrt((4.0 * ll * ll - 1.0) / (double(ll) * ll - double(m) * m));
          const double bb = sqrt(((ll - 1.0) * (ll - 1.0) - double(m) * m) / (4.0 * (ll - 1.0) * (ll - 1.0) - 1.0));
          const double pn = a * (rz * p1 - bb * p2);
          p2 = p1;
          p1 = pn;
        }
        q = p1;
      }
      double yv = q;
      if (m > 0) yv = sqrt(2.0) * q * ((mp & 1) ? cos(m * phi) : sin(m * phi));
      const float yf = float(yv);
      for (int64_t c = 0; c < C; ++c) {
        const float hv = h ? h[(b * C + c) * (L + 1) + l] : 1.0f;
        out[(b * C + c) * K + o] = hv * yf;
      }
    }
  }
}

// Fused product with the 2D convolution done directly (Sec. 3.2, eq.
// 2D-conv, without the convolution theorem), in the real form of the
// Fourier basis, one product per workgroup:
//   (1) g_t[m][u] = sum_l T1[tri(l, m)][u] (x_t[l, +m] - i x_t[l, -m]): F_t =
//       sum_{m >= 0, u} Re(g_t[m][u] e^{i m phi}) T_m(u theta), T_m = cos for
//       even m, sin for odd m (the theta series of eq. sh-fs, real form);
//   (2) c[m3][u3]: product of the two series; in phi
//       Re(a e^{i m1 phi}) Re(b e^{i m2 phi}) = 1/2 Re(a b e^{i (m1+m2) phi})
//       + 1/2 Re(a conj(b) e^{i (m1-m2) phi}), in theta the product-to-sum
//       identities of cos / sin, each output cell gathering its terms;
//   (3) y[l, +m] = n_m sum_u Z[tri(l, m)][u] Re c[m][u], y[l, -m] = n_m sum_u
//       Z[tri(l, m)][u] (-Im c[m][u]), Z = Zc (even m) or Zs (odd m),
//       n_0 = 2 pi, n_m = pi (eq. fs-sh: the phi integral of cos^2, sin^2).
// LDS: x1, x2, then g1, g2 (complex), c (complex).
struct DirectLayout {
  int K1, K2, G1, G2, C3, off_g1, off_g2, off_c, total;
};
__host__ __device__ inline DirectLayout direct_layout(const DevTables& t) {
  DirectLayout d;
  d.K1 = (t.L1 + 1) * (t.L1 + 1);
  d.K2 = (t.L2 + 1) * (t.L2 + 1);
  d.G1 = (t.L1 + 1) * (t.L1 + 1);  // [m][u], m, u <= L1
  d.G2 = (t.L2 + 1) * (t.L2 + 1);
  d.C3 = (t.Le + 1) * (t.U + 1);   // [m3][u3], m3 <= Le, u3 <= U
  d.off_g1 = d.K1 + d.K2;
  d.off_g2 = d.off_g1 + 2 * d.G1;
  d.off_c = d.off_g2 + 2 * d.G2;
  d.total = d.off_c + 2 * d.C3;
  return d;
}

// theta product-to-sum coefficient of T_{m1}(u1 t) T_{m2}(u2 t) on the output
// term T_{m1+m2}(u3 t): sum = 1 for u1 + u2 = u3, else the difference term
__device__ __forceinline__ float theta_coef(bool odd1, bool odd2, bool is_sum, int u1, int u2) {
  if (!odd1 && !odd2) return 0.5f;                       // cos cos = (cos(u1-u2) + cos(u1+u2)) / 2
  if (odd1 && odd2) return is_sum ? -0.5f : 0.5f;        // sin sin = (cos(u1-u2) - cos(u1+u2)) / 2
  if (is_sum) return 0.5f;                               // sin cos, cos sin: sin(u1+u2) / 2 ...
  const int d = odd1 ? u1 - u2 : u2 - u1;                // ... + sin(u1-u2) / 2, resp. + sin(u2-u1) / 2
  return d > 0 ? 0.5f : (d < 0 ? -0.5f : 0.0f);
}

template <typename T1, typename T2>
__global__ __launch_bounds__(kBlock) void k_full_direct(DevTables t, const T1* __restrict__ x1,
                                                        const T2* __restrict__ x2, float* __restrict__ y, int64_t n) {
  extern __shared__ float smem[];
  const DirectLayout d = direct_layout(t);
  lds_poison(smem, d.total);
  const int tid = threadIdx.x;
  const int L1 = t.L1, L2 = t.L2, Le = t.Le, U = t.U;
  const int KO = (t.Lout + 1) * (t.Lout + 1);
  float* xs1 = smem;
  float* xs2 = smem + d.K1;
  float2* g1 = reinterpret_cast<float2*>(smem + d.off_g1);
  float2* g2 = reinterpret_cast<float2*>(smem + d.off_g2);
  float2* c3 = reinterpret_cast<float2*>(smem + d.off_c);
  const float kPiF = 3.14159265358979323846f;

  for (int64_t p = blockIdx.x; p < n; p += gridDim.x) {
    for (int i = tid; i < d.K1; i += kBlock) xs1[i] = ld_in(x1, p * d.K1 + i);
    for (int i = tid; i < d.K2; i += kBlock) xs2[i] = ld_in(x2, p * d.K2 + i);
    __syncthreads();
    // (1) theta series of every phi part
    for (int e = tid; e < d.G1 + d.G2; e += kBlock) {
      const bool second = e >= d.G1;
      const int L = second ? L2 : L1;
      const int ee = second ? e - d.G1 : e;
      const int m = ee / (L + 1), u = ee % (L + 1);
      const float* xs = second ? xs2 : xs1;
      float re = 0.0f, im = 0.0f;
      for (int l = (m > u ? m : u); l <= L; ++l) {
        if ((l - u) & 1) continue;  // Theta_lm has only u = l (mod 2)
        const float c = t.T1[dtri(l, m) * t.ldT1 + u];
        re = fmaf(c, xs[l * l + l + m], re);
        if (m > 0) im = fmaf(-c, xs[l * l + l - m], im);
      }
      (second ? g2 : g1)[ee] = make_float2(re, im);
    }
    __syncthreads();
    // (2) direct convolution, gathered per output cell (m3, u3)
    for (int e = tid; e < d.C3; e += kBlock) {
      const int m3 = e / (U + 1), u3 = e % (U + 1);
      float cr = 0.0f, ci = 0.0f;
      for (int m1 = 0; m1 <= L1; ++m1) {
        // the (m2, phi factor) partners of m1: 0 = a b (m1 + m2 = m3),
        // 1 = a conj(b) (m1 - m2 = m3), 2 = conj(a) b (m2 - m1 = m3 > 0)
        for (int kind = 0; kind < 3; ++kind) {
          const int m2 = kind == 0 ? m3 - m1 : (kind == 1 ? m1 - m3 : m1 + m3);
          if (m2 < 0 || m2 > L2 || (kind == 2 && m3 == 0)) continue;
          const bool odd1 = m1 & 1, odd2 = m2 & 1;
          const float2* a = g1 + m1 * (L1 + 1);
          const float2* b = g2 + m2 * (L2 + 1);
          float sr = 0.0f, si = 0.0f;
          for (int u1 = 0; u1 <= L1; ++u1) {
            // theta partners: u1 + u2 = u3, u1 - u2 = u3, u2 - u1 = u3 (> 0)
            for (int tk = 0; tk < 3; ++tk) {
              const int u2 = tk == 0 ? u3 - u1 : (tk == 1 ? u1 - u3 : u1 + u3);
              if (u2 < 0 || u2 > L2 || (tk == 2 && u3 == 0)) continue;
              const float w = theta_coef(odd1, odd2, tk == 0, u1, u2);
              if (w == 0.0f) continue;
              const float2 av = a[u1], bv = b[u2];
              // a b, a conj(b) or conj(a) b
              const float bi = kind == 1 ? -bv.y : bv.y, ai = kind == 2 ? -av.y : av.y;
              sr = fmaf(w, av.x * bv.x - ai * bi, sr);
              si = fmaf(w, av.x * bi + ai * bv.x, si);
            }
          }
          cr = fmaf(0.5f, sr, cr);
          ci = fmaf(0.5f, si, ci);
        }
      }
      c3[e] = make_float2(cr, ci);
    }
    __syncthreads();
    // (3) projection onto the output SH
    for (int o = tid; o < KO; o += kBlock) {
      int l = 0;
      while ((l + 1) * (l + 1) <= o) ++l;
      const int ms = o - l * l - l, m = ms < 0 ? -ms : ms;
      float acc = 0.0f;
      if (l <= Le) {
        const float* Z = ((m & 1) ? t.Zs : t.Zc) + dtri(l, m) * t.ldZ;
        const float2* c = c3 + m * (U + 1);
        for (int u = 0; u <= U; ++u) acc = fmaf(Z[u], ms < 0 ? -c[u].y : c[u].x, acc);
        acc *= m == 0 ? 2.0f * kPiF : kPiF;
      }
      y[p * KO + o] = acc;
    }
    __syncthreads();
  }
}

unsigned grid_for(int64_t work_items, int per_block) {
  int64_t g = (work_items + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > (1 << 22)) g = (1 << 22);
  return unsigned(g);
}

}  // namespace

int generic_chunk(const DevTables& t, int nu, size_t* lds_bytes) {
  // largest node chunk whose LDS footprint stays within the 64 KB default
  int JC = t.NJ;
  while (JC > 1 && generic_layout(t, nu, JC).total * sizeof(float) > 64 * 1024) JC = (JC + 1) / 2;
  *lds_bytes = size_t(generic_layout(t, nu, JC).total) * sizeof(float);
  return JC;
}

hipError_t launch_full_generic(const DevTables& t, const void* x1, int type1, const void* x2, int type2, int64_t n,
                               float* y, int nu, const DegWeights& wt, hipStream_t s, const PairIdx& pi) {
  size_t lds = 0;
  const int JC = generic_chunk(t, nu, &lds);
  const dim3 grid(grid_for(n, 1)), block(kBlock);
  const bool b1 = type1 == IN_BF16, b2 = type2 == IN_BF16;
  using u16 = uint16_t;
  if (b1 && b2)
    hipLaunchKernelGGL((k_full_generic<u16, u16>), grid, block, lds, s, t, static_cast<const u16*>(x1),
                       static_cast<const u16*>(x2), y, n, nu, JC, wt, pi);
  else if (b1)
    hipLaunchKernelGGL((k_full_generic<u16, float>), grid, block, lds, s, t, static_cast<const u16*>(x1),
                       static_cast<const float*>(x2), y, n, nu, JC, wt, pi);
  else if (b2)
    hipLaunchKernelGGL((k_full_generic<float, u16>), grid, block, lds, s, t, static_cast<const float*>(x1),
                       static_cast<const u16*>(x2), y, n, nu, JC, wt, pi);
  else
    hipLaunchKernelGGL((k_full_generic<float, float>), grid, block, lds, s, t, static_cast<const float*>(x1),
                       static_cast<const float*>(x2), y, n, nu, JC, wt, pi);
  return hipGetLastError();
}

template <typename TIn>
__global__ __launch_bounds__(kBlock) void k_pad_copy(const TIn* __restrict__ x, int K, int64_t n,
                                                     float* __restrict__ y, int KO) {
  const int64_t total = n * KO;
  for (int64_t e = int64_t(blockIdx.x) * kBlock + threadIdx.x; e < total; e += int64_t(gridDim.x) * kBlock) {
    const int64_t p = e / KO;
    const int i = int(e % KO);
    y[e] = i < K ? ld_in(x, p * K + i) : 0.0f;
  }
}

hipError_t launch_pad_copy(const void* x, int in_type, int L, int64_t n, float* y, int Lout, hipStream_t s) {
  const int K = (L + 1) * (L + 1), KO = (Lout + 1) * (Lout + 1);
  const dim3 g(grid_for(n * KO, kBlock)), b(kBlock);
  if (in_type == IN_BF16)
    hipLaunchKernelGGL(k_pad_copy<uint16_t>, g, b, 0, s, static_cast<const uint16_t*>(x), K, n, y, KO);
  else
    hipLaunchKernelGGL(k_pad_copy<float>, g, b, 0, s, static_cast<const float*>(x), K, n, y, KO);
  return hipGetLastError();
}

// Lout = 0: the only output is the projection of F1 F2 onto Y_0^0, i.e.
// (1 / sqrt(4 pi)) int F1 F2 dOmega, which orthonormality of the real SH
// turns into the dot product of the coefficients both inputs have (Sec. 3.1,
// the Gaunt coefficient with (l, m) = (0, 0)).  One lane per product.
template <typename T1, typename T2>
__global__ __launch_bounds__(kBlock) void k_dot0(const T1* __restrict__ x1, int k1, const T2* __restrict__ x2,
                                                 int k2, int64_t n, float* __restrict__ y) {
  const int kc = k1 < k2 ? k1 : k2;
  for (int64_t p = int64_t(blockIdx.x) * kBlock + threadIdx.x; p < n; p += int64_t(gridDim.x) * kBlock) {
    float a = 0.0f;
    for (int i = 0; i < kc; ++i) a = fmaf(ld_in(x1, p * k1 + i), ld_in(x2, p * k2 + i), a);
    y[p] = a * 0.28209479177387814f;  // 1 / sqrt(4 pi)
  }
}

hipError_t launch_dot0(const void* x1, int it1, int k1, const void* x2, int it2, int k2, int64_t n, float* y,
                       hipStream_t s, bool* supported) {
  *supported = true;
  const dim3 g(grid_for(n, kBlock)), b(kBlock);
  if (it1 == IN_F32 && it2 == IN_F32)
    hipLaunchKernelGGL((k_dot0<float, float>), g, b, 0, s, static_cast<const float*>(x1), k1,
                       static_cast<const float*>(x2), k2, n, y);
  else if (it1 == IN_BF16 && it2 == IN_BF16)
    hipLaunchKernelGGL((k_dot0<uint16_t, uint16_t>), g, b, 0, s, static_cast<const uint16_t*>(x1), k1,
                       static_cast<const uint16_t*>(x2), k2, n, y);
  else if (it1 == IN_F32 && it2 == IN_BF16)
    hipLaunchKernelGGL((k_dot0<float, uint16_t>), g, b, 0, s, static_cast<const float*>(x1), k1,
                       static_cast<const uint16_t*>(x2), k2, n, y);
  else {
    *supported = false;
    return hipSuccess;
  }
  return hipGetLastError();
}

hipError_t launch_full_direct(const DevTables& t, const void* x1, int it1, const void* x2, int it2, int64_t n,
                              float* y, hipStream_t s) {
  const size_t lds = size_t(direct_layout(t).total) * sizeof(float);
  if (lds > 64 * 1024) return hipErrorNotSupported;  // the default LDS limit of one workgroup
  if (n <= 0) return hipSuccess;
  const dim3 grid(grid_for(n, 1)), block(kBlock);
  const float* f1 = static_cast<const float*>(x1);
  const float* f2 = static_cast<const float*>(x2);
  const uint16_t* h1 = static_cast<const uint16_t*>(x1);
  const uint16_t* h2 = static_cast<const uint16_t*>(x2);
  if (it1 == IN_BF16 && it2 == IN_BF16)
    hipLaunchKernelGGL((k_full_direct<uint16_t, uint16_t>), grid, block, lds, s, t, h1, h2, y, n);
  else if (it1 == IN_BF16)
    hipLaunchKernelGGL((k_full_direct<uint16_t, float>), grid, block, lds, s, t, h1, f2, y, n);
  else if (it2 == IN_BF16)
    hipLaunchKernelGGL((k_full_direct<float, uint16_t>), grid, block, lds, s, t, f1, h2, y, n);
  else
    hipLaunchKernelGGL((k_full_direct<float, float>), grid, block, lds, s, t, f1, f2, y, n);
  return hipGetLastError();
}

hipError_t launch_sh2fourier(const DevTables& t, int L, const void* x, int in_type, int64_t n, float* grid,
                             hipStream_t s) {
  const int64_t D = 2 * L + 1;
  const dim3 g(grid_for(n * D * D, kBlock)), b(kBlock);
  if (in_type == IN_BF16)
    hipLaunchKernelGGL(k_sh2fourier<uint16_t>, g, b, 0, s, t, L, static_cast<const uint16_t*>(x), grid, n);
  else
    hipLaunchKernelGGL(k_sh2fourier<float>, g, b, 0, s, t, L, static_cast<const float*>(x), grid, n);
  return hipGetLastError();
}

hipError_t launch_fourier_conv(int L1, int L2, const float* g1, const float* g2, int64_t n, float* g3,
                               hipStream_t s) {
  const size_t bytes = size_t(2) * ((2 * L1 + 1) * (2 * L1 + 1) + (2 * L2 + 1) * (2 * L2 + 1)) * sizeof(float);
  const int use_lds = bytes <= 64 * 1024;
  hipLaunchKernelGGL(k_fourier_conv, dim3(grid_for(n, 1)), dim3(kBlock), use_lds ? bytes : 0, s, L1, L2, g1, g2,
                     g3, n, use_lds);
  return hipGetLastError();
}

hipError_t launch_fourier2sh(const DevTables& t, const float* g3, int64_t n, float* y, hipStream_t s) {
  const int64_t KO = int64_t(t.Lout + 1) * (t.Lout + 1);
  hipLaunchKernelGGL(k_fourier2sh, dim3(grid_for(n * KO, kBlock)), dim3(kBlock), 0, s, t, g3, y, n);
  return hipGetLastError();
}

hipError_t launch_sh_filter(int L, const float* r, const float* h, int64_t B, int64_t C, float* out,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_sh_filter, dim3(grid_for(B, 1)), dim3(kBlock), 0, s, L, r, h, B, C, out);
  return hipGetLastError();
}

}  // namespace gtp
