// C ABI of the Gaunt Tensor Product library: plans, argument validation (all
// of it before the first HIP call), table upload and kernel dispatch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <new>
#include <stdexcept>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/gtp.h"
#include "gtp_device.hpp"
#include "gtp_escn.hpp"
#include "gtp_probe.hpp"
#include "gtp_small.hpp"
#include "gtp_tables.hpp"

struct gtp_plan_ {
  int L1 = 0, L2 = 0, Lout = 0;
  float* scratch = nullptr;  // this device's copy of the static scratch array (gtp_conv_escn_noalloc)
  unsigned flags = 0;
  bool host_only = true;
  int device = -1;
  int conv = GTP_CONV_DFT;
  bool force_generic = false;
  gtp::Tables tab;
  gtp::EscnHost esc;  // rotated-frame convolution tables (L1 = L2 = Lout <= 8)
  std::vector<float*> dbufs;
  gtp::DevTables dev{};
  gtp::EscnDev escd{};
  // companion plans (process-lifetime cache entries), made with the plan so
  // that no later call allocates: the equal-degree plan of the padded
  // matrix-core product, and the degree-16 plan of the rotated-frame kernel
  struct gtp_plan_* padw = nullptr;
  struct gtp_plan_* esc16 = nullptr;
};

// Device scratch of the allocation-free entry point: one copy per device,
// allocated with the library's code object and held until the process ends.
// Host code never passes this name to a kernel (on the host it is only a
// stand-in for the symbol); it uses the address hipGetSymbolAddress returns
// for the current device, kept in each plan.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

namespace {

thread_local std::string g_last_error;

gtp_status fail(gtp_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

gtp_status hip_fail(hipError_t e, const char* what) {
  return fail(GTP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

constexpr int kMaxL = 64;
constexpr int kMaxLout = 64;
// Internal flag: force the workgroup-per-product kernel (tests compare paths).
constexpr unsigned kForceGeneric = 32u;

bool ranges_overlap(const void* a, size_t na, const void* b, size_t nb) {
  const char* pa = static_cast<const char*>(a);
  const char* pb = static_cast<const char*>(b);
  return pa < pb + nb && pb < pa + na;
}

bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b < 0) return false;
  if (a != 0 && b > INT64_MAX / a) return false;
  *out = a * b;
  return true;
}

size_t dtype_size(gtp_dtype d) { return d == GTP_BF16 ? 2 : 4; }

// Whether every pointer is a multiple of `align` bytes (NULL passes).
template <typename... Ps>
bool aligned(size_t align, Ps... ps) {
  return ((reinterpret_cast<uintptr_t>(ps) % align == 0) && ...);
}

// Test hook: GTP_TEST_FAIL_ALLOC=host makes the host table build fail as if
// out of memory; GTP_TEST_FAIL_ALLOC=<n> makes the n-th device allocation of
// a plan (counting from 0) fail.  Read at every plan creation; unset in
// normal use.
long fail_alloc_hook(bool* host) {
  const char* v = std::getenv("GTP_TEST_FAIL_ALLOC");
  *host = false;
  if (!v || !*v) return -1;
  if (std::strcmp(v, "host") == 0) {
    *host = true;
    return -1;
  }
  char* end = nullptr;
  const long n = std::strtol(v, &end, 10);
  return (end && *end == '\0' && n >= 0) ? n : -1;
}
bool dtype_ok(gtp_dtype d) { return d == GTP_F32 || d == GTP_BF16; }

gtp_status upload(gtp_plan_* p, long fail_at) {
  using gtp::ntri;
  long nalloc = 0;
  // every device allocation of the plan goes through here (fail_at >= 0: the
  // test hook fails that one)
  auto dmalloc = [&](void** d, size_t bytes) -> hipError_t {
    if (nalloc++ == fail_at) return hipErrorOutOfMemory;
    return hipMalloc(d, bytes);
  };
  const gtp::Tables& t = p->tab;
  const int nmp = 2 * t.Mphi + 1;
  const int ntE = ntri(t.Le);
  const int ntS = ntri(t.Lin);
  std::vector<float> WT(size_t(t.NJ) * ntE), ST(size_t(t.NJ) * ntS), PhiT(size_t(t.NP) * nmp);
  for (int r = 0; r < ntE; ++r)
    for (int j = 0; j < t.NJ; ++j) WT[size_t(j) * ntE + r] = float(t.W[size_t(r) * t.NJ + j]);
  for (int r = 0; r < ntS; ++r)
    for (int j = 0; j < t.NJ; ++j) ST[size_t(j) * ntS + r] = float(t.S[size_t(r) * t.NJ + j]);
  for (int mp = 0; mp < nmp; ++mp)
    for (int k = 0; k < t.NP; ++k) PhiT[size_t(k) * nmp + mp] = float(t.Phi[size_t(mp) * t.NP + k]);
  auto up = [&](const std::vector<double>* src64, const std::vector<float>* src32, const float** dst) -> gtp_status {
    const size_t cnt = src64 ? src64->size() : src32->size();
    std::vector<float> h(cnt ? cnt : 1, 0.0f);
    for (size_t i = 0; i < cnt; ++i) h[i] = src64 ? float((*src64)[i]) : (*src32)[i];
    float* d = nullptr;
    hipError_t e = dmalloc(reinterpret_cast<void**>(&d), h.size() * sizeof(float));
    if (e != hipSuccess) return fail(GTP_ERR_ALLOC, std::string("hipMalloc: ") + hipGetErrorString(e));
    p->dbufs.push_back(d);
    e = hipMemcpy(d, h.data(), h.size() * sizeof(float), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy");
    *dst = d;
    return GTP_OK;
  };
  gtp_status s;
  gtp::DevTables& d = p->dev;
  d.L1 = t.L1; d.L2 = t.L2; d.Lout = t.Lout; d.U = t.U; d.Le = t.Le; d.Lin = t.Lin;
  d.NT = t.NT; d.NJ = t.NJ; d.NP = t.NP; d.Mphi = t.Mphi; d.ldT1 = t.ldT1; d.ldZ = t.ldZ;
  if ((s = up(&t.S, nullptr, &d.S)) != GTP_OK) return s;
  if ((s = up(&t.W, nullptr, &d.W)) != GTP_OK) return s;
  if ((s = up(nullptr, &WT, &d.WT)) != GTP_OK) return s;
  if ((s = up(nullptr, &ST, &d.ST)) != GTP_OK) return s;
  d.ntS = ntS;
  d.ntW = ntE;
  if ((s = up(&t.Phi, nullptr, &d.Phi)) != GTP_OK) return s;
  if ((s = up(nullptr, &PhiT, &d.PhiT)) != GTP_OK) return s;
  if ((s = up(&t.T1, nullptr, &d.T1)) != GTP_OK) return s;
  if ((s = up(&t.Zc, nullptr, &d.Zc)) != GTP_OK) return s;
  if ((s = up(&t.Zs, nullptr, &d.Zs)) != GTP_OK) return s;
  d.waveL = t.waveL;
  d.TWR = d.SMP = d.SM0P = d.WP = nullptr;
  d.XMAP = nullptr;
  d.XQUADS = t.XQUADS;
  d.phi_fft = p->conv == GTP_CONV_FFT ? 1 : 0;
  p->escd = gtp::EscnDev{nullptr, nullptr, 0, 0, 0, nullptr, nullptr, nullptr};
  if (p->esc.NPAIR) {
    gtp::EscnDev& ed = p->escd;
    if ((s = up(&p->esc.J, nullptr, &ed.J)) != GTP_OK) return s;
    if ((s = up(&p->esc.E, nullptr, &ed.E)) != GTP_OK) return s;
    ed.LM = p->esc.LM;
    ed.NPAIR = p->esc.NPAIR;
    ed.ERL = p->esc.ERL;
    if (!p->esc.A.empty()) {
      if ((s = up(&p->esc.A, nullptr, &ed.A)) != GTP_OK) return s;
      if ((s = up(&p->esc.Z, nullptr, &ed.Z)) != GTP_OK) return s;
      if ((s = up(&p->esc.JI, nullptr, &ed.JI)) != GTP_OK) return s;
    }
  }
  if (t.waveL) {
    if ((s = up(&t.TWR, nullptr, &d.TWR)) != GTP_OK) return s;
    if ((s = up(&t.SMP, nullptr, &d.SMP)) != GTP_OK) return s;
    if ((s = up(&t.SM0P, nullptr, &d.SM0P)) != GTP_OK) return s;
    if ((s = up(&t.WP, nullptr, &d.WP)) != GTP_OK) return s;
    int* dm = nullptr;
    hipError_t e = dmalloc(reinterpret_cast<void**>(&dm), t.XMAPP.size() * sizeof(int));
    if (e != hipSuccess) return fail(GTP_ERR_ALLOC, std::string("hipMalloc: ") + hipGetErrorString(e));
    p->dbufs.push_back(reinterpret_cast<float*>(dm));
    e = hipMemcpy(dm, t.XMAPP.data(), t.XMAPP.size() * sizeof(int), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy");
    d.XMAP = dm;
  }
  return GTP_OK;
}

void release(gtp_plan_* p) {
  for (float* b : p->dbufs) (void)hipFree(b);
  p->dbufs.clear();
}

gtp_status check_device() {
  int n = 0;
  hipError_t e = hipGetDeviceCount(&n);
  if (e != hipSuccess || n <= 0) return fail(GTP_ERR_NO_DEVICE, "no HIP device visible");
  return GTP_OK;
}

// The 2D-convolution algorithm of GTP_CONV_AUTO, from the measured crossover:
// the convolution theorem at every degree (faster than the direct
// convolution from L = 2 on), with the phi transforms as direct symmetric
// DFTs (unrolled, or contractions on the matrix cores) wherever they beat the
// radix-2 FFT kernels.
unsigned auto_conv(int L1, int L2, int Lout) {
  (void)L1;
  (void)L2;
  (void)Lout;
  return GTP_CONV_DFT;
}

gtp_status cached_plan(int L1, int L2, int Lout, unsigned flags, gtp_plan* out);

// Degree W of the equal-degree matrix-core kernel that runs a triple with no
// kernel of its own (run_product's padding), 0 when none is needed.
int pad_wave_degree(int L1, int L2, int Lout) {
  const int A = std::max({1, L1, L2, std::min(Lout, L1 + L2)});
  const bool own = L1 == L2 && L2 == Lout && (L1 == 16 || L1 == 32 || L1 == 64);
  if (A <= 8 || A > kMaxL || own) return 0;
  return A <= 16 ? 16 : (A <= 32 ? 32 : 64);
}
// Whether the degree-16 rotated-frame kernel serves a triple other than
// (16, 16, 16) (rows zero-padded, outputs truncated): highest degree 9..16.
bool escn_wave_padded(int L1, int L2, int Lout) {
  const int M = std::max({L1, L2, Lout});
  return M >= 9 && M <= gtp::kEscnWaveL && !(L1 == L2 && L2 == Lout && L1 == gtp::kEscnWaveL);
}

gtp_status make_plan(gtp_plan* out, int L1, int L2, int Lout, unsigned flags, int maxL) {
  if (!out) return fail(GTP_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (L1 < 0 || L2 < 0 || Lout < 0 || L1 > maxL || L2 > maxL || Lout > kMaxLout)
    return fail(GTP_ERR_INVALID_ARG, "degrees must satisfy 0 <= L1, L2, Lout <= 64");
  const unsigned conv = flags & 3u;
  if (flags & ~(3u | GTP_PLAN_HOST_ONLY | kForceGeneric)) return fail(GTP_ERR_INVALID_ARG, "unknown flag bits");
  std::unique_ptr<gtp_plan_> p(new (std::nothrow) gtp_plan_);
  if (!p) return fail(GTP_ERR_ALLOC, "host allocation failed");
  p->L1 = L1;
  p->L2 = L2;
  p->Lout = Lout;
  p->flags = flags;
  p->host_only = (flags & GTP_PLAN_HOST_ONLY) != 0;
  p->force_generic = (flags & kForceGeneric) != 0;
  p->conv = conv == GTP_CONV_AUTO ? int(auto_conv(L1, L2, Lout)) : int(conv);
  bool fail_host = false;
  const long fail_dev = fail_alloc_hook(&fail_host);
  try {
    if (fail_host) throw std::bad_alloc();
    p->tab = gtp::build_tables(L1, L2, Lout);
    // the rotated-frame convolution kernels exist for equal degrees <= 8
    // and 16 (degrees 9..15 run on a 16-plan's tables)
    if (L1 == L2 && L2 == Lout && ((L1 >= 1 && L1 <= 8) || L1 == gtp::kEscnWaveL))
      p->esc = gtp::build_escn_tables(p->tab);
  } catch (const std::bad_alloc&) {
    return fail(GTP_ERR_ALLOC, "table allocation failed");
  } catch (const std::exception& e) {
    return fail(GTP_ERR_INVALID_ARG, e.what());
  }
  if (!p->host_only) {
    gtp_status s = check_device();
    if (s != GTP_OK) return s;
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    // this device's address of the scratch array (set-up of the
    // allocation-free entry point; the plan is used only on this device)
    void* sp = nullptr;
    e = hipGetSymbolAddress(&sp, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    p->scratch = static_cast<float*>(sp);
    s = upload(p.get(), fail_dev);
    if (s != GTP_OK) {
      release(p.get());
      return s;
    }
    if (!p->force_generic && p->conv != GTP_CONV_DIRECT) {
      const int W = pad_wave_degree(L1, L2, Lout);
      if (W && (s = cached_plan(W, W, W, GTP_CONV_DFT, &p->padw)) != GTP_OK) {
        release(p.get());
        return s;
      }
      if (escn_wave_padded(L1, L2, Lout) &&
          (s = cached_plan(gtp::kEscnWaveL, gtp::kEscnWaveL, gtp::kEscnWaveL, GTP_CONV_DFT, &p->esc16)) != GTP_OK) {
        release(p.get());
        return s;
      }
    }
  }
  *out = p.release();
  return GTP_OK;
}

// Internal plan cache of the many-body and backward entry points, keyed by
// device, degrees and plan flags.
std::recursive_mutex g_cache_mu;  // make_plan, called under it, takes companion plans
std::map<std::tuple<int, int, int, int, unsigned>, gtp_plan> g_cache;

gtp_status cached_plan(int L1, int L2, int Lout, unsigned flags, gtp_plan* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::recursive_mutex> lk(g_cache_mu);
  auto key = std::make_tuple(dev, L1, L2, Lout, flags);
  auto it = g_cache.find(key);
  if (it != g_cache.end()) {
    *out = it->second;
    return GTP_OK;
  }
  gtp_plan p = nullptr;
  gtp_status s = make_plan(&p, L1, L2, Lout, flags, kMaxL);
  if (s != GTP_OK) return s;
  g_cache[key] = p;
  *out = p;
  return GTP_OK;
}

gtp_status plan_check(gtp_plan p) {
  if (!p) return fail(GTP_ERR_INVALID_ARG, "plan is NULL");
  return GTP_OK;
}

// Last step of validation, after every argument check: a plan built with
// GTP_PLAN_HOST_ONLY has no device tables.
gtp_status device_ready(gtp_plan p) {
  if (p->host_only) return fail(GTP_ERR_INVALID_ARG, "plan was created with GTP_PLAN_HOST_ONLY");
  return GTP_OK;
}

// One fused product y = P_Lout(x1 * x2) with the plan's tables: the direct
// convolution when the plan asks for it, else the thread-per-product kernel,
// the matrix-core wave kernel or the workgroup kernel, the first that has an
// instantiation for the degrees and input types.
constexpr gtp::DegWeights kNoWeights{nullptr, nullptr, nullptr, 1, 0, 0, false};

gtp_status run_product(gtp_plan p, const void* x1, int it1, const void* x2, int it2, int64_t n, float* y,
                       hipStream_t st, const char* what, const gtp::DegWeights& wt = kNoWeights) {
  hipError_t e = hipSuccess;
  if (p->conv == GTP_CONV_DIRECT) {
    if (wt.on) return fail(GTP_ERR_UNSUPPORTED, "per-degree weights are not built for the direct convolution path");
    e = gtp::launch_full_direct(p->dev, x1, it1, x2, it2, n, y, st);
    if (e == hipErrorNotSupported) return fail(GTP_ERR_UNSUPPORTED, "direct convolution path not built");
    return e == hipSuccess ? GTP_OK : hip_fail(e, what);
  }
  bool done = false;
  if (!p->force_generic) {
    e = gtp::launch_full_small(p->dev, x1, it1, x2, it2, n, y, 0, wt, st, &done);
    if (done) return e == hipSuccess ? GTP_OK : hip_fail(e, what);
    e = gtp::launch_full_wave(p->dev, x1, it1, x2, it2, n, y, wt, st, &done);
    if (done) return e == hipSuccess ? GTP_OK : hip_fail(e, what);
    if (!wt.on) {
      // no kernel for these exact degrees: the equal-degree kernel of the
      // padded degree A (the inputs read with zeros above their degrees, the
      // outputs above Lout dropped; exact, see k_full_small_pad)
      const int A = std::max({1, p->L1, p->L2, std::min(p->Lout, p->L1 + p->L2)});
      const int k1 = gtp::nsh(p->L1), k2 = gtp::nsh(p->L2), ko = gtp::nsh(p->Lout);
      if (p->Lout == 0) {
        // one output, the projection onto Y_0^0: a dot product (k_dot0)
        e = gtp::launch_dot0(x1, it1, k1, x2, it2, k2, n, y, st, &done);
        if (done) return e == hipSuccess ? GTP_OK : hip_fail(e, what);
      }
      if (A <= 8) {
        e = gtp::launch_full_small_padded(A, x1, it1, k1, x2, it2, k2, n, y, ko, st, &done);
        if (done) return e == hipSuccess ? GTP_OK : hip_fail(e, what);
      } else if (A <= kMaxL) {
        const int W = A <= 16 ? 16 : (A <= 32 ? 32 : 64);
        gtp_plan q = p->padw;  // made with the plan
        if (!q || q->L1 != W) {
          const gtp_status s = cached_plan(W, W, W, GTP_CONV_DFT, &q);
          if (s != GTP_OK) return s;
        }
        e = gtp::launch_full_wave(q->dev, x1, it1, x2, it2, n, y, wt, st, &done, k1, k2, ko);
        if (done) return e == hipSuccess ? GTP_OK : hip_fail(e, what);
      }
    }
  }
  e = gtp::launch_full_generic(p->dev, x1, it1, x2, it2, n, y, 0, wt, st);
  return e == hipSuccess ? GTP_OK : hip_fail(e, what);
}

// Argument checks shared by both rotated-frame entry points (all before any
// HIP call); *n = B C.
gtp_status escn_check(gtp_plan p, const void* x, gtp_dtype in_dtype, const float* r, const float* h, int64_t B,
                      int64_t C, float* y, int64_t* n_out) {
  gtp_status s = plan_check(p);
  if (s != GTP_OK) return s;
  if (!dtype_ok(in_dtype)) return fail(GTP_ERR_INVALID_ARG, "in_dtype must be GTP_F32 or GTP_BF16");
  int64_t n = 0, ex = 0, eh = 0, eo = 0, er = 0;
  if (!mul_ok(B, C, &n) || !mul_ok(B, 3, &er)) return fail(GTP_ERR_INVALID_ARG, "B and C must be >= 0 and B*C must fit");
  if (!mul_ok(n, gtp::nsh(p->L1), &ex) || !mul_ok(n, p->L2 + 1, &eh) || !mul_ok(n, gtp::nsh(p->Lout), &eo) ||
      ex > INT64_MAX / 4 || eh > INT64_MAX / 4 || eo > INT64_MAX / 4)
    return fail(GTP_ERR_INVALID_ARG, "B*C*(L+1)^2 overflows");
  *n_out = n;
  if (n == 0) return GTP_OK;
  if (!x || !r || !h || !y) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  const size_t es = dtype_size(in_dtype), ny = size_t(eo) * 4;
  if (ranges_overlap(y, ny, x, size_t(ex) * es) || ranges_overlap(y, ny, r, size_t(er) * 4) ||
      ranges_overlap(y, ny, h, size_t(eh) * 4))
    return fail(GTP_ERR_INVALID_ARG, "y overlaps an input");
  if (!aligned(es, x) || !aligned(4, r, h, y)) return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  return GTP_OK;
}

// Whether the plan's rotated-frame convolution runs on its own kernels
// (L1 = L2 = Lout in 1..8 or 16, convolution-theorem plan) rather than as
// filter + plain product.
bool escn_rotated(gtp_plan p) {
  return !p->force_generic && p->conv != GTP_CONV_DIRECT && p->esc.NPAIR > 0 &&
         (gtp::escn_rot_floats(p->L1) > 0 || (p->L1 == gtp::kEscnWaveL && !p->esc.JI.empty()));
}

// Other triples with highest degree 9..16: the degree-16 rotated-frame kernel
// on the companion plan's tables (rows zero-padded, outputs truncated; exact,
// as for the padded product), without workspace.
bool escn_wave16(gtp_plan p) {
  return !p->force_generic && p->conv != GTP_CONV_DIRECT && !escn_rotated(p) && p->esc16 != nullptr;
}
gtp_status escn_wave16_run(gtp_plan p, const void* x, int it, const float* r, const float* h, int64_t B, int64_t C,
                           float* y, hipStream_t st, const char* what) {
  const hipError_t e = gtp::launch_conv_escn_wave(p->esc16->escd, x, it, r, h, B, C, y, gtp::nsh(p->L1), p->L2 + 1,
                                                  gtp::nsh(p->Lout), st);
  return e == hipSuccess ? GTP_OK : hip_fail(e, what);
}

}  // namespace

extern "C" {

gtp_status gtp_plan_create(gtp_plan* out, int L1, int L2, int Lout, unsigned flags) {
  return make_plan(out, L1, L2, Lout, flags, kMaxL);
}

gtp_status gtp_plan_destroy(gtp_plan p) {
  if (!p) return GTP_OK;
  release(p);
  delete p;
  return GTP_OK;
}

gtp_status gtp_full(gtp_plan p, const void* x1, const void* x2, gtp_dtype in_dtype, int64_t B, int64_t C, float* y,
                    void* stream) {
  gtp_status s = plan_check(p);
  if (s != GTP_OK) return s;
  if (!dtype_ok(in_dtype)) return fail(GTP_ERR_INVALID_ARG, "in_dtype must be GTP_F32 or GTP_BF16");
  int64_t n = 0, e1 = 0, e2 = 0, eo = 0;
  if (!mul_ok(B, C, &n)) return fail(GTP_ERR_INVALID_ARG, "B and C must be >= 0 and B*C must fit in int64");
  if (!mul_ok(n, gtp::nsh(p->L1), &e1) || !mul_ok(n, gtp::nsh(p->L2), &e2) || !mul_ok(n, gtp::nsh(p->Lout), &eo) ||
      e1 > INT64_MAX / 4 || e2 > INT64_MAX / 4 || eo > INT64_MAX / 4)
    return fail(GTP_ERR_INVALID_ARG, "B*C*(L+1)^2 overflows");
  if (n == 0) return GTP_OK;
  if (!x1 || !x2 || !y) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  const size_t es = dtype_size(in_dtype);
  if (ranges_overlap(y, size_t(eo) * 4, x1, size_t(e1) * es) || ranges_overlap(y, size_t(eo) * 4, x2, size_t(e2) * es))
    return fail(GTP_ERR_INVALID_ARG, "y overlaps x1 or x2");
  if ((reinterpret_cast<uintptr_t>(x1) | reinterpret_cast<uintptr_t>(x2)) % es || reinterpret_cast<uintptr_t>(y) % 4)
    return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  if ((s = device_ready(p)) != GTP_OK) return s;
  const int it = in_dtype == GTP_BF16 ? gtp::IN_BF16 : gtp::IN_F32;
  return run_product(p, x1, it, x2, it, n, y, static_cast<hipStream_t>(stream), "gtp_full launch");
}

gtp_status gtp_full_weighted(gtp_plan p, const void* x1, const void* x2, gtp_dtype in_dtype, const float* w1,
                             const float* w2, const float* wout, int per_channel, int64_t B, int64_t C, float* y,
                             void* stream) {
  gtp_status s = plan_check(p);
  if (s != GTP_OK) return s;
  if (!dtype_ok(in_dtype)) return fail(GTP_ERR_INVALID_ARG, "in_dtype must be GTP_F32 or GTP_BF16");
  if (per_channel != 0 && per_channel != 1) return fail(GTP_ERR_INVALID_ARG, "per_channel must be 0 or 1");
  int64_t n = 0, e1 = 0, e2 = 0, eo = 0;
  if (!mul_ok(B, C, &n)) return fail(GTP_ERR_INVALID_ARG, "B and C must be >= 0 and B*C must fit in int64");
  if (!mul_ok(n, gtp::nsh(p->L1), &e1) || !mul_ok(n, gtp::nsh(p->L2), &e2) || !mul_ok(n, gtp::nsh(p->Lout), &eo) ||
      e1 > INT64_MAX / 4 || e2 > INT64_MAX / 4 || eo > INT64_MAX / 4)
    return fail(GTP_ERR_INVALID_ARG, "B*C*(L+1)^2 overflows");
  if (n == 0) return GTP_OK;
  if (!x1 || !x2 || !y) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  const size_t es = dtype_size(in_dtype);
  const size_t rows = per_channel ? size_t(C) : 1;
  const size_t nw1 = rows * (p->L1 + 1) * 4, nw2 = rows * (p->L2 + 1) * 4, nwo = rows * (p->Lout + 1) * 4;
  const size_t ny = size_t(eo) * 4;
  if (ranges_overlap(y, ny, x1, size_t(e1) * es) || ranges_overlap(y, ny, x2, size_t(e2) * es) ||
      (w1 && ranges_overlap(y, ny, w1, nw1)) || (w2 && ranges_overlap(y, ny, w2, nw2)) ||
      (wout && ranges_overlap(y, ny, wout, nwo)))
    return fail(GTP_ERR_INVALID_ARG, "y overlaps an input or a weight array");
  if ((reinterpret_cast<uintptr_t>(x1) | reinterpret_cast<uintptr_t>(x2)) % es ||
      (reinterpret_cast<uintptr_t>(y) | reinterpret_cast<uintptr_t>(w1) | reinterpret_cast<uintptr_t>(w2) |
       reinterpret_cast<uintptr_t>(wout)) % 4)
    return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  if ((s = device_ready(p)) != GTP_OK) return s;
  const int it = in_dtype == GTP_BF16 ? gtp::IN_BF16 : gtp::IN_F32;
  const gtp::DegWeights wt{w1, w2, wout, C, 0, per_channel, w1 || w2 || wout};
  return run_product(p, x1, it, x2, it, n, y, static_cast<hipStream_t>(stream), "gtp_full_weighted launch", wt);
}

gtp_status gtp_channel_mix(gtp_plan p, const void* x1, const void* x2, gtp_dtype in_dtype, const float* W,
                           int64_t B, int64_t C1, int64_t C2, int64_t Co, float* y, void* stream) {
  gtp_status s = plan_check(p);
  if (s != GTP_OK) return s;
  if (!dtype_ok(in_dtype)) return fail(GTP_ERR_INVALID_ARG, "in_dtype must be GTP_F32 or GTP_BF16");
  int64_t P = 0, nw = 0, n1 = 0, n2 = 0, no = 0, ex1 = 0, ex2 = 0, eo = 0, npair = 0;
  if (B < 0 || C1 < 0 || C2 < 0 || Co < 0 || !mul_ok(C1, C2, &P) || !mul_ok(Co, P, &nw) || !mul_ok(B, C1, &n1) ||
      !mul_ok(B, C2, &n2) || !mul_ok(B, Co, &no) || !mul_ok(B, P, &npair) || !mul_ok(n1, gtp::nsh(p->L1), &ex1) ||
      !mul_ok(n2, gtp::nsh(p->L2), &ex2) || !mul_ok(no, gtp::nsh(p->Lout), &eo) || eo > INT64_MAX / 4 ||
      nw > INT64_MAX / 4 || Co > 0x7fffffff)
    return fail(GTP_ERR_INVALID_ARG, "sizes must be >= 0 and their products must fit in int64");
  if (no == 0) return GTP_OK;
  if (!y || (P > 0 && (!x1 || !x2 || !W))) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  const size_t es = dtype_size(in_dtype), ny = size_t(eo) * 4;
  if (P > 0 && (ranges_overlap(y, ny, x1, size_t(ex1) * es) || ranges_overlap(y, ny, x2, size_t(ex2) * es) ||
                ranges_overlap(y, ny, W, size_t(nw) * 4)))
    return fail(GTP_ERR_INVALID_ARG, "y overlaps an input or W");
  if ((reinterpret_cast<uintptr_t>(x1) | reinterpret_cast<uintptr_t>(x2)) % es ||
      (reinterpret_cast<uintptr_t>(W) | reinterpret_cast<uintptr_t>(y)) % 4)
    return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  if ((s = device_ready(p)) != GTP_OK) return s;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const int it = in_dtype == GTP_BF16 ? gtp::IN_BF16 : gtp::IN_F32;
  const int K = gtp::nsh(p->Lout), K1 = gtp::nsh(p->L1), K2 = gtp::nsh(p->L2);
  hipError_t e = hipSuccess;
  if (P == 0) {  // no pair products: y = 0 (a fill kernel, not a memset node)
    e = gtp::launch_fill_zero(y, eo, st);
    return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_channel_mix launch");
  }
  const int nct = gtp::mix_fused_nct(int(Co));
  if (!p->force_generic && p->conv != GTP_CONV_DIRECT && nct > 0 && p->L1 == p->L2 && p->L2 == p->Lout &&
      p->L1 >= 1 && p->L1 <= 8 && B <= 0x7fffffff) {
    // one kernel: the pair products of a batch entry stay on chip; only the
    // weights in the kernel's blocked layout go through a workspace
    int64_t nwb = 0;
    if (!mul_ok((P + 255) / 256 * 256, int64_t(16) * nct, &nwb) || nwb > INT64_MAX / 4)
      return fail(GTP_ERR_INVALID_ARG, "C1*C2 too large");
    float* wb = nullptr;
    e = hipMallocAsync(reinterpret_cast<void**>(&wb), size_t(nwb) * sizeof(float), st);
    if (e != hipSuccess) return fail(GTP_ERR_ALLOC, std::string("hipMallocAsync: ") + hipGetErrorString(e));
    bool done = false;
    e = gtp::launch_mix_wt_blocks(W, wb, int(Co), P, nct, st);
    if (e == hipSuccess) e = gtp::launch_mix_fused(p->dev, x1, x2, it, wb, y, B, C1, C2, int(Co), st, &done);
    const hipError_t e2 = hipFreeAsync(wb, st);
    if (e != hipSuccess) return hip_fail(e, "gtp_channel_mix launch");
    if (e2 != hipSuccess) return hip_fail(e2, "hipFreeAsync");
    if (done) return GTP_OK;
  }
  // the transposed weights, then the pair products of a chunk of batch
  // entries (at most 256 MiB) in a stream-ordered workspace, then the mix on
  // the matrix cores
  const int64_t per_b = P * K, nwt = P * gtp::mix_cop(int(Co));
  int64_t chunk = (int64_t(256) << 20) / 4 / per_b;
  if (chunk < 1) chunk = 1;
  if (chunk > B) chunk = B;
  float* ws = nullptr;
  e = hipMallocAsync(reinterpret_cast<void**>(&ws), (size_t(chunk) * per_b + size_t(nwt)) * sizeof(float), st);
  if (e != hipSuccess) return fail(GTP_ERR_ALLOC, std::string("hipMallocAsync: ") + hipGetErrorString(e));
  float* const WT = ws;
  float* const T = ws + nwt;
  e = gtp::launch_mix_transpose(W, WT, int(Co), P, st);
  for (int64_t b0 = 0; b0 < B && e == hipSuccess; b0 += chunk) {
    const int64_t nb = B - b0 < chunk ? B - b0 : chunk;
    const char* a = static_cast<const char*>(x1) + size_t(b0) * C1 * K1 * es;
    const char* c = static_cast<const char*>(x2) + size_t(b0) * C2 * K2 * es;
    const gtp::PairIdx pi{C1, C2};
    bool done = false;
    if (!p->force_generic && p->conv != GTP_CONV_DIRECT)
      e = gtp::launch_pairs_small(p->dev, a, it, c, it, nb * P, T, pi, st, &done);
    if (!done) {
      const gtp::DegWeights nw0{nullptr, nullptr, nullptr, 1, 0, 0, false};
      e = gtp::launch_full_generic(p->dev, a, it, c, it, nb * P, T, 0, nw0, st, pi);
    }
    if (e == hipSuccess) e = gtp::launch_mix_gemm(WT, T, y + size_t(b0) * Co * K, int(Co), P, K, nb, st);
  }
  const hipError_t e2 = hipFreeAsync(ws, st);
  if (e != hipSuccess) return hip_fail(e, "gtp_channel_mix launch");
  return e2 == hipSuccess ? GTP_OK : hip_fail(e2, "hipFreeAsync");
}

gtp_status gtp_conv_escn(gtp_plan p, const void* x, gtp_dtype in_dtype, const float* r, const float* h, int64_t B,
                         int64_t C, float* y, void* stream) {
  int64_t n = 0;
  gtp_status s = escn_check(p, x, in_dtype, r, h, B, C, y, &n);
  if (s != GTP_OK || n == 0) return s;
  if ((s = device_ready(p)) != GTP_OK) return s;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const int it = in_dtype == GTP_BF16 ? gtp::IN_BF16 : gtp::IN_F32;
  const int64_t rf = gtp::escn_rot_floats(p->L1);
  if (escn_rotated(p)) {
    // per-edge rotation matrices in a stream-ordered workspace (none when the
    // kernel applies the rotations from the edge angles)
    float* dws = nullptr;
    int64_t nd = 0;
    if (!mul_ok(B, rf, &nd) || nd > INT64_MAX / 4) return fail(GTP_ERR_INVALID_ARG, "B too large");
    hipError_t e = nd > 0 ? hipMallocAsync(reinterpret_cast<void**>(&dws), size_t(nd) * sizeof(float), st)
                          : hipSuccess;
    if (e != hipSuccess) return fail(GTP_ERR_ALLOC, std::string("hipMallocAsync: ") + hipGetErrorString(e));
    bool done = false;
    e = gtp::launch_conv_escn(p->escd, p->L1, p->L2, p->Lout, x, it, r, h, B, C, y, dws, st, &done);
    const hipError_t e2 = dws ? hipFreeAsync(dws, st) : hipSuccess;
    if (done) {
      if (e != hipSuccess) return hip_fail(e, "gtp_conv_escn launch");
      return e2 == hipSuccess ? GTP_OK : hip_fail(e2, "hipFreeAsync");
    }
  }
  if (escn_wave16(p)) return escn_wave16_run(p, x, it, r, h, B, C, y, st, "gtp_conv_escn launch");
  // no rotated-frame kernel for these degrees: build the filter in a
  // stream-ordered workspace and take the plain product (same result)
  float* f = nullptr;
  hipError_t e = hipMallocAsync(reinterpret_cast<void**>(&f), size_t(n) * gtp::nsh(p->L2) * sizeof(float), st);
  if (e != hipSuccess) return fail(GTP_ERR_ALLOC, std::string("hipMallocAsync: ") + hipGetErrorString(e));
  e = gtp::launch_sh_filter(p->L2, r, h, B, C, f, st);
  s = e == hipSuccess ? run_product(p, x, it, f, gtp::IN_F32, n, y, st, "gtp_conv_escn launch")
                      : hip_fail(e, "gtp_conv_escn filter launch");
  const hipError_t e2 = hipFreeAsync(f, st);
  if (s != GTP_OK) return s;
  return e2 == hipSuccess ? GTP_OK : hip_fail(e2, "hipFreeAsync");
}

gtp_status gtp_conv_escn_noalloc(gtp_plan p, const void* x, gtp_dtype in_dtype, const float* r, const float* h,
                                 int64_t B, int64_t C, float* y, void* stream) {
  int64_t n = 0;
  gtp_status s = escn_check(p, x, in_dtype, r, h, B, C, y, &n);
  if (s != GTP_OK || n == 0) return s;
  if (escn_wave16(p)) {
    // the degree-16 rotated-frame kernel needs no scratch
    if ((s = device_ready(p)) != GTP_OK) return s;
    return escn_wave16_run(p, x, in_dtype == GTP_BF16 ? gtp::IN_BF16 : gtp::IN_F32, r, h, B, C, y,
                           static_cast<hipStream_t>(stream), "gtp_conv_escn_noalloc launch");
  }
  // scratch floats one edge needs: its rotation matrices (rotated-frame
  // kernels) or its C filter rows (filter + plain product)
  const bool rot = escn_rotated(p);
  const int64_t cap = int64_t(kScratchBytes / sizeof(float));
  const int64_t per_edge = rot ? gtp::escn_rot_floats(p->L1) : (C <= cap / gtp::nsh(p->L2) ? C * gtp::nsh(p->L2) : -1);
  if (per_edge < 0 || per_edge > cap)
    return fail(GTP_ERR_UNSUPPORTED, "one edge needs more than the " + std::to_string(kScratchBytes) +
                                         " bytes of scratch of the allocation-free entry point (C * (L2+1)^2 * 4 "
                                         "bytes of filter when no rotated-frame kernel serves the plan)");
  if ((s = device_ready(p)) != GTP_OK) return s;
  if (!p->scratch) return fail(GTP_ERR_HIP, "plan has no scratch address");
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const int it = in_dtype == GTP_BF16 ? gtp::IN_BF16 : gtp::IN_F32;
  const size_t es = dtype_size(in_dtype);
  const int64_t K1 = gtp::nsh(p->L1), Ko = gtp::nsh(p->Lout), H = p->L2 + 1;
  // edges in chunks that fit the scratch; the launches of a chunk are
  // stream-ordered after those of the previous one, so each chunk reuses the
  // whole array.  Every scratch entry a kernel reads was written earlier in
  // the same chunk: nothing needs clearing.
  // (the degree-16 rotated-frame kernel needs no scratch: one chunk)
  const int64_t chunk = per_edge == 0 ? B : (cap / per_edge < B ? cap / per_edge : B);
  for (int64_t b0 = 0; b0 < B; b0 += chunk) {
    const int64_t nb = B - b0 < chunk ? B - b0 : chunk;
    const void* xc = static_cast<const char*>(x) + size_t(b0) * C * K1 * es;
    const float* rc = r + size_t(b0) * 3;
    const float* hc = h + size_t(b0) * C * H;
    float* yc = y + size_t(b0) * C * Ko;
    hipError_t e = hipSuccess;
    if (rot) {
      bool done = false;
      e = gtp::launch_conv_escn(p->escd, p->L1, p->L2, p->Lout, xc, it, rc, hc, nb, C, yc, p->scratch, st, &done);
      if (!done) return fail(GTP_ERR_HIP, "rotated-frame kernel missing for a plan that has its tables");
      if (e != hipSuccess) return hip_fail(e, "gtp_conv_escn_noalloc launch");
    } else {
      e = gtp::launch_sh_filter(p->L2, rc, hc, nb, C, p->scratch, st);
      if (e != hipSuccess) return hip_fail(e, "gtp_conv_escn_noalloc filter launch");
      if ((s = run_product(p, xc, it, p->scratch, gtp::IN_F32, nb * C, yc, st, "gtp_conv_escn_noalloc launch")) !=
          GTP_OK)
        return s;
    }
  }
  return GTP_OK;
}

gtp_status gtp_full_backward(gtp_plan p, const void* x1, const void* x2, gtp_dtype in_dtype, const float* dy,
                             int64_t B, int64_t C, float* dx1, float* dx2, void* stream) {
  gtp_status s = plan_check(p);
  if (s != GTP_OK) return s;
  if (!dtype_ok(in_dtype)) return fail(GTP_ERR_INVALID_ARG, "in_dtype must be GTP_F32 or GTP_BF16");
  int64_t n = 0, e1 = 0, e2 = 0, eo = 0;
  if (!mul_ok(B, C, &n)) return fail(GTP_ERR_INVALID_ARG, "B and C must be >= 0 and B*C must fit in int64");
  if (!mul_ok(n, gtp::nsh(p->L1), &e1) || !mul_ok(n, gtp::nsh(p->L2), &e2) || !mul_ok(n, gtp::nsh(p->Lout), &eo) ||
      e1 > INT64_MAX / 4 || e2 > INT64_MAX / 4 || eo > INT64_MAX / 4)
    return fail(GTP_ERR_INVALID_ARG, "B*C*(L+1)^2 overflows");
  if (n == 0 || (!dx1 && !dx2)) return GTP_OK;
  if (!dy || (dx1 && !x2) || (dx2 && !x1)) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  const size_t es = dtype_size(in_dtype);
  const size_t b1 = size_t(e1) * 4, b2 = size_t(e2) * 4;
  // every output against every input it could alias, and the outputs against each other
  auto hits_inputs = [&](const void* out, size_t nb) {
    return (x1 && ranges_overlap(out, nb, x1, size_t(e1) * es)) || (x2 && ranges_overlap(out, nb, x2, size_t(e2) * es)) ||
           ranges_overlap(out, nb, dy, size_t(eo) * 4);
  };
  if ((dx1 && hits_inputs(dx1, b1)) || (dx2 && hits_inputs(dx2, b2)) || (dx1 && dx2 && ranges_overlap(dx1, b1, dx2, b2)))
    return fail(GTP_ERR_INVALID_ARG, "a gradient overlaps an input or the other gradient");
  if ((reinterpret_cast<uintptr_t>(x1) | reinterpret_cast<uintptr_t>(x2)) % es ||
      (reinterpret_cast<uintptr_t>(dy) | reinterpret_cast<uintptr_t>(dx1) | reinterpret_cast<uintptr_t>(dx2)) % 4)
    return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  if ((s = device_ready(p)) != GTP_OK) return s;
  // dx1 = P_L1(GTP(dy, x2)) and dx2 = P_L2(GTP(dy, x1)): the real Gaunt
  // coefficient is symmetric in its three (l, m) pairs, so the gradient of
  // <dy, GTP(x1, x2)> in x1 is the product of the functions of dy and x2
  // projected to degree L1 (and likewise for x2).
  const unsigned conv = p->flags & 3u;  // the same request for the gradient plans
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const int it = in_dtype == GTP_BF16 ? gtp::IN_BF16 : gtp::IN_F32;
  if (dx1 && dx2 && p->L1 == p->L2 && p->L2 == p->Lout && !p->force_generic && p->conv != GTP_CONV_DIRECT) {
    // equal degrees 1..8 (the thread-per-product kernel's): both gradients
    // in one launch that reads dy once
    bool done = false;
    const hipError_t e = gtp::launch_bwd_small(p->L1, dy, x1, x2, it, n, dx1, dx2, st, &done);
    if (done) return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_full_backward launch");
  }
  if (dx1) {
    gtp_plan q = p;  // the plan's own tables when (Lout, L2, L1) = (L1, L2, Lout)
    if (p->Lout != p->L1 && (s = cached_plan(p->Lout, p->L2, p->L1, conv, &q)) != GTP_OK) return s;
    if ((s = run_product(q, dy, gtp::IN_F32, x2, it, n, dx1, st, "gtp_full_backward launch")) != GTP_OK) return s;
  }
  if (dx2) {
    gtp_plan q = p;
    if ((p->Lout != p->L1 || p->L1 != p->L2) && (s = cached_plan(p->Lout, p->L1, p->L2, conv, &q)) != GTP_OK)
      return s;
    if ((s = run_product(q, dy, gtp::IN_F32, x1, it, n, dx2, st, "gtp_full_backward launch")) != GTP_OK) return s;
  }
  return GTP_OK;
}

gtp_status gtp_full_weighted_backward(gtp_plan p, const void* x1, const void* x2, gtp_dtype in_dtype,
                                      const float* w1, const float* w2, const float* wout, int per_channel,
                                      const float* dy, int64_t B, int64_t C, float* dx1, float* dx2, float* dw1,
                                      float* dw2, float* dwout, void* stream) {
  gtp_status s = plan_check(p);
  if (s != GTP_OK) return s;
  if (!dtype_ok(in_dtype)) return fail(GTP_ERR_INVALID_ARG, "in_dtype must be GTP_F32 or GTP_BF16");
  if (per_channel != 0 && per_channel != 1) return fail(GTP_ERR_INVALID_ARG, "per_channel must be 0 or 1");
  int64_t n = 0, e1 = 0, e2 = 0, eo = 0;
  if (!mul_ok(B, C, &n)) return fail(GTP_ERR_INVALID_ARG, "B and C must be >= 0 and B*C must fit in int64");
  if (!mul_ok(n, gtp::nsh(p->L1), &e1) || !mul_ok(n, gtp::nsh(p->L2), &e2) || !mul_ok(n, gtp::nsh(p->Lout), &eo) ||
      e1 > INT64_MAX / 4 || e2 > INT64_MAX / 4 || eo > INT64_MAX / 4)
    return fail(GTP_ERR_INVALID_ARG, "B*C*(L+1)^2 overflows");
  const bool any = dx1 || dx2 || dw1 || dw2 || dwout;
  if (n == 0 && !(dw1 || dw2 || dwout)) return GTP_OK;
  if (!any) return GTP_OK;
  if (n > 0 && (!x1 || !x2 || !dy)) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  const int64_t R = per_channel ? C : 1;
  if (R > 65535) return fail(GTP_ERR_UNSUPPORTED, "more than 65535 weight rows");
  const size_t es = dtype_size(in_dtype);
  const size_t rb1 = size_t(R) * (p->L1 + 1) * 4, rb2 = size_t(R) * (p->L2 + 1) * 4, rbo = size_t(R) * (p->Lout + 1) * 4;
  // every output against every input and every other output
  const struct {
    const void* ptr;
    size_t bytes;
  } ins[] = {{x1, size_t(e1) * es}, {x2, size_t(e2) * es}, {dy, size_t(eo) * 4}, {w1, rb1}, {w2, rb2}, {wout, rbo}},
    outs[] = {{dx1, size_t(e1) * 4}, {dx2, size_t(e2) * 4}, {dw1, rb1}, {dw2, rb2}, {dwout, rbo}};
  for (const auto& o : outs) {
    if (!o.ptr || !o.bytes) continue;
    for (const auto& in : ins)
      if (in.ptr && in.bytes && ranges_overlap(o.ptr, o.bytes, in.ptr, in.bytes))
        return fail(GTP_ERR_INVALID_ARG, "an output overlaps an input");
    for (const auto& o2 : outs)
      if (&o2 != &o && o2.ptr && o2.bytes && ranges_overlap(o.ptr, o.bytes, o2.ptr, o2.bytes))
        return fail(GTP_ERR_INVALID_ARG, "two outputs overlap");
  }
  if (!aligned(es, x1, x2) || !aligned(4, dy, w1, w2, wout, dx1, dx2, dw1, dw2, dwout))
    return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  if (p->conv == GTP_CONV_DIRECT) return fail(GTP_ERR_UNSUPPORTED, "per-degree weights are not built for the direct "
                                                                   "convolution path");
  if ((s = device_ready(p)) != GTP_OK) return s;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const int it = in_dtype == GTP_BF16 ? gtp::IN_BF16 : gtp::IN_F32;
  // y = wout GTP(w1 x1, w2 x2): with u1 = P_L1 GTP(wout dy, w2 x2) and
  // u2 = P_L2 GTP(wout dy, w1 x1) the gradients with respect to the weighted
  // inputs (the Gaunt coefficient is symmetric in its three (l, m) pairs),
  //   dx1 = w1 u1,  dw1[r, l1] = sum over row r of <x1, u1> on degree l1
  // (likewise for x2), and with z = GTP(w1 x1, w2 x2)
  //   dwout[r, l] = sum over row r of <dy, z> on degree l.
  const int64_t nchunk = gtp::wgrad_nchunk(B, C, per_channel);
  const bool need_u1 = dx1 || dw1, need_u2 = dx2 || dw2;
  // workspace: u1 / u2 where dx1 / dx2 are not given, z, and the partials
  const int64_t f_u1 = (need_u1 && !dx1) ? e1 : 0, f_u2 = (need_u2 && !dx2) ? e2 : 0, f_z = dwout ? eo : 0;
  const int64_t Lmax = std::max({p->L1, p->L2, p->Lout});
  const int64_t f_part = nchunk * R * (Lmax + 1);
  const int64_t total = f_u1 + f_u2 + f_z + f_part;
  float* ws = nullptr;
  hipError_t e = hipMallocAsync(reinterpret_cast<void**>(&ws), size_t(total > 0 ? total : 1) * sizeof(float), st);
  if (e != hipSuccess) return fail(GTP_ERR_ALLOC, std::string("hipMallocAsync: ") + hipGetErrorString(e));
  float* const u1 = dx1 ? dx1 : ws;
  float* const u2 = dx2 ? dx2 : ws + f_u1;
  float* const z = ws + f_u1 + f_u2;
  float* const part = z + f_z;
  const unsigned conv = p->flags & 3u;
  s = GTP_OK;
  if (n > 0 && need_u1) {
    gtp_plan q = p;
    if ((p->Lout != p->L1 || p->L1 != p->L2) && (s = cached_plan(p->Lout, p->L2, p->L1, conv, &q)) != GTP_OK) {
    } else {
      // slot 1 = dy weighted by wout, slot 2 = x2 weighted by w2, no output weight
      const gtp::DegWeights wt{wout, w2, nullptr, C, 0, per_channel, wout || w2};
      s = run_product(q, dy, gtp::IN_F32, x2, it, n, u1, st, "gtp_full_weighted_backward launch", wt);
      if (s == GTP_OK) {
        e = gtp::launch_wgrad(x1, it, u1, dx1, w1, B, C, p->L1, per_channel, part, dw1, st);
        if (e != hipSuccess) s = hip_fail(e, "gtp_full_weighted_backward reduction");
      }
    }
  }
  if (s == GTP_OK && n > 0 && need_u2) {
    gtp_plan q = p;
    if ((p->Lout != p->L1 || p->L1 != p->L2) && (s = cached_plan(p->Lout, p->L1, p->L2, conv, &q)) != GTP_OK) {
    } else {
      const gtp::DegWeights wt{wout, w1, nullptr, C, 0, per_channel, wout || w1};
      s = run_product(q, dy, gtp::IN_F32, x1, it, n, u2, st, "gtp_full_weighted_backward launch", wt);
      if (s == GTP_OK) {
        e = gtp::launch_wgrad(x2, it, u2, dx2, w2, B, C, p->L2, per_channel, part, dw2, st);
        if (e != hipSuccess) s = hip_fail(e, "gtp_full_weighted_backward reduction");
      }
    }
  }
  if (s == GTP_OK && n > 0 && dwout) {
    const gtp::DegWeights wt{w1, w2, nullptr, C, 0, per_channel, w1 || w2};
    s = run_product(p, x1, it, x2, it, n, z, st, "gtp_full_weighted_backward launch", wt);
    if (s == GTP_OK) {
      e = gtp::launch_wgrad(dy, gtp::IN_F32, z, nullptr, nullptr, B, C, p->Lout, per_channel, part, dwout, st);
      if (e != hipSuccess) s = hip_fail(e, "gtp_full_weighted_backward reduction");
    }
  }
  if (s == GTP_OK && n == 0) {
    // no products: the weight gradients are zero
    for (auto [dw, L] : {std::pair<float*, int>{dw1, p->L1}, {dw2, p->L2}, {dwout, p->Lout}}) {
      if (!dw) continue;
      e = gtp::launch_fill_zero(dw, R * (L + 1), st);
      if (e != hipSuccess) {
        s = hip_fail(e, "gtp_full_weighted_backward launch");
        break;
      }
    }
  }
  const hipError_t ef = hipFreeAsync(ws, st);
  if (s != GTP_OK) return s;
  return ef == hipSuccess ? GTP_OK : hip_fail(ef, "hipFreeAsync");
}

gtp_status gtp_sh2fourier(gtp_plan p, int which, const void* x, gtp_dtype in_dtype, int64_t n, float* grid,
                          void* stream) {
  gtp_status s = plan_check(p);
  if (s != GTP_OK) return s;
  if (which != 1 && which != 2) return fail(GTP_ERR_INVALID_ARG, "which must be 1 or 2");
  if (!dtype_ok(in_dtype)) return fail(GTP_ERR_INVALID_ARG, "bad in_dtype");
  const int L = which == 1 ? p->L1 : p->L2;
  int64_t ex = 0, eg = 0;
  if (!mul_ok(n, gtp::nsh(L), &ex) || !mul_ok(n, int64_t(2) * (2 * L + 1) * (2 * L + 1), &eg) || eg > INT64_MAX / 4 ||
      ex > INT64_MAX / 4)
    return fail(GTP_ERR_INVALID_ARG, "n must be >= 0 and n * grid size must fit");
  if (n == 0) return GTP_OK;
  if (!x || !grid) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  if (ranges_overlap(grid, size_t(eg) * 4, x, size_t(ex) * dtype_size(in_dtype)))
    return fail(GTP_ERR_INVALID_ARG, "grid overlaps x");
  if (!aligned(dtype_size(in_dtype), x) || !aligned(4, grid)) return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  if ((s = device_ready(p)) != GTP_OK) return s;
  hipError_t e = gtp::launch_sh2fourier(p->dev, L, x, in_dtype == GTP_BF16 ? gtp::IN_BF16 : gtp::IN_F32, n, grid,
                                        static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_sh2fourier launch");
}

gtp_status gtp_fourier_conv(gtp_plan p, const float* g1, const float* g2, int64_t n, float* g3, void* stream) {
  gtp_status s = plan_check(p);
  if (s != GTP_OK) return s;
  const int64_t D1 = 2 * p->L1 + 1, D2 = 2 * p->L2 + 1, D3 = 2 * (p->L1 + p->L2) + 1;
  int64_t e1 = 0, e2 = 0, e3 = 0;
  if (!mul_ok(n, 2 * D1 * D1, &e1) || !mul_ok(n, 2 * D2 * D2, &e2) || !mul_ok(n, 2 * D3 * D3, &e3) ||
      e3 > INT64_MAX / 4)
    return fail(GTP_ERR_INVALID_ARG, "n must be >= 0 and n * grid size must fit");
  if (n == 0) return GTP_OK;
  if (!g1 || !g2 || !g3) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  if (ranges_overlap(g3, size_t(e3) * 4, g1, size_t(e1) * 4) || ranges_overlap(g3, size_t(e3) * 4, g2, size_t(e2) * 4))
    return fail(GTP_ERR_INVALID_ARG, "g3 overlaps g1 or g2");
  if (!aligned(4, g1, g2, g3)) return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  if ((s = device_ready(p)) != GTP_OK) return s;
  hipError_t e = gtp::launch_fourier_conv(p->L1, p->L2, g1, g2, n, g3, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_fourier_conv launch");
}

gtp_status gtp_fourier2sh(gtp_plan p, const float* g3, int64_t n, float* y, void* stream) {
  gtp_status s = plan_check(p);
  if (s != GTP_OK) return s;
  const int64_t D3 = 2 * (p->L1 + p->L2) + 1;
  int64_t e3 = 0, eo = 0;
  if (!mul_ok(n, 2 * D3 * D3, &e3) || !mul_ok(n, gtp::nsh(p->Lout), &eo) || e3 > INT64_MAX / 4 || eo > INT64_MAX / 4)
    return fail(GTP_ERR_INVALID_ARG, "n must be >= 0 and n * grid size must fit");
  if (n == 0) return GTP_OK;
  if (!g3 || !y) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  if (ranges_overlap(y, size_t(eo) * 4, g3, size_t(e3) * 4)) return fail(GTP_ERR_INVALID_ARG, "y overlaps g3");
  if (!aligned(4, g3, y)) return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  if ((s = device_ready(p)) != GTP_OK) return s;
  hipError_t e = gtp::launch_fourier2sh(p->dev, g3, n, y, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_fourier2sh launch");
}

gtp_status gtp_selfproduct(int L, int nu, int Lout, unsigned mode, const void* x, gtp_dtype in_dtype, int64_t B,
                           int64_t C, float* y, void* stream) {
  if (L < 0 || L > kMaxL || Lout < 0 || Lout > kMaxLout) return fail(GTP_ERR_INVALID_ARG, "degree out of range");
  if (nu < 1) return fail(GTP_ERR_INVALID_ARG, "nu must be >= 1");
  if (mode != GTP_SELF_STEPWISE && mode != GTP_SELF_FUSED) return fail(GTP_ERR_INVALID_ARG, "bad mode");
  if (mode == GTP_SELF_FUSED && int64_t(nu) * L > kMaxL)
    return fail(GTP_ERR_UNSUPPORTED, "fused mode needs nu * L <= 64");
  if (!dtype_ok(in_dtype)) return fail(GTP_ERR_INVALID_ARG, "bad in_dtype");
  int64_t n = 0, ex = 0, eo = 0;
  if (!mul_ok(B, C, &n) || !mul_ok(n, gtp::nsh(L), &ex) || !mul_ok(n, gtp::nsh(Lout), &eo) || eo > INT64_MAX / 4 ||
      ex > INT64_MAX / 4)
    return fail(GTP_ERR_INVALID_ARG, "B and C must be >= 0 and sizes must fit");
  if (n == 0) return GTP_OK;
  if (!x || !y) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  if (ranges_overlap(y, size_t(eo) * 4, x, size_t(ex) * dtype_size(in_dtype)))
    return fail(GTP_ERR_INVALID_ARG, "y overlaps x");
  if (!aligned(dtype_size(in_dtype), x) || !aligned(4, y)) return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  gtp_status s = check_device();
  if (s != GTP_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int it = in_dtype == GTP_BF16 ? gtp::IN_BF16 : gtp::IN_F32;
  hipError_t e = hipSuccess;
  if (nu == 1) {
    // B_1 = P_Lout(A): truncate or zero-pad the input
    e = gtp::launch_pad_copy(x, it, L, n, y, Lout, st);
    return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_selfproduct launch");
  }
  if (mode == GTP_SELF_STEPWISE && nu == 2) {
    gtp_plan p = nullptr;
    if ((s = cached_plan(L, L, Lout, 0u, &p)) != GTP_OK) return s;
    bool done = false;
    e = gtp::launch_full_small(p->dev, x, it, x, it, n, y, 0, kNoWeights, st, &done);
    if (!done) e = gtp::launch_full_generic(p->dev, x, it, x, it, n, y, 0, kNoWeights, st);
    return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_selfproduct launch");
  }
  if (mode == GTP_SELF_FUSED) {
    gtp_plan p = nullptr;
    if ((s = cached_plan(L, (nu - 1) * L, Lout, 0u, &p)) != GTP_OK) return s;
    bool done = false;
    e = gtp::launch_full_small(p->dev, x, it, x, it, n, y, nu, kNoWeights, st, &done);
    if (!done) e = gtp::launch_full_generic(p->dev, x, it, nullptr, it, n, y, nu, kNoWeights, st);
    return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_selfproduct launch");
  }
  // stepwise, nu >= 3
  gtp_plan p1 = nullptr, p2 = nullptr;
  if ((s = cached_plan(L, L, Lout, 0u, &p1)) != GTP_OK) return s;
  if ((s = cached_plan(Lout, L, Lout, 0u, &p2)) != GTP_OK) return s;
  bool done = false;
  e = gtp::launch_self_stepwise_small(p1->dev, p2->dev, nu, x, it, n, y, st, &done);
  if (done) return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_selfproduct launch");
  // generic chain through a stream-ordered workspace
  float* work = nullptr;
  e = hipMallocAsync(reinterpret_cast<void**>(&work), size_t(eo) * sizeof(float), st);
  if (e != hipSuccess) return fail(GTP_ERR_ALLOC, std::string("hipMallocAsync: ") + hipGetErrorString(e));
  float* cur = (nu % 2 == 1) ? work : y;  // the last product lands in y
  float* nxt = (nu % 2 == 1) ? y : work;
  e = gtp::launch_full_generic(p1->dev, x, it, x, it, n, cur, 0, kNoWeights, st);
  for (int step = 3; e == hipSuccess && step <= nu; ++step) {
    // B_k (fp32, degree Lout) times A
    e = gtp::launch_full_generic(p2->dev, cur, gtp::IN_F32, x, it, n, nxt, 0, kNoWeights, st);
    std::swap(cur, nxt);
  }
  hipError_t e2 = hipFreeAsync(work, st);
  if (e != hipSuccess) return hip_fail(e, "gtp_selfproduct launch");
  return e2 == hipSuccess ? GTP_OK : hip_fail(e2, "hipFreeAsync");
}

gtp_status gtp_sh_filter(int L, const float* r, const float* h, int64_t B, int64_t C, float* out, void* stream) {
  if (L < 0 || L > kMaxL) return fail(GTP_ERR_INVALID_ARG, "degree out of range");
  int64_t n = 0, eo = 0;
  if (!mul_ok(B, C, &n) || !mul_ok(n, gtp::nsh(L), &eo) || eo > INT64_MAX / 4)
    return fail(GTP_ERR_INVALID_ARG, "B and C must be >= 0 and sizes must fit");
  if (!h && C != 1) return fail(GTP_ERR_INVALID_ARG, "h == NULL requires C == 1");
  if (n == 0) return GTP_OK;
  if (!r || !out) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  if (ranges_overlap(out, size_t(eo) * 4, r, size_t(B) * 12) ||
      (h && ranges_overlap(out, size_t(eo) * 4, h, size_t(n) * (L + 1) * 4)))
    return fail(GTP_ERR_INVALID_ARG, "out overlaps an input");
  if (!aligned(4, r, h, out)) return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  gtp_status s = check_device();
  if (s != GTP_OK) return s;
  hipError_t e = gtp::launch_sh_filter(L, r, h, B, C, out, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_sh_filter launch");
}

gtp_status gtp_stream_probe(int mode, const void* src, void* dst, int64_t nbytes, void* stream) {
  if (mode < 0 || mode > 3)
    return fail(GTP_ERR_INVALID_ARG, "mode must be 0 (read), 1 (write), 2 (copy) or 3 (two reads, one write)");
  if (nbytes < 0 || nbytes % (mode == 3 ? 32 : 16))
    return fail(GTP_ERR_INVALID_ARG, "nbytes must be a non-negative multiple of 16 (32 for mode 3)");
  if (nbytes == 0) return GTP_OK;
  if (!dst || (mode != 1 && !src)) return fail(GTP_ERR_INVALID_ARG, "NULL data pointer");
  if (!aligned(16, src, dst)) return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  if ((mode == 2 || mode == 3) &&
      ranges_overlap(src, size_t(nbytes), dst, size_t(mode == 3 ? nbytes / 2 : nbytes)))
    return fail(GTP_ERR_INVALID_ARG, "src and dst overlap");
  gtp_status s = check_device();
  if (s != GTP_OK) return s;
  const hipError_t e = gtp::launch_stream_probe(mode, src, dst, nbytes, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_stream_probe launch");
}

gtp_status gtp_compute_probe(int mode, int64_t iters, float* sink, double* flops, void* stream) {
  if (mode < 0 || mode > 1) return fail(GTP_ERR_INVALID_ARG, "mode must be 0 (VALU FMA) or 1 (MFMA)");
  if (iters < 1 || iters > (int64_t(1) << 30)) return fail(GTP_ERR_INVALID_ARG, "iters must be in 1..2^30");
  if (!sink || !flops) return fail(GTP_ERR_INVALID_ARG, "NULL pointer");
  if (!aligned(4, sink)) return fail(GTP_ERR_INVALID_ARG, "misaligned pointer");
  gtp_status s = check_device();
  if (s != GTP_OK) return s;
  const hipError_t e = gtp::launch_compute_probe(mode, iters, sink, flops, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? GTP_OK : hip_fail(e, "gtp_compute_probe launch");
}

int64_t gtp_grid_floats(gtp_plan p, int which) {
  if (!p || which < 1 || which > 3) return -1;
  const int64_t L = which == 1 ? p->L1 : (which == 2 ? p->L2 : p->L1 + p->L2);
  return 2 * (2 * L + 1) * (2 * L + 1);
}

gtp_status gtp_plan_info(gtp_plan p, int64_t* out8) {
  if (!p || !out8) return fail(GTP_ERR_INVALID_ARG, "NULL argument");
  const gtp::Tables& t = p->tab;
  // the FFT request is served by the radix-FFT kernels at equal degrees 16, 32
  const bool radix = p->conv == GTP_CONV_FFT && !p->force_generic && t.waveL > 0;
  const int64_t used = p->conv == GTP_CONV_FFT && !radix ? GTP_CONV_DFT : p->conv;
  const int64_t v[8] = {t.L1, t.L2, t.Lout, t.U, t.Le, t.NT, t.NP, used};
  std::memcpy(out8, v, sizeof(v));
  return GTP_OK;
}

gtp_status gtp_plan_table(gtp_plan p, int which, double* buf, int64_t* count) {
  if (!p || !count) return fail(GTP_ERR_INVALID_ARG, "NULL argument");
  const std::vector<double>* src = nullptr;
  std::vector<double> tmp;
  switch (which) {
    case 0: src = &p->tab.T1; break;
    case 1: src = &p->tab.Zc; break;
    case 2: src = &p->tab.Zs; break;
    case 3: src = &p->tab.S; break;
    case 4: src = &p->tab.W; break;
    case 5: src = &p->tab.TWR; break;
    case 6: src = &p->tab.SMP; break;
    case 7: src = &p->tab.SM0P; break;
    case 8: src = &p->tab.WP; break;
    case 9: {
      tmp.assign(p->tab.XMAPP.begin(), p->tab.XMAPP.end());
      src = &tmp;
      break;
    }
    case 10: src = &p->esc.J; break;
    case 11: src = &p->esc.E; break;
    case 12: src = &p->esc.A; break;
    case 13: src = &p->esc.Z; break;
    case 14: src = &p->esc.JI; break;
    default: return fail(GTP_ERR_INVALID_ARG, "which must be 0..14");
  }
  if (!buf) {
    *count = int64_t(src->size());
    return GTP_OK;
  }
  if (*count < int64_t(src->size())) return fail(GTP_ERR_INVALID_ARG, "buffer too small");
  std::memcpy(buf, src->data(), src->size() * sizeof(double));
  *count = int64_t(src->size());
  return GTP_OK;
}

gtp_status gtp_debug_host_pipeline(gtp_plan p, const double* x1, const double* x2, int64_t n, double* y) {
  if (!p || n < 0 || (n > 0 && (!x1 || !x2 || !y))) return fail(GTP_ERR_INVALID_ARG, "bad argument");
  try {
    gtp::host_pipeline(p->tab, x1, x2, n, y);
  } catch (const std::bad_alloc&) {
    return fail(GTP_ERR_ALLOC, "host allocation failed");
  }
  return GTP_OK;
}

const char* gtp_status_str(gtp_status s) {
  switch (s) {
    case GTP_OK: return "GTP_OK";
    case GTP_ERR_INVALID_ARG: return "GTP_ERR_INVALID_ARG";
    case GTP_ERR_UNSUPPORTED: return "GTP_ERR_UNSUPPORTED";
    case GTP_ERR_NO_DEVICE: return "GTP_ERR_NO_DEVICE";
    case GTP_ERR_HIP: return "GTP_ERR_HIP";
    case GTP_ERR_ALLOC: return "GTP_ERR_ALLOC";
  }
  return "GTP_ERR_UNKNOWN";
}

const char* gtp_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
