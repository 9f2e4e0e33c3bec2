// C ABI of libfdc: argument validation, plans, workspace layout and kernel
// sequencing.  Every entry point validates on the host first and returns
// before enqueuing anything when an argument is wrong.
#include "fdc.h"
#include "internal.h"

#include <cmath>
#include <cstdlib>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <algorithm>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <unordered_set>
#include <vector>

namespace {

thread_local std::string g_last_error;

fdc_status fail(fdc_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

fdc_status check_hip(hipError_t e, const char *what) {
  if (e == hipSuccess) return FDC_OK;
  return fail(FDC_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool even_pos(long long v) { return v > 0 && v % 2 == 0; }

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }
bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

constexpr uint32_t kFftMagic = 0xFDC0FF70u;
constexpr uint32_t kLayerMagic = 0xFDC01A7Eu;
constexpr uint32_t kStackMagic = 0xFDC05AC4u;

// Registry of live plan handles.  A handle is dereferenced only after it is found
// here, so a destroyed or never-created handle is refused without reading freed
// memory; the magic word then tells the three plan types apart.
std::mutex g_plans_mu;
std::unordered_set<const void *> &live_plans() {
  static std::unordered_set<const void *> s;
  return s;
}
bool plan_register(const void *p) {
  std::lock_guard<std::mutex> g(g_plans_mu);
  try {
    live_plans().insert(p);
  } catch (...) {
    return false;
  }
  return true;
}
bool plan_live(const void *p) {
  if (p == nullptr) return false;
  std::lock_guard<std::mutex> g(g_plans_mu);
  return live_plans().count(p) != 0;
}
// Removes p; false when p was not a live plan.
bool plan_unregister(const void *p) {
  std::lock_guard<std::mutex> g(g_plans_mu);
  return live_plans().erase(p) != 0;
}

}  // namespace

struct fdc_fft_plan {
  uint32_t magic;
  int64_t count;
  int h, w;
};

struct fdc_layer_plan {
  uint32_t magic;
  int kind;  // 0: CIC + FDP, 1: Full FDC
  int B, C, S, N, M, artifact, kn, out;
  int ksz;  // CIC: spatial kernel size for the spatial-kernel calls (0: none given)
  size_t fwd_ws, saved, bwd_ws;
  float2 *tw;  // Full FDC: device table W^j = exp(-2 pi i j / N), j < N (owned by the plan)
};

// ---------------------------------------------------------------------------
// kernel timing
// ---------------------------------------------------------------------------
namespace {
struct Timing {
  std::mutex mu;
  bool enabled = false;
  int max = 0;
  int used = 0;
  std::vector<hipEvent_t> start, stop;
  std::vector<const char *> names;
  std::string only;  // record only launches of this kernel name (empty: all)
};
Timing &timing() {
  static Timing t;
  return t;
}
void timing_release(Timing &t) {
  for (auto e : t.start) (void)hipEventDestroy(e);
  for (auto e : t.stop) (void)hipEventDestroy(e);
  t.start.clear();
  t.stop.clear();
  t.names.clear();
  t.used = 0;
  t.max = 0;
}
}  // namespace

namespace fdc {
bool timing_slot(const char *name, hipEvent_t *start, hipEvent_t *stop) {
  Timing &t = timing();
  if (!t.enabled) return false;
  std::lock_guard<std::mutex> g(t.mu);
  if (t.used >= t.max) return false;
  if (!t.only.empty() && t.only != name) return false;
  t.names[t.used] = name;
  *start = t.start[t.used];
  *stop = t.stop[t.used];
  ++t.used;
  return true;
}
}  // namespace fdc

using fdc::ImgView;

extern "C" {

const char *fdc_status_string(int status) {
  switch (status) {
    case FDC_OK: return "FDC_OK";
    case FDC_EINVAL: return "FDC_EINVAL: invalid argument";
    case FDC_EUNSUPPORTED: return "FDC_EUNSUPPORTED: size or mode not supported";
    case FDC_EWORKSPACE: return "FDC_EWORKSPACE: workspace missing or too small";
    case FDC_EHIP: return "FDC_EHIP: HIP runtime error";
    default: return "unknown fdc_status";
  }
}

const char *fdc_last_error(void) { return g_last_error.c_str(); }

int fdc_version(void) { return 100; }

// ---------------------------------------------------------------------------
// 2-D real FFT plans
// ---------------------------------------------------------------------------
static fdc_status check_fft_plan(const fdc_fft_plan *p) {
  if (!plan_live(p) || p->magic != kFftMagic) return fail(FDC_EINVAL, "invalid or destroyed fft plan");
  return FDC_OK;
}

static size_t fft_spec_bytes(const fdc_fft_plan *p) {
  return (size_t)p->count * p->h * (p->w / 2 + 1) * sizeof(fdc_c64);
}

fdc_status fdc_fft_plan_create(fdc_fft_plan **plan, int64_t count, int h, int w) {
  if (plan == nullptr) return fail(FDC_EINVAL, "plan out-pointer is NULL");
  *plan = nullptr;
  if (count < 1) return fail(FDC_EINVAL, "count must be >= 1 (got %lld)", (long long)count);
  if (!even_pos(h) || !even_pos(w)) return fail(FDC_EINVAL, "h and w must be positive and even (%d x %d)", h, w);
  if (!fdc::size_supported(h) || !fdc::size_supported(w))
    return fail(FDC_EUNSUPPORTED, "transform size %d x %d not supported", h, w);
  if (!fdc::index_fits(count, h) || !fdc::index_fits(count, w / 2 + 1))
    return fail(FDC_EUNSUPPORTED, "count %lld of %d x %d images exceeds the kernels' 32-bit row indexing",
                (long long)count, h, w);
  auto *p = new (std::nothrow) fdc_fft_plan{kFftMagic, count, h, w};
  if (p == nullptr) return fail(FDC_EINVAL, "out of host memory");
  if (!plan_register(p)) {
    delete p;
    return fail(FDC_EINVAL, "out of host memory");
  }
  *plan = p;
  return FDC_OK;
}

fdc_status fdc_fft_plan_destroy(fdc_fft_plan *plan) {
  if (plan == nullptr) return FDC_OK;
  if (!plan_live(plan) || plan->magic != kFftMagic) return fail(FDC_EINVAL, "invalid or destroyed fft plan");
  plan_unregister(plan);
  delete plan;
  return FDC_OK;
}

fdc_status fdc_fft_workspace_size(const fdc_fft_plan *plan, size_t *bytes) {
  if (fdc_status st = check_fft_plan(plan)) return st;
  if (bytes == nullptr) return fail(FDC_EINVAL, "bytes is NULL");
  *bytes = fft_spec_bytes(plan);
  return FDC_OK;
}

static fdc_status check_ws(void *ws, size_t have, size_t need) {
  if (need == 0) return FDC_OK;
  if (ws == nullptr || have < need)
    return fail(FDC_EWORKSPACE, "workspace needs %zu bytes (got %zu, ptr %p)", need, have, ws);
  return FDC_OK;
}

fdc_status fdc_rfft2(const fdc_fft_plan *p, const float *x, fdc_c64 *X, void *, size_t, hipStream_t s) {
  if (fdc_status st = check_fft_plan(p)) return st;
  if (!x || !X) return fail(FDC_EINVAL, "NULL tensor");
  const int h = p->h, w = p->w, wf = w / 2 + 1;
  ImgView id{0, 0, h, w};
  auto *out = reinterpret_cast<float2 *>(X);
  if (fdc::fft2_small_supported(h, w))
    return check_hip(fdc::launch_fft2_small(h, false, x, out, nullptr, nullptr, p->count, 1.f, 1.f, s), "rfft2");
  if (fdc_status st = check_hip(fdc::launch_row_r2c(w, x, fdc::plain_layout(out, h, wf), p->count, h, id,
                                                    (long long)h * w, wf, 1.f, 1.f, s), "rfft2 rows"))
    return st;
  return check_hip(fdc::launch_col_fft(h, -1, out, out, p->count, wf, wf, (long long)h * wf, (long long)h * wf, s),
                   "rfft2 columns");
}

fdc_status fdc_rfft2_pooled(const fdc_fft_plan *p, const float *x, fdc_c64 *X, int mh, int mw, hipStream_t s) {
  if (fdc_status st = check_fft_plan(p)) return st;
  if (!x || !X) return fail(FDC_EINVAL, "NULL tensor");
  const int h = p->h, w = p->w, wf = w / 2 + 1;
  if (mh < 2 || mw < 2 || mh > h || mw > w || (mh & 1) || (mw & 1))
    return fail(FDC_EINVAL, "pooled size %d x %d must be even, >= 2 and within %d x %d", mh, mw, h, w);
  auto *out = reinterpret_cast<float2 *>(X);
  if (fdc::fft2_small_supported(h, w))  // one launch forms every bin
    return check_hip(fdc::launch_fft2_small(h, false, x, out, nullptr, nullptr, p->count, 1.f, 1.f, s),
                     "rfft2_pooled");
  const int L = mw / 2 + 1;
  // the plain layout's row stride with only the first L bins of each row written
  const fdc::SpecLayout lay{out, (long long)h * wf, wf, 8, out + (L - 1), (long long)h * wf, wf};
  ImgView id{0, 0, h, w};
  if (fdc_status st = check_hip(fdc::launch_row_r2c(w, x, lay, p->count, h, id, (long long)h * w, L, 1.f, 1.f, s),
                                "rfft2_pooled rows"))
    return st;
  return check_hip(fdc::launch_col_fft(h, -1, out, out, p->count, L, wf, (long long)h * wf, (long long)h * wf, s, mh),
                   "rfft2_pooled columns");
}

fdc_status fdc_rfft2_pooled_ws(const fdc_fft_plan *p, const float *x, fdc_c64 *X, int mh, int mw, void *ws,
                               size_t ws_bytes, hipStream_t s) {
  if (fdc_status st = check_fft_plan(p)) return st;
  if (!x || !X) return fail(FDC_EINVAL, "NULL tensor");
  const int h = p->h, w = p->w, wf = w / 2 + 1;
  if (mh < 2 || mw < 2 || mh > h || mw > w || (mh & 1) || (mw & 1))
    return fail(FDC_EINVAL, "pooled size %d x %d must be even, >= 2 and within %d x %d", mh, mw, h, w);
  auto *out = reinterpret_cast<float2 *>(X);
  if (fdc::fft2_small_supported(h, w))  // one launch forms every bin, no workspace
    return check_hip(fdc::launch_fft2_small(h, false, x, out, nullptr, nullptr, p->count, 1.f, 1.f, s),
                     "rfft2_pooled");
  const int L = mw / 2 + 1;
  if (fdc_status st = check_ws(ws, ws_bytes, (size_t)p->count * h * L * sizeof(fdc_c64))) return st;
  // rows into the tiled layout in the workspace (whole runs of 8 bins per row), then the
  // column pass reads those tiles and stores the kept rows into X
  const fdc::SpecLayout t = fdc::tiled_layout(static_cast<const float2 *>(ws), p->count, h, L);
  ImgView id{0, 0, h, w};
  if (fdc_status st = check_hip(fdc::launch_row_r2c(w, x, t, p->count, h, id, (long long)h * w, L, 1.f, 1.f, s),
                                "rfft2_pooled rows"))
    return st;
  return check_hip(fdc::launch_col_fft_keep(h, t, out, p->count, L, wf, mh, s), "rfft2_pooled columns");
}

static fdc_status inverse_like(const fdc_fft_plan *p, const fdc_c64 *X, float *x, void *ws, size_t ws_bytes,
                               hipStream_t s, float alpha, float beta, const char *what) {
  if (fdc_status st = check_fft_plan(p)) return st;
  if (!x || !X) return fail(FDC_EINVAL, "NULL tensor");
  if (fdc_status st = check_ws(ws, ws_bytes, fft_spec_bytes(p))) return st;
  const int h = p->h, w = p->w, wf = w / 2 + 1;
  if (fdc::fft2_small_supported(h, w))
    return check_hip(fdc::launch_fft2_small(h, true, nullptr, nullptr, x, reinterpret_cast<const float2 *>(X),
                                            p->count, alpha, beta, s), what);
  auto *tmp = reinterpret_cast<float2 *>(ws);
  if (fdc_status st = check_hip(fdc::launch_col_fft(h, +1, reinterpret_cast<const float2 *>(X), tmp, p->count, wf,
                                                    wf, (long long)h * wf, (long long)h * wf, s), what))
    return st;
  ImgView id{0, 0, h, w};
  return check_hip(fdc::launch_row_c2r(w, fdc::plain_layout(tmp, h, wf), x, p->count, h, wf, alpha, beta, id,
                                       (long long)h * w, s), what);
}

fdc_status fdc_irfft2(const fdc_fft_plan *p, const fdc_c64 *X, float *x, void *ws, size_t ws_bytes,
                      hipStream_t s) {
  if (fdc_status st = check_fft_plan(p)) return st;
  return inverse_like(p, X, x, ws, ws_bytes, s, 1.f / ((float)p->h * (float)p->w), 1.f, "irfft2");
}

fdc_status fdc_rfft2_backward(const fdc_fft_plan *p, const fdc_c64 *gX, float *gx, void *ws, size_t ws_bytes,
                              hipStream_t s) {
  return inverse_like(p, gX, gx, ws, ws_bytes, s, 1.f, 0.5f, "rfft2_backward");
}

fdc_status fdc_irfft2_backward(const fdc_fft_plan *p, const float *gx, fdc_c64 *gX, void *, size_t,
                               hipStream_t s) {
  if (fdc_status st = check_fft_plan(p)) return st;
  if (!gx || !gX) return fail(FDC_EINVAL, "NULL tensor");
  const int h = p->h, w = p->w, wf = w / 2 + 1;
  ImgView id{0, 0, h, w};
  auto *out = reinterpret_cast<float2 *>(gX);
  if (fdc::fft2_small_supported(h, w))
    return check_hip(fdc::launch_fft2_small(h, false, gx, out, nullptr, nullptr, p->count,
                                            1.f / ((float)h * (float)w), 2.f, s), "irfft2_backward");
  if (fdc_status st = check_hip(fdc::launch_row_r2c(w, gx, fdc::plain_layout(out, h, wf), p->count, h, id,
                                                    (long long)h * w, wf, 1.f / ((float)h * (float)w), 2.f, s),
                                "irfft2_backward rows"))
    return st;
  return check_hip(fdc::launch_col_fft(h, -1, out, out, p->count, wf, wf, (long long)h * wf, (long long)h * wf, s),
                   "irfft2_backward columns");
}

// ---------------------------------------------------------------------------
// spectral CIC and FDP
// ---------------------------------------------------------------------------
static fdc_status check_cic_dims(int B, int C, int S, int H, int Wf) {
  if (B < 1 || C < 1 || S < 1 || H < 1 || Wf < 1)
    return fail(FDC_EINVAL, "sizes must be >= 1 (B=%d C=%d S=%d H=%d Wf=%d)", B, C, S, H, Wf);
  if (S % C) return fail(FDC_EINVAL, "CIC needs S mod C == 0 (S=%d C=%d)", S, C);
  return FDC_OK;
}

fdc_status fdc_cic_forward(const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *Y, int B, int C, int S, int H, int Wf,
                           hipStream_t s) {
  if (fdc_status st = check_cic_dims(B, C, S, H, Wf)) return st;
  if (!X || !K || !Y) return fail(FDC_EINVAL, "NULL tensor");
  return check_hip(fdc::launch_cic_fwd(reinterpret_cast<const float2 *>(X), reinterpret_cast<const float2 *>(K),
                                       reinterpret_cast<float2 *>(Y), B, C, S, (long long)H * Wf, s),
                   "cic_forward");
}

fdc_status fdc_cic_backward(const fdc_c64 *gY, const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *gX, fdc_c64 *gK,
                            int B, int C, int S, int H, int Wf, hipStream_t s) {
  if (fdc_status st = check_cic_dims(B, C, S, H, Wf)) return st;
  if (!gY || (gX && !K) || (gK && !X)) return fail(FDC_EINVAL, "NULL tensor");
  const long long P = (long long)H * Wf;
  if (gX) {
    if (fdc_status st = check_hip(fdc::launch_cic_bwd_gx(reinterpret_cast<const float2 *>(gY),
                                                         reinterpret_cast<const float2 *>(K),
                                                         reinterpret_cast<float2 *>(gX), B, C, S, P, s),
                                  "cic_backward gX"))
      return st;
  }
  if (gK) {
    return check_hip(fdc::launch_cic_bwd_gk(reinterpret_cast<const float2 *>(gY), reinterpret_cast<const float2 *>(X),
                                            reinterpret_cast<float2 *>(gK), B, C, S, P, s),
                     "cic_backward gK");
  }
  return FDC_OK;
}

static fdc_status check_cic_fdp(int B, int C, int S, int N, int M) {
  if (B < 1 || C < 1 || S < 1) return fail(FDC_EINVAL, "B, C, S must be >= 1 (B=%d C=%d S=%d)", B, C, S);
  if (S % C) return fail(FDC_EINVAL, "CIC needs S mod C == 0 (S=%d C=%d)", S, C);
  if (!even_pos(N) || !even_pos(M) || M > N)
    return fail(FDC_EINVAL, "N and M must be positive and even with M <= N (N=%d M=%d)", N, M);
  if (!fdc::cic_fdp_size_supported(N))
    return fail(FDC_EUNSUPPORTED, "spectrum of %d x %d bins exceeds the kernels' bin indexing", N, N / 2 + 1);
  // the backward's one-dimensional grid: 256-bin blocks of an N-plane times S channels
  // (dK), 256-pair blocks times C channels (dX) and, projected, a thread per bin of
  // dX's columns 0 and N/2; the projected forward adds a thread per bin of Y's columns
  // 0 and M/2 to its grid, which is smaller than the backward's
  const long long pe = (long long)N * (N / 2 + 1);
  if (((pe + 255) / 256) * S + ((pe / 2 + 255) / 256) * C + ((long long)B * C * N * 2 + 255) / 256 +
          ((long long)B * S * M * 2 + 255) / 256 >= (1LL << 31))
    return fail(FDC_EUNSUPPORTED, "B = %d, S = %d channels of %d x %d bins exceed the kernels' grid", B, S, N,
                N / 2 + 1);
  return FDC_OK;
}

static fdc_status cic_fdp_forward(const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *Y, int B, int C, int S, int N, int M,
                                  bool project, hipStream_t s) {
  if (fdc_status st = check_cic_fdp(B, C, S, N, M)) return st;
  if (!X || !K || !Y) return fail(FDC_EINVAL, "NULL tensor");
  if (!aligned16(Y)) return fail(FDC_EINVAL, "Y must be 16-byte aligned");
  return check_hip(fdc::launch_cic_fdp_fwd(reinterpret_cast<const float2 *>(X), reinterpret_cast<const float2 *>(K),
                                           reinterpret_cast<float2 *>(Y), B, C, S, N, M, project, s),
                   "cic_fdp_forward");
}

fdc_status fdc_cic_fdp_forward(const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *Y, int B, int C, int S, int N, int M,
                               hipStream_t s) {
  return cic_fdp_forward(X, K, Y, B, C, S, N, M, false, s);
}

fdc_status fdc_cic_fdp_forward_projected(const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *Y, int B, int C, int S, int N,
                                         int M, hipStream_t s) {
  return cic_fdp_forward(X, K, Y, B, C, S, N, M, true, s);
}

static fdc_status cic_fdp_backward(const fdc_c64 *gY, const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *gX, fdc_c64 *gK,
                                   int B, int C, int S, int N, int M, bool project, bool kept, hipStream_t s) {
  if (fdc_status st = check_cic_fdp(B, C, S, N, M)) return st;
  if (!gY || (gX && !K) || (gK && !X)) return fail(FDC_EINVAL, "NULL tensor");
  if (gX && !aligned16(gX)) return fail(FDC_EINVAL, "gX must be 16-byte aligned");
  return check_hip(fdc::launch_cic_fdp_bwd(reinterpret_cast<const float2 *>(gY), reinterpret_cast<const float2 *>(K),
                                           reinterpret_cast<float2 *>(gX), reinterpret_cast<const float2 *>(X),
                                           reinterpret_cast<float2 *>(gK), B, C, S, N, M, project, kept, s),
                   "cic_fdp_backward");
}

fdc_status fdc_cic_fdp_backward(const fdc_c64 *gY, const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *gX, fdc_c64 *gK,
                                int B, int C, int S, int N, int M, hipStream_t s) {
  return cic_fdp_backward(gY, X, K, gX, gK, B, C, S, N, M, false, false, s);
}

fdc_status fdc_cic_fdp_backward_projected(const fdc_c64 *gY, const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *gX,
                                          fdc_c64 *gK, int B, int C, int S, int N, int M, hipStream_t s) {
  return cic_fdp_backward(gY, X, K, gX, gK, B, C, S, N, M, true, false, s);
}

fdc_status fdc_cic_fdp_backward_kept(const fdc_c64 *gY, const fdc_c64 *X, const fdc_c64 *K, fdc_c64 *gX, fdc_c64 *gK,
                                     int B, int C, int S, int N, int M, hipStream_t s) {
  return cic_fdp_backward(gY, X, K, gX, gK, B, C, S, N, M, false, true, s);
}

fdc_status fdc_cic_fdp_backward_projected_kept(const fdc_c64 *gY, const fdc_c64 *X, const fdc_c64 *K,
                                               fdc_c64 *gX, fdc_c64 *gK, int B, int C, int S, int N, int M,
                                               hipStream_t s) {
  return cic_fdp_backward(gY, X, K, gX, gK, B, C, S, N, M, true, true, s);
}

fdc_status fdc_hermitian_project(fdc_c64 *Y, int64_t count, int H, int W, hipStream_t s) {
  if (count < 1 || !even_pos(H) || !even_pos(W))
    return fail(FDC_EINVAL, "count >= 1 and even H, W required (count=%lld H=%d W=%d)", (long long)count, H, W);
  if (!Y) return fail(FDC_EINVAL, "Y is NULL");
  if (count > (1LL << 40) / H) return fail(FDC_EUNSUPPORTED, "too many planes (%lld)", (long long)count);
  return check_hip(fdc::launch_hermitian_columns(reinterpret_cast<float2 *>(Y), count, H, W / 2 + 1, s),
                   "hermitian_project");
}

static fdc_status check_fdp(int64_t count, int H, int W, int Mh, int Mw) {
  if (count < 1) return fail(FDC_EINVAL, "count must be >= 1");
  if (!even_pos(H) || !even_pos(W) || !even_pos(Mh) || !even_pos(Mw))
    return fail(FDC_EINVAL, "FDP sizes must be positive and even (%d x %d -> %d x %d)", H, W, Mh, Mw);
  if (Mh > H || Mw > W) return fail(FDC_EINVAL, "FDP output %d x %d larger than input %d x %d", Mh, Mw, H, W);
  return FDC_OK;
}

fdc_status fdp_forward(const fdc_c64 *X, fdc_c64 *Y, int64_t count, int H, int W, int Mh, int Mw, hipStream_t s) {
  if (fdc_status st = check_fdp(count, H, W, Mh, Mw)) return st;
  if (!X || !Y) return fail(FDC_EINVAL, "NULL tensor");
  return check_hip(fdc::launch_fdp_gather(reinterpret_cast<const float2 *>(X), reinterpret_cast<float2 *>(Y), count,
                                          H, W / 2 + 1, Mh, Mw / 2 + 1, s),
                   "fdp_forward");
}

fdc_status fdp_backward(const fdc_c64 *gY, fdc_c64 *gX, int64_t count, int H, int W, int Mh, int Mw,
                        hipStream_t s) {
  if (fdc_status st = check_fdp(count, H, W, Mh, Mw)) return st;
  if (!gY || !gX) return fail(FDC_EINVAL, "NULL tensor");
  return check_hip(fdc::launch_fdp_scatter(reinterpret_cast<const float2 *>(gY), reinterpret_cast<float2 *>(gX),
                                           count, H, W / 2 + 1, Mh, Mw / 2 + 1, s),
                   "fdp_backward");
}

// ---------------------------------------------------------------------------
// layer plans
// ---------------------------------------------------------------------------
static fdc_status check_any_layer_plan(const fdc_layer_plan *p) {
  if (!plan_live(p) || p->magic != kLayerMagic) return fail(FDC_EINVAL, "invalid or destroyed layer plan");
  return FDC_OK;
}

static fdc_status check_layer_plan(const fdc_layer_plan *p, int kind) {
  if (fdc_status st = check_any_layer_plan(p)) return st;
  if (p->kind != kind) return fail(FDC_EINVAL, "layer plan is of the other layer kind");
  return FDC_OK;
}

static int artifact_out(int m, int artifact, int kn) { return artifact == FDC_ARTIFACT_CROP ? m - kn + 1 : m; }

fdc_status fdc_cic_layer_plan_create(fdc_layer_plan **plan, int B, int C, int S, int N, int M, int artifact,
                                     int kernel_n) {
  if (plan == nullptr) return fail(FDC_EINVAL, "plan out-pointer is NULL");
  *plan = nullptr;
  if (B < 1 || C < 1 || S < 1) return fail(FDC_EINVAL, "B, C, S must be >= 1 (B=%d C=%d S=%d)", B, C, S);
  if (S % C) return fail(FDC_EINVAL, "CIC needs S mod C == 0 (S=%d C=%d)", S, C);
  if (!even_pos(N) || !even_pos(M)) return fail(FDC_EINVAL, "N and M must be positive and even (N=%d M=%d)", N, M);
  if (M > N) return fail(FDC_EINVAL, "FDP output M=%d larger than N=%d", M, N);
  if (artifact < FDC_ARTIFACT_NONE || artifact > FDC_ARTIFACT_ROLL) return fail(FDC_EINVAL, "bad artifact mode");
  if (artifact != FDC_ARTIFACT_NONE && (kernel_n < 1 || kernel_n > M))
    return fail(FDC_EINVAL, "kernel_n must be in [1, M] for crop/roll (got %d)", kernel_n);
  if (!fdc::cic_pair_supported(N, M))
    return fail(FDC_EUNSUPPORTED, "layer size %d -> %d not supported (N in the supported set, M in {N, N/2, N/4})",
                N, M);
  if (!fdc::index_fits((long long)B * C, N) || !fdc::index_fits((long long)B * S, M) ||
      !fdc::index_fits((long long)S * N, N / 2 + 1))
    return fail(FDC_EUNSUPPORTED, "B * C * N or B * S * M rows, or the S * N * (N/2+1) bins of gK, exceed the "
                "kernels' 32-bit indexing");
  auto *p = new (std::nothrow) fdc_layer_plan{};
  if (p == nullptr) return fail(FDC_EINVAL, "out of host memory");
  p->magic = kLayerMagic;
  p->kind = 0;
  p->B = B, p->C = C, p->S = S, p->N = N, p->M = M;
  p->artifact = artifact;
  p->kn = artifact == FDC_ARTIFACT_NONE ? 1 : kernel_n;
  p->ksz = kernel_n >= 1 && kernel_n <= M ? kernel_n : 0;
  p->out = artifact_out(M, artifact, p->kn);
  // split-layout spectra (fdc::SpecLayout) of L = M/2 + 1 bins per row
  const size_t L = (size_t)M / 2 + 1;
  const size_t c64 = sizeof(fdc_c64);
  p->fwd_ws = ((size_t)B * C * N * L + (size_t)B * S * M * L + (size_t)B * C * M * L) * c64;  // T, U, Xh
  p->saved = (size_t)B * C * M * L * c64;                             // pooled input spectrum
  p->bwd_ws = ((size_t)B * S * M * L + (size_t)B * C * N * L) * c64;  // Tg, V
  if (!plan_register(p)) {
    delete p;
    return fail(FDC_EINVAL, "out of host memory");
  }
  *plan = p;
  return FDC_OK;
}

fdc_status fdc_layer_plan_destroy(fdc_layer_plan *plan) {
  if (plan == nullptr) return FDC_OK;
  if (fdc_status st = check_any_layer_plan(plan)) return st;
  plan_unregister(plan);
  if (plan->tw != nullptr) (void)hipFree(plan->tw);
  delete plan;
  return FDC_OK;
}

fdc_status fdc_layer_workspace_size(const fdc_layer_plan *p, size_t *fwd_ws, size_t *saved, size_t *bwd_ws) {
  if (fdc_status st = check_any_layer_plan(p)) return st;
  if (fwd_ws) *fwd_ws = p->fwd_ws;
  if (saved) *saved = p->saved;
  if (bwd_ws) *bwd_ws = p->bwd_ws;
  return FDC_OK;
}

fdc_status fdc_layer_output_size(const fdc_layer_plan *p, int *out_size) {
  if (fdc_status st = check_any_layer_plan(p)) return st;
  if (out_size == nullptr) return fail(FDC_EINVAL, "out_size is NULL");
  *out_size = p->out;
  return FDC_OK;
}

static ImgView artifact_view(const fdc_layer_plan *p) {
  switch (p->artifact) {
    case FDC_ARTIFACT_CROP: return ImgView{1, p->kn - 1, p->M, p->out};
    case FDC_ARTIFACT_ROLL: return ImgView{2, (p->kn - 1) / 2, p->M, p->M};
    default: return ImgView{0, 0, p->M, p->M};
  }
}

fdc_status fdc_cic_layer_forward(const fdc_layer_plan *p, const float *x, const fdc_c64 *K, float *y, void *saved,
                                 void *ws, size_t ws_bytes, hipStream_t s) {
  if (fdc_status st = check_layer_plan(p, 0)) return st;
  if (!x || !K || !y) return fail(FDC_EINVAL, "NULL tensor");
  if (fdc_status st = check_ws(ws, ws_bytes, p->fwd_ws)) return st;
  const int B = p->B, C = p->C, S = p->S, N = p->N, M = p->M, L = M / 2 + 1;
  auto *T = reinterpret_cast<float2 *>(ws);
  auto *U = T + (size_t)B * C * N * L;
  // the pooled input spectrum goes to `saved` when the caller keeps it, else to the workspace
  auto *Xh = saved != nullptr ? reinterpret_cast<float2 *>(saved) : U + (size_t)B * S * M * L;
  ImgView id{0, 0, N, N};
  if (fdc_status st = check_hip(fdc::launch_row_r2c(N, x, fdc::tiled_layout(T, (long long)B * C, N, L),
                                                    (long long)B * C, N, id, (long long)N * N, L, 1.f, 1.f, s),
                                "layer forward rows"))
    return st;
  if (fdc_status st = check_hip(fdc::launch_col_fwd_cic(N, M, T, reinterpret_cast<const float2 *>(K), U, Xh, B, C,
                                                        S, s),
                                "layer forward columns"))
    return st;
  return check_hip(fdc::launch_row_c2r(M, fdc::tiled_layout(U, (long long)B * S, M, L), y, (long long)B * S, M, L,
                                       1.f / ((float)M * (float)M), 1.f, artifact_view(p),
                                       (long long)p->out * p->out, s),
                   "layer forward inverse rows");
}

fdc_status fdc_cic_layer_backward(const fdc_layer_plan *p, const float *gy, const void *saved, const fdc_c64 *K,
                                  float *gx, fdc_c64 *gK, void *ws, size_t ws_bytes, hipStream_t s) {
  if (fdc_status st = check_layer_plan(p, 0)) return st;
  if (!gy) return fail(FDC_EINVAL, "gy is NULL");
  if (gK && !saved) return fail(FDC_EINVAL, "saved is NULL but gK was requested");
  if (gx && !K) return fail(FDC_EINVAL, "K is NULL but gx was requested");
  if (!gx && !gK) return FDC_OK;
  if (fdc_status st = check_ws(ws, ws_bytes, p->bwd_ws)) return st;
  const int B = p->B, C = p->C, S = p->S, N = p->N, M = p->M, L = M / 2 + 1;
  auto *Tg = reinterpret_cast<float2 *>(ws);
  auto *V = Tg + (size_t)B * S * M * L;
  if (fdc_status st = check_hip(fdc::launch_row_r2c(M, gy, fdc::tiled_layout(Tg, (long long)B * S, M, L),
                                                    (long long)B * S, M, artifact_view(p),
                                                    (long long)p->out * p->out, L, 1.f / ((float)M * (float)M),
                                                    2.f, s),
                                "layer backward rows"))
    return st;
  if (gK) {
    auto *gk = reinterpret_cast<float2 *>(gK);
    // the dX buffer V (written only after dK) holds dK's batch-range sums
    if (fdc_status st = check_hip(fdc::launch_col_bwd_gk(N, M, Tg, reinterpret_cast<const float2 *>(saved), gk, B,
                                                         C, S, V, (long long)B * C * N * L, s),
                                  "layer backward dK"))
      return st;
  }
  if (gx) {
    if (fdc_status st = check_hip(fdc::launch_col_bwd_gx(N, M, Tg, reinterpret_cast<const float2 *>(K), V, B, C, S,
                                                         s), "layer backward dx columns"))
      return st;
    ImgView id{0, 0, N, N};
    return check_hip(fdc::launch_row_c2r(N, fdc::tiled_layout(V, (long long)B * C, N, L), gx, (long long)B * C, N,
                                         L, 1.f, 0.5f, id, (long long)N * N, s),
                     "layer backward dx rows");
  }
  return FDC_OK;
}

// ---------------------------------------------------------------------------
// CIC layer with spatial kernels
// ---------------------------------------------------------------------------
namespace {
struct SpatialWs {
  size_t k, gk, part, layer, fwd, bwd;  // byte offsets and totals
};
SpatialWs spatial_layout(const fdc_layer_plan *p) {
  SpatialWs w{};
  const size_t kbytes = align256((size_t)p->S * p->N * (p->N / 2 + 1) * sizeof(fdc_c64));
  w.k = 0;
  w.fwd = kbytes + align256(p->fwd_ws);
  w.gk = kbytes;
  w.part = w.gk + kbytes;
  w.layer = w.part + align256((size_t)p->S * fdc::cic_wgrad_blocks(p->M) * p->ksz * p->ksz * sizeof(float));
  w.bwd = w.layer + align256(p->bwd_ws);
  return w;
}
fdc_status check_spatial_plan(const fdc_layer_plan *p) {
  if (fdc_status st = check_layer_plan(p, 0)) return st;
  if (!fdc::spatial_kernel_size_supported(p->ksz))
    return fail(FDC_EUNSUPPORTED, "spatial kernels need a plan with kernel_n in [1, %d] and <= M (got %d)", 8,
                p->ksz);
  if (!fdc::spatial_channels_supported(p->S))
    return fail(FDC_EUNSUPPORTED, "spatial kernels: too many output channels (%d)", p->S);
  return FDC_OK;
}
}  // namespace

fdc_status fdc_cic_spatial_workspace_size(const fdc_layer_plan *p, size_t *fwd_ws, size_t *bwd_ws) {
  if (fdc_status st = check_spatial_plan(p)) return st;
  const SpatialWs w = spatial_layout(p);
  if (fwd_ws) *fwd_ws = w.fwd;
  if (bwd_ws) *bwd_ws = w.bwd;
  return FDC_OK;
}

fdc_status fdc_cic_spatial_layer_forward(const fdc_layer_plan *p, const float *x, const float *w, float *y,
                                         void *saved, void *ws, size_t ws_bytes, hipStream_t s) {
  if (fdc_status st = check_spatial_plan(p)) return st;
  if (!x || !w || !y) return fail(FDC_EINVAL, "NULL tensor");
  const SpatialWs L = spatial_layout(p);
  if (fdc_status st = check_ws(ws, ws_bytes, L.fwd)) return st;
  char *base = static_cast<char *>(ws);
  auto *K = reinterpret_cast<float2 *>(base + L.k);
  if (fdc_status st = check_hip(fdc::launch_cic_kspec(p->N, w, K, p->S, p->ksz, p->M, s), "spatial kernel spectra"))
    return st;
  const size_t layer_off = L.fwd - align256(p->fwd_ws);  // the layer workspace follows the spectra
  return fdc_cic_layer_forward(p, x, reinterpret_cast<const fdc_c64 *>(K), y, saved, base + layer_off,
                               align256(p->fwd_ws), s);
}

fdc_status fdc_cic_spatial_layer_backward(const fdc_layer_plan *p, const float *gy, const void *saved, const float *w,
                                          float *gx, float *gw, void *ws, size_t ws_bytes, hipStream_t s) {
  if (fdc_status st = check_spatial_plan(p)) return st;
  if (!gy) return fail(FDC_EINVAL, "gy is NULL");
  if (gw && !saved) return fail(FDC_EINVAL, "saved is NULL but gw was requested");
  if (gx && !w) return fail(FDC_EINVAL, "w is NULL but gx was requested");
  if (!gx && !gw) return FDC_OK;
  const SpatialWs L = spatial_layout(p);
  if (fdc_status st = check_ws(ws, ws_bytes, L.bwd)) return st;
  char *base = static_cast<char *>(ws);
  auto *K = reinterpret_cast<float2 *>(base + L.k);
  auto *gK = reinterpret_cast<float2 *>(base + L.gk);
  auto *part = reinterpret_cast<float *>(base + L.part);
  if (gx) {
    if (fdc_status st = check_hip(fdc::launch_cic_kspec(p->N, w, K, p->S, p->ksz, p->M, s), "spatial kernel spectra"))
      return st;
  }
  if (fdc_status st = fdc_cic_layer_backward(p, gy, saved, reinterpret_cast<const fdc_c64 *>(K), gx,
                                             gw ? reinterpret_cast<fdc_c64 *>(gK) : nullptr, base + L.layer,
                                             align256(p->bwd_ws), s))
    return st;
  if (gw)
    return check_hip(fdc::launch_cic_wgrad(p->N, gK, part, gw, p->S, p->ksz, p->M, s), "spatial kernel gradient");
  return FDC_OK;
}

// ---------------------------------------------------------------------------
// Stack of CIC + FDP layers
// ---------------------------------------------------------------------------
struct fdc_stack_plan {
  uint32_t magic;
  int B, layers;
  std::vector<int> N, C;  // sizes[0..layers], channels[0..layers]
  size_t ws_a, ws_b, ws_x;  // complex elements: T / Tg buffer, U / V buffer, Xh when `saved` is NULL
  std::vector<size_t> saved;
  int tail;  // first of the two last layers run by the LDS-resident tail kernels, or -1
};

namespace {
// per-layer geometry: planes and bins of the four spectra of layer i
struct StackLayer {
  int N, M, L, C, S;
};
StackLayer stack_layer(const fdc_stack_plan *p, int i) {
  return StackLayer{p->N[i], p->N[i + 1], p->N[i + 1] / 2 + 1, p->C[i], p->C[i + 1]};
}
fdc_status check_stack_plan(const fdc_stack_plan *p) {
  if (!plan_live(p) || p->magic != kStackMagic) return fail(FDC_EINVAL, "invalid or destroyed stack plan");
  return FDC_OK;
}
// The layer where the stack's LDS-resident tail starts (the last two layers, when
// their sizes and fan-outs are an instantiated tail), or -1.  FDC_STACK_TAIL=0 in the
// environment at plan creation keeps every layer on the per-layer kernels.
int stack_tail(int layers, const int *N, const int *C) {
  const char *env = std::getenv("FDC_STACK_TAIL");
  if (env != nullptr && env[0] == '0') return -1;
  if (layers < 2) return -1;
  const int a = layers - 2;
  return fdc::tail_supported(N[a], N[a + 1], N[a + 2], C[a + 1] / C[a], C[a + 2] / C[a + 1]) ? a : -1;
}
}  // namespace

fdc_status fdc_cic_stack_plan_create(fdc_stack_plan **plan, int B, int layers, const int *sizes, const int *channels) {
  if (plan == nullptr) return fail(FDC_EINVAL, "plan out-pointer is NULL");
  *plan = nullptr;
  if (B < 1 || layers < 1) return fail(FDC_EINVAL, "B and layers must be >= 1 (B=%d layers=%d)", B, layers);
  if (!sizes || !channels) return fail(FDC_EINVAL, "sizes or channels is NULL");
  for (int i = 0; i < layers; ++i) {
    const int N = sizes[i], M = sizes[i + 1], C = channels[i], S = channels[i + 1];
    if (C < 1 || S < 1 || S % C) return fail(FDC_EINVAL, "layer %d: channels %d -> %d (need S mod C == 0)", i, C, S);
    if (!even_pos(N) || !even_pos(M) || M > N)
      return fail(FDC_EINVAL, "layer %d: sizes %d -> %d (even, positive, non-increasing)", i, N, M);
    if (!fdc::cic_pair_supported(N, M))
      return fail(FDC_EUNSUPPORTED, "layer %d: size %d -> %d not supported", i, N, M);
    if (!fdc::index_fits((long long)B * C, N) || !fdc::index_fits((long long)B * S, M) ||
        !fdc::index_fits((long long)S * N, N / 2 + 1))
      return fail(FDC_EUNSUPPORTED, "layer %d: B * C * N or B * S * M rows, or the bins of gK, exceed the kernels' "
                  "32-bit indexing", i);
  }
  auto *p = new (std::nothrow) fdc_stack_plan{};
  if (p == nullptr) return fail(FDC_EINVAL, "out of host memory");
  p->magic = kStackMagic;
  p->B = B, p->layers = layers;
  p->N.assign(sizes, sizes + layers + 1);
  p->C.assign(channels, channels + layers + 1);
  for (int i = 0; i < layers; ++i) {
    const StackLayer g = stack_layer(p, i);
    const size_t t = (size_t)B * g.C * g.N * g.L, u = (size_t)B * g.S * g.M * g.L, x = (size_t)B * g.C * g.M * g.L;
    // forward: T (in A) and U (in B); backward: Tg = [B S M L] (in A) and V = [B C N L] (in B)
    p->ws_a = std::max(p->ws_a, std::max(t, u));
    p->ws_b = std::max(p->ws_b, std::max(u, t));
    p->ws_x = std::max(p->ws_x, x);
    p->saved.push_back(x * sizeof(fdc_c64));
  }
  p->tail = stack_tail(layers, sizes, channels);
  if (p->tail >= 0) {
    // the tail keeps both layers' pooled spectra (in Xw when `saved` is NULL) and
    // writes both layers' per-image dK products to the U / V buffer
    const StackLayer ga = stack_layer(p, p->tail), gb = stack_layer(p, p->tail + 1);
    const size_t xa = (size_t)B * ga.C * ga.M * ga.L, xb = (size_t)B * gb.C * gb.M * gb.L;
    const size_t pa = (size_t)B * ga.S * ga.M * ga.L, pb = (size_t)B * gb.S * gb.M * gb.L;
    p->ws_x = std::max(p->ws_x, xa + xb);
    p->ws_b = std::max(p->ws_b, pa + pb);
  }
  if (!plan_register(p)) {
    delete p;
    return fail(FDC_EINVAL, "out of host memory");
  }
  *plan = p;
  return FDC_OK;
}

fdc_status fdc_cic_stack_plan_destroy(fdc_stack_plan *plan) {
  if (plan == nullptr) return FDC_OK;
  if (fdc_status st = check_stack_plan(plan)) return st;
  plan_unregister(plan);
  delete plan;
  return FDC_OK;
}

fdc_status fdc_cic_stack_workspace_size(const fdc_stack_plan *p, size_t *fwd_ws, size_t *bwd_ws) {
  if (fdc_status st = check_stack_plan(p)) return st;
  if (fwd_ws) *fwd_ws = (p->ws_a + p->ws_b + p->ws_x) * sizeof(fdc_c64);
  if (bwd_ws) *bwd_ws = (p->ws_a + p->ws_b) * sizeof(fdc_c64);
  return FDC_OK;
}

fdc_status fdc_cic_stack_saved_size(const fdc_stack_plan *p, int layer, size_t *bytes) {
  if (fdc_status st = check_stack_plan(p)) return st;
  if (layer < 0 || layer >= p->layers) return fail(FDC_EINVAL, "layer %d outside [0, %d)", layer, p->layers);
  if (bytes == nullptr) return fail(FDC_EINVAL, "bytes is NULL");
  *bytes = p->saved[layer];
  return FDC_OK;
}

fdc_status fdc_cic_stack_forward(const fdc_stack_plan *p, const float *x, const fdc_c64 *const *K, float *y,
                                 void *const *saved, void *ws, size_t ws_bytes, hipStream_t s) {
  if (fdc_status st = check_stack_plan(p)) return st;
  if (!x || !K || !y) return fail(FDC_EINVAL, "NULL tensor");
  for (int i = 0; i < p->layers; ++i)
    if (!K[i] || (saved && !saved[i])) return fail(FDC_EINVAL, "layer %d: NULL kernel or saved buffer", i);
  if (fdc_status st = check_ws(ws, ws_bytes, (p->ws_a + p->ws_b + p->ws_x) * sizeof(fdc_c64))) return st;
  const int B = p->B;
  auto *A = reinterpret_cast<float2 *>(ws);
  auto *U = A + p->ws_a;
  auto *Xw = U + p->ws_b;
  for (int i = 0; i < p->layers; ++i) {
    const StackLayer g = stack_layer(p, i);
    const long long cin = (long long)B * g.C, cout = (long long)B * g.S;
    auto *Xh = saved ? reinterpret_cast<float2 *>(saved[i]) : Xw;
    if (i == p->tail) {
      // the last two layers in one launch, from the previous layer's column-inverted
      // spectra in U (or from x when the tail is the whole stack)
      const StackLayer h = stack_layer(p, i + 1);
      auto *Xh2 = saved ? reinterpret_cast<float2 *>(saved[i + 1]) : Xw + (size_t)cin * g.M * g.L;
      fdc::SpecLayout in{};
      float a_in = 1.f;
      if (i > 0) {
        const StackLayer f = stack_layer(p, i - 1);
        in = fdc::tiled_layout(U, (long long)B * f.S, f.M, f.L);
        a_in = 1.f / ((float)f.M * (float)f.M);
      }
      return check_hip(fdc::launch_tail_fwd(g.N, g.M, h.M, g.S / g.C, h.S / h.C, in, i == 0 ? x : nullptr, a_in,
                                            reinterpret_cast<const float2 *>(K[i]),
                                            reinterpret_cast<const float2 *>(K[i + 1]),
                                            fdc::tiled_layout(Xh, cin, g.M, g.L),
                                            fdc::tiled_layout(Xh2, cout, h.M, h.L), y, B, g.C, s),
                       "stack forward tail");
    }
    if (i == 0) {
      ImgView id{0, 0, g.N, g.N};
      if (fdc_status st = check_hip(fdc::launch_row_r2c(g.N, x, fdc::tiled_layout(A, cin, g.N, g.L), cin, g.N, id,
                                                        (long long)g.N * g.N, g.L, 1.f, 1.f, s),
                                    "stack forward rows"))
        return st;
    }
    if (fdc_status st = check_hip(fdc::launch_col_fwd_cic(g.N, g.M, A, reinterpret_cast<const float2 *>(K[i]), U, Xh,
                                                          B, g.C, g.S, s),
                                  "stack forward columns"))
      return st;
    const float inv = 1.f / ((float)g.M * (float)g.M);
    if (i + 1 == p->tail) continue;  // the tail starts from this layer's column-inverted spectra
    if (i + 1 < p->layers) {
      // this layer's inverse rows and the next layer's forward rows on the same rows
      const StackLayer h = stack_layer(p, i + 1);
      if (fdc_status st = check_hip(fdc::launch_row_c2r_r2c(g.M, fdc::tiled_layout(U, cout, g.M, g.L), g.L, inv, 1.f,
                                                            fdc::tiled_layout(A, cout, h.N, h.L), h.L, 1.f, 1.f,
                                                            cout, g.M, s),
                                    "stack forward boundary rows"))
        return st;
    } else {
      ImgView id{0, 0, g.M, g.M};
      if (fdc_status st = check_hip(fdc::launch_row_c2r(g.M, fdc::tiled_layout(U, cout, g.M, g.L), y, cout, g.M, g.L,
                                                        inv, 1.f, id, (long long)g.M * g.M, s),
                                    "stack forward inverse rows"))
        return st;
    }
  }
  return FDC_OK;
}

namespace {
// The stack's backward; kept: gK's dropped bins are left as they are (the caller's
// buffers hold zeros there), only the kept bins are written.
fdc_status stack_backward(const fdc_stack_plan *p, const float *gy, const void *const *saved, const fdc_c64 *const *K,
                          float *gx, fdc_c64 *const *gK, void *ws, size_t ws_bytes, hipStream_t s, bool kept) {
  if (fdc_status st = check_stack_plan(p)) return st;
  if (!gy || !saved || !K || !gK) return fail(FDC_EINVAL, "NULL tensor or array");
  for (int i = 0; i < p->layers; ++i)
    if (!saved[i] || !K[i] || !gK[i]) return fail(FDC_EINVAL, "layer %d: NULL saved, kernel or dK", i);
  if (fdc_status st = check_ws(ws, ws_bytes, (p->ws_a + p->ws_b) * sizeof(fdc_c64))) return st;
  const int B = p->B;
  auto *Tg = reinterpret_cast<float2 *>(ws);
  auto *V = Tg + p->ws_a;
  // Layer i's dK and dX in one launch (k_col_bwd_dk_dx), else dK alone.
  auto dk_merged = [&](int i) {
    const StackLayer g = stack_layer(p, i);
    return (i > 0 || gx) && fdc::gk_batch_ranges(g.N, g.M, B, g.S, (long long)p->ws_b) == 1 &&
           fdc::col_bwd_dk_dx_supported(g.N, g.M);
  };
  // Layer i's gK zeros written by the boundary row launch of layer i + 1 (which runs
  // just before layer i's dK): for a dK launch of one batch range below the tail.
  auto zeros_early = [&](int i) {
    if (kept || i + 1 >= p->layers || (p->tail >= 0 && i + 1 >= p->tail)) return false;
    const StackLayer g = stack_layer(p, i);
    return !dk_merged(i) && fdc::gk_batch_ranges(g.N, g.M, B, g.S, (long long)p->ws_b) == 1;
  };
  for (int i = p->layers - 1; i >= 0; --i) {
    if (p->tail >= 0 && i == p->tail + 1) {
      // the last two layers in one launch: their dK products per image go to V and are
      // summed over the images in order; the output is the previous layer's
      // upstream-gradient row spectrum in Tg (or the input gradient)
      const int a = p->tail;
      const StackLayer ga = stack_layer(p, a), gb = stack_layer(p, a + 1);
      auto *part_a = V, *part_b = V + (size_t)B * ga.S * ga.M * ga.L;
      const int out_mode = a > 0 ? 0 : (gx ? 1 : 2);
      fdc::SpecLayout tg{};
      if (a > 0) {
        const StackLayer f = stack_layer(p, a - 1);
        tg = fdc::tiled_layout(Tg, (long long)B * ga.C, f.M, f.L);
      }
      const float a_out = 1.f / ((float)ga.N * (float)ga.N);
      if (fdc_status st = check_hip(
              fdc::launch_tail_bwd(ga.N, ga.M, gb.M, ga.S / ga.C, gb.S / gb.C, gy,
                                   fdc::tiled_layout(static_cast<const float2 *>(saved[a]), (long long)B * ga.C, ga.M, ga.L),
                                   fdc::tiled_layout(static_cast<const float2 *>(saved[a + 1]), (long long)B * gb.C, gb.M, gb.L),
                                   reinterpret_cast<const float2 *>(K[a]), reinterpret_cast<const float2 *>(K[a + 1]),
                                   part_a, part_b, out_mode, tg, a_out, gx, B, ga.C, s),
              "stack backward tail"))
        return st;
      if (fdc_status st = check_hip(fdc::launch_gk_reduce2(part_a, reinterpret_cast<float2 *>(gK[a]), ga.S, ga.M,
                                                           ga.N, part_b, reinterpret_cast<float2 *>(gK[a + 1]), gb.S,
                                                           gb.M, gb.N, B, s, !kept),
                                    "stack backward tail dK sums"))
        return st;
      i = a;  // continue with layer a - 1
      continue;
    }
    const StackLayer g = stack_layer(p, i);
    const long long cin = (long long)B * g.C, cout = (long long)B * g.S;
    const float inv = 1.f / ((float)g.M * (float)g.M);
    if (i == p->layers - 1) {
      ImgView id{0, 0, g.M, g.M};
      if (fdc_status st = check_hip(fdc::launch_row_r2c(g.M, gy, fdc::tiled_layout(Tg, cout, g.M, g.L), cout, g.M, id,
                                                        (long long)g.M * g.M, g.L, inv, 2.f, s),
                                    "stack backward rows"))
        return st;
    }
    const bool need_dx = i > 0 || gx;
    if (dk_merged(i)) {
      // dK and dX columns side by side in one launch
      if (fdc_status st = check_hip(fdc::launch_col_bwd_dk_dx(g.N, g.M, Tg, reinterpret_cast<const float2 *>(saved[i]),
                                                              reinterpret_cast<const float2 *>(K[i]),
                                                              reinterpret_cast<float2 *>(gK[i]), V, B, g.C, g.S, s,
                                                              !kept),
                                    "stack backward dK and dx columns"))
        return st;
    } else {
      // V is free until the dX columns below: dK's batch-range sums go there
      if (fdc_status st = check_hip(fdc::launch_col_bwd_gk(g.N, g.M, Tg, reinterpret_cast<const float2 *>(saved[i]),
                                                           reinterpret_cast<float2 *>(gK[i]), B, g.C, g.S, V,
                                                           (long long)p->ws_b, s, !kept && !zeros_early(i)),
                                    "stack backward dK"))
        return st;
      if (!need_dx) break;
      if (fdc_status st = check_hip(fdc::launch_col_bwd_gx(g.N, g.M, Tg, reinterpret_cast<const float2 *>(K[i]), V,
                                                           B, g.C, g.S, s),
                                    "stack backward dx columns"))
        return st;
    }
    if (i > 0) {
      // this layer's adjoint inverse rows and the previous layer's upstream-gradient rows
      const StackLayer h = stack_layer(p, i - 1);
      const float hinv = 1.f / ((float)h.M * (float)h.M);
      // with layer i - 1's gK zeros, when its dK launch leaves them to this one
      const fdc::ZeroBins zb = zeros_early(i - 1) ? fdc::ZeroBins{reinterpret_cast<float2 *>(gK[i - 1]), h.S, h.N, h.M}
                                                  : fdc::ZeroBins{nullptr, 0, 0, 0};
      if (fdc_status st = check_hip(fdc::launch_row_c2r_r2c(g.N, fdc::tiled_layout(V, cin, g.N, g.L), g.L, 1.f, 0.5f,
                                                            fdc::tiled_layout(Tg, cin, h.M, h.L), h.L, hinv, 2.f,
                                                            cin, g.N, s, zb),
                                    "stack backward boundary rows"))
        return st;
    } else {
      ImgView id{0, 0, g.N, g.N};
      if (fdc_status st = check_hip(fdc::launch_row_c2r(g.N, fdc::tiled_layout(V, cin, g.N, g.L), gx, cin, g.N, g.L,
                                                        1.f, 0.5f, id, (long long)g.N * g.N, s),
                                    "stack backward dx rows"))
        return st;
    }
  }
  return FDC_OK;
}
}  // namespace

fdc_status fdc_cic_stack_backward(const fdc_stack_plan *p, const float *gy, const void *const *saved,
                                  const fdc_c64 *const *K, float *gx, fdc_c64 *const *gK, void *ws, size_t ws_bytes,
                                  hipStream_t s) {
  return stack_backward(p, gy, saved, K, gx, gK, ws, ws_bytes, s, false);
}

fdc_status fdc_cic_stack_backward_kept(const fdc_stack_plan *p, const float *gy, const void *const *saved,
                                       const fdc_c64 *const *K, float *gx, fdc_c64 *const *gK, void *ws,
                                       size_t ws_bytes, hipStream_t s) {
  return stack_backward(p, gy, saved, K, gx, gK, ws, ws_bytes, s, true);
}

// ---------------------------------------------------------------------------
// Full FDC
// ---------------------------------------------------------------------------
namespace {
struct FullWs {  // byte offsets inside the forward / backward workspaces
  size_t x, y, wf;         // forward: X (when `saved` is NULL), Y, rearranged weights
  size_t g, gx, wg, part;  // backward: G, dL/dX spectrum, rearranged weights, dL/dw partials
};
FullWs full_layout(int B, int Cin, int Cout, int P, int kn, size_t *fwd, size_t *bwd) {
  const size_t xs = (size_t)fdc::full_spec_elems((long long)B * Cin, P) * sizeof(fdc_c64);
  const size_t ys = (size_t)fdc::full_spec_elems((long long)B * Cout, P) * sizeof(fdc_c64);
  FullWs w{};
  w.x = 0;
  w.y = align256(w.x + xs);
  w.wf = align256(w.y + ys);
  *fwd = align256(w.wf + fdc::full_weight_floats(Cin, Cout, kn) * sizeof(float));
  w.g = 0;
  w.gx = align256(w.g + ys);
  w.wg = align256(w.gx + xs);
  w.part = align256(w.wg + fdc::full_weight_floats(Cout, Cin, kn) * sizeof(float));
  *bwd = align256(w.part + (size_t)fdc::full_gw_chunks(B, Cout, Cin, P, kn) * Cout * Cin * kn * kn * sizeof(float));
  return w;
}
}  // namespace

fdc_status fdc_full_layer_plan_create(fdc_layer_plan **plan, int B, int Cin, int Cout, int P, int kernel_n,
                                      int artifact) {
  if (plan == nullptr) return fail(FDC_EINVAL, "plan out-pointer is NULL");
  *plan = nullptr;
  if (B < 1 || Cin < 1 || Cout < 1) return fail(FDC_EINVAL, "B, Cin, Cout must be >= 1 (%d, %d, %d)", B, Cin, Cout);
  if (B > 65535 * 16) return fail(FDC_EUNSUPPORTED, "B = %d exceeds the contraction grid (at most %d)", B, 65535 * 16);
  if (!even_pos(P)) return fail(FDC_EINVAL, "P must be positive and even (got %d)", P);
  if (artifact < FDC_ARTIFACT_NONE || artifact > FDC_ARTIFACT_ROLL) return fail(FDC_EINVAL, "bad artifact mode");
  if (kernel_n < 1 || kernel_n > P) return fail(FDC_EINVAL, "kernel_n must be in [1, P] (got %d)", kernel_n);
  if (!fdc::size_supported(P) || P % 8 != 0)
    return fail(FDC_EUNSUPPORTED, "image size %d not supported (Full FDC needs a multiple of 8 in the FFT set)", P);
  if (!fdc::full_kernel_size_supported(kernel_n))
    return fail(FDC_EUNSUPPORTED, "Full FDC supports kernel_n 1..5 (got %d)", kernel_n);
  if (!fdc::index_fits((long long)B * Cin, P) || !fdc::index_fits((long long)B * Cout, P) ||
      !fdc::full_launch_fits(B, Cin, Cout, P, kernel_n))
    return fail(FDC_EUNSUPPORTED, "B = %d, %d -> %d channels at %d^2 exceed the kernels' grid or row indexing", B,
                Cin, Cout, P);
  auto *p = new (std::nothrow) fdc_layer_plan{};
  if (p == nullptr) return fail(FDC_EINVAL, "out of host memory");
  p->magic = kLayerMagic;
  p->kind = 1;
  p->B = B, p->C = Cin, p->S = Cout, p->N = P, p->M = P;
  p->artifact = artifact;
  p->kn = kernel_n;
  p->out = artifact == FDC_ARTIFACT_CROP ? P - kernel_n + 1 : P;
  full_layout(B, Cin, Cout, P, kernel_n, &p->fwd_ws, &p->bwd_ws);
  p->saved = (size_t)fdc::full_spec_elems((long long)B * Cin, P) * sizeof(fdc_c64);
  std::vector<float2> tw(P);
  for (int j = 0; j < P; ++j) {
    const double ang = -2.0 * 3.14159265358979323846 * (double)j / (double)P;
    tw[j] = make_float2((float)std::cos(ang), (float)std::sin(ang));
  }
  if (hipMalloc(&p->tw, P * sizeof(float2)) != hipSuccess) {
    delete p;
    return fail(FDC_EHIP, "hipMalloc of the %d-entry twiddle table failed", P);
  }
  if (hipMemcpy(p->tw, tw.data(), P * sizeof(float2), hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipFree(p->tw);
    delete p;
    return fail(FDC_EHIP, "copy of the twiddle table failed");
  }
  if (!plan_register(p)) {
    (void)hipFree(p->tw);
    delete p;
    return fail(FDC_EINVAL, "out of host memory");
  }
  *plan = p;
  return FDC_OK;
}

fdc_status fdc_full_forward(const fdc_layer_plan *p, const float *x, const float *w, float *y, void *saved, void *ws,
                            size_t ws_bytes, hipStream_t s) {
  if (fdc_status st = check_layer_plan(p, 1)) return st;
  if (!x || !w || !y) return fail(FDC_EINVAL, "NULL tensor");
  if (fdc_status st = check_ws(ws, ws_bytes, p->fwd_ws)) return st;
  const int B = p->B, Cin = p->C, Cout = p->S, P = p->N, Pf = P / 2 + 1;
  size_t fwd, bwd;
  const FullWs L = full_layout(B, Cin, Cout, P, p->kn, &fwd, &bwd);
  char *base = static_cast<char *>(ws);
  auto *X = saved != nullptr ? static_cast<float2 *>(saved) : reinterpret_cast<float2 *>(base + L.x);
  auto *Y = reinterpret_cast<float2 *>(base + L.y);
  auto *wf = reinterpret_cast<float *>(base + L.wf);
  const long long Xp = (long long)B * Cin, Yp = (long long)B * Cout;
  const fdc::SpecLayout XL = fdc::full_spec_layout(X, Xp, P), YL = fdc::full_spec_layout(Y, Yp, P);
  ImgView id{0, 0, P, P};
  if (fdc_status st = check_hip(fdc::launch_row_r2c(P, x, XL, Xp, P, id, (long long)P * P, Pf, 1.f, 1.f, s),
                                "full forward rows"))
    return st;
  if (fdc_status st = check_hip(fdc::launch_col_fft_split(P, -1, XL, XL, Xp, s), "full forward columns")) return st;
  if (fdc_status st = check_hip(fdc::launch_full_weights(w, wf, false, Cout, Cin, p->kn, s), "full weights"))
    return st;
  if (fdc_status st = check_hip(fdc::launch_full_contract(false, p->kn, XL, wf, p->tw, YL, B, Cin, Cout, P, s),
                                "full forward contraction"))
    return st;
  if (fdc_status st = check_hip(fdc::launch_col_fft_split(P, +1, YL, YL, Yp, s), "full forward inverse columns"))
    return st;
  return check_hip(fdc::launch_row_c2r(P, YL, y, Yp, P, Pf, 1.f / ((float)P * (float)P), 1.f, artifact_view(p),
                                       (long long)p->out * p->out, s),
                   "full forward inverse rows");
}

fdc_status fdc_full_backward(const fdc_layer_plan *p, const float *gy, const void *saved, const float *w, float *gx,
                             float *gw, void *ws, size_t ws_bytes, hipStream_t s) {
  if (fdc_status st = check_layer_plan(p, 1)) return st;
  if (!gy) return fail(FDC_EINVAL, "gy is NULL");
  if (gx && !w) return fail(FDC_EINVAL, "w is NULL but gx was requested");
  if (gw && !saved) return fail(FDC_EINVAL, "saved is NULL but gw was requested");
  if (!gx && !gw) return FDC_OK;
  if (fdc_status st = check_ws(ws, ws_bytes, p->bwd_ws)) return st;
  const int B = p->B, Cin = p->C, Cout = p->S, P = p->N, Pf = P / 2 + 1;
  size_t fwd, bwd;
  const FullWs L = full_layout(B, Cin, Cout, P, p->kn, &fwd, &bwd);
  char *base = static_cast<char *>(ws);
  auto *G = reinterpret_cast<float2 *>(base + L.g);
  auto *gX = reinterpret_cast<float2 *>(base + L.gx);
  auto *wg = reinterpret_cast<float *>(base + L.wg);
  auto *part = reinterpret_cast<float *>(base + L.part);
  const long long Xp = (long long)B * Cin, Gp = (long long)B * Cout;
  const fdc::SpecLayout GL = fdc::full_spec_layout(G, Gp, P), gXL = fdc::full_spec_layout(gX, Xp, P);
  // G = adjoint of the inverse transform and the artifact step: (c_l / P^2) rfft2 of gy placed in P x P
  if (fdc_status st = check_hip(fdc::launch_row_r2c(P, gy, GL, Gp, P, artifact_view(p), (long long)p->out * p->out,
                                                    Pf, 1.f / ((float)P * (float)P), 2.f, s),
                                "full backward rows"))
    return st;
  if (fdc_status st = check_hip(fdc::launch_col_fft_split(P, -1, GL, GL, Gp, s), "full backward columns")) return st;
  if (gw) {
    const fdc::SpecLayout XL = fdc::full_spec_layout(static_cast<const float2 *>(saved), Xp, P);
    if (fdc_status st = check_hip(fdc::launch_full_gw(p->kn, GL, XL, p->tw, part, gw, B, Cout, Cin, P, s),
                                  "full backward dw"))
      return st;
  }
  if (gx) {
    if (fdc_status st = check_hip(fdc::launch_full_weights(w, wg, true, Cout, Cin, p->kn, s), "full weights"))
      return st;
    if (fdc_status st = check_hip(fdc::launch_full_contract(true, p->kn, GL, wg, p->tw, gXL, B, Cout, Cin, P, s),
                                  "full backward dx contraction"))
      return st;
    // rfft2 adjoint: P^2 irfft2(gX / c_l)
    if (fdc_status st = check_hip(fdc::launch_col_fft_split(P, +1, gXL, gXL, Xp, s), "full backward dx columns"))
      return st;
    ImgView id{0, 0, P, P};
    return check_hip(fdc::launch_row_c2r(P, gXL, gx, Xp, P, Pf, 1.f, 0.5f, id, (long long)P * P, s),
                     "full backward dx rows");
  }
  return FDC_OK;
}

// ---------------------------------------------------------------------------
// FDCNN classifier head and Adam
// ---------------------------------------------------------------------------
static fdc_status check_head(int B, int64_t F, int classes) {
  if (B < 1 || F < 1) return fail(FDC_EINVAL, "B and F must be positive (got %d, %lld)", B, (long long)F);
  if (classes < 1 || classes > fdc::kHeadMaxClasses)
    return fail(FDC_EUNSUPPORTED, "classes must be in [1, %d] (got %d)", fdc::kHeadMaxClasses, classes);
  if ((long long)B * classes > fdc::kHeadMaxPairs)
    return fail(FDC_EUNSUPPORTED, "B * classes = %lld exceeds the head's LDS (%d)", (long long)B * classes,
                fdc::kHeadMaxPairs);
  if ((long long)B * F >= (1LL << 40) || F >= (1LL << 38)) return fail(FDC_EUNSUPPORTED, "B * F or F too large");
  return FDC_OK;
}

fdc_status fdc_head_workspace_size(int B, int64_t F, int classes, size_t *bytes) {
  if (fdc_status st = check_head(B, F, classes)) return st;
  if (!bytes) return fail(FDC_EINVAL, "bytes is NULL");
  *bytes = (size_t)fdc::head_chunks(F) * B * classes * sizeof(float);
  return FDC_OK;
}

fdc_status fdc_head_forward(const float *y, const float *W, const float *bias, const int32_t *labels, float *logits,
                            float *loss, int B, int64_t F, int classes, void *ws, size_t ws_bytes, hipStream_t s) {
  size_t need = 0;
  if (fdc_status st = fdc_head_workspace_size(B, F, classes, &need)) return st;
  if (!y || !W || !bias || !labels || !logits || !loss) return fail(FDC_EINVAL, "NULL tensor");
  if (!ws || ws_bytes < need) return fail(FDC_EWORKSPACE, "head workspace: need %zu bytes, got %zu", need, ws_bytes);
  return check_hip(fdc::launch_head_forward(y, W, bias, labels, logits, loss, static_cast<float *>(ws), B, F, classes,
                                            s),
                   "head forward");
}

fdc_status fdc_head_forward_noalloc(const float *y, const float *W, const float *bias, const int32_t *labels,
                                    float *logits, float *loss, int B, int64_t F, int classes, hipStream_t s) {
  if (fdc_status st = check_head(B, F, classes)) return st;
  if (!y || !W || !bias || !labels || !logits || !loss) return fail(FDC_EINVAL, "NULL tensor");
  const long long need = fdc::head_chunks(F) * B * classes;
  if (need > fdc::kHeadScratchFloats)
    return fail(FDC_EUNSUPPORTED,
                "head_forward_noalloc: ceil(F / 1024) * B * classes = %lld partial logits exceed the library's "
                "static scratch of %lld floats; use fdc_head_forward with a workspace",
                need, (long long)fdc::kHeadScratchFloats);
  return check_hip(fdc::launch_head_forward_noalloc(y, W, bias, labels, logits, loss, B, F, classes, s),
                   "head forward (static scratch)");
}

fdc_status fdc_head_backward(const float *y, const float *W, const float *logits, const int32_t *labels, float *gy,
                             float *gW, float *gbias, int B, int64_t F, int classes, hipStream_t s) {
  if (fdc_status st = check_head(B, F, classes)) return st;
  if (!y || !W || !logits || !labels || !gW || !gbias) return fail(FDC_EINVAL, "NULL tensor");
  return check_hip(fdc::launch_head_backward(y, W, logits, labels, gy, gW, gbias, B, F, classes, s), "head backward");
}

fdc_status fdc_adam_step(float *p, const float *g, float *m, float *v, int64_t n, int32_t *step_count, float lr,
                         float beta1, float beta2, float eps, float weight_decay, hipStream_t s) {
  if (n < 0) return fail(FDC_EINVAL, "n must be >= 0 (got %lld)", (long long)n);
  if (n > 0 && (!p || !g || !m || !v)) return fail(FDC_EINVAL, "NULL tensor");
  if (!step_count) return fail(FDC_EINVAL, "step_count is NULL");
  if (!(beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f))
    return fail(FDC_EINVAL, "betas must be in [0, 1) (got %g, %g)", (double)beta1, (double)beta2);
  return check_hip(fdc::launch_adam(p, g, m, v, n, step_count, lr, beta1, beta2, eps, weight_decay, s), "adam");
}

// ---------------------------------------------------------------------------
// kernel timing
// ---------------------------------------------------------------------------
fdc_status fdc_kernel_timing_enable(int max_launches, const char *only_kernel) {
  if (max_launches < 1) return fail(FDC_EINVAL, "max_launches must be >= 1");
  Timing &t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  timing_release(t);
  t.start.resize(max_launches);
  t.stop.resize(max_launches);
  t.names.assign(max_launches, nullptr);
  for (int i = 0; i < max_launches; ++i) {
    if (hipEventCreate(&t.start[i]) != hipSuccess || hipEventCreate(&t.stop[i]) != hipSuccess) {
      t.start.resize(i);
      t.stop.resize(i);
      timing_release(t);
      return fail(FDC_EHIP, "hipEventCreate failed");
    }
  }
  t.max = max_launches;
  t.used = 0;
  t.only = only_kernel ? only_kernel : "";
  t.enabled = true;
  return FDC_OK;
}

fdc_status fdc_kernel_timing_disable(void) {
  Timing &t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  t.enabled = false;
  return FDC_OK;
}

fdc_status fdc_kernel_timing_report(char *buf, size_t buf_bytes) {
  if (buf == nullptr || buf_bytes == 0) return fail(FDC_EINVAL, "buffer is NULL or empty");
  Timing &t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  std::map<std::string, std::pair<int, double>> acc;
  for (int i = 0; i < t.used; ++i) {
    if (hipEventSynchronize(t.stop[i]) != hipSuccess) return fail(FDC_EHIP, "hipEventSynchronize failed");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, t.start[i], t.stop[i]) != hipSuccess)
      return fail(FDC_EHIP, "hipEventElapsedTime failed");
    auto &e = acc[t.names[i]];
    e.first += 1;
    e.second += ms;
  }
  std::string out;
  for (auto &kv : acc) {
    char line[256];
    snprintf(line, sizeof line, "%s %d %.6f\n", kv.first.c_str(), kv.second.first, kv.second.second);
    out += line;
  }
  if (out.size() + 1 > buf_bytes) return fail(FDC_EINVAL, "report needs %zu bytes", out.size() + 1);
  memcpy(buf, out.c_str(), out.size() + 1);
  return FDC_OK;
}

fdc_status fdc_cic_layer_dk_ranges(const fdc_layer_plan *p, int *ranges) {
  if (fdc_status st = check_layer_plan(p, 0)) return st;
  if (ranges == nullptr) return fail(FDC_EINVAL, "ranges is NULL");
  // the same scratch as fdc_cic_layer_backward: the dX buffer
  *ranges = fdc::gk_batch_ranges(p->N, p->M, p->B, p->S, (long long)p->B * p->C * p->N * (p->M / 2 + 1));
  return FDC_OK;
}

fdc_status fdc_cic_stack_tail(const fdc_stack_plan *p, int *first_layer) {
  if (fdc_status st = check_stack_plan(p)) return st;
  if (first_layer == nullptr) return fail(FDC_EINVAL, "first_layer is NULL");
  *first_layer = p->tail;
  return FDC_OK;
}

fdc_status fdc_cic_stack_dk_ranges(const fdc_stack_plan *p, int layer, int *ranges) {
  if (fdc_status st = check_stack_plan(p)) return st;
  if (layer < 0 || layer >= p->layers) return fail(FDC_EINVAL, "layer %d outside [0, %d)", layer, p->layers);
  if (ranges == nullptr) return fail(FDC_EINVAL, "ranges is NULL");
  const StackLayer g = stack_layer(p, layer);
  // the same scratch as fdc_cic_stack_backward: the dX buffer
  *ranges = fdc::gk_batch_ranges(g.N, g.M, p->B, g.S, (long long)p->ws_b);
  return FDC_OK;
}

// ---------------------------------------------------------------------------
// Stack with spatial kernels: the kernel spectra of every layer (with the ROLL shift
// folded in as a phase) in one launch, the stack executor on them, and dL/dw of every
// layer from the executor's dK in one launch (plus the in-order sum of its partials).
// ---------------------------------------------------------------------------
namespace {
struct SpatialStackWs {
  std::vector<size_t> k, gk, part;  // byte offsets per layer
  size_t stack_fwd, stack_bwd, fwd, bwd;
};
SpatialStackWs spatial_stack_layout(const fdc_stack_plan *p, int n) {
  SpatialStackWs w;
  size_t off = 0;
  for (int i = 0; i < p->layers; ++i) {
    const StackLayer g = stack_layer(p, i);
    w.k.push_back(off);
    off += align256((size_t)g.S * g.N * (g.N / 2 + 1) * sizeof(fdc_c64));
  }
  w.stack_fwd = off;
  w.fwd = off + align256((p->ws_a + p->ws_b + p->ws_x) * sizeof(fdc_c64));
  for (int i = 0; i < p->layers; ++i) {
    const StackLayer g = stack_layer(p, i);
    w.gk.push_back(off);
    off += align256((size_t)g.S * g.N * (g.N / 2 + 1) * sizeof(fdc_c64));
  }
  for (int i = 0; i < p->layers; ++i) {
    const StackLayer g = stack_layer(p, i);
    w.part.push_back(off);
    off += align256((size_t)g.S * fdc::cic_wgrad_stack_blocks(g.M) * n * n * sizeof(float));
  }
  w.stack_bwd = off;
  w.bwd = off + align256((p->ws_a + p->ws_b) * sizeof(fdc_c64));
  return w;
}
fdc_status check_spatial_stack(const fdc_stack_plan *p, int n) {
  if (fdc_status st = check_stack_plan(p)) return st;
  if (!fdc::spatial_kernel_size_supported(n)) return fail(FDC_EUNSUPPORTED, "kernel_n must be in [1, 8] (got %d)", n);
  for (int i = 0; i < p->layers; ++i)
    if (n > p->N[i + 1]) return fail(FDC_EINVAL, "kernel_n %d larger than layer %d's output %d", n, i, p->N[i + 1]);
  return FDC_OK;
}
// kernel spectra of every layer into the workspace (batches of fdc::kSpatialBatch layers)
fdc_status spatial_stack_kspec(const fdc_stack_plan *p, int n, const float *const *w, char *base,
                               const SpatialStackWs &L, std::vector<const fdc_c64 *> &K, hipStream_t s) {
  K.assign(p->layers, nullptr);
  for (int i0 = 0; i0 < p->layers; i0 += fdc::kSpatialBatch) {
    fdc::SpatialBatch sb{};
    for (int i = i0; i < p->layers && i < i0 + fdc::kSpatialBatch; ++i) {
      const StackLayer g = stack_layer(p, i);
      auto *Ki = reinterpret_cast<float2 *>(base + L.k[i]);
      K[i] = reinterpret_cast<const fdc_c64 *>(Ki);
      fdc::SpatialLayer &d = sb.layer[sb.count++];
      d.w = w[i], d.K = Ki, d.N = g.N, d.M = g.M, d.S = g.S, d.n = n, d.roll = (n - 1) / 2;
    }
    if (fdc_status st = check_hip(fdc::launch_cic_kspec_stack(sb, s), "spatial stack kernel spectra")) return st;
  }
  return FDC_OK;
}
}  // namespace

fdc_status fdc_cic_spatial_stack_workspace_size(const fdc_stack_plan *p, int kernel_n, size_t *fwd_ws,
                                                size_t *bwd_ws) {
  if (fdc_status st = check_spatial_stack(p, kernel_n)) return st;
  const SpatialStackWs L = spatial_stack_layout(p, kernel_n);
  if (fwd_ws) *fwd_ws = L.fwd;
  if (bwd_ws) *bwd_ws = L.bwd;
  return FDC_OK;
}

fdc_status fdc_cic_spatial_stack_forward(const fdc_stack_plan *p, int kernel_n, const float *x, const float *const *w,
                                         float *y, void *const *saved, void *ws, size_t ws_bytes, hipStream_t s) {
  if (fdc_status st = check_spatial_stack(p, kernel_n)) return st;
  if (!x || !w || !y) return fail(FDC_EINVAL, "NULL tensor or array");
  for (int i = 0; i < p->layers; ++i)
    if (!w[i] || (saved && !saved[i])) return fail(FDC_EINVAL, "layer %d: NULL weights or saved buffer", i);
  const SpatialStackWs L = spatial_stack_layout(p, kernel_n);
  if (fdc_status st = check_ws(ws, ws_bytes, L.fwd)) return st;
  char *base = static_cast<char *>(ws);
  std::vector<const fdc_c64 *> K;
  if (fdc_status st = spatial_stack_kspec(p, kernel_n, w, base, L, K, s)) return st;
  return fdc_cic_stack_forward(p, x, K.data(), y, saved, base + L.stack_fwd, L.fwd - L.stack_fwd, s);
}

fdc_status fdc_cic_spatial_stack_backward(const fdc_stack_plan *p, int kernel_n, const float *gy,
                                          const void *const *saved, const float *const *w, float *gx,
                                          float *const *gw, void *ws, size_t ws_bytes, hipStream_t s) {
  if (fdc_status st = check_spatial_stack(p, kernel_n)) return st;
  if (!gy || !saved || !w || !gw) return fail(FDC_EINVAL, "NULL tensor or array");
  for (int i = 0; i < p->layers; ++i)
    if (!saved[i] || !w[i] || !gw[i]) return fail(FDC_EINVAL, "layer %d: NULL saved, weights or dL/dw", i);
  const SpatialStackWs L = spatial_stack_layout(p, kernel_n);
  if (fdc_status st = check_ws(ws, ws_bytes, L.bwd)) return st;
  char *base = static_cast<char *>(ws);
  std::vector<const fdc_c64 *> K;
  if (fdc_status st = spatial_stack_kspec(p, kernel_n, w, base, L, K, s)) return st;
  std::vector<fdc_c64 *> gK(p->layers);
  for (int i = 0; i < p->layers; ++i) gK[i] = reinterpret_cast<fdc_c64 *>(base + L.gk[i]);
  if (fdc_status st = fdc_cic_stack_backward(p, gy, saved, K.data(), gx, gK.data(), base + L.stack_bwd,
                                             L.bwd - L.stack_bwd, s))
    return st;
  for (int i0 = 0; i0 < p->layers; i0 += fdc::kSpatialBatch) {
    fdc::SpatialBatch sb{};
    for (int i = i0; i < p->layers && i < i0 + fdc::kSpatialBatch; ++i) {
      const StackLayer g = stack_layer(p, i);
      fdc::SpatialLayer &d = sb.layer[sb.count++];
      d.gK = reinterpret_cast<const float2 *>(gK[i]);
      d.part = reinterpret_cast<float *>(base + L.part[i]);
      d.gw = gw[i];
      d.N = g.N, d.M = g.M, d.S = g.S, d.n = kernel_n, d.roll = (kernel_n - 1) / 2;
    }
    if (fdc_status st = check_hip(fdc::launch_cic_wgrad_stack(sb, s), "spatial stack kernel gradients")) return st;
  }
  return FDC_OK;
}

fdc_status fdc_kernel_timing_launches(char *buf, size_t buf_bytes) {
  if (buf == nullptr || buf_bytes == 0) return fail(FDC_EINVAL, "buffer is NULL or empty");
  Timing &t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  std::string out;
  for (int i = 0; i < t.used; ++i) {
    if (hipEventSynchronize(t.stop[i]) != hipSuccess) return fail(FDC_EHIP, "hipEventSynchronize failed");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, t.start[i], t.stop[i]) != hipSuccess)
      return fail(FDC_EHIP, "hipEventElapsedTime failed");
    char line[256];
    snprintf(line, sizeof line, "%s %.6f\n", t.names[i], ms);
    out += line;
  }
  if (out.size() + 1 > buf_bytes) return fail(FDC_EINVAL, "report needs %zu bytes", out.size() + 1);
  memcpy(buf, out.c_str(), out.size() + 1);
  return FDC_OK;
}

}  // extern "C"
