// C ABI of liboq: argument validation, workspace carving, the launch sequence
// of one calibration step and the optional per-kernel event timing.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <mutex>
#include <string>
#include <vector>

#include "oq.h"
#include "oq_internal.h"
#include "packed.h"

namespace {

thread_local std::string g_err;

oq_status fail(oq_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define OQ_HIP(expr, what)                                                            \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess) return fail(OQ_ERR_HIP, "%s: %s", what, hipGetErrorString(e_)); \
  } while (0)

#define OQ_REQ(cond, ...)                                    \
  do {                                                       \
    if (!(cond)) return fail(OQ_ERR_INVALID_ARG, __VA_ARGS__); \
  } while (0)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool dtype_ok(oq_dtype d) { return d == OQ_F32 || d == OQ_BF16; }
size_t esize(oq_dtype d) { return d == OQ_BF16 ? 2 : 4; }

// ------------------------------------------------------------------ profiling
struct ProfRec {
  int kind;
  hipEvent_t e0, e1;
  double work;
};
std::mutex g_pm;
std::vector<ProfRec> g_pending;
bool g_prof_on = false;
struct ProfAcc {
  int64_t n = 0;
  double ms = 0, work = 0;
} g_acc[OQ_PROF_KINDS];

void drain_pending() {
  for (auto& r : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(r.e1) == hipSuccess && hipEventElapsedTime(&ms, r.e0, r.e1) == hipSuccess) {
      g_acc[r.kind].n += 1;
      g_acc[r.kind].ms += ms;
      g_acc[r.kind].work += r.work;
    }
    (void)hipEventDestroy(r.e0);
    (void)hipEventDestroy(r.e1);
  }
  g_pending.clear();
}

// ------------------------------------------------------------------ workspace carving
struct Carver {
  char* base;
  size_t off = 0;
  template <class T>
  T* take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

}  // namespace

namespace oq {
ProfScope::ProfScope(int k, hipStream_t s, double w) : kind(k), stream(s), work(w), on(g_prof_on) {
  if (on) {
    on = hipEventCreate(&e0) == hipSuccess && hipEventCreate(&e1) == hipSuccess &&
         hipEventRecord(e0, s) == hipSuccess;
  }
}
ProfScope::~ProfScope() {
  if (!on) return;
  (void)hipEventRecord(e1, stream);
  std::lock_guard<std::mutex> lk(g_pm);
  g_pending.push_back({kind, e0, e1, work});
}
}  // namespace oq

using namespace oq;

extern "C" {

const char* oq_status_str(oq_status s) {
  switch (s) {
    case OQ_OK: return "OQ_OK";
    case OQ_ERR_INVALID_ARG: return "OQ_ERR_INVALID_ARG";
    case OQ_ERR_UNSUPPORTED: return "OQ_ERR_UNSUPPORTED";
    case OQ_ERR_WORKSPACE: return "OQ_ERR_WORKSPACE";
    case OQ_ERR_HIP: return "OQ_ERR_HIP";
  }
  return "OQ_ERR_UNKNOWN";
}

const char* oq_last_error(void) { return g_err.c_str(); }
int oq_version(void) { return 1; }

oq_status oq_profile_enable(int on) {
  std::lock_guard<std::mutex> lk(g_pm);
  g_prof_on = on != 0;
  return OQ_OK;
}

oq_status oq_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_pm);
  drain_pending();
  for (auto& a : g_acc) a = ProfAcc{};
  return OQ_OK;
}

oq_status oq_profile_read(int kind, int64_t* launches, double* total_ms, double* work) {
  if (kind < 0 || kind >= OQ_PROF_KINDS) return fail(OQ_ERR_INVALID_ARG, "profile kind %d", kind);
  std::lock_guard<std::mutex> lk(g_pm);
  drain_pending();
  if (launches) *launches = g_acc[kind].n;
  if (total_ms) *total_ms = g_acc[kind].ms;
  if (work) *work = g_acc[kind].work;
  return OQ_OK;
}

// ------------------------------------------------------------------ quantisers
static oq_status check_lwc(const void* W, oq_dtype w_dt, int64_t c_out, int64_t c_in,
                           const float* gl, const float* bl, int bits, int64_t group) {
  OQ_REQ(W && gl && bl, "W, gamma_logit and beta_logit are required");
  OQ_REQ(dtype_ok(w_dt), "bad weight dtype %d", int(w_dt));
  OQ_REQ(c_out >= 0 && c_in > 0, "bad shape c_out=%lld c_in=%lld", (long long)c_out, (long long)c_in);
  OQ_REQ(c_in % 8 == 0, "c_in=%lld must be a multiple of 8", (long long)c_in);
  OQ_REQ(aligned16(W), "W must be 16-byte aligned");
  if (bits < 2 || bits > 8) return fail(OQ_ERR_UNSUPPORTED, "bits=%d outside [2, 8]", bits);
  if (group <= 0 || c_in % group)
    return fail(OQ_ERR_INVALID_ARG, "group=%lld must divide c_in=%lld", (long long)group, (long long)c_in);
  if (!quant_shape_supported(c_in, group))
    return fail(OQ_ERR_UNSUPPORTED,
                "group=%lld with c_in=%lld: need a power of two in [8, 512] or group == c_in "
                "(c_in <= 32768)",
                (long long)group, (long long)c_in);
  return OQ_OK;
}

static oq_status wquant_fwd(int quant, const void* W, oq_dtype w_dt, int64_t c_out, int64_t c_in,
                            const float* s, const float* gamma_logit, const float* beta_logit,
                            int bits, int64_t group, void* W_dq, oq_dtype dq_dt, uint8_t* codes,
                            float* h, float* z, hipStream_t stream);
static oq_status wquant_bwd(int quant, const void* W, oq_dtype w_dt, int64_t c_out, int64_t c_in,
                            const float* s, const float* gamma_logit, const float* beta_logit,
                            int bits, int64_t group, const float* dW_dq, float* d_gamma_logit,
                            float* d_beta_logit, float* d_s, float* dW_tilde, void* ws,
                            size_t ws_bytes, hipStream_t stream);

oq_status oq_lwc_fakequant_fwd(const void* W, oq_dtype w_dt, int64_t c_out, int64_t c_in,
                               const float* s, const float* gamma_logit, const float* beta_logit,
                               int bits, int64_t group, void* W_dq, oq_dtype dq_dt,
                               uint8_t* codes, float* h, float* z, hipStream_t stream) {
  return wquant_fwd(OQ_WQ_LWC, W, w_dt, c_out, c_in, s, gamma_logit, beta_logit, bits, group, W_dq,
                    dq_dt, codes, h, z, stream);
}

oq_status oq_wquant_fakequant_fwd(int quantizer, const void* W, oq_dtype w_dt, int64_t c_out,
                                  int64_t c_in, const float* s, const float* p1, const float* p2,
                                  int bits, int64_t group, void* W_dq, oq_dtype dq_dt,
                                  uint8_t* codes, float* h, float* z, hipStream_t stream) {
  return wquant_fwd(quantizer, W, w_dt, c_out, c_in, s, p1, p2, bits, group, W_dq, dq_dt, codes, h,
                    z, stream);
}

static oq_status wquant_fwd(int quant, const void* W, oq_dtype w_dt, int64_t c_out, int64_t c_in,
                            const float* s, const float* gamma_logit, const float* beta_logit,
                            int bits, int64_t group, void* W_dq, oq_dtype dq_dt, uint8_t* codes,
                            float* h, float* z, hipStream_t stream) {
  OQ_REQ(quant >= OQ_WQ_LWC && quant <= OQ_WQ_LSQ, "quantizer=%d", quant);
  oq_status e = check_lwc(W, w_dt, c_out, c_in, gamma_logit, beta_logit, bits, group);
  if (e != OQ_OK) return e;
  OQ_REQ(!W_dq || dtype_ok(dq_dt), "bad W_dq dtype");
  OQ_REQ(!W_dq || aligned16(W_dq), "W_dq must be 16-byte aligned");
  OQ_REQ(!codes || (reinterpret_cast<uintptr_t>(codes) & 7u) == 0, "codes must be 8-byte aligned");
  OQ_REQ(!s || aligned16(s), "s must be 16-byte aligned");
  ProfScope ps(PK_LWC_FWD, stream,
               double(c_out) * c_in * (esize(w_dt) + (W_dq ? esize(dq_dt) : 0) + (codes ? 1 : 0)));
  OQ_HIP(lwc_fwd(W, w_dt == OQ_BF16, c_out, c_in, s, gamma_logit, beta_logit, bits, group, W_dq,
                 dq_dt == OQ_BF16, codes, h, z, stream, nullptr, quant),
         "lwc_fwd");
  return OQ_OK;
}

oq_status oq_lwc_fakequant_bwd_workspace_size(int64_t c_out, int64_t c_in, int64_t group,
                                              int want_d_s, size_t* bytes) {
  (void)group;
  OQ_REQ(bytes, "bytes is required");
  *bytes = want_d_s ? size_t(lwc_bwd_nparts(c_out)) * size_t(c_in) * 4 + 256 : 0;
  return OQ_OK;
}

oq_status oq_lwc_fakequant_bwd(const void* W, oq_dtype w_dt, int64_t c_out, int64_t c_in,
                               const float* s, const float* gamma_logit, const float* beta_logit,
                               int bits, int64_t group, const float* dW_dq,
                               float* d_gamma_logit, float* d_beta_logit, float* d_s,
                               float* dW_tilde, void* ws, size_t ws_bytes, hipStream_t stream) {
  return wquant_bwd(OQ_WQ_LWC, W, w_dt, c_out, c_in, s, gamma_logit, beta_logit, bits, group, dW_dq,
                    d_gamma_logit, d_beta_logit, d_s, dW_tilde, ws, ws_bytes, stream);
}

oq_status oq_wquant_fakequant_bwd(int quantizer, const void* W, oq_dtype w_dt, int64_t c_out,
                                  int64_t c_in, const float* s, const float* p1, const float* p2,
                                  int bits, int64_t group, const float* dW_dq, float* d_p1,
                                  float* d_p2, float* d_s, float* dW_tilde, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
  return wquant_bwd(quantizer, W, w_dt, c_out, c_in, s, p1, p2, bits, group, dW_dq, d_p1, d_p2,
                    d_s, dW_tilde, ws, ws_bytes, stream);
}

oq_status oq_wquant_init(int quantizer, const void* W, oq_dtype w_dt, int64_t c_out, int64_t c_in,
                         const float* s, int bits, int64_t group, float* p1, float* p2,
                         hipStream_t stream) {
  OQ_REQ(quantizer >= OQ_WQ_LWC && quantizer <= OQ_WQ_LSQ, "quantizer=%d", quantizer);
  OQ_REQ(p1 && p2, "p1 and p2 are required");
  oq_status e = check_lwc(W, w_dt, c_out, c_in, p1, p2, bits, group);
  if (e != OQ_OK) return e;
  OQ_REQ(!s || aligned16(s), "s must be 16-byte aligned");
  ProfScope ps(PK_OTHER, stream, double(c_out) * c_in * esize(w_dt));
  OQ_HIP(wquant_init(W, w_dt == OQ_BF16, c_out, c_in, s, bits, group, quantizer, p1, p2, stream),
         "wquant_init");
  return OQ_OK;
}

static oq_status wquant_bwd(int quant, const void* W, oq_dtype w_dt, int64_t c_out, int64_t c_in,
                            const float* s, const float* gamma_logit, const float* beta_logit,
                            int bits, int64_t group, const float* dW_dq, float* d_gamma_logit,
                            float* d_beta_logit, float* d_s, float* dW_tilde, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
  OQ_REQ(quant >= OQ_WQ_LWC && quant <= OQ_WQ_LSQ, "quantizer=%d", quant);
  oq_status e = check_lwc(W, w_dt, c_out, c_in, gamma_logit, beta_logit, bits, group);
  if (e != OQ_OK) return e;
  OQ_REQ(dW_dq && d_gamma_logit && d_beta_logit, "dW_dq, d_gamma_logit, d_beta_logit are required");
  OQ_REQ(aligned16(dW_dq) && (!dW_tilde || aligned16(dW_tilde)), "dW_dq/dW_tilde must be 16-byte aligned");
  size_t need = 0;
  oq_lwc_fakequant_bwd_workspace_size(c_out, c_in, group, d_s != nullptr, &need);
  if (need && (!ws || ws_bytes < need))
    return fail(OQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws_bytes);
  Carver cv{static_cast<char*>(ws)};
  float* parts = d_s ? cv.take<float>(size_t(lwc_bwd_nparts(c_out)) * c_in) : nullptr;
  {
    ProfScope ps(PK_LWC_BWD, stream, double(c_out) * c_in * (esize(w_dt) + 4 + (dW_tilde ? 4 : 0)));
    OQ_HIP(lwc_bwd(W, w_dt == OQ_BF16, c_out, c_in, s, gamma_logit, beta_logit, bits, group, dW_dq,
                   d_gamma_logit, d_beta_logit, dW_tilde, parts, stream, 1, 0, quant),
           "lwc_bwd");
  }
  if (d_s) {
    ProfScope ps(PK_OTHER, stream, 0);
    OQ_HIP(let_grad_finish(c_in, nullptr, parts, lwc_bwd_nparts(c_out), nullptr, nullptr, 0,
                           nullptr, 0, d_s, nullptr, stream),
           "ds finish");
  }
  return OQ_OK;
}

oq_status oq_let_fold(const void* W, oq_dtype w_dt, const float* B, int64_t c_out, int64_t c_in,
                      const float* s, const float* delta, void* W_tilde, oq_dtype wt_dt,
                      float* B_tilde, hipStream_t stream) {
  OQ_REQ(W, "W is required");
  OQ_REQ(dtype_ok(w_dt) && (!W_tilde || dtype_ok(wt_dt)), "bad dtype");
  OQ_REQ(c_out >= 0 && c_in > 0 && c_in % 8 == 0, "bad shape");
  OQ_REQ(aligned16(W) && (!W_tilde || aligned16(W_tilde)) && (!s || aligned16(s)) &&
             (!delta || aligned16(delta)),
         "pointers must be 16-byte aligned");
  ProfScope ps(PK_OTHER, stream, double(c_out) * c_in * (esize(w_dt) + (W_tilde ? esize(wt_dt) : 0)));
  OQ_HIP(let_fold(W, w_dt == OQ_BF16, B, c_out, c_in, s, delta, W_tilde, wt_dt == OQ_BF16, B_tilde,
                  stream),
         "let_fold");
  return OQ_OK;
}

// Splits the activation bits argument: the bit width and OQ_ACT_SYM.
static void act_mode(int bits_arg, int* bits, bool* sym) {
  *sym = (bits_arg & OQ_ACT_SYM) != 0;
  *bits = bits_arg & ~OQ_ACT_SYM;
}

static oq_status check_act(const void* X, oq_dtype x_dt, int64_t T, int64_t C, int bits_arg,
                           const float* s, const float* delta) {
  int bits;
  bool sym;
  act_mode(bits_arg, &bits, &sym);
  if (sym && bits == 16) return fail(OQ_ERR_UNSUPPORTED, "OQ_ACT_SYM needs bits in [2, 8]");
  OQ_REQ(X, "X is required");
  OQ_REQ(dtype_ok(x_dt), "bad dtype");
  OQ_REQ(T >= 0 && C > 0 && C % 8 == 0, "bad shape T=%lld C=%lld", (long long)T, (long long)C);
  OQ_REQ(aligned16(X) && (!s || aligned16(s)) && (!delta || aligned16(delta)),
         "pointers must be 16-byte aligned");
  if (!(bits == 16 || (bits >= 2 && bits <= 8)))
    return fail(OQ_ERR_UNSUPPORTED, "activation bits=%d (need 2..8 or 16)", bits);
  if (C > 32768) return fail(OQ_ERR_UNSUPPORTED, "C=%lld > 32768", (long long)C);
  return OQ_OK;
}

oq_status oq_act_fakequant_fwd(const void* X, oq_dtype x_dt, int64_t T, int64_t C, int bits,
                               const float* s, const float* delta, void* X_dq, oq_dtype dq_dt,
                               uint8_t* codes, float* h, float* z, hipStream_t stream) {
  oq_status e = check_act(X, x_dt, T, C, bits, s, delta);
  if (e != OQ_OK) return e;
  OQ_REQ(!X_dq || (dtype_ok(dq_dt) && aligned16(X_dq)), "bad X_dq");
  OQ_REQ(!codes || (reinterpret_cast<uintptr_t>(codes) & 7u) == 0, "codes must be 8-byte aligned");
  int nb;
  bool sym;
  act_mode(bits, &nb, &sym);
  OQ_REQ(!codes || nb < 16, "codes need bits < 16");
  ProfScope ps(PK_ACT_FWD, stream,
               double(T) * C * (esize(x_dt) + (X_dq ? esize(dq_dt) : 0) + (codes ? 1 : 0)));
  OQ_HIP(act_fwd(X, x_dt == OQ_BF16, T, C, nb, s, delta, X_dq, dq_dt == OQ_BF16, codes, h, z,
                 stream, sym),
         "act_fwd");
  return OQ_OK;
}

oq_status oq_act_fakequant_bwd_workspace_size(int64_t T, int64_t C, size_t* bytes) {
  OQ_REQ(bytes, "bytes is required");
  *bytes = 2 * (size_t(act_bwd_nparts(T)) * size_t(C) * 4 + 256);
  return OQ_OK;
}

oq_status oq_act_fakequant_bwd(const void* X, oq_dtype x_dt, int64_t T, int64_t C, int bits,
                               const float* s, const float* delta, const float* dX_dq,
                               float* dX_tilde, float* d_s, float* d_delta, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  oq_status e = check_act(X, x_dt, T, C, bits, s, delta);
  if (e != OQ_OK) return e;
  OQ_REQ(dX_dq && aligned16(dX_dq), "dX_dq is required and 16-byte aligned");
  OQ_REQ(!dX_tilde || aligned16(dX_tilde), "dX_tilde must be 16-byte aligned");
  const bool parts = d_s || d_delta;
  size_t need = 0;
  if (parts) oq_act_fakequant_bwd_workspace_size(T, C, &need);
  if (need && (!ws || ws_bytes < need))
    return fail(OQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws_bytes);
  Carver cv{static_cast<char*>(ws)};
  const int64_t np = act_bwd_nparts(T);
  float* psx = parts ? cv.take<float>(size_t(np) * C) : nullptr;
  float* ps1 = parts ? cv.take<float>(size_t(np) * C) : nullptr;
  {
    int nb;
    bool sym;
    act_mode(bits, &nb, &sym);
    ProfScope ps(PK_ACT_BWD, stream, double(T) * C * (esize(x_dt) + 4 + (dX_tilde ? 4 : 0)));
    OQ_HIP(act_bwd(X, x_dt == OQ_BF16, T, C, nb, s, delta, dX_dq, dX_tilde, psx, ps1, stream, sym),
           "act_bwd");
  }
  if (parts) {
    ProfScope ps(PK_OTHER, stream, 0);
    OQ_HIP(let_grad_finish(C, s, nullptr, 0, psx, ps1, np, nullptr, 0, d_s, d_delta, stream),
           "act finish");
  }
  return OQ_OK;
}

}  // extern "C"

// ------------------------------------------------------------------ no-allocation variant
// File-scope device array that holds the column partials of
// oq_act_fakequant_bwd_noalloc.  Each GPU has its own copy at its own
// address; host code uses the address hipGetSymbolAddress returns for the
// current device, never the array's name (a host-side stand-in).
static __device__ __align__(256) unsigned char scratch[OQ_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The scratch array's device address on the current device, looked up once
// per device (with that device current) and kept.
oq_status scratch_for_current_device(void** out) {
  int dev = 0;
  OQ_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(OQ_ERR_UNSUPPORTED, "device %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    OQ_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (!p) return fail(OQ_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return OQ_OK;
}
}  // namespace

extern "C" {

oq_status oq_act_fakequant_bwd_noalloc(const void* X, oq_dtype x_dt, int64_t T, int64_t C, int bits,
                                       const float* s, const float* delta, const float* dX_dq,
                                       float* dX_tilde, float* d_s, float* d_delta,
                                       hipStream_t stream) {
  oq_status e = check_act(X, x_dt, T, C, bits, s, delta);
  if (e != OQ_OK) return e;
  OQ_REQ(dX_dq && aligned16(dX_dq), "dX_dq is required and 16-byte aligned");
  OQ_REQ(!dX_tilde || aligned16(dX_tilde), "dX_tilde must be 16-byte aligned");
  const bool parts = d_s || d_delta;
  size_t need = 0;
  if (parts) oq_act_fakequant_bwd_workspace_size(T, C, &need);
  if (need > size_t(OQ_NOALLOC_SCRATCH_BYTES))
    return fail(OQ_ERR_UNSUPPORTED,
                "T=%lld C=%lld needs %zu bytes of partials, more than the %zu-byte scratch",
                (long long)T, (long long)C, need, size_t(OQ_NOALLOC_SCRATCH_BYTES));
  float *psx = nullptr, *ps1 = nullptr;
  const int64_t np = act_bwd_nparts(T);
  if (parts) {
    void* base = nullptr;
    e = scratch_for_current_device(&base);
    if (e != OQ_OK) return e;
    Carver cv{static_cast<char*>(base)};
    psx = cv.take<float>(size_t(np) * C);
    ps1 = cv.take<float>(size_t(np) * C);
  }
  {
    int nb;
    bool sym;
    act_mode(bits, &nb, &sym);
    ProfScope ps(PK_ACT_BWD, stream, double(T) * C * (esize(x_dt) + 4 + (dX_tilde ? 4 : 0)));
    OQ_HIP(act_bwd(X, x_dt == OQ_BF16, T, C, nb, s, delta, dX_dq, dX_tilde, psx, ps1, stream, sym),
           "act_bwd");
  }
  if (parts) {
    ProfScope ps(PK_OTHER, stream, 0);
    OQ_HIP(let_grad_finish(C, s, nullptr, 0, psx, ps1, np, nullptr, 0, d_s, d_delta, stream),
           "act finish");
  }
  return OQ_OK;
}

static size_t let_init_ws(int64_t T, int64_t C, const int64_t* c_out_site, int n_site) {
  size_t naw = 0;
  for (int i = 0; i < n_site; ++i) naw += size_t(colstat_nparts(c_out_site[i]));
  return size_t(colstat_nparts(T)) * C * 12 + naw * C * 4 + 3 * 256;
}

oq_status oq_let_init_workspace_size(int64_t T, int64_t C, const int64_t* c_out_site, int n_site,
                                     size_t* bytes) {
  OQ_REQ(bytes && c_out_site, "bytes and c_out_site are required");
  OQ_REQ(n_site >= 1 && n_site <= OQ_MAX_LINEARS, "n_site=%d", n_site);
  *bytes = let_init_ws(T, C, c_out_site, n_site);
  return OQ_OK;
}

oq_status oq_let_init(const void* X, oq_dtype x_dt, int64_t T, int64_t C,
                      const void* const* W_site, const int64_t* c_out_site, int n_site,
                      oq_dtype w_dt, float* s, float* delta, void* ws, size_t ws_bytes,
                      hipStream_t stream) {
  OQ_REQ(X && W_site && c_out_site && s && delta, "X, W_site, c_out_site, s, delta are required");
  OQ_REQ(n_site >= 1 && n_site <= OQ_MAX_LINEARS, "n_site=%d", n_site);
  OQ_REQ(dtype_ok(x_dt) && dtype_ok(w_dt), "bad dtype");
  OQ_REQ(T > 0 && C > 0 && C % 8 == 0, "bad shape");
  OQ_REQ(aligned16(X), "X must be 16-byte aligned");
  int64_t naw = 0;
  for (int i = 0; i < n_site; ++i) {
    OQ_REQ(W_site[i] && aligned16(W_site[i]) && c_out_site[i] > 0, "bad site weight %d", i);
    naw += colstat_nparts(c_out_site[i]);
  }
  const size_t need = let_init_ws(T, C, c_out_site, n_site);
  if (!ws || ws_bytes < need)
    return fail(OQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws_bytes);
  Carver cv{static_cast<char*>(ws)};
  const int64_t nax = colstat_nparts(T);
  float* ax = cv.take<float>(size_t(nax) * C);
  double* sm = cv.take<double>(size_t(nax) * C);
  float* aw = cv.take<float>(size_t(naw) * C);
  ProfScope ps(PK_OTHER, stream, double(T) * C * esize(x_dt));
  OQ_HIP(colstat(X, x_dt == OQ_BF16, T, C, ax, sm, stream), "colstat X");
  int64_t off = 0;
  for (int i = 0; i < n_site; ++i) {
    OQ_HIP(colstat(W_site[i], w_dt == OQ_BF16, c_out_site[i], C, aw + off * C, nullptr, stream),
           "colstat W");
    off += colstat_nparts(c_out_site[i]);
  }
  OQ_HIP(let_init_finish(C, T, ax, nax, sm, aw, naw, s, delta, stream), "let_init_finish");
  return OQ_OK;
}

oq_status oq_fp_target(const void* X, const void* W, oq_dtype dt, const float* B, int64_t T,
                       int64_t c_in, int64_t c_out, void* Y_T, hipStream_t stream) {
  OQ_REQ(X && W && Y_T, "X, W, Y_T are required");
  OQ_REQ(dtype_ok(dt), "bad dtype");
  OQ_REQ(T >= 0 && c_out >= 0 && c_in > 0 && c_in % 8 == 0, "bad shape");
  OQ_REQ(aligned16(X) && aligned16(W), "X and W must be 16-byte aligned");
  ProfScope ps(PK_OTHER, stream, 2.0 * double(T) * c_in * c_out);
  OQ_HIP(gemm_nt_store(W, X, dt == OQ_BF16, c_out, T, c_in, c_in, c_in, Y_T, dt == OQ_BF16, T, B,
                       stream),
         "fp_target");
  return OQ_OK;
}

oq_status oq_matmul_nt(const void* A, const void* B, oq_dtype in_dt, int64_t M, int64_t N,
                       int64_t K, void* C, oq_dtype out_dt, hipStream_t stream) {
  OQ_REQ(A && B && C, "A, B, C are required");
  OQ_REQ(dtype_ok(in_dt) && dtype_ok(out_dt), "bad dtype");
  OQ_REQ(M >= 0 && N >= 0 && K >= 0 && K % 8 == 0, "bad shape (K must be a multiple of 8)");
  OQ_REQ(aligned16(A) && aligned16(B), "A and B must be 16-byte aligned");
  ProfScope ps(PK_OTHER, stream, 2.0 * double(M) * N * K);
  if (out_dt == OQ_F32)
    OQ_HIP(gemm_nt_f32out(A, B, in_dt == OQ_BF16, M, N, K, K, K, static_cast<float*>(C), N, stream),
           "matmul");
  else
    OQ_HIP(gemm_nt_store(A, B, in_dt == OQ_BF16, M, N, K, K, K, C, true, N, nullptr, stream),
           "matmul");
  return OQ_OK;
}

oq_status oq_matmul(const void* A, int a_mn, const void* B, int b_mn, int64_t M, int64_t N,
                    int64_t K, float* C, hipStream_t stream) {
  OQ_REQ(A && B && C, "A, B, C are required");
  OQ_REQ(M >= 0 && N >= 0 && K >= 0, "bad shape");
  OQ_REQ(aligned16(A) && aligned16(B), "A and B must be 16-byte aligned");
  const int64_t lda = a_mn ? M : K, ldb = b_mn ? N : K;
  ProfScope ps(PK_OTHER, stream, 2.0 * double(M) * N * K);
  if (!a_mn && !b_mn) {
    OQ_REQ(K % 8 == 0, "K must be a multiple of 8");
    OQ_HIP(gemm_nt_f32out(A, B, true, M, N, K, K, K, C, N, stream), "matmul");
    return OQ_OK;
  }
  if (M == 0 || N == 0) return OQ_OK;
  if (!gemm_mn_supported(a_mn != 0, b_mn != 0, M, N, K, lda, ldb))
    return fail(OQ_ERR_UNSUPPORTED, "MN-major operand needs K %% 64 == 0 and M, N %% 8 == 0");
  OQ_HIP(gemm_f32out_mn(A, a_mn != 0, B, b_mn != 0, M, N, K, lda, ldb, C, N, stream), "matmul");
  return OQ_OK;
}

oq_status oq_pack_codes(const uint8_t* codes, int64_t c_out, int64_t c_in, int bits,
                        uint8_t* packed, hipStream_t stream) {
  OQ_REQ(c_out >= 0 && c_in > 0 && c_in % 32 == 0, "bad shape c_out=%lld c_in=%lld (need c_in %% 32 == 0)",
         (long long)c_out, (long long)c_in);
  if (bits < 2 || bits > 8) return fail(OQ_ERR_UNSUPPORTED, "bits=%d (need 2..8)", bits);
  if (c_out == 0) return OQ_OK;                   // empty: pointers may be NULL
  OQ_REQ(codes && packed, "codes and packed are required");
  OQ_REQ(aligned16(codes) && aligned16(packed), "pointers must be 16-byte aligned");
  ProfScope ps(PK_OTHER, stream, double(c_out) * c_in * (1.0 + bits / 8.0));
  OQ_HIP(pack_codes(codes, c_out, c_in, bits, packed, stream), "pack_codes");
  return OQ_OK;
}

oq_status oq_packed_linear(const void* X, oq_dtype x_dt, int64_t n_tok, int64_t c_in,
                           const uint8_t* packed, int bits, int64_t group, const float* h,
                           const float* z, const float* B, int64_t c_out, void* Y,
                           oq_dtype y_dt, hipStream_t stream) {
  if (x_dt != OQ_BF16) return fail(OQ_ERR_UNSUPPORTED, "the packed linear takes bf16 activations");
  OQ_REQ(dtype_ok(y_dt), "bad Y dtype");
  OQ_REQ(n_tok >= 0 && c_out >= 0 && c_in > 0 && c_in % 32 == 0,
         "bad shape n_tok=%lld c_in=%lld c_out=%lld (need c_in %% 32 == 0)", (long long)n_tok,
         (long long)c_in, (long long)c_out);
  OQ_REQ(group > 0 && group % 32 == 0 && c_in % group == 0,
         "group=%lld must be a multiple of 32 that divides c_in=%lld", (long long)group, (long long)c_in);
  if (bits < 2 || bits > 7) return fail(OQ_ERR_UNSUPPORTED, "bits=%d (need 2..7)", bits);
  if (c_in > PACKED_MAX_C_IN)
    return fail(OQ_ERR_UNSUPPORTED, "c_in=%lld > %lld", (long long)c_in, (long long)PACKED_MAX_C_IN);
  if (n_tok == 0 || c_out == 0) return OQ_OK;     // empty: pointers may be NULL
  OQ_REQ(X && packed && h && z && Y, "X, packed, h, z and Y are required");
  OQ_REQ(aligned16(X) && aligned16(packed) && aligned16(h) && aligned16(z) && (!B || aligned16(B)) &&
             aligned16(Y),
         "pointers must be 16-byte aligned");
  const double bytes = double(c_out) * c_in * bits / 8.0 + double(c_out) * (c_in / group) * 8.0 +
                       double(n_tok) * (2.0 * c_in + double(esize(y_dt)) * c_out) + (B ? 4.0 * c_out : 0.0);
  ProfScope ps(PK_PACKED_LINEAR, stream, bytes);
  OQ_HIP(packed_linear(static_cast<const uint16_t*>(X), n_tok, c_in, packed, bits, group, h, z, B, c_out,
                       Y, y_dt == OQ_BF16, stream),
         "packed_linear");
  return OQ_OK;
}

oq_status oq_adamw_step(float* p, const float* g, float* m, float* v, int64_t n, double lr,
                        double beta1, double beta2, double eps, double wd, int step,
                        hipStream_t stream) {
  OQ_REQ(p && g && m && v, "p, g, m, v are required");
  OQ_REQ(n >= 0 && step >= 1, "bad n or step");
  ProfScope ps(PK_OTHER, stream, double(n) * 28);
  OQ_HIP(adamw(p, g, m, v, n, adam_coef(lr, beta1, beta2, eps, wd, step), stream), "adamw");
  return OQ_OK;
}

}  // extern "C"

// ------------------------------------------------------------------ block step
namespace {

struct SitePlan {
  int k, l0, l1;
  int64_t C, M;
  bool let, act, sym;   // sym: symmetric absmax activation quantiser
  int act_bits;         // 2..8, or 16 = no activation quantisation
  bool lwc_only;        // every linear of the site quantised by LWC
};

struct BlockWs {
  void *what, *xhat, *xhatT, *dyT, *dy, *whatT;
  float *dW, *dX, *psq, *pdy, *dbt, *bt, *pw, *psx, *ps1, *pb;
  double* rl;
  float4* gstat;
};

oq_status plan_block(const oq_block_desc* d, std::vector<SitePlan>& plan) {
  OQ_REQ(d, "desc is required");
  OQ_REQ(d->n_sites >= 1 && d->n_sites <= OQ_MAX_SITES, "n_sites=%d", d->n_sites);
  OQ_REQ(d->n_linears >= 1 && d->n_linears <= OQ_MAX_LINEARS, "n_linears=%d", d->n_linears);
  OQ_REQ(dtype_ok(d->dtype), "bad dtype");
  OQ_REQ(d->tokens > 0 && d->tokens % 8 == 0, "tokens=%lld must be a positive multiple of 8",
         (long long)d->tokens);
  plan.clear();
  int prev_site = -1;
  for (int l = 0; l < d->n_linears; ++l) {
    const int k = d->lin_site[l];
    OQ_REQ(k >= 0 && k < d->n_sites, "linear %d: site %d out of range", l, k);
    OQ_REQ(k >= prev_site, "linears of one site must be consecutive (linear %d)", l);
    OQ_REQ(d->lin_c_out[l] > 0 && d->lin_c_out[l] % 8 == 0, "linear %d: c_out must be a positive multiple of 8", l);
    if (k != prev_site) {
      for (auto& p : plan) OQ_REQ(p.k != k, "linears of site %d are not consecutive", k);
      const int64_t C = d->site_width[k];
      OQ_REQ(C > 0 && C % 8 == 0, "site %d: width must be a positive multiple of 8", k);
      const int ab = d->site_act_bits[k] & ~OQ_ACT_SYM;
      const bool sym = (d->site_act_bits[k] & OQ_ACT_SYM) != 0;
      if (sym && ab == 16) return fail(OQ_ERR_UNSUPPORTED, "site %d: OQ_ACT_SYM needs bits 2..8", k);
      if (!(ab == 16 || (ab >= 2 && ab <= 8)))
        return fail(OQ_ERR_UNSUPPORTED, "site %d: activation bits %d", k, ab);
      if (C > 32768) return fail(OQ_ERR_UNSUPPORTED, "site %d: width %lld > 32768", k, (long long)C);
      plan.push_back(SitePlan{k, l, l + 1, C, 0, d->site_let[k] != 0, ab < 16, sym, ab, true});
      prev_site = k;
    } else {
      plan.back().l1 = l + 1;
    }
    SitePlan& sp = plan.back();
    sp.M += d->lin_c_out[l];
    if (sp.l1 - sp.l0 > MAX_SEG)
      return fail(OQ_ERR_UNSUPPORTED, "site %d has more than %d linears", k, MAX_SEG);
    if (d->lin_bits[l] < 2 || d->lin_bits[l] > 8)
      return fail(OQ_ERR_UNSUPPORTED, "linear %d: bits %d", l, d->lin_bits[l]);
    if (d->lin_quant[l] < OQ_WQ_LWC || d->lin_quant[l] > OQ_WQ_LSQ)
      return fail(OQ_ERR_UNSUPPORTED, "linear %d: quantizer %d", l, d->lin_quant[l]);
    sp.lwc_only = sp.lwc_only && d->lin_quant[l] == OQ_WQ_LWC;
    if (d->lin_group[l] <= 0 || sp.C % d->lin_group[l])
      return fail(OQ_ERR_INVALID_ARG, "linear %d: group %lld does not divide %lld", l,
                  (long long)d->lin_group[l], (long long)sp.C);
    if (!quant_shape_supported(sp.C, d->lin_group[l]))
      return fail(OQ_ERR_UNSUPPORTED, "linear %d: group %lld unsupported for width %lld", l,
                  (long long)d->lin_group[l], (long long)sp.C);
  }
  return OQ_OK;
}

// The weight gradient reads X^ token-major and the input gradient reads dY^T
// as stored (no transposes of the token-sized operands) when the 8-wave kernel takes the shapes
// with MN-major operands (bf16, T and the site's stacked rows multiples of 64).
bool direct_grads(const oq_block_desc* d, const SitePlan& p) {
  if (d->dtype != OQ_BF16) return false;
  const int64_t T = d->tokens;
  bool ok = gemm_mn_supported(false, true, p.M, p.C, T, T, p.C);
  if (p.let) ok = ok && gemm_mn_supported(true, true, T, p.C, p.M, T, p.C);
  return ok;
}

// The direct input gradient reads W^ through a transposed copy when the
// tokens are many enough for the faster product to repay the copy.
bool direct_wt_copy(const oq_block_desc* d, const SitePlan& p) {
  return p.let && d->tokens >= 65536 && direct_grads(d, p) &&
         gemm_mn_supported(true, false, d->tokens, p.C, p.M, d->tokens, p.M);
}

// K-split count of the weight gradient (its K is the token count); only the
// direct path splits.
int wgrad_splits(const oq_block_desc* d, const SitePlan& p) {
  if (!direct_grads(d, p)) return 1;
  const int64_t T = d->tokens;
  return gemm_mn_splits(false, true, p.M, p.C, T, T, p.C);
}

// K-split count of the forward product (bf16 only): few output tiles and a
// long K, as at the paper's 2048-token step.
int fwd_splits(const oq_block_desc* d, const SitePlan& p) {
  if (d->dtype != OQ_BF16) return 1;
  return gemm_resid_splits(p.M, d->tokens, p.C);
}

// The LWC straight-through backward runs in the weight gradient's epilogue
// when that product is not split, the site has no LET, and every linear of it
// shares one power-of-two group of at most 256 weights and one bit width.
bool fused_lwc(const oq_block_desc* d, const SitePlan& p) {
  if (p.let || !p.lwc_only || !direct_grads(d, p) || wgrad_splits(d, p) != 1) return false;
  const int64_t g = d->lin_group[p.l0];
  for (int l = p.l0; l < p.l1; ++l)
    if (d->lin_group[l] != g || d->lin_bits[l] != d->lin_bits[p.l0]) return false;
  return p.l1 - p.l0 <= MAX_SEG && gemm_wgrad_lwc_supported(p.M, p.C, d->tokens, int(g));
}

// Side streams (non-blocking, default priority) and fork / join events for
// concurrent sites: created once per device and host thread, kept for the
// life of the process.
constexpr int MAX_SIDE = 3;
struct SiteStreams {
  hipStream_t s[MAX_SIDE];
  hipEvent_t fork, join[MAX_SIDE];
  bool ok;
};

hipError_t site_streams(SiteStreams** out) {
  thread_local SiteStreams cache[16] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 16) return hipErrorInvalidDevice;
  SiteStreams& c = cache[dev];
  if (!c.ok) {
    for (int i = 0; i < MAX_SIDE; ++i) {
      if ((e = hipStreamCreateWithFlags(&c.s[i], hipStreamNonBlocking)) != hipSuccess) return e;
      if ((e = hipEventCreateWithFlags(&c.join[i], hipEventDisableTiming)) != hipSuccess) return e;
    }
    if ((e = hipEventCreateWithFlags(&c.fork, hipEventDisableTiming)) != hipSuccess) return e;
    c.ok = true;
  }
  *out = &c;
  return hipSuccess;
}

// The whole-block step's weight side (weight gradients, LWC backward, LET
// weight and bias paths) runs on a side stream of its own beside the input
// gradients: one per device and host thread, kept for the life of the
// process, with its fork and join events.
struct BlockSide {
  hipStream_t s;
  hipEvent_t fork, join;
  bool ok;
};

hipError_t block_side(BlockSide** out) {
  thread_local BlockSide cache[16] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 16) return hipErrorInvalidDevice;
  BlockSide& c = cache[dev];
  if (!c.ok) {
    if ((e = hipStreamCreateWithFlags(&c.s, hipStreamNonBlocking)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&c.fork, hipEventDisableTiming)) != hipSuccess) return e;
    if ((e = hipEventCreateWithFlags(&c.join, hipEventDisableTiming)) != hipSuccess) return e;
    c.ok = true;
  }
  *out = &c;
  return hipSuccess;
}

// Sites run concurrently (one stream each) at small token counts, where a
// site's products leave CUs idle in their last wave of tiles; each site then
// has its own buffers.  At large token counts the sites share one set.
bool concurrent_sites(const oq_block_desc* d, const std::vector<SitePlan>& plan) {
  if (plan.size() < 2 || plan.size() > size_t(MAX_SIDE) + 1 || d->dtype != OQ_BF16 ||
      d->tokens > 16384)
    return false;
  // only when every site's forward product is at most four waves of 256 x 256
  // tiles over 256 CUs: larger concurrent products measured slower (the
  // 70B block at 2048 tokens, 9%), smaller ones faster (the 7B and 13B, 5-14%)
  for (const auto& p : plan)
    if (((p.M + 255) / 256) * ((d->tokens + 255) / 256) > 4 * 256) return false;
  return true;
}

// Buffer sizes (elements) one site needs.
struct SiteSizes {
  size_t what = 0, xhat = 0, xhatT = 0, dyT = 0, dy = 0, whatT = 0, dW = 0, dX = 0, parts = 0,
         rows = 0, pw = 0, pa = 0, pb = 0, gs = 0;
  void max_with(const SiteSizes& o) {
    what = std::max(what, o.what); xhat = std::max(xhat, o.xhat); xhatT = std::max(xhatT, o.xhatT);
    dyT = std::max(dyT, o.dyT); dy = std::max(dy, o.dy); whatT = std::max(whatT, o.whatT);
    dW = std::max(dW, o.dW); dX = std::max(dX, o.dX); parts = std::max(parts, o.parts);
    rows = std::max(rows, o.rows); pw = std::max(pw, o.pw); pa = std::max(pa, o.pa);
    pb = std::max(pb, o.pb); gs = std::max(gs, o.gs);
  }
};

SiteSizes site_sizes(const oq_block_desc* d, const SitePlan& p) {
  const bool bf = d->dtype == OQ_BF16;
  const int64_t T = d->tokens;
  const int ptn = gemm_part_tile_n(bf);
  const int64_t ntn = (T + ptn - 1) / ptn;
  const bool direct = direct_grads(d, p);
  SiteSizes z;
  z.what = size_t(p.M * p.C);
  if (!direct) z.xhatT = size_t(T * p.C);
  z.dyT = size_t(p.M * T);
  z.dW = size_t(p.M * p.C) * size_t(wgrad_splits(d, p));
  // a split forward's parts live there too (the weight gradient comes later)
  const int sf = fwd_splits(d, p);
  if (sf > 1) z.dW = std::max(z.dW, size_t(p.M * T) * size_t(sf));
  if (fused_lwc(d, p)) z.gs = size_t(2 * p.M * (p.C / d->lin_group[p.l0]));
  z.parts = size_t(p.M * ntn);
  z.rows = size_t(p.M);
  if (p.let || p.act) z.xhat = size_t(T * p.C);
  if (p.let) {
    if (!direct) z.dy = size_t(p.M * T);
    if (!direct || direct_wt_copy(d, p)) z.whatT = size_t(p.M * p.C);
    z.dX = size_t(T * p.C);
    z.pa = size_t(act_bwd_nparts(T) * p.C);
    size_t a = 0, b = 0;
    for (int l = p.l0; l < p.l1; ++l) {
      a += size_t(lwc_bwd_nparts(d->lin_c_out[l]));
      b += size_t(wcolsum_nparts(d->lin_c_out[l]));
    }
    z.pw = a * p.C;
    z.pb = b * p.C;
  }
  return z;
}

BlockWs carve_set(Carver& cv, const SiteSizes& z, size_t es) {
  BlockWs t{};
  t.what = cv.take<char>(z.what * es);
  t.xhat = z.xhat ? cv.take<char>(z.xhat * es) : nullptr;
  t.xhatT = z.xhatT ? cv.take<char>(z.xhatT * es) : nullptr;
  t.dyT = cv.take<char>(z.dyT * es);
  t.dy = z.dy ? cv.take<char>(z.dy * es) : nullptr;
  t.whatT = z.whatT ? cv.take<char>(z.whatT * es) : nullptr;
  t.dW = cv.take<float>(z.dW);
  t.dX = z.dX ? cv.take<float>(z.dX) : nullptr;
  t.psq = cv.take<float>(z.parts);
  t.pdy = cv.take<float>(z.parts);
  t.dbt = cv.take<float>(z.rows);
  t.bt = cv.take<float>(z.rows);
  t.pw = z.pw ? cv.take<float>(z.pw) : nullptr;
  t.psx = z.pa ? cv.take<float>(z.pa) : nullptr;
  t.ps1 = z.pa ? cv.take<float>(z.pa) : nullptr;
  t.pb = z.pb ? cv.take<float>(z.pb) : nullptr;
  t.gstat = z.gs ? cv.take<float4>(z.gs) : nullptr;
  return t;
}

// Workspace layout: one buffer set per site when the sites run concurrently,
// else one set sized for the largest site; the row losses (fp64, every row
// of the block) after them.  w (one entry per site) may be null.
size_t carve_block(const oq_block_desc* d, const std::vector<SitePlan>& plan, char* base,
                   std::vector<BlockWs>* w) {
  const size_t es = d->dtype == OQ_BF16 ? 2 : 4;
  int64_t mtot = 0;
  for (const auto& p : plan) mtot += p.M;
  Carver cv{base};
  std::vector<BlockWs> sets;
  if (concurrent_sites(d, plan)) {
    for (const auto& p : plan) sets.push_back(carve_set(cv, site_sizes(d, p), es));
  } else {
    SiteSizes z;
    for (const auto& p : plan) z.max_with(site_sizes(d, p));
    const BlockWs t = carve_set(cv, z, es);
    sets.assign(plan.size(), t);
  }
  double* rl = cv.take<double>(size_t(mtot));
  for (auto& t : sets) t.rl = rl;
  if (w) *w = sets;
  return cv.off + 256;
}

}  // namespace

extern "C" {

oq_status oq_block_plan(const oq_block_desc* desc, int* info, int n_info) {
  OQ_REQ(info, "info is required");
  std::vector<SitePlan> plan;
  oq_status e = plan_block(desc, plan);
  if (e != OQ_OK) return e;
  OQ_REQ(n_info >= OQ_PLAN_FIELDS * desc->n_sites, "info holds %d ints, %d needed", n_info,
         OQ_PLAN_FIELDS * desc->n_sites);
  const bool conc = concurrent_sites(desc, plan);
  for (const auto& p : plan) {
    int* r = info + OQ_PLAN_FIELDS * p.k;
    const bool direct = direct_grads(desc, p);
    r[0] = conc;
    r[1] = direct;
    r[2] = direct && !fused_lwc(desc, p) ? wgrad_splits(desc, p) : 1;
    r[3] = fwd_splits(desc, p);
    r[4] = fused_lwc(desc, p);
    r[5] = p.let && direct_wt_copy(desc, p);
  }
  return OQ_OK;
}

oq_status oq_block_workspace_size(const oq_block_desc* desc, size_t* bytes) {
  OQ_REQ(bytes, "bytes is required");
  std::vector<SitePlan> plan;
  oq_status e = plan_block(desc, plan);
  if (e != OQ_OK) return e;
  *bytes = carve_block(desc, plan, nullptr, nullptr);
  return OQ_OK;
}

oq_status oq_block_calib_step(const oq_block_desc* d, const void* const* Y_fp_T,
                              const void* const* X_q, const oq_block_params* prm,
                              const oq_block_grads* gr, const oq_block_optim* opt, float* loss,
                              void* ws, size_t ws_bytes, hipStream_t st0) {
  std::vector<SitePlan> plan;
  oq_status e = plan_block(d, plan);
  if (e != OQ_OK) return e;
  OQ_REQ(Y_fp_T && X_q && prm && gr && loss, "Y_fp_T, X_q, params, grads, loss are required");
  const int frozen = opt ? opt->frozen : 0;
  OQ_REQ(frozen >= 0 && frozen <= (OQ_FREEZE_LWC | OQ_FREEZE_LET), "optim frozen=%d", frozen);
  const bool lwc_train = !(frozen & OQ_FREEZE_LWC), let_train = !(frozen & OQ_FREEZE_LET);
  for (const auto& p : plan) {
    OQ_REQ(X_q[p.k] && aligned16(X_q[p.k]), "X_q[%d] missing or misaligned", p.k);
    if (p.let) {
      OQ_REQ(prm->s[p.k] && prm->delta[p.k] && aligned16(prm->s[p.k]) && aligned16(prm->delta[p.k]),
             "site %d: LET needs 16-byte aligned s and delta", p.k);
      if (let_train)
        OQ_REQ(gr->d_s[p.k] && gr->d_delta[p.k], "site %d: d_s and d_delta are required", p.k);
    }
  }
  for (int l = 0; l < d->n_linears; ++l) {
    OQ_REQ(prm->W[l] && aligned16(prm->W[l]), "W[%d] missing or misaligned", l);
    OQ_REQ(prm->gamma_logit[l] && prm->beta_logit[l], "logits of linear %d missing", l);
    OQ_REQ(gr->d_gamma_logit[l] && gr->d_beta_logit[l], "gradients of linear %d missing", l);
    OQ_REQ(Y_fp_T[l], "Y_fp_T[%d] missing", l);
  }
  if (opt) {
    OQ_REQ(opt->step >= 1, "optim step must be >= 1");
    for (int l = 0; l < d->n_linears && lwc_train; ++l)
      OQ_REQ(opt->m_gamma[l] && opt->v_gamma[l] && opt->m_beta[l] && opt->v_beta[l],
             "AdamW state of linear %d missing", l);
    for (const auto& p : plan)
      if (p.let && let_train)
        OQ_REQ(opt->m_s[p.k] && opt->v_s[p.k] && opt->m_delta[p.k] && opt->v_delta[p.k],
               "AdamW state of site %d missing", p.k);
  }
  const size_t need = carve_block(d, plan, nullptr, nullptr);
  if (!ws || ws_bytes < need)
    return fail(OQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws_bytes);
  std::vector<BlockWs> wsets;
  carve_block(d, plan, static_cast<char*>(ws), &wsets);
  // concurrent sites: site 0 on the caller's stream, the others on side
  // streams forked from it here and joined before the loss
  const bool conc = concurrent_sites(d, plan);
  SiteStreams* ss = nullptr;
  if (conc) {
    OQ_HIP(site_streams(&ss), "site streams");
    OQ_HIP(hipEventRecord(ss->fork, st0), "fork");
    for (size_t i = 1; i < plan.size(); ++i)
      OQ_HIP(hipStreamWaitEvent(ss->s[i - 1], ss->fork, 0), "fork");
  }

  const bool bf = d->dtype == OQ_BF16;
  const size_t es = bf ? 2 : 4;
  const int64_t T = d->tokens;
  const int ptn = gemm_part_tile_n(bf);
  const int ntn = int((T + ptn - 1) / ptn);
  int64_t row_base = 0;
  LossArgs la{};
  la.nlin = d->n_linears;

  for (size_t si = 0; si < plan.size(); ++si) {
    const SitePlan& p = plan[si];
    hipStream_t st = conc && si > 0 ? ss->s[si - 1] : st0;
    const BlockWs& w = wsets[si];
    const int k = p.k;
    const int64_t C = p.C, M = p.M;
    const float* s = p.let ? prm->s[k] : nullptr;
    const float* dl = p.let ? prm->delta[k] : nullptr;
    // LET gradients (the input-gradient path) only for a trained LET; the
    // weight gradient only when some trained parameter needs it
    const bool let_grads = p.let && let_train;
    const bool wgrad = lwc_train || let_grads;
    bool any_bias = p.let;
    for (int l = p.l0; l < p.l1; ++l) any_bias = any_bias || prm->B[l];

    // 1. LWC forward of every linear of the site into the stacked W^ [M, C]
    //    (and, for the fused backward, each group's max, min, h and z)
    const bool fused = fused_lwc(d, p);
    const int64_t ngs = C / d->lin_group[p.l0];
    int64_t off = 0;
    for (int l = p.l0; l < p.l1; ++l) {
      const int64_t co = d->lin_c_out[l];
      ProfScope ps(PK_LWC_FWD, st, double(co) * C * 2 * es);
      OQ_HIP(lwc_fwd(prm->W[l], bf, co, C, s, prm->gamma_logit[l], prm->beta_logit[l],
                     d->lin_bits[l], d->lin_group[l], static_cast<char*>(w.what) + off * C * es, bf,
                     nullptr, nullptr, nullptr, st, fused ? w.gstat + 2 * off * ngs : nullptr,
                     d->lin_quant[l]),
             "lwc_fwd");
      la.row_begin[l] = row_base + off;
      la.row_end[l] = row_base + off + co;
      la.inv_n[l] = 1.0 / (double(T) * double(co));
      la.row_loss[l] = gr->row_loss[l];
      off += co;
    }
    // 2. folded bias B~ = B + W delta
    if (any_bias) {
      ProfScope ps(PK_OTHER, st, double(M) * C * es);
      off = 0;
      for (int l = p.l0; l < p.l1; ++l) {
        const int64_t co = d->lin_c_out[l];
        OQ_HIP(let_fold(prm->W[l], bf, prm->B[l], co, C, nullptr, dl, nullptr, false, w.bt + off, st),
               "let_fold");
        off += co;
      }
    }
    // 3. quantised-model input X^ = Q_a((X - delta)/s)
    const void* xsrc = X_q[k];
    if (p.let || p.act) {
      ProfScope ps(PK_ACT_FWD, st, double(T) * C * 2 * es);
      OQ_HIP(act_fwd(X_q[k], bf, T, C, p.act ? p.act_bits : 16, s, dl, w.xhat, bf,
                     nullptr, nullptr, nullptr, st, p.sym),
             "act_fwd");
      xsrc = w.xhat;
    }
    // 4. token-contiguous copy of X^ for the weight gradient (only where the
    //    gradient products cannot read X^ as stored)
    const bool direct = direct_grads(d, p);
    if (!direct) {
      ProfScope ps(PK_TRANSPOSE, st, double(T) * C * 2 * es);
      OQ_HIP(transpose(xsrc, T, C, C, w.xhatT, T, int(es), st), "transpose X");
    }
    // 5. forward: Y^T = W^ X^T + B~, residual, dY^T, row partials
    {
      ResidArgs ra{};
      ra.nseg = p.l1 - p.l0;
      int64_t b = 0;
      for (int i = 0; i < ra.nseg; ++i) {
        const int l = p.l0 + i;
        ra.seg_begin[i] = b;
        b += d->lin_c_out[l];
        ra.seg_end[i] = b;
        ra.yfp[i] = Y_fp_T[l];
        ra.scale[i] = 2.0f / float(T * d->lin_c_out[l]);
      }
      ra.ld_yfp = T;
      ra.bias = any_bias ? w.bt : nullptr;
      ra.dy = w.dyT;
      ra.ld_dy = T;
      ra.part_sq = w.psq;
      ra.part_dy = let_grads ? w.pdy : nullptr;
      ProfScope ps(PK_GEMM_FWD, st, 2.0 * double(M) * T * C);
      const int SF = fwd_splits(d, p);
      if (SF > 1)
        OQ_HIP(gemm_nt_resid_split(w.what, xsrc, M, T, C, C, C, ra, w.dW, SF, st),
               "forward gemm (K split)");
      else
        OQ_HIP(gemm_nt_resid(w.what, xsrc, bf, M, T, C, C, C, ra, st), "forward gemm");
    }
    {
      ProfScope ps(PK_OTHER, st, double(M) * ntn * 8);
      OQ_HIP(row_partials(w.psq, let_grads ? w.pdy : nullptr, M, ntn, w.rl + row_base, w.dbt, st),
             "row partials");
    }
    if (!wgrad) {            // every parameter this site feeds is frozen
      row_base += M;
      continue;
    }
    // 6. weight gradient dW^ = dY^T X^  [M, C]; over a K (token) split of S
    //    parts when that fills the last wave of tiles better, the parts
    //    summed in a fixed order (by the LWC backward's loads where it can)
    const int S = direct && !fused ? wgrad_splits(d, p) : 1;
    bool parts_in_bwd = S > 1 && p.lwc_only;
    for (int l = p.l0; l < p.l1; ++l)
      parts_in_bwd = parts_in_bwd && lwc_bwd_sums_parts(d->lin_c_out[l], C, d->lin_group[l], s,
                                                        p.let);
    {
      ProfScope ps(PK_GEMM_WGRAD, st, 2.0 * double(M) * T * C);
      if (fused) {
        // with the LWC straight-through backward in the epilogue (step 7)
        LwcArgs la{};
        la.nseg = p.l1 - p.l0;
        int64_t b = 0;
        for (int i = 0; i < la.nseg; ++i) {
          const int l = p.l0 + i;
          la.seg_begin[i] = b;
          b += d->lin_c_out[l];
          la.seg_end[i] = b;
          la.W[i] = static_cast<const uint16_t*>(prm->W[l]);
          la.dgl[i] = gr->d_gamma_logit[l];
          la.dbl[i] = gr->d_beta_logit[l];
        }
        la.gstat = w.gstat;
        la.C = C;
        la.group = int(d->lin_group[p.l0]);
        la.ng = int(ngs);
        la.qmax = float((1 << d->lin_bits[p.l0]) - 1);
        OQ_HIP(gemm_wgrad_lwc(w.dyT, xsrc, M, C, T, T, C, la, st), "wgrad gemm with LWC backward");
      } else if (direct) {
        OQ_HIP(gemm_f32out_mn(w.dyT, false, xsrc, true, M, C, T, T, C, w.dW, C, st, S, M * C),
               "wgrad gemm");
        if (S > 1 && !parts_in_bwd) OQ_HIP(sum_partials(w.dW, M * C, S, M * C, st), "wgrad split sum");
      } else
        OQ_HIP(gemm_nt_f32out(w.dyT, w.xhatT, bf, M, C, T, T, T, w.dW, C, st), "wgrad gemm");
    }
    // 7. LWC backward per linear (+ weight-path LET scale partials), unless
    //    the weight gradient's epilogue did it
    off = 0;
    int64_t pwo = 0;
    for (int l = p.l0; l < p.l1 && !fused; ++l) {
      const int64_t co = d->lin_c_out[l];
      ProfScope ps(PK_LWC_BWD, st, double(co) * C * (es + 4.0 * (parts_in_bwd ? S : 1)));
      OQ_HIP(lwc_bwd(prm->W[l], bf, co, C, s, prm->gamma_logit[l], prm->beta_logit[l],
                     d->lin_bits[l], d->lin_group[l], w.dW + off * C, gr->d_gamma_logit[l],
                     gr->d_beta_logit[l], nullptr, let_grads ? w.pw + pwo * C : nullptr, st,
                     parts_in_bwd ? S : 1, M * C, d->lin_quant[l]),
             "lwc_bwd");
      off += co;
      pwo += lwc_bwd_nparts(co);
    }
    // 8. LET: input gradient through Q_a and (X - delta)/s, bias path, finish
    if (let_grads) {
      const bool wt_copy = direct_wt_copy(d, p);
      if (direct && wt_copy) {
        // dX^ [T, C] = dY W^ with dY read from dY^T [M, T] as stored and W^
        // from a K-contiguous copy W^T [C, M] (its fragments then load as
        // plain 128-bit LDS reads: 3-9% faster than reading W^ as stored, for
        // a copy of M C bf16 that pays off only over many tokens)
        {
          ProfScope ps(PK_TRANSPOSE, st, double(M) * C * 2 * es);
          OQ_HIP(transpose(w.what, M, C, C, w.whatT, M, int(es), st), "transpose W^");
        }
        ProfScope ps(PK_GEMM_DGRAD, st, 2.0 * double(M) * T * C);
        OQ_HIP(gemm_f32out_mn(w.dyT, true, w.whatT, false, T, C, M, T, M, w.dX, C, st),
               "dgrad gemm");
      } else if (direct) {
        // dX^ [T, C] = dY W^ with dY^T [M, T] and W^ [M, C] read as stored
        ProfScope ps(PK_GEMM_DGRAD, st, 2.0 * double(M) * T * C);
        OQ_HIP(gemm_f32out_mn(w.dyT, true, w.what, true, T, C, M, T, C, w.dX, C, st),
               "dgrad gemm");
      } else {
        {
          ProfScope ps(PK_TRANSPOSE, st, double(M) * (T + C) * 2 * es);
          OQ_HIP(transpose(w.dyT, M, T, T, w.dy, M, int(es), st), "transpose dY");
          OQ_HIP(transpose(w.what, M, C, C, w.whatT, M, int(es), st), "transpose W^");
        }
        ProfScope ps(PK_GEMM_DGRAD, st, 2.0 * double(M) * T * C);
        OQ_HIP(gemm_nt_f32out(w.dy, w.whatT, bf, T, C, M, M, M, w.dX, C, st), "dgrad gemm");
      }
      {
        ProfScope ps(PK_ACT_BWD, st, double(T) * C * (es + 4));
        OQ_HIP(act_bwd(X_q[k], bf, T, C, p.act ? p.act_bits : 16, s, dl, w.dX, nullptr,
                       w.psx, w.ps1, st, p.sym),
               "act_bwd");
      }
      ProfScope ps(PK_OTHER, st, double(M) * C * es);
      off = 0;
      int64_t pbo = 0;
      for (int l = p.l0; l < p.l1; ++l) {
        const int64_t co = d->lin_c_out[l];
        OQ_HIP(wcolsum(prm->W[l], bf, co, C, w.dbt + off, w.pb + pbo * C, st), "bias path");
        off += co;
        pbo += wcolsum_nparts(co);
      }
      OQ_HIP(let_grad_finish(C, s, w.pw, pwo, w.psx, w.ps1, act_bwd_nparts(T), w.pb, pbo,
                             gr->d_s[k], gr->d_delta[k], st),
             "LET finish");
    }
    row_base += M;
  }
  if (conc) {
    for (size_t i = 1; i < plan.size(); ++i) {
      OQ_HIP(hipEventRecord(ss->join[i - 1], ss->s[i - 1]), "join");
      OQ_HIP(hipStreamWaitEvent(st0, ss->join[i - 1], 0), "join");
    }
  }
  hipStream_t st = st0;
  {
    ProfScope ps(PK_OTHER, st, double(row_base) * 8);
    OQ_HIP(loss_finish(wsets[0].rl, la, loss, st), "loss");
  }
  if (opt) {
    const AdamCoef cl = adam_coef(opt->lr_lwc, opt->beta1, opt->beta2, opt->eps, opt->wd, opt->step);
    const AdamCoef ce = adam_coef(opt->lr_let, opt->beta1, opt->beta2, opt->eps, opt->wd, opt->step);
    // every parameter tensor of the block in one launch (set 0: LWC, set 1: LET)
    ProfScope ps(PK_OTHER, st, 0);
    AdamList L{};
    auto add = [&](float* pp, const float* g, float* m, float* v, int64_t n, int set) {
      L.p[L.n] = pp; L.g[L.n] = g; L.m[L.n] = m; L.v[L.n] = v; L.len[L.n] = n; L.set[L.n] = set;
      ++L.n;
    };
    for (int l = 0; l < d->n_linears && lwc_train; ++l) {
      const int64_t n = d->lin_c_out[l] * (d->site_width[d->lin_site[l]] / d->lin_group[l]);
      add(prm->gamma_logit[l], gr->d_gamma_logit[l], opt->m_gamma[l], opt->v_gamma[l], n, 0);
      add(prm->beta_logit[l], gr->d_beta_logit[l], opt->m_beta[l], opt->v_beta[l], n, 0);
    }
    for (const auto& p : plan) {
      if (!p.let || !let_train) continue;
      add(prm->s[p.k], gr->d_s[p.k], opt->m_s[p.k], opt->v_s[p.k], p.C, 1);
      add(prm->delta[p.k], gr->d_delta[p.k], opt->m_delta[p.k], opt->v_delta[p.k], p.C, 1);
    }
    OQ_HIP(adamw_multi(L, cl, ce, st), "adamw");
  }
  return OQ_OK;
}

oq_status oq_block_export_workspace_size(const oq_block_desc* d, size_t* bytes) {
  OQ_REQ(bytes, "bytes is required");
  std::vector<SitePlan> plan;
  oq_status e = plan_block(d, plan);
  if (e != OQ_OK) return e;
  size_t mx = 0;
  for (int l = 0; l < d->n_linears; ++l)
    mx = std::max(mx, size_t(d->lin_c_out[l]) * size_t(d->site_width[d->lin_site[l]]));
  *bytes = (mx + 255) & ~size_t(255);
  return OQ_OK;
}

oq_status oq_block_export(const oq_block_desc* d, const oq_block_params* prm,
                          uint8_t* const* packed, float* const* h, float* const* z,
                          float* const* B_tilde, void* ws, size_t ws_bytes, hipStream_t st) {
  size_t need = 0;
  oq_status e = oq_block_export_workspace_size(d, &need);
  if (e != OQ_OK) return e;
  OQ_REQ(prm && packed && h && z, "params, packed, h and z are required");
  if (!ws || ws_bytes < need || !aligned16(ws))
    return fail(OQ_ERR_WORKSPACE, "workspace of %zu bytes (16-byte aligned) needed, %zu given", need,
                ws_bytes);
  for (int l = 0; l < d->n_linears; ++l) {
    const int k = d->lin_site[l];
    OQ_REQ(d->site_width[k] % 32 == 0, "linear %d: C_in=%lld is not a multiple of 32", l,
           (long long)d->site_width[k]);
    // the packed linear consumes the export: codes of 2..7 bits, groups of
    // whole 32-code runs
    if (d->lin_bits[l] > 7 || d->lin_group[l] % 32 != 0)
      return fail(OQ_ERR_UNSUPPORTED,
                  "linear %d: bits %d / group %lld cannot be deployed by oq_packed_linear "
                  "(bits 2..7, group a multiple of 32)",
                  l, d->lin_bits[l], (long long)d->lin_group[l]);
    OQ_REQ(prm->W[l] && aligned16(prm->W[l]), "W[%d] missing or misaligned", l);
    OQ_REQ(prm->gamma_logit[l] && prm->beta_logit[l], "logits of linear %d missing", l);
    OQ_REQ(packed[l] && aligned16(packed[l]) && h[l] && z[l], "outputs of linear %d missing or misaligned", l);
    if (d->site_let[k])
      OQ_REQ(prm->s[k] && prm->delta[k] && aligned16(prm->s[k]) && aligned16(prm->delta[k]),
             "site %d: LET needs 16-byte aligned s and delta", k);
  }
  const bool bf = d->dtype == OQ_BF16;
  uint8_t* codes = static_cast<uint8_t*>(ws);
  for (int l = 0; l < d->n_linears; ++l) {
    const int k = d->lin_site[l];
    const int64_t c_out = d->lin_c_out[l], c_in = d->site_width[k];
    const bool let = d->site_let[k] != 0;
    ProfScope ps(PK_OTHER, st, double(c_out) * c_in * (esize(d->dtype) + 1.0 + d->lin_bits[l] / 8.0));
    OQ_HIP(lwc_fwd(prm->W[l], bf, c_out, c_in, let ? prm->s[k] : nullptr, prm->gamma_logit[l],
                   prm->beta_logit[l], d->lin_bits[l], d->lin_group[l], nullptr, false, codes, h[l],
                   z[l], st, nullptr, d->lin_quant[l]),
           "export lwc_fwd");
    OQ_HIP(pack_codes(codes, c_out, c_in, d->lin_bits[l], packed[l], st), "export pack_codes");
    if (B_tilde && B_tilde[l])
      OQ_HIP(let_fold(prm->W[l], bf, prm->B[l], c_out, c_in, let ? prm->s[k] : nullptr,
                      let ? prm->delta[k] : nullptr, nullptr, false, B_tilde[l], st),
             "export let_fold");
  }
  return OQ_OK;
}

oq_status oq_let_absorb(const void* P, oq_dtype p_dt, const float* b, int64_t C, int64_t n,
                        const float* s, const float* delta, void* P_out, float* b_out,
                        hipStream_t stream) {
  OQ_REQ(dtype_ok(p_dt), "bad dtype");
  OQ_REQ(C >= 0 && n >= 0, "bad shape C=%lld n=%lld", (long long)C, (long long)n);
  OQ_REQ(!P_out || P, "P_out needs P");
  OQ_REQ(P_out || b_out, "nothing to write: P_out and b_out are both NULL");
  ProfScope ps(PK_OTHER, stream, double(C) * n * 2 * esize(p_dt));
  OQ_HIP(let_absorb(P, p_dt == OQ_BF16, b, C, n, s, delta, P_out, b_out, stream), "let_absorb");
  return OQ_OK;
}

}  // extern "C"

// ------------------------------------------------------------------ checkpoint / resume
namespace {

constexpr char kCkptMagic[8] = {'O', 'Q', 'C', 'K', 'P', 'T', '\0', '\1'};
constexpr uint32_t kCkptVersion = 1;

uint64_t fnv1a64(const void* data, size_t n) {
  const unsigned char* p = static_cast<const unsigned char*>(data);
  uint64_t h = 1469598103934665603ull;
  for (size_t i = 0; i < n; ++i) {
    h ^= p[i];
    h *= 1099511628211ull;
  }
  return h;
}

// One calibrated tensor of the block: kind (0 gamma_logit, 1 beta_logit,
// 2 s, 3 delta, 4 m_gamma, 5 v_gamma, 6 m_beta, 7 v_beta, 8 m_s, 9 v_s,
// 10 m_delta, 11 v_delta), the linear or site it belongs to, its device
// pointer and element count.
struct CkptTensor {
  uint32_t kind, index;
  float* ptr;
  uint64_t count;
};

std::vector<CkptTensor> ckpt_tensors(const oq_block_desc* d, const std::vector<SitePlan>& plan,
                                     const oq_block_params* prm, const oq_block_optim* opt) {
  std::vector<CkptTensor> t;
  for (int l = 0; l < d->n_linears; ++l) {
    const uint64_t n = uint64_t(d->lin_c_out[l]) * uint64_t(d->site_width[d->lin_site[l]] / d->lin_group[l]);
    t.push_back({0, uint32_t(l), prm->gamma_logit[l], n});
    t.push_back({1, uint32_t(l), prm->beta_logit[l], n});
    if (opt) {
      t.push_back({4, uint32_t(l), opt->m_gamma[l], n});
      t.push_back({5, uint32_t(l), opt->v_gamma[l], n});
      t.push_back({6, uint32_t(l), opt->m_beta[l], n});
      t.push_back({7, uint32_t(l), opt->v_beta[l], n});
    }
  }
  for (const auto& p : plan) {
    if (!p.let) continue;
    const uint64_t n = uint64_t(p.C);
    t.push_back({2, uint32_t(p.k), prm->s[p.k], n});
    t.push_back({3, uint32_t(p.k), prm->delta[p.k], n});
    if (opt) {
      t.push_back({8, uint32_t(p.k), opt->m_s[p.k], n});
      t.push_back({9, uint32_t(p.k), opt->v_s[p.k], n});
      t.push_back({10, uint32_t(p.k), opt->m_delta[p.k], n});
      t.push_back({11, uint32_t(p.k), opt->v_delta[p.k], n});
    }
  }
  return t;
}

// The descriptor fields a checkpoint must agree on (the token count and the
// data type of X and W may differ between the saving and the resuming run).
struct CkptShape {
  int32_t n_sites, n_linears;
  int64_t site_width[OQ_MAX_SITES];
  int32_t site_let[OQ_MAX_SITES], site_act_bits[OQ_MAX_SITES];
  int32_t lin_site[OQ_MAX_LINEARS];
  int64_t lin_c_out[OQ_MAX_LINEARS];
  int32_t lin_bits[OQ_MAX_LINEARS];
  int64_t lin_group[OQ_MAX_LINEARS];
  int32_t lin_quant[OQ_MAX_LINEARS];
};

CkptShape ckpt_shape(const oq_block_desc* d) {
  CkptShape c;
  memset(&c, 0, sizeof c);
  c.n_sites = d->n_sites;
  c.n_linears = d->n_linears;
  for (int k = 0; k < d->n_sites; ++k) {
    c.site_width[k] = d->site_width[k];
    c.site_let[k] = d->site_let[k];
    c.site_act_bits[k] = d->site_act_bits[k];
  }
  for (int l = 0; l < d->n_linears; ++l) {
    c.lin_site[l] = d->lin_site[l];
    c.lin_c_out[l] = d->lin_c_out[l];
    c.lin_bits[l] = d->lin_bits[l];
    c.lin_quant[l] = d->lin_quant[l];
    c.lin_group[l] = d->lin_group[l];
  }
  return c;
}

struct FileCloser {
  FILE* f;
  ~FileCloser() {
    if (f) fclose(f);
  }
};

}  // namespace

extern "C" {

oq_status oq_block_state_save(const oq_block_desc* d, const oq_block_params* prm,
                              const oq_block_optim* opt, int completed_steps, const char* path,
                              hipStream_t stream) {
  std::vector<SitePlan> plan;
  oq_status e = plan_block(d, plan);
  if (e != OQ_OK) return e;
  OQ_REQ(prm && path, "params and path are required");
  OQ_REQ(completed_steps >= 0, "completed_steps=%d", completed_steps);
  const auto ts = ckpt_tensors(d, plan, prm, opt);
  for (const auto& t : ts) OQ_REQ(t.ptr, "tensor kind %u of %u is missing", t.kind, t.index);
  OQ_HIP(hipStreamSynchronize(stream), "synchronise before saving");
  const std::string tmp = std::string(path) + ".tmp";
  {
    FileCloser fc{fopen(tmp.c_str(), "wb")};
    if (!fc.f) return fail(OQ_ERR_INVALID_ARG, "cannot open %s for writing", tmp.c_str());
    const CkptShape shape = ckpt_shape(d);
    const int32_t head[4] = {int32_t(kCkptVersion), int32_t(sizeof(CkptShape)), completed_steps,
                             opt ? 1 : 0};
    const uint64_t nt = ts.size();
    bool ok = fwrite(kCkptMagic, 1, 8, fc.f) == 8 && fwrite(head, sizeof head, 1, fc.f) == 1 &&
              fwrite(&shape, sizeof shape, 1, fc.f) == 1 && fwrite(&nt, 8, 1, fc.f) == 1;
    if (opt) {
      const double hp[6] = {opt->lr_lwc, opt->lr_let, opt->beta1, opt->beta2, opt->eps, opt->wd};
      ok = ok && fwrite(hp, sizeof hp, 1, fc.f) == 1;
    }
    std::vector<float> buf;
    for (const auto& t : ts) {
      if (!ok) break;
      buf.resize(t.count);
      OQ_HIP(hipMemcpy(buf.data(), t.ptr, t.count * 4, hipMemcpyDeviceToHost), "copy to host");
      const uint64_t sum = fnv1a64(buf.data(), t.count * 4);
      const uint32_t ki[2] = {t.kind, t.index};
      ok = fwrite(ki, sizeof ki, 1, fc.f) == 1 && fwrite(&t.count, 8, 1, fc.f) == 1 &&
           fwrite(&sum, 8, 1, fc.f) == 1 &&
           (t.count == 0 || fwrite(buf.data(), 4, t.count, fc.f) == t.count);
    }
    if (!ok) return fail(OQ_ERR_INVALID_ARG, "write to %s failed", tmp.c_str());
    if (fflush(fc.f) != 0) return fail(OQ_ERR_INVALID_ARG, "flush of %s failed", tmp.c_str());
  }
  if (rename(tmp.c_str(), path) != 0)
    return fail(OQ_ERR_INVALID_ARG, "cannot rename %s to %s", tmp.c_str(), path);
  return OQ_OK;
}

oq_status oq_block_state_load(const oq_block_desc* d, const oq_block_params* prm,
                              oq_block_optim* opt, int* completed_steps, const char* path,
                              hipStream_t stream) {
  std::vector<SitePlan> plan;
  oq_status e = plan_block(d, plan);
  if (e != OQ_OK) return e;
  OQ_REQ(prm && path && completed_steps, "params, path and completed_steps are required");
  FileCloser fc{fopen(path, "rb")};
  if (!fc.f) return fail(OQ_ERR_INVALID_ARG, "cannot open %s", path);
  char magic[8];
  int32_t head[4];
  CkptShape shape;
  uint64_t nt = 0;
  if (fread(magic, 1, 8, fc.f) != 8 || memcmp(magic, kCkptMagic, 8) != 0)
    return fail(OQ_ERR_INVALID_ARG, "%s is not a block checkpoint", path);
  if (fread(head, sizeof head, 1, fc.f) != 1 || head[0] != int32_t(kCkptVersion) ||
      head[1] != int32_t(sizeof(CkptShape)))
    return fail(OQ_ERR_INVALID_ARG, "%s: unsupported checkpoint version", path);
  if (fread(&shape, sizeof shape, 1, fc.f) != 1 || fread(&nt, 8, 1, fc.f) != 1)
    return fail(OQ_ERR_INVALID_ARG, "%s: truncated header", path);
  const CkptShape want = ckpt_shape(d);
  if (memcmp(&shape, &want, sizeof shape) != 0)
    return fail(OQ_ERR_INVALID_ARG, "%s: the checkpoint's block shape differs from desc", path);
  const bool has_opt = head[3] != 0;
  if (opt && !has_opt) return fail(OQ_ERR_INVALID_ARG, "%s holds no AdamW state", path);
  double hp[6];
  if (has_opt && fread(hp, sizeof hp, 1, fc.f) != 1)
    return fail(OQ_ERR_INVALID_ARG, "%s: truncated header", path);
  const auto ts = ckpt_tensors(d, plan, prm, has_opt ? opt : nullptr);
  for (const auto& t : ts) OQ_REQ(t.ptr, "tensor kind %u of %u is missing", t.kind, t.index);
  // read and verify everything before any device buffer is written
  std::vector<std::vector<float>> data;
  std::vector<const CkptTensor*> dst;
  for (uint64_t i = 0; i < nt; ++i) {
    uint32_t ki[2];
    uint64_t cnt = 0, sum = 0;
    if (fread(ki, sizeof ki, 1, fc.f) != 1 || fread(&cnt, 8, 1, fc.f) != 1 ||
        fread(&sum, 8, 1, fc.f) != 1)
      return fail(OQ_ERR_INVALID_ARG, "%s: truncated at tensor %llu", path, (unsigned long long)i);
    const CkptTensor* match = nullptr;
    for (const auto& t : ts)
      if (t.kind == ki[0] && t.index == ki[1]) match = &t;
    if (cnt > (uint64_t(1) << 40))
      return fail(OQ_ERR_INVALID_ARG, "%s: tensor %llu has an implausible size", path,
                  (unsigned long long)i);
    std::vector<float> v(cnt);
    if (cnt && fread(v.data(), 4, cnt, fc.f) != cnt)
      return fail(OQ_ERR_INVALID_ARG, "%s: truncated in tensor %llu", path, (unsigned long long)i);
    if (fnv1a64(v.data(), cnt * 4) != sum)
      return fail(OQ_ERR_INVALID_ARG, "%s: checksum mismatch in tensor kind %u of %u", path, ki[0],
                  ki[1]);
    if (!match) continue;               // AdamW state the caller does not restore
    if (match->count != cnt)
      return fail(OQ_ERR_INVALID_ARG, "%s: tensor kind %u of %u has %llu elements, %llu expected",
                  path, ki[0], ki[1], (unsigned long long)cnt, (unsigned long long)match->count);
    data.push_back(std::move(v));
    dst.push_back(match);
  }
  if (data.size() != ts.size())
    return fail(OQ_ERR_INVALID_ARG, "%s holds %zu of the %zu tensors needed", path, data.size(),
                ts.size());
  for (size_t i = 0; i < data.size(); ++i)
    OQ_HIP(hipMemcpyAsync(dst[i]->ptr, data[i].data(), dst[i]->count * 4, hipMemcpyHostToDevice,
                          stream),
           "copy to device");
  OQ_HIP(hipStreamSynchronize(stream), "synchronise after loading");
  *completed_steps = head[2];
  if (opt) {
    opt->step = head[2] + 1;
    opt->lr_lwc = hp[0];
    opt->lr_let = hp[1];
    opt->beta1 = hp[2];
    opt->beta2 = hp[3];
    opt->eps = hp[4];
    opt->wd = hp[5];
  }
  return OQ_OK;
}

oq_status oq_block_calibrate(const oq_block_desc* d, int n_segments, int epochs,
                             const void* const* Y_fp_T, const void* const* X_q,
                             const oq_block_params* prm, const oq_block_grads* gr,
                             const oq_block_optim* opt, float* losses, void* ws, size_t ws_bytes,
                             hipStream_t stream) {
  OQ_REQ(d && Y_fp_T && X_q && prm && gr && opt && losses,
         "desc, Y_fp_T, X_q, params, grads, optim and losses are required");
  OQ_REQ(n_segments >= 1 && epochs >= 1, "need n_segments >= 1 and epochs >= 1 (got %d, %d)",
         n_segments, epochs);
  OQ_REQ(opt->step >= 1 && int64_t(opt->step) + int64_t(epochs) * n_segments - 1 <= INT32_MAX,
         "optim step %d out of range for %d steps", opt->step, epochs * n_segments);
  size_t need = 0;
  oq_status e = oq_block_workspace_size(d, &need);
  if (e != OQ_OK) return e;
  if (ws_bytes < need || !ws)
    return fail(OQ_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, need);
  // every segment's pointers before the first launch; the first step checks the rest
  for (int g = 0; g < n_segments; ++g) {
    for (int l = 0; l < d->n_linears; ++l)
      OQ_REQ(Y_fp_T[size_t(g) * d->n_linears + l], "segment %d: Y_fp_T[%d] missing", g, l);
    for (int k = 0; k < d->n_sites; ++k) {
      const void* x = X_q[size_t(g) * d->n_sites + k];
      OQ_REQ(x && aligned16(x), "segment %d: X_q[%d] missing or misaligned", g, k);
    }
  }
  oq_block_optim o = *opt;
  for (int ep = 0; ep < epochs; ++ep)
    for (int g = 0; g < n_segments; ++g) {
      const int64_t i = int64_t(ep) * n_segments + g;
      o.step = int(opt->step + i);
      e = oq_block_calib_step(d, Y_fp_T + size_t(g) * d->n_linears, X_q + size_t(g) * d->n_sites,
                              prm, gr, &o, losses + i, ws, ws_bytes, stream);
      if (e != OQ_OK) return e;
    }
  return OQ_OK;
}

}  // extern "C"

// ------------------------------------------------------------------ whole LLaMA block
namespace {

constexpr int NL = OQ_LLAMA_LINEARS;
constexpr int L_SITE[NL] = {0, 0, 0, 1, 2, 2, 3};

struct LlamaDims {
  int64_t T, S, D, F, H, Hkv, dh, Hd, Kd, Mqkv;
  int64_t c_out[NL], c_in[NL];
  int ab;     // activation bits without the symmetric flag
  int pb;     // softmax-output bits (16 = unquantised)
  bool sym, let;
};

oq_status llama_dims(const oq_llama_desc* d, LlamaDims* o) {
  OQ_REQ(d, "desc is required");
  LlamaDims& m = *o;
  m.T = d->tokens;
  m.S = d->seq_len;
  m.D = d->hidden;
  m.F = d->ffn;
  m.H = d->heads;
  m.Hkv = d->kv_heads;
  OQ_REQ(m.T > 0 && m.S > 0 && m.D > 0 && m.F > 0 && m.H > 0 && m.Hkv > 0, "bad shape");
  OQ_REQ(m.D % m.H == 0, "hidden %lld not a multiple of heads %lld", (long long)m.D, (long long)m.H);
  m.dh = m.D / m.H;
  m.Hd = m.H * m.dh;
  m.Kd = m.Hkv * m.dh;
  m.Mqkv = m.Hd + 2 * m.Kd;
  if (!attn_supported(m.T, int(m.S), int(m.H), int(m.Hkv), int(m.dh)))
    return fail(OQ_ERR_UNSUPPORTED,
                "attention: head_dim %lld (need 64 or 128), S %lld (multiple of 64), T %lld "
                "(multiple of S), H %lld / Hkv %lld",
                (long long)m.dh, (long long)m.S, (long long)m.T, (long long)m.H, (long long)m.Hkv);
  if (m.D % 64 || m.F % 64) return fail(OQ_ERR_UNSUPPORTED, "hidden and ffn must be multiples of 64");
  m.sym = (d->act_bits & OQ_ACT_SYM) != 0;
  m.ab = d->act_bits & ~OQ_ACT_SYM;
  if (!(m.ab == 16 || (m.ab >= 2 && m.ab <= 8)) || (m.sym && m.ab == 16))
    return fail(OQ_ERR_UNSUPPORTED, "activation bits %d", d->act_bits);
  m.let = d->let != 0;
  m.pb = d->softmax_bits;
  if (!(m.pb == 16 || (m.pb >= 2 && m.pb <= 8)))
    return fail(OQ_ERR_UNSUPPORTED, "softmax bits %d", d->softmax_bits);
  const int64_t co[NL] = {m.Hd, m.Kd, m.Kd, m.D, m.F, m.F, m.D};
  const int64_t ci[NL] = {m.D, m.D, m.D, m.Hd, m.D, m.D, m.F};
  for (int l = 0; l < NL; ++l) {
    m.c_out[l] = co[l];
    m.c_in[l] = ci[l];
    if (d->w_bits[l] < 2 || d->w_bits[l] > 8)
      return fail(OQ_ERR_UNSUPPORTED, "linear %d: bits %d", l, d->w_bits[l]);
    if (d->w_group[l] <= 0 || ci[l] % d->w_group[l])
      return fail(OQ_ERR_INVALID_ARG, "linear %d: group %lld does not divide %lld", l,
                  (long long)d->w_group[l], (long long)ci[l]);
    if (!quant_shape_supported(ci[l], d->w_group[l]))
      return fail(OQ_ERR_UNSUPPORTED, "linear %d: group %lld for width %lld", l,
                  (long long)d->w_group[l], (long long)ci[l]);
  }
  return OQ_OK;
}

struct LlamaWs {
  float *x1, *rstd1, *qkv, *qt, *kt, *vv, *att, *lse, *pstat, *o, *h1, *x3, *rstd2, *gu, *x4, *dn, *h2;
  void *xh1, *wqkv, *qh, *kh, *vh, *xh2, *wo, *xh3, *wgu, *xh4, *wd;
  float *dh2, *dW, *dxh, *dxt, *dh1, *Dl, *dQ, *dK, *dV, *dqt, *dkt, *dvt;
  void *dh2_16, *dh1_16, *dgu16, *datt16, *dqkv16;
  double* rows;
  float* rope;                        // RoPE table [S, dh/2] (cos, sin)
  float* part;                        // K-split partial products
  float *bt_qkv, *bt_o, *bt_gu;       // folded biases B~ of the LET sites
  float *dbt, *psx, *ps1, *psxq, *psxk, *pw, *pb, *amax;
  double* csum;
};

size_t llama_carve(const LlamaDims& m, char* base, LlamaWs* w) {
  Carver cv{base};
  LlamaWs t{};
  const int64_t T = m.T, D = m.D, F = m.F;
  const int64_t maxC = std::max(std::max(D, m.Hd), F);
  int64_t maxWC = 0, maxM = 0;
  for (int l = 0; l < NL; ++l) maxWC = std::max(maxWC, m.c_out[l] * m.c_in[l]);
  maxWC = std::max(maxWC, std::max(m.Mqkv * D, 2 * F * D));
  maxM = std::max(std::max(m.Mqkv, 2 * F), std::max(D, m.Hd));
  t.x1 = cv.take<float>(T * D);
  t.rstd1 = cv.take<float>(T);
  t.xh1 = cv.take<uint16_t>(T * D);
  t.wqkv = cv.take<uint16_t>(m.Mqkv * D);
  t.qkv = cv.take<float>(T * m.Mqkv);
  t.qt = cv.take<float>(T * m.Hd);
  t.kt = cv.take<float>(T * m.Kd);
  t.vv = cv.take<float>(T * m.Kd);
  t.qh = cv.take<uint16_t>(T * m.Hd);
  t.kh = cv.take<uint16_t>(T * m.Kd);
  t.vh = cv.take<uint16_t>(T * m.Kd);
  t.att = cv.take<float>(T * m.Hd);
  t.lse = cv.take<float>(m.H * T);
  t.pstat = cv.take<float>(m.pb < 16 ? 4 * m.H * T : 0);
  t.xh2 = cv.take<uint16_t>(T * m.Hd);
  t.wo = cv.take<uint16_t>(D * m.Hd);
  t.o = cv.take<float>(T * D);
  t.h1 = cv.take<float>(T * D);
  t.x3 = cv.take<float>(T * D);
  t.rstd2 = cv.take<float>(T);
  t.xh3 = cv.take<uint16_t>(T * D);
  t.wgu = cv.take<uint16_t>(2 * F * D);
  t.gu = cv.take<float>(T * 2 * F);
  t.x4 = cv.take<float>(T * F);
  t.xh4 = cv.take<uint16_t>(T * F);
  t.wd = cv.take<uint16_t>(D * F);
  t.dn = cv.take<float>(T * D);
  t.h2 = cv.take<float>(T * D);
  t.dh2 = cv.take<float>(T * D);
  t.dh2_16 = cv.take<uint16_t>(T * D);
  t.rows = cv.take<double>(T);
  t.rope = cv.take<float>(m.S * m.dh);
  t.bt_qkv = cv.take<float>(m.Mqkv);
  t.bt_o = cv.take<float>(D);
  t.bt_gu = cv.take<float>(2 * F);
  t.dW = cv.take<float>(maxWC);
  t.dxh = cv.take<float>(T * maxC);
  t.dxt = cv.take<float>(T * maxC);
  t.dh1 = cv.take<float>(T * D);
  t.dh1_16 = cv.take<uint16_t>(T * D);
  t.dgu16 = cv.take<uint16_t>(T * 2 * F);
  t.datt16 = cv.take<uint16_t>(T * m.Hd);
  t.Dl = cv.take<float>(int64_t(attn_bwd_ws_floats(T, int(m.H), m.pb)));
  t.dQ = cv.take<float>(T * m.Hd);
  t.dK = cv.take<float>(T * m.Kd);
  t.dV = cv.take<float>(T * m.Kd);
  t.dqt = cv.take<float>(T * m.Hd);
  t.dkt = cv.take<float>(T * m.Kd);
  t.dvt = cv.take<float>(T * m.Kd);
  t.dqkv16 = cv.take<uint16_t>(T * m.Mqkv);
  const int64_t npa = act_bwd_nparts(T);
  t.psx = cv.take<float>(npa * maxC);
  t.ps1 = cv.take<float>(npa * maxC);
  t.psxq = cv.take<float>(npa * m.Hd);
  t.psxk = cv.take<float>(npa * m.Kd);
  int64_t npw = 0, npb = 0;
  for (int l = 0; l < NL; ++l) {
    npw = std::max(npw, lwc_bwd_nparts(m.c_out[l]));
    npb = std::max(npb, wcolsum_nparts(m.c_out[l]));
  }
  t.pw = cv.take<float>(3 * npw * maxC);        // up to three linears per site
  t.pb = cv.take<float>(3 * npb * maxC);
  t.dbt = cv.take<float>(maxM);
  const int64_t nc = colstat_nparts(T);
  t.amax = cv.take<float>(nc * maxM);
  t.csum = cv.take<double>(nc * maxM);
  // partial products of the K-split forward and input-gradient products
  // (llama_mm takes the same decisions)
  int64_t part = 0;
  const int64_t fwd[4][2] = {{m.Mqkv, D}, {D, m.Hd}, {2 * F, D}, {D, F}};   // (N = c_out, K = c_in)
  for (const auto& f : fwd) {
    const int sf = gemm_mn_splits(false, false, T, f[0], f[1], f[1], f[1]);
    if (sf > 1) part = std::max(part, sf * T * f[0]);
    const int sd = gemm_mn_splits(false, true, T, f[1], f[0], f[0], f[1]);
    if (sd > 1) part = std::max(part, sd * T * f[1]);
  }
  t.part = cv.take<float>(part);
  if (w) *w = t;
  return cv.off + 256;
}

// C [M, N] fp32 = A B with the K split gemm_mn_splits models fastest: the
// parts go to w.part and are summed into C in fixed order (deterministic).
oq_status llama_mm(const LlamaWs& w, const void* A, bool a_mn, const void* B, bool b_mn,
                   int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, float* C,
                   hipStream_t st, const char* what) {
  const int sp = gemm_mn_splits(a_mn, b_mn, M, N, K, lda, ldb);
  if (sp > 1) {
    OQ_HIP(gemm_f32out_mn(A, a_mn, B, b_mn, M, N, K, lda, ldb, w.part, N, st, sp, M * N), what);
    OQ_HIP(sum_partials_to(w.part, C, M * N, sp, M * N, st), what);
  } else {
    OQ_HIP(gemm_f32out_mn(A, a_mn, B, b_mn, M, N, K, lda, ldb, C, N, st), what);
  }
  return OQ_OK;
}

}  // namespace

extern "C" {

oq_status oq_llama_workspace_size(const oq_llama_desc* d, size_t* bytes) {
  OQ_REQ(bytes, "bytes is required");
  LlamaDims m;
  oq_status e = llama_dims(d, &m);
  if (e != OQ_OK) return e;
  *bytes = llama_carve(m, nullptr, nullptr);
  return OQ_OK;
}

}  // extern "C"

namespace {

// The quantised (or full-precision) forward of the block into the workspace,
// up to h2.  Returns the LWC'd weights and the site tensors the backward reads.
oq_status llama_forward(const LlamaDims& m, const oq_llama_desc* d, const void* h0,
                        const oq_llama_params* p, bool quant, const LlamaWs& w, hipStream_t st) {
  const int64_t T = m.T, D = m.D, F = m.F;
  const bool let = quant && m.let;
  const int ab = quant ? m.ab : 16;
  const bool sym = quant && m.sym;
  const float* s1 = let ? p->s[0] : nullptr;
  const float* d1 = let ? p->delta[0] : nullptr;
  // LWC'd weights of the linears stacked per site (or the plain weights)
  auto weights = [&](int l0, int l1, void* dst) -> oq_status {
    int64_t off = 0;
    for (int l = l0; l < l1; ++l) {
      const int k = L_SITE[l];
      const float* s = let && k < 3 ? p->s[k] : nullptr;
      char* out = static_cast<char*>(dst) + off * m.c_in[l] * 2;
      if (quant) {
        ProfScope ps(PK_LWC_FWD, st, double(m.c_out[l]) * m.c_in[l] * 4);
        OQ_HIP(lwc_fwd(p->W[l], true, m.c_out[l], m.c_in[l], s, p->gamma_logit[l], p->beta_logit[l],
                       d->w_bits[l], d->w_group[l], out, true, nullptr, nullptr, nullptr, st),
               "lwc_fwd");
      } else {
        OQ_HIP(hipMemcpyAsync(out, p->W[l], size_t(m.c_out[l] * m.c_in[l]) * 2,
                              hipMemcpyDeviceToDevice, st),
               "weight copy");
      }
      off += m.c_out[l];
    }
    return OQ_OK;
  };
  auto biases = [&](int l0, int l1, float* bt) -> oq_status {
    int64_t off = 0;
    for (int l = l0; l < l1; ++l) {
      const int k = L_SITE[l];
      OQ_HIP(let_fold(p->W[l], true, nullptr, m.c_out[l], m.c_in[l], nullptr, p->delta[k], nullptr,
                      false, bt + off, st),
             "let_fold");
      off += m.c_out[l];
    }
    return OQ_OK;
  };
  auto product = [&](const void* x, const void* wt, int64_t M, int64_t K, float* out) -> oq_status {
    ProfScope ps(PK_GEMM_FWD, st, 2.0 * double(T) * M * K);
    return llama_mm(w, x, false, wt, false, T, M, K, K, K, out, st, "forward product");
  };
  oq_status e;
  // ---- attention half
  OQ_HIP(rmsnorm_fwd(h0, true, p->norm1, T, D, d->norm_eps, w.x1, w.rstd1, st), "rmsnorm");
  {
    ProfScope ps(PK_ACT_FWD, st, double(T) * D * 6);
    OQ_HIP(act_fwd(w.x1, false, T, D, ab, s1, d1, w.xh1, true, nullptr, nullptr, nullptr, st, sym),
           "act_fwd site 1");
  }
  if ((e = weights(0, 3, w.wqkv)) != OQ_OK) return e;
  if (let && (e = biases(0, 3, w.bt_qkv)) != OQ_OK) return e;
  if ((e = product(w.xh1, w.wqkv, m.Mqkv, D, w.qkv)) != OQ_OK) return e;
  OQ_HIP(rope_table(int(m.S), int(m.dh), d->rope_base, w.rope, st), "RoPE table");
  OQ_HIP(qkv_post(w.qkv, let ? w.bt_qkv : nullptr, T, int(m.S), int(m.H), int(m.Hkv), int(m.dh),
                  w.rope, let ? p->s_a : nullptr, w.qt, w.kt, w.vv, st),
         "qkv epilogue");
  {
    ProfScope ps(PK_ACT_FWD, st, double(T) * m.Mqkv * 6);
    OQ_HIP(act_fwd(w.qt, false, T, m.Hd, ab, nullptr, nullptr, w.qh, true, nullptr, nullptr, nullptr,
                   st, sym),
           "act_fwd Q");
    OQ_HIP(act_fwd(w.kt, false, T, m.Kd, ab, nullptr, nullptr, w.kh, true, nullptr, nullptr, nullptr,
                   st, sym),
           "act_fwd K");
    OQ_HIP(act_fwd(w.vv, false, T, m.Kd, ab, nullptr, nullptr, w.vh, true, nullptr, nullptr, nullptr,
                   st, sym),
           "act_fwd V");
  }
  {
    ProfScope ps(PK_ATTN_FWD, st, 2.0 * double(T) * m.S * m.Hd);   // causal: QK^T and PV, half each
    OQ_HIP(attn_fwd(w.qh, w.kh, w.vh, T, int(m.S), int(m.H), int(m.Hkv), int(m.dh),
                    quant ? m.pb : 16, w.att, w.lse, w.pstat, st),
           "attention");
  }
  {
    ProfScope ps(PK_ACT_FWD, st, double(T) * m.Hd * 6);
    OQ_HIP(act_fwd(w.att, false, T, m.Hd, ab, let ? p->s[1] : nullptr, let ? p->delta[1] : nullptr,
                   w.xh2, true, nullptr, nullptr, nullptr, st, sym),
           "act_fwd site 2");
  }
  if ((e = weights(3, 4, w.wo)) != OQ_OK) return e;
  if (let && (e = biases(3, 4, w.bt_o)) != OQ_OK) return e;
  if ((e = product(w.xh2, w.wo, D, m.Hd, w.o)) != OQ_OK) return e;
  OQ_HIP(resid_add(h0, true, w.o, let ? w.bt_o : nullptr, T, D, w.h1, st), "residual 1");
  // ---- feed-forward half
  OQ_HIP(rmsnorm_fwd(w.h1, false, p->norm2, T, D, d->norm_eps, w.x3, w.rstd2, st), "rmsnorm 2");
  {
    ProfScope ps(PK_ACT_FWD, st, double(T) * D * 6);
    OQ_HIP(act_fwd(w.x3, false, T, D, ab, let ? p->s[2] : nullptr, let ? p->delta[2] : nullptr,
                   w.xh3, true, nullptr, nullptr, nullptr, st, sym),
           "act_fwd site 3");
  }
  if ((e = weights(4, 6, w.wgu)) != OQ_OK) return e;
  if (let && (e = biases(4, 6, w.bt_gu)) != OQ_OK) return e;
  if ((e = product(w.xh3, w.wgu, 2 * F, D, w.gu)) != OQ_OK) return e;
  OQ_HIP(silu_mul(w.gu, let ? w.bt_gu : nullptr, T, F, w.x4, st), "silu");
  {
    ProfScope ps(PK_ACT_FWD, st, double(T) * F * 6);
    OQ_HIP(act_fwd(w.x4, false, T, F, ab, nullptr, nullptr, w.xh4, true, nullptr, nullptr, nullptr,
                   st, sym),
           "act_fwd site 4");
  }
  if ((e = weights(6, 7, w.wd)) != OQ_OK) return e;
  if ((e = product(w.xh4, w.wd, D, F, w.dn)) != OQ_OK) return e;
  OQ_HIP(resid_add(w.h1, false, w.dn, nullptr, T, D, w.h2, st), "residual 2");
  return OQ_OK;
}

oq_status llama_check(const LlamaDims& m, const oq_llama_params* p, bool quant) {
  OQ_REQ(p, "params are required");
  for (int l = 0; l < NL; ++l) {
    OQ_REQ(p->W[l] && aligned16(p->W[l]), "W[%d] missing or misaligned", l);
    if (quant) OQ_REQ(p->gamma_logit[l] && p->beta_logit[l], "logits of linear %d missing", l);
  }
  OQ_REQ(p->norm1 && p->norm2, "norm gains are required");
  if (quant && m.let) {
    for (int k = 0; k < 3; ++k)
      OQ_REQ(p->s[k] && p->delta[k] && aligned16(p->s[k]) && aligned16(p->delta[k]),
             "LET site %d: s and delta (16-byte aligned) are required", k);
    OQ_REQ(p->s_a, "s_a is required with LET");
  }
  return OQ_OK;
}

}  // namespace

extern "C" {

oq_status oq_attention_fwd(const void* Q, const void* K, const void* V, int64_t T, int64_t S,
                           int H, int Hkv, int head_dim, int softmax_bits, float* O, float* LSE,
                           float* pstat, hipStream_t st) {
  OQ_REQ(Q && K && V && O && LSE, "Q, K, V, O and LSE are required");
  OQ_REQ(aligned16(Q) && aligned16(K) && aligned16(V) && aligned16(O), "pointers must be 16-byte aligned");
  OQ_REQ(softmax_bits == 16 || (softmax_bits >= 2 && softmax_bits <= 8), "softmax bits %d",
         softmax_bits);
  OQ_REQ(softmax_bits == 16 || (pstat && aligned16(pstat)),
         "pstat (16-byte aligned) is required with softmax quantisation");
  if (!attn_supported(T, int(S), H, Hkv, head_dim) || S > INT32_MAX)
    return fail(OQ_ERR_UNSUPPORTED, "attention shape T=%lld S=%lld H=%d Hkv=%d d=%d", (long long)T,
                (long long)S, H, Hkv, head_dim);
  // causal: QK^T and PV, half each (a quantised softmax recomputes QK^T once more)
  ProfScope ps(PK_ATTN_FWD, st, 2.0 * double(T) * S * H * head_dim);
  OQ_HIP(attn_fwd(Q, K, V, T, int(S), H, Hkv, head_dim, softmax_bits, O, LSE, pstat, st), "attention");
  return OQ_OK;
}

oq_status oq_attention_bwd_workspace_size(int64_t T, int H, int softmax_bits, size_t* bytes) {
  OQ_REQ(bytes && T >= 0 && H > 0, "bad arguments");
  *bytes = attn_bwd_ws_floats(T, H, softmax_bits) * 4 + 256;
  return OQ_OK;
}

oq_status oq_attention_bwd(const void* Q, const void* K, const void* V, const void* dO,
                           const float* LSE, const float* pstat, int64_t T, int64_t S, int H,
                           int Hkv, int head_dim, int softmax_bits, float* dQ, float* dK, float* dV,
                           void* ws, size_t ws_bytes, hipStream_t st) {
  OQ_REQ(Q && K && V && dO && LSE && dQ && dK && dV, "every tensor is required");
  OQ_REQ(aligned16(Q) && aligned16(K) && aligned16(V) && aligned16(dO),
         "pointers must be 16-byte aligned");
  OQ_REQ(softmax_bits == 16 || (softmax_bits >= 2 && softmax_bits <= 8), "softmax bits %d",
         softmax_bits);
  OQ_REQ(softmax_bits == 16 || (pstat && aligned16(pstat)),
         "pstat (16-byte aligned) is required with softmax quantisation");
  OQ_REQ(!ws || aligned16(ws), "workspace must be 16-byte aligned");
  if (!attn_supported(T, int(S), H, Hkv, head_dim) || S > INT32_MAX)
    return fail(OQ_ERR_UNSUPPORTED, "attention shape T=%lld S=%lld H=%d Hkv=%d d=%d", (long long)T,
                (long long)S, H, Hkv, head_dim);
  size_t need = 0;
  oq_attention_bwd_workspace_size(T, H, softmax_bits, &need);
  if (!ws || ws_bytes < need) return fail(OQ_ERR_WORKSPACE, "workspace of %zu bytes needed", need);
  ProfScope ps(PK_ATTN_BWD, st, 4.0 * double(T) * S * H * head_dim);   // dV, dP, dQ, dK (causal halves)
  OQ_HIP(attn_bwd(Q, K, V, dO, LSE, pstat, T, int(S), H, Hkv, head_dim, softmax_bits,
                  static_cast<float*>(ws), dQ, dK, dV, st),
         "attention backward");
  return OQ_OK;
}

oq_status oq_llama_block_forward(const oq_llama_desc* d, const void* h0,
                                 const oq_llama_params* p, int quantised, void* h_out, void* ws,
                                 size_t ws_bytes, hipStream_t st) {
  LlamaDims m;
  oq_status e = llama_dims(d, &m);
  if (e != OQ_OK) return e;
  if ((e = llama_check(m, p, quantised != 0)) != OQ_OK) return e;
  OQ_REQ(h0 && h_out && aligned16(h0) && aligned16(h_out) && h0 != h_out, "h0, h_out");
  const size_t need = llama_carve(m, nullptr, nullptr);
  if (!ws || ws_bytes < need)
    return fail(OQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws_bytes);
  LlamaWs w;
  llama_carve(m, static_cast<char*>(ws), &w);
  if ((e = llama_forward(m, d, h0, p, quantised != 0, w, st)) != OQ_OK) return e;
  OQ_HIP(scale_to_bf16(w.h2, nullptr, m.T, m.D, h_out, st), "output");
  return OQ_OK;
}

oq_status oq_llama_block_step(const oq_llama_desc* d, const void* h0, const void* target,
                              const oq_llama_params* p, const oq_llama_grads* g,
                              const oq_llama_optim* opt, float* loss, void* ws, size_t ws_bytes,
                              hipStream_t st) {
  LlamaDims m;
  oq_status e = llama_dims(d, &m);
  if (e != OQ_OK) return e;
  if ((e = llama_check(m, p, true)) != OQ_OK) return e;
  OQ_REQ(h0 && target && aligned16(h0) && aligned16(target) && loss && g,
         "h0, target, grads and loss are required");
  for (int l = 0; l < NL; ++l)
    OQ_REQ(g->d_gamma_logit[l] && g->d_beta_logit[l], "gradients of linear %d missing", l);
  if (m.let) {
    for (int k = 0; k < 3; ++k) OQ_REQ(g->d_s[k] && g->d_delta[k], "LET gradients of site %d", k);
    OQ_REQ(g->d_s_a, "d_s_a is required with LET");
  }
  if (opt) {
    OQ_REQ(opt->step >= 1, "optim step must be >= 1");
    for (int l = 0; l < NL; ++l)
      OQ_REQ(opt->m_gamma[l] && opt->v_gamma[l] && opt->m_beta[l] && opt->v_beta[l],
             "AdamW state of linear %d missing", l);
    if (m.let) {
      for (int k = 0; k < 3; ++k)
        OQ_REQ(opt->m_s[k] && opt->v_s[k] && opt->m_delta[k] && opt->v_delta[k],
               "AdamW state of site %d missing", k);
      OQ_REQ(opt->m_s_a && opt->v_s_a, "AdamW state of s_a missing");
    }
  }
  const size_t need = llama_carve(m, nullptr, nullptr);
  if (!ws || ws_bytes < need)
    return fail(OQ_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need, ws_bytes);
  LlamaWs w;
  llama_carve(m, static_cast<char*>(ws), &w);
  const int64_t T = m.T, D = m.D, F = m.F;
  const bool let = m.let;
  const int ab = m.ab;
  const bool sym = m.sym;
  if ((e = llama_forward(m, d, h0, p, true, w, st)) != OQ_OK) return e;
  {
    ProfScope ps(PK_OTHER, st, double(T) * D * 12);
    OQ_HIP(block_loss(w.h2, target, T, D, w.dh2, w.dh2_16, w.rows, loss, st), "loss");
  }
  const int64_t npa = act_bwd_nparts(T);
  // The weight side of each site runs on a side stream sw, forked from st
  // once the site's dY is ready and joined back where its outputs are read
  // (the LET finish, and before AdamW).  Its buffers (dW, the ds and bias
  // partials, the column sums) are its own; the next site's weight side is
  // forked after this site's LET finish, which reads them.
  BlockSide* sd = nullptr;
  OQ_HIP(block_side(&sd), "side stream");
  const hipStream_t sw = sd->s;
  // dX^ = dY W^ (on st) and dW^ = dY^T X^ (on sw) of the linears [l0, l1)
  // stacked on one site, then their LWC backward (with LET: the weight-path
  // ds partials and the bias-path partials of ddelta); dy16 bf16 [T, M],
  // xh bf16 [T, C].
  int64_t npw = 0, npb = 0;
  auto linears_bwd = [&](int l0, int l1, const void* dy16, const void* wst, const void* xh,
                         float* dxh) -> oq_status {
    const int k = L_SITE[l0];
    const int64_t C = m.c_in[l0];
    int64_t M = 0;
    for (int l = l0; l < l1; ++l) M += m.c_out[l];
    const bool let_site = let && k < 3;
    OQ_HIP(hipEventRecord(sd->fork, st), "fork");
    OQ_HIP(hipStreamWaitEvent(sw, sd->fork, 0), "fork");
    {
      ProfScope ps(PK_GEMM_DGRAD, st, 2.0 * double(T) * M * C);
      oq_status e2 = llama_mm(w, dy16, false, wst, true, T, C, M, M, C, dxh, st, "input gradient");
      if (e2 != OQ_OK) return e2;
    }
    {
      ProfScope ps(PK_GEMM_WGRAD, sw, 2.0 * double(T) * M * C);
      OQ_HIP(gemm_f32out_mn(dy16, true, xh, true, M, C, T, M, C, w.dW, C, sw), "weight gradient");
    }
    npw = npb = 0;
    int64_t off = 0;
    for (int l = l0; l < l1; ++l) {
      ProfScope ps(PK_LWC_BWD, sw, double(m.c_out[l]) * C * 6);
      OQ_HIP(lwc_bwd(p->W[l], true, m.c_out[l], C, let_site ? p->s[k] : nullptr, p->gamma_logit[l],
                     p->beta_logit[l], d->w_bits[l], d->w_group[l], w.dW + off * C,
                     g->d_gamma_logit[l], g->d_beta_logit[l], nullptr,
                     let_site ? w.pw + npw * C : nullptr, sw),
             "lwc_bwd");
      if (let_site) npw += lwc_bwd_nparts(m.c_out[l]);
      off += m.c_out[l];
    }
    if (let_site) {
      ProfScope ps(PK_OTHER, sw, double(T) * M * 2 + double(M) * C * 2);
      const int64_t nc = colstat_nparts(T);
      OQ_HIP(colstat(dy16, true, T, M, w.amax, w.csum, sw), "bias-path column sums");
      OQ_HIP(colsum_finish(w.csum, nc, M, w.dbt, sw), "bias-path finish");
      off = 0;
      for (int l = l0; l < l1; ++l) {
        OQ_HIP(wcolsum(p->W[l], true, m.c_out[l], C, w.dbt + off, w.pb + npb * C, sw), "bias path");
        npb += wcolsum_nparts(m.c_out[l]);
        off += m.c_out[l];
      }
    }
    OQ_HIP(hipEventRecord(sd->join, sw), "join");
    return OQ_OK;
  };
  // through Q_a and the LET transform of site k: dxt = dL/dX~ (and the LET
  // gradients of the site)
  auto site_bwd = [&](int k, const float* x, int64_t C, const float* dxh, float* dxt) -> oq_status {
    const bool let_site = let && k < 3;
    {
      ProfScope ps(PK_ACT_BWD, st, double(T) * C * 8);
      OQ_HIP(act_bwd(x, false, T, C, ab, let_site ? p->s[k] : nullptr,
                     let_site ? p->delta[k] : nullptr, dxh, dxt, let_site ? w.psx : nullptr,
                     let_site ? w.ps1 : nullptr, st, sym),
             "act_bwd");
    }
    if (let_site) {
      OQ_HIP(hipStreamWaitEvent(st, sd->join, 0), "join");
      OQ_HIP(let_grad_finish(C, p->s[k], w.pw, npw, w.psx, w.ps1, npa, w.pb, npb, g->d_s[k],
                             g->d_delta[k], st),
             "LET finish");
    }
    return OQ_OK;
  };
  // ---- feed-forward half
  if ((e = linears_bwd(6, 7, w.dh2_16, w.wd, w.xh4, w.dxh)) != OQ_OK) return e;
  if ((e = site_bwd(3, w.x4, F, w.dxh, w.dxt)) != OQ_OK) return e;
  OQ_HIP(silu_mul_bwd(w.gu, w.dxt, T, F, w.dgu16, st), "silu backward");
  if ((e = linears_bwd(4, 6, w.dgu16, w.wgu, w.xh3, w.dxh)) != OQ_OK) return e;
  if ((e = site_bwd(2, w.x3, D, w.dxh, w.dxt)) != OQ_OK) return e;
  OQ_HIP(rmsnorm_bwd(w.h1, false, p->norm2, w.rstd2, w.dxt, let ? p->s[2] : nullptr, w.dh2, T, D,
                     w.dh1, st),
         "rmsnorm backward");
  OQ_HIP(scale_to_bf16(w.dh1, nullptr, T, D, w.dh1_16, st), "dh1");
  // ---- attention half
  if ((e = linears_bwd(3, 4, w.dh1_16, w.wo, w.xh2, w.dxh)) != OQ_OK) return e;
  if ((e = site_bwd(1, w.att, m.Hd, w.dxh, w.dxt)) != OQ_OK) return e;
  OQ_HIP(scale_to_bf16(w.dxt, let ? p->s[1] : nullptr, T, m.Hd, w.datt16, st), "dO");
  {
    ProfScope ps(PK_ATTN_BWD, st, 4.0 * double(T) * m.S * m.Hd);   // dV, dP, dQ, dK (causal halves)
    OQ_HIP(attn_bwd(w.qh, w.kh, w.vh, w.datt16, w.lse, w.pstat, T, int(m.S), int(m.H),
                    int(m.Hkv), int(m.dh), m.pb, w.Dl, w.dQ, w.dK, w.dV, st),
           "attention backward");
  }
  {
    ProfScope ps(PK_ACT_BWD, st, double(T) * m.Mqkv * 8);
    OQ_HIP(act_bwd(w.qt, false, T, m.Hd, ab, nullptr, nullptr, w.dQ, w.dqt, let ? w.psxq : nullptr,
                   let ? w.ps1 : nullptr, st, sym),
           "act_bwd Q");
    OQ_HIP(act_bwd(w.kt, false, T, m.Kd, ab, nullptr, nullptr, w.dK, w.dkt, let ? w.psxk : nullptr,
                   let ? w.ps1 : nullptr, st, sym),
           "act_bwd K");
    OQ_HIP(act_bwd(w.vv, false, T, m.Kd, ab, nullptr, nullptr, w.dV, w.dvt, nullptr, nullptr, st, sym),
           "act_bwd V");
  }
  if (let)
    OQ_HIP(sa_grad_finish(w.psxq, npa, w.psxk, npa, int(m.H), int(m.Hkv), int(m.dh), p->s_a,
                          g->d_s_a, st),
           "s_a finish");
  OQ_HIP(qkv_post_bwd(w.dqt, w.dkt, w.dvt, T, int(m.S), int(m.H), int(m.Hkv), int(m.dh), w.rope,
                      let ? p->s_a : nullptr, w.dqkv16, st),
         "qkv epilogue backward");
  if ((e = linears_bwd(0, 3, w.dqkv16, w.wqkv, w.xh1, w.dxh)) != OQ_OK) return e;
  if ((e = site_bwd(0, w.x1, D, w.dxh, w.dxt)) != OQ_OK) return e;
  // the last weight side (the clipping-logit gradients of q, k, v) back on st
  OQ_HIP(hipStreamWaitEvent(st, sd->join, 0), "join");
  // ---- AdamW over every trained tensor
  if (opt) {
    const AdamCoef cl = adam_coef(opt->lr_lwc, opt->beta1, opt->beta2, opt->eps, opt->wd, opt->step);
    const AdamCoef ce = adam_coef(opt->lr_let, opt->beta1, opt->beta2, opt->eps, opt->wd, opt->step);
    ProfScope ps(PK_OTHER, st, 0);
    AdamList L{};
    auto add = [&](float* pp, const float* gg, float* mm, float* vv, int64_t n, int set) {
      L.p[L.n] = pp; L.g[L.n] = gg; L.m[L.n] = mm; L.v[L.n] = vv; L.len[L.n] = n; L.set[L.n] = set;
      ++L.n;
    };
    for (int l = 0; l < NL; ++l) {
      const int64_t n = m.c_out[l] * (m.c_in[l] / d->w_group[l]);
      add(p->gamma_logit[l], g->d_gamma_logit[l], opt->m_gamma[l], opt->v_gamma[l], n, 0);
      add(p->beta_logit[l], g->d_beta_logit[l], opt->m_beta[l], opt->v_beta[l], n, 0);
    }
    if (let) {
      const int64_t cs[3] = {D, m.Hd, D};
      for (int k = 0; k < 3; ++k) {
        add(p->s[k], g->d_s[k], opt->m_s[k], opt->v_s[k], cs[k], 1);
        add(p->delta[k], g->d_delta[k], opt->m_delta[k], opt->v_delta[k], cs[k], 1);
      }
      add(p->s_a, g->d_s_a, opt->m_s_a, opt->v_s_a, m.Kd, 1);
    }
    OQ_HIP(adamw_multi(L, cl, ce, st), "adamw");
  }
  return OQ_OK;
}

oq_status oq_llama_calibrate(const oq_llama_desc* d, int n_samples, int epochs,
                             const void* const* h0, const void* const* target,
                             const oq_llama_params* p, const oq_llama_grads* g,
                             const oq_llama_optim* opt, float* losses, void* ws, size_t ws_bytes,
                             hipStream_t st) {
  OQ_REQ(d && h0 && target && p && g && opt && losses,
         "desc, h0, target, params, grads, optim and losses are required");
  OQ_REQ(n_samples >= 1 && epochs >= 1, "need n_samples >= 1 and epochs >= 1 (got %d, %d)",
         n_samples, epochs);
  OQ_REQ(opt->step >= 1 && int64_t(opt->step) + int64_t(epochs) * n_samples - 1 <= INT32_MAX,
         "optim step %d out of range for %d steps", opt->step, epochs * n_samples);
  // every sample's pointers before the first launch; the first step checks the rest
  for (int j = 0; j < n_samples; ++j)
    OQ_REQ(h0[j] && target[j] && aligned16(h0[j]) && aligned16(target[j]),
           "sample %d: h0 or target missing or misaligned", j);
  oq_llama_optim o = *opt;
  for (int ep = 0; ep < epochs; ++ep)
    for (int j = 0; j < n_samples; ++j) {
      const int64_t i = int64_t(ep) * n_samples + j;
      o.step = int(opt->step + i);
      const oq_status e = oq_llama_block_step(d, h0[j], target[j], p, g, &o, losses + i, ws,
                                              ws_bytes, st);
      if (e != OQ_OK) return e;
    }
  return OQ_OK;
}

}  // extern "C"
