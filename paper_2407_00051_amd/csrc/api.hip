// C ABI of libsagips.so (declared in include/sagips.h): context, argument
// validation, workspace, kernel timing and dispatch to the kernel files.
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/sagips.h"
#include "kernels.hpp"

using namespace sagips;

// Workspace of sagips_disc_fwd_bwd_noalloc: one array per device, which every
// call of that entry point on the device shares (calls that overlap on one
// device race on it).  In host code `scratch` names a host-side stand-in, not
// device memory: kernels only ever receive the device address taken with
// hipGetSymbolAddress in sagips_create.
constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

thread_local std::string g_create_error = "no error";

// Device address of `scratch` per device (taken once, with that device current).
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};
hipError_t g_scratch_err[kMaxDevices] = {};

hipError_t scratch_address(int dev, char** ptr) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev] && g_scratch_err[dev] == hipSuccess) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e == hipSuccess && p) g_scratch_ptr[dev] = static_cast<char*>(p);
    else g_scratch_err[dev] = e != hipSuccess ? e : hipErrorInvalidSymbol;
  }
  *ptr = g_scratch_ptr[dev];
  return g_scratch_err[dev];
}

struct EventTimer final : Timer {
  struct Rec {
    const char* name;
    hipEvent_t a, b;
  };
  hipStream_t stream = nullptr;
  std::vector<hipEvent_t> pool;
  std::vector<Rec> recs;
  const char* open_name = nullptr;
  hipEvent_t open_a = nullptr;

  hipEvent_t take() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
  void begin(const char* name) override {
    open_name = name;
    open_a = take();
    if (open_a) (void)hipEventRecord(open_a, stream);
  }
  void end() override {
    hipEvent_t b = take();
    if (open_a && b) {
      (void)hipEventRecord(b, stream);
      recs.push_back({open_name, open_a, b});
    }
    open_a = nullptr;
  }
  void release() {
    for (auto& r : recs) {
      pool.push_back(r.a);
      pool.push_back(r.b);
    }
    recs.clear();
  }
  ~EventTimer() override {
    release();
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
  }
};

}  // namespace

struct sagips_ctx {
  int device = 0;
  hipStream_t stream = nullptr;
  int n_cu = 0;
  void* ws = nullptr;
  size_t ws_cap = 0;
  std::string err = "no error";
  bool timing = false;
  int bf16_chunk_rows = 0;      // 0: the library's default
  EventTimer timer;
};

namespace {

sagips_status fail(sagips_ctx* c, sagips_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  if (c) c->err = buf;
  else g_create_error = buf;
  return s;
}

sagips_status hip_fail(sagips_ctx* c, hipError_t e, const char* what) {
  return fail(c, SAGIPS_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) == hipSuccess && prev != dev) (void)hipSetDevice(dev);
    else prev = -1;
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

Timer* timer_of(sagips_ctx* c) { return c->timing ? &c->timer : nullptr; }

sagips_status ensure_ws(sagips_ctx* c, size_t bytes) {
  if (bytes <= c->ws_cap) return SAGIPS_OK;
  if (c->ws) {
    hipError_t e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize before workspace growth");
    (void)hipFree(c->ws);
    c->ws = nullptr;
    c->ws_cap = 0;
  }
  size_t want = (bytes + ((size_t)1 << 20) - 1) & ~(((size_t)1 << 20) - 1);
  if (hipMalloc(&c->ws, want) != hipSuccess) {
    (void)hipGetLastError();
    c->ws = nullptr;
    return fail(c, SAGIPS_E_NOMEM, "workspace allocation of %zu bytes failed", want);
  }
  c->ws_cap = want;
  return SAGIPS_OK;
}

// Where a call's workspace comes from: the context's (grown on demand with
// hipMalloc), or a fixed device buffer that is never reallocated.
struct WsFrom {
  char* fixed = nullptr;   // fixed buffer on the context's device, or NULL
  size_t fixed_cap = 0;
};

sagips_status acquire_ws(sagips_ctx* c, const WsFrom& from, size_t bytes, char** ws) {
  if (from.fixed) {
    if (bytes > from.fixed_cap)
      return fail(c, SAGIPS_E_INVAL,
                  "this call needs %zu bytes of workspace; the no-allocation entry point has %zu (use the allocating call)",
                  bytes, from.fixed_cap);
    *ws = from.fixed;
    return SAGIPS_OK;
  }
  sagips_status s = ensure_ws(c, bytes);
  if (s == SAGIPS_OK) *ws = static_cast<char*>(c->ws);
  return s;
}

sagips_status check_source(sagips_ctx* c, const sagips_source* s, const char* name) {
  if (!s) return fail(c, SAGIPS_E_INVAL, "%s is NULL", name);
  if (!s->theta) return fail(c, SAGIPS_E_INVAL, "%s.theta is NULL", name);
  if (((uintptr_t)s->theta) & 3u) return fail(c, SAGIPS_E_INVAL, "%s.theta is not 4-byte aligned", name);
  if (s->n_theta < 1 || s->n_theta > 65535) return fail(c, SAGIPS_E_INVAL, "%s.n_theta = %d outside [1, 65535]", name, s->n_theta);
  if (s->d != 2 && s->d != 3) return fail(c, SAGIPS_E_INVAL, "%s.d = %d, must be 2 or 3", name, s->d);
  if (s->events_per_theta < 1) return fail(c, SAGIPS_E_INVAL, "%s.events_per_theta must be >= 1", name);
  const int64_t N = (int64_t)s->n_theta * s->events_per_theta;
  if (s->events_per_theta > ((int64_t)1 << 31) || N >= ((int64_t)1 << 31))
    return fail(c, SAGIPS_E_INVAL, "%s: n_theta * events_per_theta = %lld must be < 2^31", name, (long long)N);
  if (s->counter_base > UINT64_MAX - (uint64_t)N) return fail(c, SAGIPS_E_INVAL, "%s: counter_base + N overflows 2^64", name);
  return SAGIPS_OK;
}

int64_t source_events(const sagips_source* s) { return (int64_t)s->n_theta * s->events_per_theta; }

// bf16 path: one chunked launcher; dL_G/dtheta by the reduction kernel over dL_G/dx.
sagips_status disc_bf16(sagips_ctx* c, const sagips_mlp* D, const float* fake_x, const sagips_source* fake_src,
                        int64_t n_fake, const float* real_x, int64_t n_real, const sagips_disc_out* out, int d,
                        const WsFrom& from, Timer* tm) {
  const char* why = nullptr;
  if (!disc_bf16_supported(*D, d, &why)) return fail(c, SAGIPS_E_UNSUPPORTED, "%s", why);
  SourceArgs sa{};
  if (fake_src) sa = source_args(*fake_src);
  DiscArgs a;
  a.D = D;
  a.fake_x = fake_x;
  a.fake_src = fake_src ? &sa : nullptr;
  a.n_fake = n_fake;
  a.real_x = real_x;
  a.n_real = n_real;
  a.d = d;
  a.chunk_rows = c->bf16_chunk_rows;
  sagips_disc_out o2 = *out;
  o2.dLg_dtheta = nullptr;
  a.out = &o2;
  const size_t disc_ws = (disc_bf16_workspace(a, c->n_cu) + 255) & ~(size_t)255;
  size_t off_g = disc_ws, off_pg = disc_ws, total = disc_ws;
  const bool want_theta = out->dLg_dtheta != nullptr;
  if (want_theta) {
    off_pg = off_g + (((size_t)n_fake * d * sizeof(float) + 255) & ~(size_t)255);
    total = off_pg + param_grad_workspace(sa);
  }
  char* ws = nullptr;
  sagips_status s = acquire_ws(c, from, total, &ws);
  if (s != SAGIPS_OK) return s;
  if (want_theta && !o2.dLg_dx) o2.dLg_dx = reinterpret_cast<float*>(ws + off_g);
  hipError_t e = launch_disc_bf16(a, ws, c->n_cu, c->stream, tm);
  if (e != hipSuccess) return hip_fail(c, e, "disc_fwd_bwd (bf16) launch");
  if (want_theta) {
    e = launch_param_grad(sa, o2.dLg_dx, out->dLg_dtheta, nullptr, ws + off_pg, c->stream, tm);
    if (e != hipSuccess) return hip_fail(c, e, "param_grad launch");
  }
  return SAGIPS_OK;
}

sagips_status check_gen(sagips_ctx* c, const sagips_gen* G, const float* noise, int64_t k) {
  if (!G) return fail(c, SAGIPS_E_INVAL, "G is NULL");
  if (!noise) return fail(c, SAGIPS_E_INVAL, "noise is NULL");
  if (G->n_members < 1 || G->n_members > 65535) return fail(c, SAGIPS_E_INVAL, "n_members = %d outside [1, 65535]", G->n_members);
  if (G->n_layers < 2 || G->n_layers > SAGIPS_MAX_LAYERS)
    return fail(c, SAGIPS_E_INVAL, "n_layers = %d outside [2, %d]", G->n_layers, SAGIPS_MAX_LAYERS);
  for (int l = 0; l <= G->n_layers; ++l)
    if (G->width[l] < 1) return fail(c, SAGIPS_E_INVAL, "width[%d] < 1", l);
  for (int l = 0; l < G->n_layers; ++l) {
    if (!G->W[l] || !G->b[l]) return fail(c, SAGIPS_E_INVAL, "W[%d] or b[%d] is NULL", l, l);
    if (!aligned16(G->W[l]) || !aligned16(G->b[l])) return fail(c, SAGIPS_E_INVAL, "W[%d] or b[%d] is not 16-byte aligned", l, l);
  }
  if (k < 1 || k >= ((int64_t)1 << 30)) return fail(c, SAGIPS_E_INVAL, "k = %lld outside [1, 2^30)", (long long)k);
  const char* why = nullptr;
  if (!sagips::gen_supported(*G, &why)) return fail(c, SAGIPS_E_UNSUPPORTED, "%s", why);
  return SAGIPS_OK;
}

sagips_status check_bootstrap(sagips_ctx* c, const float* data, int64_t n_data, int d, int64_t n_out, float* out,
                              int64_t* idx_out) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  if (!data || !out) return fail(c, SAGIPS_E_INVAL, "data or out is NULL");
  if (d != 2 && d != 3) return fail(c, SAGIPS_E_INVAL, "d = %d, must be 2 or 3", d);
  if (n_data < 1 || n_data > ((int64_t)1 << 32)) return fail(c, SAGIPS_E_INVAL, "n_data = %lld outside [1, 2^32]", (long long)n_data);
  if (n_out < 1) return fail(c, SAGIPS_E_INVAL, "n_out must be >= 1");
  if (!aligned16(data) || !aligned16(out) || (idx_out && !aligned16(idx_out)))
    return fail(c, SAGIPS_E_INVAL, "data, out and idx_out must be 16-byte aligned");
  const uintptr_t d0 = reinterpret_cast<uintptr_t>(data), d1 = d0 + (uintptr_t)n_data * d * sizeof(float);
  const uintptr_t o0 = reinterpret_cast<uintptr_t>(out), o1 = o0 + (uintptr_t)n_out * d * sizeof(float);
  if (o0 < d1 && d0 < o1) return fail(c, SAGIPS_E_INVAL, "out overlaps data");
  if (idx_out) {
    const uintptr_t i0 = reinterpret_cast<uintptr_t>(idx_out), i1 = i0 + (uintptr_t)n_out * sizeof(int64_t);
    if ((i0 < d1 && d0 < i1) || (i0 < o1 && o0 < i1)) return fail(c, SAGIPS_E_INVAL, "idx_out overlaps data or out");
  }
  return SAGIPS_OK;
}

}  // namespace

extern "C" {

sagips_status sagips_create(sagips_ctx** out, int hip_device, void* hip_stream) {
  if (!out) return fail(nullptr, SAGIPS_E_INVAL, "out is NULL");
  *out = nullptr;
  int n = 0;
  hipError_t e = hipGetDeviceCount(&n);
  if (e != hipSuccess) return fail(nullptr, SAGIPS_E_HIP, "hipGetDeviceCount: %s", hipGetErrorString(e));
  if (hip_device < 0 || hip_device >= n) return fail(nullptr, SAGIPS_E_INVAL, "device %d outside [0, %d)", hip_device, n);
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, hip_device);
  if (e != hipSuccess) return fail(nullptr, SAGIPS_E_HIP, "hipGetDeviceProperties: %s", hipGetErrorString(e));
  if (strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(nullptr, SAGIPS_E_ARCH, "device %d is %s; this library is built for gfx950 only", hip_device, prop.gcnArchName);
  if (hip_device >= kMaxDevices) return fail(nullptr, SAGIPS_E_INVAL, "device %d beyond %d devices", hip_device, kMaxDevices);
  {
    // The scratch array's address on this device, for the no-allocation entry
    // point.  A failure is kept (and reported by that entry point); the other
    // calls do not use the array.
    DeviceGuard g(hip_device);
    char* p = nullptr;
    (void)scratch_address(hip_device, &p);
  }
  sagips_ctx* c = new (std::nothrow) sagips_ctx;
  if (!c) return fail(nullptr, SAGIPS_E_NOMEM, "context allocation failed");
  c->device = hip_device;
  c->stream = static_cast<hipStream_t>(hip_stream);
  c->n_cu = prop.multiProcessorCount;
  c->timer.stream = c->stream;
  *out = c;
  return SAGIPS_OK;
}

sagips_status sagips_destroy(sagips_ctx* c) {
  if (!c) return SAGIPS_OK;
  {
    DeviceGuard g(c->device);
    (void)hipStreamSynchronize(c->stream);
    if (c->ws) (void)hipFree(c->ws);
  }
  delete c;
  return SAGIPS_OK;
}

sagips_status sagips_set_stream(sagips_ctx* c, void* hip_stream) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  hipStream_t next = static_cast<hipStream_t>(hip_stream);
  if (next != c->stream) {
    // Work already queued on the old stream may still read the workspace the
    // next call reuses: the new stream waits for it (without blocking the host).
    DeviceGuard g(c->device);
    hipEvent_t ev = nullptr;
    hipError_t e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventCreateWithFlags");
    e = hipEventRecord(ev, c->stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(next, ev, 0);
    (void)hipEventDestroy(ev);
    if (e != hipSuccess) return hip_fail(c, e, "ordering the new stream after the old one");
  }
  c->stream = next;
  c->timer.stream = c->stream;
  return SAGIPS_OK;
}

sagips_status sagips_set_bf16_chunk_rows(sagips_ctx* c, int64_t rows) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  const int64_t max_rows = disc_bf16_max_chunk_rows();
  if (rows != 0 && (rows < 128 || rows > max_rows || rows % 128 != 0))
    return fail(c, SAGIPS_E_INVAL, "bf16 chunk rows = %lld: must be 0 (default) or a multiple of 128 in [128, %lld]",
                (long long)rows, (long long)max_rows);
  c->bf16_chunk_rows = (int)rows;
  return SAGIPS_OK;
}

const char* sagips_last_error(const sagips_ctx* c) { return c ? c->err.c_str() : g_create_error.c_str(); }

sagips_status sagips_set_timing(sagips_ctx* c, int enable) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  c->timing = enable != 0;
  return SAGIPS_OK;
}

int sagips_kernel_times(sagips_ctx* c, const char** names, int64_t* launches, double* total_ms, int cap) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  DeviceGuard g(c->device);
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(c, e, "hipStreamSynchronize");
  std::vector<std::pair<const char*, std::pair<int64_t, double>>> agg;
  for (auto& r : c->timer.recs) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) continue;
    size_t i = 0;
    for (; i < agg.size(); ++i)
      if (strcmp(agg[i].first, r.name) == 0) break;
    if (i == agg.size()) agg.push_back({r.name, {0, 0.0}});
    agg[i].second.first += 1;
    agg[i].second.second += ms;
  }
  c->timer.release();
  const int n = (int)agg.size();
  for (int i = 0; i < n && i < cap; ++i) {
    if (names) names[i] = agg[i].first;
    if (launches) launches[i] = agg[i].second.first;
    if (total_ms) total_ms[i] = agg[i].second.second;
  }
  return n;
}

sagips_status sagips_sample_events(sagips_ctx* c, const sagips_source* src, float* x_out, uint32_t* words_out) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  sagips_status s = check_source(c, src, "src");
  if (s != SAGIPS_OK) return s;
  if (!x_out && !words_out) return fail(c, SAGIPS_E_INVAL, "x_out and words_out are both NULL");
  if (x_out && !aligned16(x_out)) return fail(c, SAGIPS_E_INVAL, "x_out is not 16-byte aligned");
  if (words_out && !aligned16(words_out)) return fail(c, SAGIPS_E_INVAL, "words_out is not 16-byte aligned");
  DeviceGuard g(c->device);
  hipError_t e = launch_sample(source_args(*src), x_out, words_out, c->stream, timer_of(c));
  return e == hipSuccess ? SAGIPS_OK : hip_fail(c, e, "sample_events launch");
}

sagips_status sagips_param_grad(sagips_ctx* c, const sagips_source* src, sagips_critic critic, const float* dL_dx,
                                float* dL_dtheta, float* loss_out) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  sagips_status s = check_source(c, src, "src");
  if (s != SAGIPS_OK) return s;
  if (!dL_dtheta) return fail(c, SAGIPS_E_INVAL, "dL_dtheta is NULL");
  if (critic == SAGIPS_CRITIC_BUFFER) {
    if (!dL_dx) return fail(c, SAGIPS_E_INVAL, "critic BUFFER needs dL_dx");
    if (!aligned16(dL_dx)) return fail(c, SAGIPS_E_INVAL, "dL_dx is not 16-byte aligned");
    if (loss_out) return fail(c, SAGIPS_E_INVAL, "loss_out must be NULL with critic BUFFER");
  } else if (critic == SAGIPS_CRITIC_QUADRATIC) {
    if (dL_dx) return fail(c, SAGIPS_E_INVAL, "dL_dx must be NULL with critic QUADRATIC");
  } else {
    return fail(c, SAGIPS_E_INVAL, "unknown critic %d", (int)critic);
  }
  DeviceGuard g(c->device);
  const SourceArgs a = source_args(*src);
  s = ensure_ws(c, param_grad_workspace(a));
  if (s != SAGIPS_OK) return s;
  hipError_t e = launch_param_grad(a, critic == SAGIPS_CRITIC_BUFFER ? dL_dx : nullptr, dL_dtheta, loss_out, c->ws,
                                   c->stream, timer_of(c));
  return e == hipSuccess ? SAGIPS_OK : hip_fail(c, e, "param_grad launch");
}

}  // extern "C"

namespace {

// The discriminator step behind sagips_disc_fwd_bwd and its no-allocation
// variant: validation, then the fp32 or the bf16 path.
sagips_status disc_call(sagips_ctx* c, const sagips_mlp* D, const float* fake_x, const sagips_source* fake_src,
                        int64_t n_fake, const float* real_x, int64_t n_real, sagips_disc_out* out,
                        const WsFrom& from, Timer* tm) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  if (!D) return fail(c, SAGIPS_E_INVAL, "D is NULL");
  if (!out) return fail(c, SAGIPS_E_INVAL, "out is NULL");
  if (D->n_layers < 2 || D->n_layers > SAGIPS_MAX_LAYERS)
    return fail(c, SAGIPS_E_INVAL, "n_layers = %d outside [2, %d]", D->n_layers, SAGIPS_MAX_LAYERS);
  for (int l = 0; l < D->n_layers; ++l) {
    if (!D->W[l] || !D->b[l]) return fail(c, SAGIPS_E_INVAL, "W[%d] or b[%d] is NULL", l, l);
    if (!aligned16(D->W[l]) || !aligned16(D->b[l])) return fail(c, SAGIPS_E_INVAL, "W[%d] or b[%d] is not 16-byte aligned", l, l);
    if (D->width[l] < 1) return fail(c, SAGIPS_E_INVAL, "width[%d] < 1", l);
  }
  if (D->width[D->n_layers] != 1) return fail(c, SAGIPS_E_INVAL, "last width must be 1 (a logit)");
  if (D->features != SAGIPS_FEAT_IDENTITY && D->features != SAGIPS_FEAT_HD8 && D->features != SAGIPS_FEAT_PROXY2)
    return fail(c, SAGIPS_E_INVAL, "unknown features %d", D->features);
  if (D->precision != SAGIPS_F32 && D->precision != SAGIPS_BF16)
    return fail(c, SAGIPS_E_INVAL, "unknown precision %d", D->precision);
  if ((fake_x == nullptr) == (fake_src == nullptr))
    return fail(c, SAGIPS_E_INVAL, "exactly one of fake_x and fake_src must be given");
  if (!real_x) return fail(c, SAGIPS_E_INVAL, "real_x is NULL");
  if (!aligned16(real_x) || (fake_x && !aligned16(fake_x))) return fail(c, SAGIPS_E_INVAL, "event buffers must be 16-byte aligned");
  if (n_fake < 1 || n_real < 1) return fail(c, SAGIPS_E_INVAL, "n_fake and n_real must be >= 1");
  if (n_fake >= ((int64_t)1 << 30) || n_real >= ((int64_t)1 << 30))
    return fail(c, SAGIPS_E_INVAL, "n_fake and n_real must be < 2^30");
  int d;
  if (fake_src) {
    sagips_status s = check_source(c, fake_src, "fake_src");
    if (s != SAGIPS_OK) return s;
    if (n_fake != source_events(fake_src))
      return fail(c, SAGIPS_E_INVAL, "n_fake = %lld but fake_src holds %lld events", (long long)n_fake,
                  (long long)source_events(fake_src));
    d = fake_src->d;
  } else {
    d = D->features == SAGIPS_FEAT_IDENTITY ? D->width[0] : 3;
  }
  if (D->features == SAGIPS_FEAT_HD8 && (d != 3 || D->width[0] != 8))
    return fail(c, SAGIPS_E_INVAL, "HD8 features need d = 3 and width[0] = 8");
  if (D->features == SAGIPS_FEAT_PROXY2 && (d != 3 || D->width[0] != 2))
    return fail(c, SAGIPS_E_INVAL, "PROXY2 features need d = 3 and width[0] = 2");
  if (D->features == SAGIPS_FEAT_IDENTITY && D->width[0] != d)
    return fail(c, SAGIPS_E_INVAL, "IDENTITY features need width[0] == d (%d vs %d)", D->width[0], d);
  const bool any_dW = out->dW[0] != nullptr;
  for (int l = 0; l < D->n_layers; ++l)
    if ((out->dW[l] != nullptr) != any_dW || (out->db[l] != nullptr) != any_dW)
      return fail(c, SAGIPS_E_INVAL, "dW/db outputs must be given for all layers or none");
  if (out->dLg_dtheta && !fake_src) return fail(c, SAGIPS_E_INVAL, "dLg_dtheta needs a fake source");

  DeviceGuard g(c->device);
  const char* why = nullptr;
  if (D->precision == SAGIPS_BF16) return disc_bf16(c, D, fake_x, fake_src, n_fake, real_x, n_real, out, d, from, tm);
  if (!disc_f32_supported(*D, d, &why)) return fail(c, SAGIPS_E_UNSUPPORTED, "%s", why);

  // The in-kernel sampler lets a tile straddle at most two parameter rows;
  // with fewer events per row than a tile holds, sample first, run on the
  // buffer, and reduce dL/dtheta after.
  const bool fused_src = fake_src && (fake_src->events_per_theta >= disc_f32_tile());
  SourceArgs sa{};
  if (fake_src) sa = source_args(*fake_src);
  DiscArgs a;
  a.D = D;
  a.fake_x = fake_x;
  a.fake_src = fused_src ? &sa : nullptr;
  a.n_fake = n_fake;
  a.real_x = real_x;
  a.n_real = n_real;
  a.d = d;
  sagips_disc_out o2 = *out;
  a.out = &o2;

  const size_t disc_ws = (disc_f32_workspace(a, c->n_cu) + 255) & ~(size_t)255;
  size_t extra = 0, off_x = 0, off_g = 0, off_pg = 0;
  const bool split = fake_src && !fused_src;
  if (split) {
    off_x = disc_ws;
    off_g = off_x + (((size_t)n_fake * d * sizeof(float) + 255) & ~(size_t)255);
    off_pg = off_g + (((size_t)n_fake * d * sizeof(float) + 255) & ~(size_t)255);
    extra = off_pg - disc_ws + param_grad_workspace(sa);
  }
  char* ws = nullptr;
  sagips_status s = acquire_ws(c, from, disc_ws + extra, &ws);
  if (s != SAGIPS_OK) return s;
  hipError_t e;
  if (split) {
    float* xs = reinterpret_cast<float*>(ws + off_x);
    e = launch_sample(sa, xs, nullptr, c->stream, tm);
    if (e != hipSuccess) return hip_fail(c, e, "sample_events launch");
    a.fake_x = xs;
    if (!o2.dLg_dx && o2.dLg_dtheta) o2.dLg_dx = reinterpret_cast<float*>(ws + off_g);
    o2.dLg_dtheta = nullptr;
  }
  e = launch_disc_f32(a, ws, c->n_cu, c->stream, tm);
  if (e != hipSuccess) return hip_fail(c, e, "disc_fwd_bwd launch");
  if (split && out->dLg_dtheta) {
    e = launch_param_grad(sa, o2.dLg_dx, out->dLg_dtheta, nullptr, ws + off_pg, c->stream, tm);
    if (e != hipSuccess) return hip_fail(c, e, "param_grad launch");
  }
  return SAGIPS_OK;
}

}  // namespace

extern "C" {

sagips_status sagips_disc_fwd_bwd(sagips_ctx* c, const sagips_mlp* D, const float* fake_x,
                                  const sagips_source* fake_src, int64_t n_fake, const float* real_x, int64_t n_real,
                                  sagips_disc_out* out) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  return disc_call(c, D, fake_x, fake_src, n_fake, real_x, n_real, out, WsFrom{}, timer_of(c));
}

sagips_status sagips_disc_fwd_bwd_noalloc(sagips_ctx* c, const sagips_mlp* D, const float* fake_x,
                                          const sagips_source* fake_src, int64_t n_fake, const float* real_x,
                                          int64_t n_real, sagips_disc_out* out) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  WsFrom from;
  hipError_t e = scratch_address(c->device, &from.fixed);
  if (e != hipSuccess || !from.fixed) return hip_fail(c, e != hipSuccess ? e : hipErrorInvalidSymbol, "scratch address");
  from.fixed_cap = kScratchBytes;
  // no per-kernel timing here: its events are created on demand
  return disc_call(c, D, fake_x, fake_src, n_fake, real_x, n_real, out, from, nullptr);
}

size_t sagips_noalloc_scratch_bytes(void) { return kScratchBytes; }

sagips_status sagips_bootstrap(sagips_ctx* c, const float* data, int64_t n_data, int d, uint64_t seed, uint32_t step,
                               int64_t n_out, float* out, int64_t* idx_out) {
  sagips_status s = check_bootstrap(c, data, n_data, d, n_out, out, idx_out);
  if (s != SAGIPS_OK) return s;
  DeviceGuard g(c->device);
  hipError_t e = launch_bootstrap(data, (uint64_t)n_data, d, (uint32_t)(seed & 0xffffffffu), (uint32_t)(seed >> 32),
                                  step, n_out, out, idx_out, c->n_cu, c->stream, timer_of(c));
  return e == hipSuccess ? SAGIPS_OK : hip_fail(c, e, "bootstrap launch");
}

sagips_status sagips_bootstrap_rows(sagips_ctx* c, const float* data, int64_t n_data, int d, uint64_t seed,
                                    uint32_t step, int64_t n_out, float* out, int64_t* idx_out) {
  sagips_status s = check_bootstrap(c, data, n_data, d, n_out, out, idx_out);
  if (s != SAGIPS_OK) return s;
  if (n_data > ((int64_t)1 << 27)) return fail(c, SAGIPS_E_UNSUPPORTED, "row order supports n_data <= 2^27");
  if (n_out >= ((int64_t)1 << 31)) return fail(c, SAGIPS_E_UNSUPPORTED, "row order supports n_out < 2^31");
  DeviceGuard g(c->device);
  s = ensure_ws(c, bootstrap_rows_workspace((uint64_t)n_data, n_out, nullptr, nullptr, nullptr));
  if (s != SAGIPS_OK) return s;
  hipError_t e = launch_bootstrap_rows(data, (uint64_t)n_data, d, (uint32_t)(seed & 0xffffffffu),
                                       (uint32_t)(seed >> 32), step, n_out, out, idx_out, c->ws, c->stream, timer_of(c));
  return e == hipSuccess ? SAGIPS_OK : hip_fail(c, e, "bootstrap_rows launch");
}

sagips_status sagips_gen_forward(sagips_ctx* c, const sagips_gen* G, const float* noise, int64_t k, float* theta) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  sagips_status s = check_gen(c, G, noise, k);
  if (s != SAGIPS_OK) return s;
  if (!theta) return fail(c, SAGIPS_E_INVAL, "theta is NULL");
  DeviceGuard g(c->device);
  hipError_t e = launch_gen_forward(*G, noise, k, theta, c->n_cu, c->stream, timer_of(c));
  return e == hipSuccess ? SAGIPS_OK : hip_fail(c, e, "gen_forward launch");
}

sagips_status sagips_gen_backward(sagips_ctx* c, const sagips_gen* G, const float* noise, int64_t k,
                                  const float* dL_dtheta, float* const* dW, float* const* db) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  sagips_status s = check_gen(c, G, noise, k);
  if (s != SAGIPS_OK) return s;
  if (!dL_dtheta || !dW || !db) return fail(c, SAGIPS_E_INVAL, "dL_dtheta, dW or db is NULL");
  for (int l = 0; l < G->n_layers; ++l)
    if (!dW[l] || !db[l]) return fail(c, SAGIPS_E_INVAL, "dW[%d] or db[%d] is NULL", l, l);
  DeviceGuard g(c->device);
  s = ensure_ws(c, gen_backward_workspace(*G, k, c->n_cu));
  if (s != SAGIPS_OK) return s;
  hipError_t e = launch_gen_backward(*G, noise, k, dL_dtheta, dW, db, c->ws, c->n_cu, c->stream, timer_of(c));
  return e == hipSuccess ? SAGIPS_OK : hip_fail(c, e, "gen_backward launch");
}

sagips_status sagips_ensemble_response(sagips_ctx* c, const sagips_gen* G, const float* noise, int64_t k,
                                       const float* p_true, float* p_hat, float* sigma, float* r_hat) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  sagips_status s = check_gen(c, G, noise, k);
  if (s != SAGIPS_OK) return s;
  if (!p_hat || !sigma) return fail(c, SAGIPS_E_INVAL, "p_hat or sigma is NULL");
  if ((p_true == nullptr) != (r_hat == nullptr)) return fail(c, SAGIPS_E_INVAL, "p_true and r_hat must be given together");
  if ((int64_t)G->n_members * k * G->width[G->n_layers] >= ((int64_t)1 << 31))
    return fail(c, SAGIPS_E_INVAL, "n_members * k * output width must be < 2^31");
  DeviceGuard g(c->device);
  s = ensure_ws(c, ensemble_workspace(*G, k));
  if (s != SAGIPS_OK) return s;
  hipError_t e = launch_ensemble(*G, noise, k, p_true, p_hat, sigma, r_hat, c->ws, c->n_cu, c->stream, timer_of(c));
  return e == hipSuccess ? SAGIPS_OK : hip_fail(c, e, "ensemble launch");
}

sagips_status sagips_adam_step(sagips_ctx* c, const sagips_param_set* ps, int32_t step, double lr, double beta1,
                               double beta2, double eps) {
  if (!c) return fail(nullptr, SAGIPS_E_INVAL, "ctx is NULL");
  if (!ps) return fail(c, SAGIPS_E_INVAL, "set is NULL");
  if (ps->n_tensors < 1 || ps->n_tensors > SAGIPS_MAX_TENSORS)
    return fail(c, SAGIPS_E_INVAL, "n_tensors = %d outside [1, %d]", ps->n_tensors, SAGIPS_MAX_TENSORS);
  for (int i = 0; i < ps->n_tensors; ++i) {
    if (!ps->param[i] || !ps->grad[i] || !ps->m[i] || !ps->v[i])
      return fail(c, SAGIPS_E_INVAL, "tensor %d has a NULL array", i);
    if (ps->size[i] < 0) return fail(c, SAGIPS_E_INVAL, "size[%d] < 0", i);
  }
  if (step < 1) return fail(c, SAGIPS_E_INVAL, "step must be >= 1");
  if (!(lr >= 0.0) || !(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) || !(eps >= 0.0))
    return fail(c, SAGIPS_E_INVAL, "need lr >= 0, 0 <= beta1, beta2 < 1, eps >= 0");
  DeviceGuard g(c->device);
  hipError_t e = launch_adam(*ps, step, lr, beta1, beta2, eps, c->stream, timer_of(c));
  return e == hipSuccess ? SAGIPS_OK : hip_fail(c, e, "adam launch");
}

}  // extern "C"
