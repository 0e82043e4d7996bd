// Internal launch interface between the C ABI (api.hip) and the kernel files.
// Every launcher enqueues on `stream`, validates nothing (the ABI layer has
// already done so) and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/sagips.h"

namespace sagips {

// Records HIP events around one launch when timing is on (api.hip).
struct Timer {
  virtual ~Timer() = default;
  virtual void begin(const char* name) = 0;
  virtual void end() = 0;
};

struct SourceArgs {
  const float* theta;
  int n_theta;
  int d;
  int64_t E;
  uint32_t k0, k1;
  uint64_t base;
  uint32_t stream;
};

inline SourceArgs source_args(const sagips_source& s) {
  SourceArgs a;
  a.theta = s.theta;
  a.n_theta = s.n_theta;
  a.d = s.d;
  a.E = s.events_per_theta;
  a.k0 = (uint32_t)(s.seed & 0xffffffffu);
  a.k1 = (uint32_t)(s.seed >> 32);
  a.base = s.counter_base;
  a.stream = s.stream;
  return a;
}

// sampler.hip ---------------------------------------------------------------
hipError_t launch_sample(const SourceArgs& s, float* x, uint32_t* words, hipStream_t st, Timer* tm);

// Bytes of workspace launch_param_grad needs.
size_t param_grad_workspace(const SourceArgs& s);
// dL/dx from a buffer (dLdx != NULL) or the quadratic critic (dLdx == NULL).
hipError_t launch_param_grad(const SourceArgs& s, const float* dLdx, float* dLdtheta, float* loss,
                             void* ws, hipStream_t st, Timer* tm);

// Bootstrap draws: out[i] = data[floor(w0(i) * n_data / 2^32)], idx_out optional.
size_t bootstrap_rows_workspace(uint64_t n_data, int64_t n_out, int* n_slabs, int* n_chunks, int64_t* per_chunk);
hipError_t launch_bootstrap_rows(const float* data, uint64_t n_data, int d, uint32_t k0, uint32_t k1, uint32_t step,
                                 int64_t n_out, float* out, int64_t* idx_out, void* ws, hipStream_t st, Timer* tm);
hipError_t launch_bootstrap(const float* data, uint64_t n_data, int d, uint32_t k0, uint32_t k1, uint32_t step,
                            int64_t n_out, float* out, int64_t* idx_out, int n_cu, hipStream_t st, Timer* tm);

// disc_f32.hip ---------------------------------------------------------------
struct DiscArgs {
  const sagips_mlp* D;
  const float* fake_x;         // or NULL with a source
  const SourceArgs* fake_src;  // or NULL
  int64_t n_fake;
  const float* real_x;
  int64_t n_real;
  const sagips_disc_out* out;
  int d;
  int chunk_rows = 0;          // bf16 path: rows per chunk (multiple of 128), 0 = the default
};
bool disc_f32_supported(const sagips_mlp& D, int d, const char** why);
int disc_f32_tile();   // events per tile; the in-kernel sampler needs E >= tile
size_t disc_f32_workspace(const DiscArgs& a, int n_cu);
hipError_t launch_disc_f32(const DiscArgs& a, void* ws, int n_cu, hipStream_t st, Timer* tm);

// generator.hip --------------------------------------------------------------
constexpr int kMaxGenLayers = 5;
bool gen_supported(const sagips_gen& G, const char** why);
size_t gen_backward_workspace(const sagips_gen& G, int64_t k, int n_cu);
size_t ensemble_workspace(const sagips_gen& G, int64_t k);
hipError_t launch_gen_forward(const sagips_gen& G, const float* noise, int64_t k, float* theta, int n_cu,
                              hipStream_t st, Timer* tm);
hipError_t launch_gen_backward(const sagips_gen& G, const float* noise, int64_t k, const float* dtheta,
                               float* const* dW, float* const* db, void* ws, int n_cu, hipStream_t st, Timer* tm);
hipError_t launch_ensemble(const sagips_gen& G, const float* noise, int64_t k, const float* p_true, float* p_hat,
                           float* sigma, float* r_hat, void* ws, int n_cu, hipStream_t st, Timer* tm);

// optim.hip ------------------------------------------------------------------
hipError_t launch_adam(const sagips_param_set& ps, int step, double lr, double beta1, double beta2, double eps,
                       hipStream_t st, Timer* tm);

// disc_bf16.hip --------------------------------------------------------------
// Samples the fake events itself when a.fake_src is set (any E); never writes dLg_dtheta.
bool disc_bf16_supported(const sagips_mlp& D, int d, const char** why);
size_t disc_bf16_workspace(const DiscArgs& a, int n_cu);
// Default (and largest) rows per chunk of the bf16 path.
int disc_bf16_max_chunk_rows();
hipError_t launch_disc_bf16(const DiscArgs& a, void* ws, int n_cu, hipStream_t st, Timer* tm);

}  // namespace sagips
