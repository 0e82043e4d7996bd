// Adam step over a set of parameter tensors, one launch per set: blockIdx.y
// picks the tensor, the x blocks stride over its elements.  Element-wise and
// deterministic; the bias corrections are formed on the host in double.
#include "kernels.hpp"

namespace sagips {
namespace {

struct AdamArgs {
  float* p[SAGIPS_MAX_TENSORS];
  const float* g[SAGIPS_MAX_TENSORS];
  float* m[SAGIPS_MAX_TENSORS];
  float* v[SAGIPS_MAX_TENSORS];
  int64_t n[SAGIPS_MAX_TENSORS];
  float beta1, beta2, eps;
  float omb1, omb2;  // 1 - beta1, 1 - beta2, formed in double and rounded once
  float step_size;   // lr / (1 - beta1^t)
  float inv_sqrt_bc2;  // 1 / sqrt(1 - beta2^t)
};

__global__ __launch_bounds__(256) void k_adam(AdamArgs a) {
  const int t = blockIdx.y;
  float* __restrict__ p = a.p[t];
  const float* __restrict__ g = a.g[t];
  float* __restrict__ m = a.m[t];
  float* __restrict__ v = a.v[t];
  const int64_t n = a.n[t];
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) {
    const float gi = g[i];
    const float mi = a.beta1 * m[i] + a.omb1 * gi;
    const float vi = a.beta2 * v[i] + a.omb2 * gi * gi;
    m[i] = mi;
    v[i] = vi;
    p[i] -= a.step_size * mi / (sqrtf(vi) * a.inv_sqrt_bc2 + a.eps);
  }
}

}  // namespace

hipError_t launch_adam(const sagips_param_set& ps, int step, double lr, double beta1, double beta2, double eps,
                       hipStream_t st, Timer* tm) {
  AdamArgs a;
  int64_t most = 0;
  for (int i = 0; i < ps.n_tensors; ++i) {
    a.p[i] = ps.param[i];
    a.g[i] = ps.grad[i];
    a.m[i] = ps.m[i];
    a.v[i] = ps.v[i];
    a.n[i] = ps.size[i];
    most = ps.size[i] > most ? ps.size[i] : most;
  }
  a.beta1 = (float)beta1;
  a.beta2 = (float)beta2;
  a.eps = (float)eps;
  a.omb1 = (float)(1.0 - beta1);
  a.omb2 = (float)(1.0 - beta2);
  a.step_size = (float)(lr / (1.0 - pow(beta1, step)));
  a.inv_sqrt_bc2 = (float)(1.0 / sqrt(1.0 - pow(beta2, step)));
  int64_t bx = (most + 255) / 256;
  if (bx > 1024) bx = 1024;
  if (bx < 1) bx = 1;
  if (tm) tm->begin("adam");
  hipLaunchKernelGGL(k_adam, dim3((unsigned)bx, ps.n_tensors), dim3(256), 0, st, a);
  if (tm) tm->end();
  return hipGetLastError();
}

}  // namespace sagips
