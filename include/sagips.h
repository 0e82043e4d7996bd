/*
 * sagips.h -- C ABI of libsagips.so: one rank's sample -> discriminate ->
 * backward step of SAGIPS (arXiv 2407.00051) on an AMD Instinct MI355X (gfx950).
 *
 * The calls follow the paper's problem statement (Sec. II, eqs. def_inv,
 * def_x_hat, def_optim): parameters p are turned into events by a pipeline
 * whose sampler module uses an inverse CDF (Sec. V-A); an objective (the GAN
 * discriminator, Sec. II-B.2 and III-A) scores synthetic against reference
 * events; gradients flow back through every differentiable module to p
 * (Sec. III-B).
 *
 * Conventions shared by every call
 *   - Pointers are DEVICE pointers on the context's device unless marked
 *     "host".  The caller allocates and owns every input and output; the
 *     library owns only the context and its workspace.
 *   - Every call is asynchronous on the context's HIP stream.  Arguments are
 *     validated before anything is launched; on a validation error nothing is
 *     launched, a negative status is returned and sagips_last_error() says why.
 *     Faults during execution surface at the caller's stream synchronisation.
 *   - Outputs are overwritten, never accumulated.  Results are bitwise
 *     reproducible for fixed inputs (fixed reduction order, no float atomics).
 *   - Device arrays must be 16-byte aligned and densely packed, row-major;
 *     the one exception is theta, which needs only 4-byte alignment so that a
 *     caller can pass the rows of one shard (theta + r * 2d).
 *   - Several contexts may share a device; each owns its own workspace.
 *   - A context is not thread-safe; calls on one context must not overlap
 *     from several host threads.
 *
 * Event sampling (shared by all calls that take a sagips_source)
 *   Event k of parameter row i has id = counter_base + i*E + k.  Its random
 *   block is Philox4x32-10 (Salmon et al., SC'11) with
 *       key = (seed & 0xffffffff, seed >> 32),
 *       counter = (id & 0xffffffff, id >> 32, stream, 0),
 *   words w0..w3.  Coordinate j < d uses u_j = ((w_j >> 9) + 1/2) * 2^-23 and
 *   the Kumaraswamy quantile x_j = (1 - (1 - u_j)^(1/b_j))^(1/a_j) with
 *   (a_j, b_j) = (theta[i][2j], theta[i][2j+1]).
 */
#ifndef SAGIPS_H
#define SAGIPS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SAGIPS_MAX_LAYERS 8

typedef struct sagips_ctx sagips_ctx;

typedef enum {
  SAGIPS_OK = 0,
  SAGIPS_E_INVAL = -1,       /* bad argument: NULL, size, alignment, unsupported shape */
  SAGIPS_E_ARCH = -2,        /* device is not gfx950 */
  SAGIPS_E_NOMEM = -3,       /* workspace allocation failed */
  SAGIPS_E_HIP = -4,         /* a HIP runtime call or a launch failed */
  SAGIPS_E_UNSUPPORTED = -5  /* valid request the library does not implement */
} sagips_status;

typedef enum { SAGIPS_F32 = 0, SAGIPS_BF16 = 1 } sagips_precision;
typedef enum { SAGIPS_FEAT_IDENTITY = 0, SAGIPS_FEAT_HD8 = 1, SAGIPS_FEAT_PROXY2 = 2 } sagips_features;
/* The last enumerator widens the type to 32 bits, so that a value a C caller
 * passes outside the list is still a value of the type, and the library can
 * reject it with SAGIPS_E_INVAL.                                           */
typedef enum {
  SAGIPS_CRITIC_BUFFER = 0,
  SAGIPS_CRITIC_QUADRATIC = 1,
  SAGIPS_CRITIC_MAX_ENUM = 0x7fffffff
} sagips_critic;

/* Parameters -> events source (host struct holding a device pointer).
 *   theta            device, [n_theta][2d] fp32, rows (a1,b1,a2,b2[,a3,b3]),
 *                    4-byte aligned; shape parameters must be > 0 (the
 *                    workloads use >= 1).
 *   n_theta          >= 1
 *   d                observables per event, 2 or 3
 *   events_per_theta E >= 1; n_theta * E < 2^31 and counter_base + n_theta*E < 2^64
 *   seed, counter_base, stream   see "Event sampling" above            */
typedef struct {
  const float* theta;
  int32_t n_theta;
  int32_t d;
  int64_t events_per_theta;
  uint64_t seed;
  uint64_t counter_base;
  uint32_t stream;
} sagips_source;

/* Discriminator (paper Sec. V-A: LeakyReLU hidden layers).  Layer l maps
 * width[l] -> width[l+1]; W[l] is [width[l+1]][width[l]] fp32 (torch.nn.Linear
 * layout), b[l] is [width[l+1]] fp32.  Hidden layers apply
 * LeakyReLU(leaky_slope); the last layer has width 1 and emits a logit.
 *   features   IDENTITY: width[0] == d;  HD8 (d == 3): width[0] == 8 and the
 *              input is [x1,x2,x3,x1x2,x2x3,x1x3,ln x1,ln(1-x3)];
 *              PROXY2 (d == 3, F32 only): width[0] == 2 and the input is the
 *              two observables (x1 + x3, x2 + x3) of the six-parameter,
 *              two-observable pipeline (Sec. V; the sum form is this
 *              library's reading, the paper does not give the mapping).
 *              Event buffers hold the d raw coordinates in every mode, and
 *              dLg_dx is the gradient with respect to them.
 *   precision  F32: every product in fp32.  BF16: hidden-to-hidden layers use
 *              bf16 operands (weights rounded once per call, activations and
 *              backward signals rounded to nearest even) with fp32 accumulate;
 *              the first and the logit layer stay fp32.
 * Supported shapes (SAGIPS_E_UNSUPPORTED otherwise): all hidden widths equal,
 * one of 64, 128 (F32) or 256, 512 (BF16); width[0] in {2, 3, 8}.  F32
 * IDENTITY with d = 2: width 64 with 1-3 or 128 with 1-2 hidden-to-hidden
 * layers; with d = 3: width 64 with 1-2 or 128 with 2.  F32 PROXY2: width 128
 * with 3 (the paper's 2-128-128-128-128-1 network).  BF16: 1-4
 * hidden-to-hidden layers and 0 <= leaky_slope <= 1.                      */
typedef struct {
  int32_t n_layers;
  int32_t width[SAGIPS_MAX_LAYERS + 1];
  const float* W[SAGIPS_MAX_LAYERS];
  const float* b[SAGIPS_MAX_LAYERS];
  float leaky_slope;
  int32_t precision;  /* sagips_precision */
  int32_t features;   /* sagips_features  */
} sagips_mlp;

/* Discriminator outputs; any pointer may be NULL ("not requested").
 *   logits_fake [n_fake], logits_real [n_real]
 *   loss_d [1]  L_D = mean_real softplus(-z) + mean_fake softplus(z)
 *   loss_g [1]  L_G = mean_fake softplus(-z)   (non-saturating generator loss)
 *   dW[l], db[l]  gradients of L_D, shaped like W[l], b[l] (all or none)
 *   dLg_dx [n_fake][d]  dL_G / d fake event
 *   dLg_dtheta [n_theta][2d]  dL_G / d theta; only with a fake source      */
typedef struct {
  float* logits_fake;
  float* logits_real;
  float* loss_d;
  float* loss_g;
  float* dW[SAGIPS_MAX_LAYERS];
  float* db[SAGIPS_MAX_LAYERS];
  float* dLg_dx;
  float* dLg_dtheta;
} sagips_disc_out;

/* Create a context on HIP device `hip_device` using `hip_stream` (a
 * hipStream_t; NULL = the device's null stream).  Fails with SAGIPS_E_ARCH
 * unless the device is gfx950.  *out is set to NULL on failure.          */
sagips_status sagips_create(sagips_ctx** out, int hip_device, void* hip_stream);

/* Release the context and its workspace.  Synchronises the context's stream
 * first.  NULL is accepted.                                               */
sagips_status sagips_destroy(sagips_ctx* ctx);

/* Switch subsequent calls to another stream of the same device.  The new
 * stream is made to wait (on the device, not the host) for the work already
 * queued on the old one, which may still use the context's workspace.     */
sagips_status sagips_set_stream(sagips_ctx* ctx, void* hip_stream);

/* Rows per chunk of the bf16 discriminator (which runs the fake and the real
 * batch in chunks whose activations and signals it stages in the workspace):
 * 0 restores the default, 4,194,304 rows, which is also the largest allowed;
 * otherwise a multiple of 128 in [128, 4194304].  Results do not depend on
 * it beyond the order of the fp32 sums across chunks; smaller chunks need a
 * smaller workspace.  SAGIPS_E_INVAL for other values.                    */
sagips_status sagips_set_bf16_chunk_rows(sagips_ctx* ctx, int64_t rows);

/* Message of the last failed call on ctx (ctx may be NULL: message of the
 * last failed sagips_create in this process).  Never NULL.               */
const char* sagips_last_error(const sagips_ctx* ctx);

/* Kernel timing: when enabled, each kernel launch of the following calls is
 * bracketed by HIP events on the context's stream.  sagips_kernel_times()
 * synchronises the stream and returns, per kernel name, the number of
 * launches and the summed milliseconds since the last reset (host arrays of
 * `cap` entries; names point to static strings).  Returns the number of
 * distinct kernels, or a negative status.                                 */
sagips_status sagips_set_timing(sagips_ctx* ctx, int enable);
int sagips_kernel_times(sagips_ctx* ctx, const char** names, int64_t* launches, double* total_ms, int cap);

/* 1. Parameters -> events (paper Sec. V-A, inverse-CDF sampler module).
 *   x_out      [N][d] fp32, N = n_theta * E; may be NULL if words_out is set
 *   words_out  [N][4] uint32 raw Philox words, or NULL                     */
sagips_status sagips_sample_events(sagips_ctx* ctx, const sagips_source* src, float* x_out,
                                   uint32_t* words_out);

/* 2. Events -> discriminator -> BCE loss -> backward (paper Sec. II-B.2,
 * Sec. III-A; the discriminator labels reference events 1 and synthetic 0).
 * Fake events come either as a buffer fake_x [n_fake][d] or as a source
 * fake_src that is sampled inside the kernel (exactly one of the two is
 * non-NULL; with a source, n_fake must equal n_theta * E and the call can
 * also return dLg_dtheta).  real_x is [n_real][d] fp32.  d is taken from
 * fake_src, or from width[0] for IDENTITY features, or is 3 for HD8.       */
sagips_status sagips_disc_fwd_bwd(sagips_ctx* ctx, const sagips_mlp* D, const float* fake_x,
                                  const sagips_source* fake_src, int64_t n_fake,
                                  const float* real_x, int64_t n_real, sagips_disc_out* out);

/* 2b. The same step for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Arguments, results and errors are those of
 * sagips_disc_fwd_bwd (the same kernels), except:
 *   - the workspace is a fixed scratch array of
 *     sagips_noalloc_scratch_bytes() bytes (64 MiB) per device, reserved by
 *     the library when it is loaded and held until the process ends; this
 *     call never allocates (no hipMalloc, hipFree or allocating library call);
 *   - a call whose workspace would exceed it returns SAGIPS_E_INVAL before
 *     launching anything (the small-batch workload needs about 35 MB, the
 *     paper's 2-128-128-128-128-1 shape about 52 MB);
 *   - every call on one device shares that device's array and leaves its
 *     contents behind: calls that overlap on one device (several streams or
 *     contexts) race and must be ordered by the caller;
 *   - per-kernel timing (sagips_set_timing) does not apply to it.          */
sagips_status sagips_disc_fwd_bwd_noalloc(sagips_ctx* ctx, const sagips_mlp* D, const float* fake_x,
                                          const sagips_source* fake_src, int64_t n_fake,
                                          const float* real_x, int64_t n_real, sagips_disc_out* out);
size_t sagips_noalloc_scratch_bytes(void);

/* 3. dL/dx -> pathwise dx/dtheta -> per-parameter reduction (paper Sec. II,
 * gradient of the objective with respect to p through the sampler).  The
 * events are regenerated from the source, never read.  With
 * critic == BUFFER, dL_dx is [N][d] fp32 and loss_out must be NULL; with
 * critic == QUADRATIC the critic is L = sum over events and coordinates of
 * (x - 1/2)^2, dL_dx must be NULL, and loss_out [1] (may be NULL) gets L.
 *   dL_dtheta  [n_theta][2d]: sum over the row's events of
 *              dL/dx_j * (dx_j/da_j, dx_j/db_j)                            */
sagips_status sagips_param_grad(sagips_ctx* ctx, const sagips_source* src, sagips_critic critic,
                                const float* dL_dx, float* dL_dtheta, float* loss_out);

/* 4. Reference data -> the step's bootstrapped sub-sample (paper Sec. IV-B:
 * every rank draws its training sub-samples from its data by bootstrapping,
 * i.e. uniformly with replacement).  Draw i < n_out copies row
 *     idx_i = floor(w0 * n_data / 2^32)
 * of data, where w0 is the first word of Philox4x32-10 with
 *     key = (seed & 0xffffffff, seed >> 32),
 *     counter = (i & 0xffffffff, i >> 32, SAGIPS_STREAM_BOOTSTRAP, step),
 * so every step draws a fresh sub-sample that depends only on (seed, step, i).
 *   data     [n_data][d] fp32, 1 <= n_data <= 2^32, d in {2, 3}
 *   out      [n_out][d] fp32, n_out >= 1; must not overlap data
 *   idx_out  [n_out] int64 (the drawn rows), or NULL
 * The result is typically passed as real_x to sagips_disc_fwd_bwd.         */
#define SAGIPS_STREAM_BOOTSTRAP 4u
sagips_status sagips_bootstrap(sagips_ctx* ctx, const float* data, int64_t n_data, int d, uint64_t seed,
                               uint32_t step, int64_t n_out, float* out, int64_t* idx_out);

/* 4b. The same sub-sample listed in ascending row order: row r of data
 * appears as often as sagips_bootstrap draws it with the same (seed, step,
 * n_out).  A batch used as a whole (the discriminator's mean loss and summed
 * gradients) does not depend on the order of its rows, and this order lets
 * the reference data be read once, in order, instead of one random line per
 * draw.  Arguments as for sagips_bootstrap, with 1 <= n_data <= 2^27 and
 * n_out < 2^31 (SAGIPS_E_UNSUPPORTED beyond); idx_out receives the rows in
 * the same ascending order.  Uses the context's workspace (6 bytes per draw
 * plus per-slab counts).                                                  */
sagips_status sagips_bootstrap_rows(sagips_ctx* ctx, const float* data, int64_t n_data, int d, uint64_t seed,
                                    uint32_t step, int64_t n_out, float* out, int64_t* idx_out);

/* A stack of M generators of one shape (paper Sec. III: the optimiser is a GAN
 * generator mapping noise to parameters; Sec. V-A: LeakyReLU hidden layers).
 * Layer l maps width[l] -> width[l+1]; member m's weight is the
 * [width[l+1]][width[l]] block at W[l] + m * width[l+1] * width[l] and its
 * bias the [width[l+1]] block at b[l] + m * width[l+1] (torch.nn.Linear
 * layout, members stacked in front).  Hidden layers apply
 * LeakyReLU(leaky_slope); the output is theta = 1 + softplus(last layer).
 * Supported: 3..5 layers, all hidden widths 128, width[0] and the output
 * width in [1, 8] (the paper's 51,206-parameter generator is
 * 6-128-128-128-128-6).  Every W[l], b[l] must be 16-byte aligned.         */
typedef struct {
  int32_t n_layers;
  int32_t width[SAGIPS_MAX_LAYERS + 1];
  const float* W[SAGIPS_MAX_LAYERS];
  const float* b[SAGIPS_MAX_LAYERS];
  int32_t n_members;  /* M >= 1 */
  float leaky_slope;
} sagips_gen;

/* 5. Generator forward: theta[m][r] = G_m(noise[r]) for every member m.
 *   noise  [k][width[0]] fp32, shared by all members, k >= 1
 *   theta  [M][k][out] fp32                                                */
sagips_status sagips_gen_forward(sagips_ctx* ctx, const sagips_gen* G, const float* noise, int64_t k,
                                 float* theta);

/* 6. Generator backward: given dL/dtheta [M][k][out] (e.g. dLg_dtheta of
 * sagips_disc_fwd_bwd), the gradients of sum_r <dL/dtheta[m][r], theta[m][r]>
 * with respect to member m's parameters, through 1 + softplus and the
 * LeakyReLU layers (the generator's step of Sec. III).
 *   dW[l], db[l]  shaped like W[l], b[l] (all members); overwritten.
 * The forward pass is recomputed from noise; nothing from sagips_gen_forward
 * is needed.                                                                */
sagips_status sagips_gen_backward(sagips_ctx* ctx, const sagips_gen* G, const float* noise, int64_t k,
                                  const float* dL_dtheta, float* const* dW, float* const* db);

/* 7. Ensemble response (paper Sec. VI-A, eqs. def_ens_mean, def_ens_std and
 * def_param_res): for each noise vector n_r the member mean
 * p_hat(n_r) = (1/M) sum_m G_m(n_r) and the spread
 * sigma(n_r) = sqrt((1/M) sum_m (G_m(n_r) - p_hat(n_r))^2), both averaged
 * over the k noise vectors; with p_true the normalised residual
 * r_hat = (p_true - p_hat) / p_true.
 *   p_hat, sigma  [out] fp32
 *   p_true, r_hat [out] fp32, both given or both NULL                       */
sagips_status sagips_ensemble_response(sagips_ctx* ctx, const sagips_gen* G, const float* noise, int64_t k,
                                       const float* p_true, float* p_hat, float* sigma, float* r_hat);

/* 8. Optimiser step (Sec. V-A gives the learning rates, generator 1e-5 and
 * discriminator 1e-4, not the optimiser; this library reads it as Adam,
 * Kingma and Ba 2015, Algorithm 1): for t = step >= 1, every element of every
 * tensor of the set gets
 *   m <- beta1 m + (1 - beta1) g,  v <- beta2 v + (1 - beta2) g^2,
 *   p <- p - lr / (1 - beta1^t) * m / (sqrt(v) / sqrt(1 - beta2^t) + eps).
 * param, m, v are updated in place (m, v start at zero); grad is read only.
 * Every array holds size[i] fp32 elements; 1 <= n_tensors <= 16.
 * 0 <= beta1, beta2 < 1, eps >= 0, lr >= 0.  The scalars are double so that
 * 1 - beta and the bias corrections are formed before rounding to fp32.   */
#define SAGIPS_MAX_TENSORS 16
typedef struct {
  int32_t n_tensors;
  float* param[SAGIPS_MAX_TENSORS];
  const float* grad[SAGIPS_MAX_TENSORS];
  float* m[SAGIPS_MAX_TENSORS];
  float* v[SAGIPS_MAX_TENSORS];
  int64_t size[SAGIPS_MAX_TENSORS];
} sagips_param_set;

sagips_status sagips_adam_step(sagips_ctx* ctx, const sagips_param_set* set, int32_t step, double lr,
                               double beta1, double beta2, double eps);

#ifdef __cplusplus
}
#endif

#endif /* SAGIPS_H */
