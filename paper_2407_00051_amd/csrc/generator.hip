// The GAN generator (noise -> parameters) of Sec. III, for a stack of M
// members of the same shape, and the ensemble response of Sec. VI-A.
//
// Network: IN -> H -> (H -> H) x NH -> OUT, LeakyReLU on the hidden layers,
// theta = 1 + softplus(last layer), so that every shape parameter is above 1.
// The paper's generator (51,206 parameters) is 6 -> 128 x 4 -> 6, i.e.
// H = 128, NH = 3.  Member m's parameters sit at W[l] + m * |W[l]|.
//
// Work decomposition: one workgroup of 8 waves per (tile of T rows of the
// noise batch, member), T = 64, or 16 when 64-row tiles would leave most CUs
// idle (a single generator on 1,024 rows).  The tile's activations
// A_1 .. A_{NH+1} live in LDS as [T][H+4] fp32; the H x H products run on the fp32 matrix cores
// (v_mfma_f32_16x16x4_f32) as out^T = W * in^T, each wave owning 16 output
// features of all T rows.  The first layer (K = IN) and the last (N = OUT)
// are VALU work.
//
// The backward kernel recomputes the tile's forward pass into LDS (cheaper
// than storing it), then runs the backward pass from dL/dtheta: each backward
// signal overwrites the activation it replaces.  Weight gradients of the tile
// go to a per-tile partial; a second kernel sums the partials over tiles in
// a fixed order, so results are deterministic.
#include "device_math.hpp"
#include "kernels.hpp"

#include <string.h>

namespace sagips {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kGThreads = 512;   // 8 waves
constexpr int kGMaxIO = 8;       // largest IN / OUT

__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ float g_leaky(float v, float s) { return v > 0.0f ? v : s * v; }
__device__ __forceinline__ float g_leaky_grad(float h, float s) { return h > 0.0f ? 1.0f : s; }
__device__ __forceinline__ float g_softplus(float t) { return fmaxf(t, 0.0f) + log1pf(expf(-fabsf(t))); }
__device__ __forceinline__ float g_sigmoid(float t) { return 1.0f / (1.0f + expf(-t)); }

// Workgroups are numbered L = x + y * gridDim.x and dealt to the 8 XCDs in
// turn (XCD = L mod 8); each XCD has its own L2.  The first 8 * floor(M / 8)
// members are placed so that all tiles of a member run on one XCD (member =
// 8 (j / tiles) + L mod 8, tile = j mod tiles, j = L / 8), so its weights are
// fetched into one L2 only; the remaining members are laid out in order.
__device__ __forceinline__ void gen_block(int tiles, int members, int& m, int& tile) {
  const int L = blockIdx.x + blockIdx.y * gridDim.x;
  const int m8 = members - members % 8;
  if (L < tiles * m8) {
    const int j = L >> 3;
    m = 8 * (j / tiles) + (L & 7);
    tile = j % tiles;
  } else {
    const int r = L - tiles * m8;
    m = m8 + r / tiles;
    tile = r % tiles;
  }
}

struct GenParams {
  const float* W[kMaxGenLayers];   // layer l of member 0; member m at + m * wsz[l]
  const float* b[kMaxGenLayers];
  int64_t wsz[kMaxGenLayers], bsz[kMaxGenLayers];
  int in, out;
  int64_t k;                       // rows of the noise batch
  float slope;
  const float* noise;              // [k][in], shared by every member
  float* theta;                    // forward: [M][k][out]
  const float* dtheta;             // backward: [M][k][out]
  float* part;                     // backward: [M][tiles][P]
  int64_t P;                       // floats per partial (all parameters of one member)
  int64_t poff_w[kMaxGenLayers], poff_b[kMaxGenLayers];
};

// kKeep: keep every activation for a backward pass; otherwise the forward
// pass alternates between two buffers (half the LDS, two workgroups per CU).
template <int H, int NH, int kGT, bool kKeep>
struct Gen {
  static constexpr int LD = H + 4;
  static constexpr int WAVES = kGThreads / 64;
  static constexpr int KB = H / 16;
  static constexpr int CB = kGT / 16;
  static_assert(kGT == 16 || kGT == 64, "row tile");
  static constexpr int PPO = kGThreads / H;     // threads per feature in the VALU loops
  static_assert(H == 16 * WAVES, "one wave per 16 features");

  static constexpr int NBUF = kKeep ? NH + 1 : 2;
  static constexpr __device__ int buf(int l) { return kKeep ? l : (l & 1); }

  struct Smem {
    float act[NBUF][kGT][LD];
    float n[kGT][kGMaxIO];
    float o[kGT][kGMaxIO];     // last-layer pre-activation
    float dout[kGT][kGMaxIO];  // dL/d(pre-activation of the last layer)
  };

  // out^T (16 features of this wave x 64 rows) = W[o][k] in[ev][k]; W row-major [H][H].
  static __device__ __forceinline__ void gemm_fwd(const float* __restrict__ W, const float* in, f32x4 (&acc)[CB],
                                                  int o0, int lr, int lg) {
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    const float* wrow = W + (o0 + lr) * H + 4 * lg;
#pragma unroll 2
    for (int kb = 0; kb < KB; ++kb) {
      const f32x4 a = *reinterpret_cast<const f32x4*>(wrow + 16 * kb);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        const f32x4 bv = *reinterpret_cast<const f32x4*>(in + (16 * cb + lr) * LD + 16 * kb + 4 * lg);
#pragma unroll
        for (int s = 0; s < 4; ++s) acc[cb] = mfma4(a[s], bv[s], acc[cb]);
      }
    }
  }

  // out^T (16 input features k of this wave x 64 rows) = sum_o W[o][k] dl[ev][o]:
  // the backward-data product, reading W column-wise.
  static __device__ __forceinline__ void gemm_bwd(const float* __restrict__ W, const float* dl, f32x4 (&acc)[CB],
                                                  int k0, int lr, int lg) {
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 2
    for (int kb = 0; kb < KB; ++kb) {
      const int o = 16 * kb + 4 * lg;
      f32x4 a;
#pragma unroll
      for (int s = 0; s < 4; ++s) a[s] = W[(o + s) * H + k0 + lr];
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        const f32x4 bv = *reinterpret_cast<const f32x4*>(dl + (16 * cb + lr) * LD + o);
#pragma unroll
        for (int s = 0; s < 4; ++s) acc[cb] = mfma4(a[s], bv[s], acc[cb]);
      }
    }
  }

  // Forward pass of member m on rows [row0, row0 + 64) into LDS; rows past k
  // carry zero noise.  Leaves A_1..A_{NH+1} in act and the last layer's
  // pre-activation in o.
  static __device__ void forward(const GenParams& p, Smem& sm, int m, int64_t row0) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lr = lane & 15, lg = lane >> 4;
    const float slope = p.slope;
    for (int i = tid; i < kGT * kGMaxIO; i += kGThreads) {
      const int ev = i / kGMaxIO, j = i % kGMaxIO;
      const int64_t r = row0 + ev;
      sm.n[ev][j] = (j < p.in && r < p.k) ? p.noise[r * p.in + j] : 0.0f;
    }
    __syncthreads();
    {   // first layer: thread (feature o, part) over rows part, part + PPO, ...
      const int o = tid % H, part = tid / H;
      const float* W0 = p.W[0] + m * p.wsz[0];
      float w[kGMaxIO];
#pragma unroll
      for (int j = 0; j < kGMaxIO; ++j) w[j] = j < p.in ? W0[o * p.in + j] : 0.0f;
      const float bias = p.b[0][m * p.bsz[0] + o];
      for (int ev = part; ev < kGT; ev += PPO) {
        float v = bias;
#pragma unroll
        for (int j = 0; j < kGMaxIO; ++j) v = fmaf(w[j], sm.n[ev][j], v);
        sm.act[buf(0)][ev][o] = g_leaky(v, slope);
      }
    }
    __syncthreads();
    const int o0 = 16 * wave;
#pragma unroll
    for (int l = 0; l < NH; ++l) {
      f32x4 acc[CB];
      gemm_fwd(p.W[1 + l] + m * p.wsz[1 + l], &sm.act[buf(l)][0][0], acc, o0, lr, lg);
      const int o = o0 + 4 * lg;
      const f32x4 bias = *reinterpret_cast<const f32x4*>(p.b[1 + l] + m * p.bsz[1 + l] + o);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        f32x4 v = acc[cb] + bias;
        v.x = g_leaky(v.x, slope); v.y = g_leaky(v.y, slope);
        v.z = g_leaky(v.z, slope); v.w = g_leaky(v.w, slope);
        *reinterpret_cast<f32x4*>(&sm.act[buf(l + 1)][16 * cb + lr][o]) = v;
      }
      __syncthreads();
    }
    if ((tid >> 3) < kGT) {   // last layer: thread (row ev, part) sums features 4 part + 32 c (c < H / 32)
      const int ev = tid >> 3, part = tid & 7;
      const float* Wl = p.W[NH + 1] + m * p.wsz[NH + 1];
      const float* hrow = &sm.act[buf(NH)][ev][0];
      for (int j = 0; j < p.out; ++j) {
        float z = 0.f;
#pragma unroll
        for (int c = 0; c < H / 32; ++c) {
          const int f = 4 * part + 32 * c;
          const f32x4 hv = *reinterpret_cast<const f32x4*>(hrow + f);
          const f32x4 wv = *reinterpret_cast<const f32x4*>(Wl + j * H + f);
          z = fmaf(hv.x, wv.x, z); z = fmaf(hv.y, wv.y, z);
          z = fmaf(hv.z, wv.z, z); z = fmaf(hv.w, wv.w, z);
        }
#pragma unroll
        for (int s = 1; s < 8; s <<= 1) z += __shfl_xor(z, s, 64);
        if (part == 0) sm.o[ev][j] = z + p.b[NH + 1][m * p.bsz[NH + 1] + j];
      }
    }
    __syncthreads();
  }

  static __device__ void run_forward(const GenParams& p) {
    __shared__ Smem sm;
    int m, tile;
    gen_block(gridDim.x, gridDim.y, m, tile);
    const int64_t row0 = (int64_t)tile * kGT;
    forward(p, sm, m, row0);
    for (int i = threadIdx.x; i < kGT * p.out; i += kGThreads) {
      const int ev = i / p.out, j = i % p.out;
      const int64_t r = row0 + ev;
      if (r < p.k) p.theta[((int64_t)m * p.k + r) * p.out + j] = 1.0f + g_softplus(sm.o[ev][j]);
    }
  }

  static __device__ void run_backward(const GenParams& p) {
    __shared__ Smem sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lr = lane & 15, lg = lane >> 4;
    int m, tile;
    gen_block(gridDim.x, gridDim.y, m, tile);
    const int64_t row0 = (int64_t)tile * kGT;
    const float slope = p.slope;
    forward(p, sm, m, row0);
    float* part = p.part + ((int64_t)m * gridDim.x + tile) * p.P;

    // dL/d(last pre-activation) = dL/dtheta * sigmoid(o); zero on rows past k
    for (int i = tid; i < kGT * kGMaxIO; i += kGThreads) {
      const int ev = i / kGMaxIO, j = i % kGMaxIO;
      const int64_t r = row0 + ev;
      float d = 0.f;
      if (j < p.out && r < p.k) d = p.dtheta[((int64_t)m * p.k + r) * p.out + j] * g_sigmoid(sm.o[ev][j]);
      sm.dout[ev][j] = d;
    }
    __syncthreads();
    const int L = NH + 1;   // index of the last layer
    const float* WL = p.W[L] + m * p.wsz[L];
    {   // last layer: dW[j][k] = sum_ev dout[ev][j] A_{NH+1}[ev][k]; db[j] = sum_ev dout[ev][j]
      const int k = tid % H, g = tid / H;
      for (int j = g; j < p.out; j += PPO) {
        float s = 0.f;
        for (int ev = 0; ev < kGT; ++ev) s = fmaf(sm.dout[ev][j], sm.act[NH][ev][k], s);
        part[p.poff_w[L] + j * H + k] = s;
      }
      if (tid < p.out) {
        float s = 0.f;
        for (int ev = 0; ev < kGT; ++ev) s += sm.dout[ev][tid];
        part[p.poff_b[L] + tid] = s;
      }
    }
    __syncthreads();
    {   // delta_{NH+1} = (dout W_L) * leaky'(A_{NH+1}), in place
      const int k = tid % H, g = tid / H;
      float w[kGMaxIO];
#pragma unroll
      for (int j = 0; j < kGMaxIO; ++j) w[j] = j < p.out ? WL[j * H + k] : 0.0f;
      for (int ev = g; ev < kGT; ev += PPO) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < kGMaxIO; ++j) s = fmaf(sm.dout[ev][j], w[j], s);
        float& h = sm.act[NH][ev][k];
        h = s * g_leaky_grad(h, slope);
      }
    }
    __syncthreads();
    const int o0 = 16 * wave;
#pragma unroll
    for (int l = NH - 1; l >= 0; --l) {
      // layer 1 + l maps A_{l+1} (act[l]) -> A_{l+2}; its output signal delta_{l+2} is in act[l+1]
      const float* dl = &sm.act[l + 1][0][0];
      float* A = &sm.act[l][0][0];
      {   // dW[o][k] = sum_ev delta[ev][o] A[ev][k]: rows o0.., 8 column blocks, K = 64 rows
        f32x4 acc[KB];
#pragma unroll
        for (int nb = 0; nb < KB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
        for (int q = 0; q < kGT / 4; ++q) {
          const int ev = 4 * q + lg;
          const float a = dl[ev * LD + o0 + lr];
#pragma unroll
          for (int nb = 0; nb < KB; ++nb) acc[nb] = mfma4(a, A[ev * LD + 16 * nb + lr], acc[nb]);
        }
        float* dW = part + p.poff_w[1 + l];
#pragma unroll
        for (int nb = 0; nb < KB; ++nb)
#pragma unroll
          for (int r = 0; r < 4; ++r) dW[(o0 + 4 * lg + r) * H + 16 * nb + lr] = acc[nb][r];
        if (tid < H) {
          float s = 0.f;
          for (int ev = 0; ev < kGT; ++ev) s += dl[ev * LD + tid];
          part[p.poff_b[1 + l] + tid] = s;
        }
      }
      __syncthreads();   // delta_{l+1} overwrites A_{l+1}, which every wave just read
      f32x4 acc[CB];
      gemm_bwd(p.W[1 + l] + m * p.wsz[1 + l], dl, acc, o0, lr, lg);
      const int k = o0 + 4 * lg;
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        const int ev = 16 * cb + lr;
        f32x4 h = *reinterpret_cast<const f32x4*>(A + ev * LD + k);
        f32x4 v = acc[cb];
        v.x *= g_leaky_grad(h.x, slope); v.y *= g_leaky_grad(h.y, slope);
        v.z *= g_leaky_grad(h.z, slope); v.w *= g_leaky_grad(h.w, slope);
        *reinterpret_cast<f32x4*>(A + ev * LD + k) = v;
      }
      __syncthreads();
    }
    {   // first layer: dW[o][j] = sum_ev delta_1[ev][o] n[ev][j]; db[o] = sum_ev delta_1[ev][o]
      const int o = tid % H, g = tid / H;
      for (int j = g; j < p.in; j += PPO) {
        float s = 0.f;
        for (int ev = 0; ev < kGT; ++ev) s = fmaf(sm.act[0][ev][o], sm.n[ev][j], s);
        part[p.poff_w[0] + o * p.in + j] = s;
      }
      if (g == 0) {
        float s = 0.f;
        for (int ev = 0; ev < kGT; ++ev) s += sm.act[0][ev][o];
        part[p.poff_b[0] + o] = s;
      }
    }
  }
};

template <int H, int NH, int T>
__global__ __launch_bounds__(kGThreads, 2) void k_gen_forward(GenParams p) {
  Gen<H, NH, T, false>::run_forward(p);
}

template <int H, int NH, int T>
__global__ __launch_bounds__(kGThreads, 1) void k_gen_backward(GenParams p) {
  Gen<H, NH, T, true>::run_backward(p);
}

// Sum of the per-tile partials of member blockIdx.y in a fixed order (tile
// slices t = s mod 4 summed side by side, then the four slices in order),
// scattered to the caller's gradient arrays.
struct GenReduceArgs {
  const float* part;
  int64_t P;
  int tiles;
  int n_layers;
  int64_t poff_w[kMaxGenLayers], poff_b[kMaxGenLayers], wsz[kMaxGenLayers], bsz[kMaxGenLayers];
  float* dW[kMaxGenLayers];
  float* db[kMaxGenLayers];
};

constexpr int kRedSlices = 4;   // tile slices summed side by side, then combined in order

__global__ __launch_bounds__(256) void k_gen_reduce(GenReduceArgs r) {
  __shared__ float red[kRedSlices][256 / kRedSlices];
  const int m = blockIdx.y;
  const int le = threadIdx.x % (256 / kRedSlices), sl = threadIdx.x / (256 / kRedSlices);
  const int64_t e = (int64_t)blockIdx.x * (256 / kRedSlices) + le;
  float s = 0.f;
  if (e < r.P) {
    const float* src = r.part + (int64_t)m * r.tiles * r.P + e;
    for (int t = sl; t < r.tiles; t += kRedSlices) s += src[(int64_t)t * r.P];
  }
  red[sl][le] = s;
  __syncthreads();
  if (sl != 0 || e >= r.P) return;
  float v = 0.f;
#pragma unroll
  for (int q = 0; q < kRedSlices; ++q) v += red[q][le];
  for (int l = 0; l < r.n_layers; ++l) {
    if (e >= r.poff_w[l] && e < r.poff_w[l] + r.wsz[l]) { r.dW[l][m * r.wsz[l] + (e - r.poff_w[l])] = v; return; }
    if (e >= r.poff_b[l] && e < r.poff_b[l] + r.bsz[l]) { r.db[l][m * r.bsz[l] + (e - r.poff_b[l])] = v; return; }
  }
}

// Ensemble statistics of theta[M][k][out]: per (row, component) the member
// mean and the population standard deviation about it (two passes over the
// members); rowstat[0][r][c] = mean, rowstat[1][r][c] = sigma.  Sixteen lanes
// share one (row, component): lane j takes members j, j + 16, ..., and the
// sixteen partial sums are added by shuffles in a fixed pattern.
constexpr int kEnsLanes = 16;

__global__ __launch_bounds__(256) void k_ens_rows(const float* __restrict__ theta, int M, int64_t k, int out,
                                                  float* __restrict__ rowstat) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t i = t / kEnsLanes;              // (row, component), uniform across the 16 lanes
  const int j = (int)(t % kEnsLanes);
  const int64_t stride = k * out;
  const bool live = i < stride;
  float s = 0.f;
  if (live)
    for (int m = j; m < M; m += kEnsLanes) s += theta[m * stride + i];
#pragma unroll
  for (int w = 1; w < kEnsLanes; w <<= 1) s += __shfl_xor(s, w, 64);
  const float mean = s / (float)M;
  float q = 0.f;
  if (live)
    for (int m = j; m < M; m += kEnsLanes) {
      const float dv = theta[m * stride + i] - mean;
      q = fmaf(dv, dv, q);
    }
#pragma unroll
  for (int w = 1; w < kEnsLanes; w <<= 1) q += __shfl_xor(q, w, 64);
  if (live && j == 0) {
    rowstat[i] = mean;
    rowstat[stride + i] = sqrtf(q / (float)M);
  }
}

// Batch averages of the row statistics (one workgroup): thread (component
// c, slice q) sums rows q, q + 32, ... of component c (out <= 8); the 32
// slices of a component are then added in a fixed tree.
__global__ __launch_bounds__(256) void k_ens_final(const float* __restrict__ rowstat, int64_t k, int out,
                                                   const float* __restrict__ p_true, float* __restrict__ p_hat,
                                                   float* __restrict__ sigma, float* __restrict__ r_hat) {
  constexpr int kSlices = 256 / kGMaxIO;   // 32
  __shared__ float red[2][kSlices][kGMaxIO];
  const int c = threadIdx.x % kGMaxIO, q = threadIdx.x / kGMaxIO;
  float a = 0.f, b = 0.f;
  if (c < out) {
    // unrolled so that eight rows' loads are in flight at once (the adds keep
    // their order)
#pragma unroll 8
    for (int64_t r = q; r < k; r += kSlices) {
      a += rowstat[r * out + c];
      b += rowstat[k * out + r * out + c];
    }
  }
  red[0][q][c] = a;
  red[1][q][c] = b;
  __syncthreads();
  for (int w = kSlices / 2; w > 0; w >>= 1) {
    if (q < w) {
      red[0][q][c] += red[0][q + w][c];
      red[1][q][c] += red[1][q + w][c];
    }
    __syncthreads();
  }
  if (q == 0 && c < out) {
    const float ph = red[0][0][c] / (float)k;
    p_hat[c] = ph;
    sigma[c] = red[1][0][c] / (float)k;
    if (r_hat) r_hat[c] = (p_true[c] - ph) / p_true[c];
  }
}

struct GenVariant {
  int H, NH;
  void (*fwd[2])(GenParams);   // 64-row, 16-row tiles
  void (*bwd[2])(GenParams);
};

#define SAGIPS_GEN_VARIANT(H_, NH_)                                               \
  {                                                                              \
    H_, NH_, {k_gen_forward<H_, NH_, 64>, k_gen_forward<H_, NH_, 16>},           \
        {k_gen_backward<H_, NH_, 64>, k_gen_backward<H_, NH_, 16> }              \
  }

const GenVariant kGenVariants[] = {SAGIPS_GEN_VARIANT(128, 1), SAGIPS_GEN_VARIANT(128, 2), SAGIPS_GEN_VARIANT(128, 3)};

const GenVariant* find_gen(const sagips_gen& G) {
  const int H = G.width[1], NH = G.n_layers - 2;
  for (const GenVariant& v : kGenVariants)
    if (v.H == H && v.NH == NH) return &v;
  return nullptr;
}

GenParams gen_params(const sagips_gen& G, const float* noise, int64_t k) {
  GenParams p;
  memset(&p, 0, sizeof(p));
  int64_t off = 0;
  for (int l = 0; l < G.n_layers; ++l) {
    p.W[l] = G.W[l];
    p.b[l] = G.b[l];
    p.wsz[l] = (int64_t)G.width[l + 1] * G.width[l];
    p.bsz[l] = G.width[l + 1];
    p.poff_w[l] = off;
    off += p.wsz[l];
    p.poff_b[l] = off;
    off += p.bsz[l];
  }
  p.P = off;
  p.in = G.width[0];
  p.out = G.width[G.n_layers];
  p.k = k;
  p.slope = G.leaky_slope;
  p.noise = noise;
  return p;
}

// Row tile: 64, unless 64-row tiles of all members would not cover the CUs.
inline int gen_rows(const sagips_gen& G, int64_t k, int n_cu) {
  return ((k + 63) / 64) * G.n_members >= n_cu ? 64 : 16;
}
inline int gen_tiles(int64_t k, int T) { return (int)((k + T - 1) / T); }

}  // namespace

bool gen_supported(const sagips_gen& G, const char** why) {
  if (G.n_layers < 3 || G.n_layers > kMaxGenLayers) { *why = "generator needs 3 to 5 layers"; return false; }
  if (G.width[0] < 1 || G.width[0] > kGMaxIO || G.width[G.n_layers] < 1 || G.width[G.n_layers] > kGMaxIO) {
    *why = "generator input and output widths must be in [1, 8]";
    return false;
  }
  for (int l = 1; l < G.n_layers; ++l)
    if (G.width[l] != G.width[1]) { *why = "all hidden widths must be equal"; return false; }
  if (!find_gen(G)) { *why = "unsupported generator shape (hidden width 128 with 1-3 hidden-to-hidden layers)"; return false; }
  return true;
}

size_t gen_backward_workspace(const sagips_gen& G, int64_t k, int n_cu) {
  const GenParams p = gen_params(G, nullptr, k);
  return sizeof(float) * (size_t)p.P * gen_tiles(k, gen_rows(G, k, n_cu)) * G.n_members;
}

size_t ensemble_workspace(const sagips_gen& G, int64_t k) {
  const size_t th = (sizeof(float) * (size_t)G.n_members * k * G.width[G.n_layers] + 255) & ~(size_t)255;
  return th + sizeof(float) * 2 * (size_t)k * G.width[G.n_layers];
}

hipError_t launch_gen_forward(const sagips_gen& G, const float* noise, int64_t k, float* theta, int n_cu,
                              hipStream_t st, Timer* tm) {
  GenParams p = gen_params(G, noise, k);
  p.theta = theta;
  const GenVariant* v = find_gen(G);
  const int T = gen_rows(G, k, n_cu);
  if (tm) tm->begin("gen_forward");
  hipLaunchKernelGGL(v->fwd[T == 64 ? 0 : 1], dim3(gen_tiles(k, T), G.n_members), dim3(kGThreads), 0, st, p);
  if (tm) tm->end();
  return hipGetLastError();
}

hipError_t launch_gen_backward(const sagips_gen& G, const float* noise, int64_t k, const float* dtheta,
                               float* const* dW, float* const* db, void* ws, int n_cu, hipStream_t st, Timer* tm) {
  GenParams p = gen_params(G, noise, k);
  p.dtheta = dtheta;
  p.part = static_cast<float*>(ws);
  const GenVariant* v = find_gen(G);
  const int T = gen_rows(G, k, n_cu);
  const int tiles = gen_tiles(k, T);
  if (tm) tm->begin("gen_backward");
  hipLaunchKernelGGL(v->bwd[T == 64 ? 0 : 1], dim3(tiles, G.n_members), dim3(kGThreads), 0, st, p);
  if (tm) tm->end();
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  GenReduceArgs r;
  memset(&r, 0, sizeof(r));
  r.part = p.part;
  r.P = p.P;
  r.tiles = tiles;
  r.n_layers = G.n_layers;
  for (int l = 0; l < G.n_layers; ++l) {
    r.poff_w[l] = p.poff_w[l];
    r.poff_b[l] = p.poff_b[l];
    r.wsz[l] = p.wsz[l];
    r.bsz[l] = p.bsz[l];
    r.dW[l] = dW[l];
    r.db[l] = db[l];
  }
  if (tm) tm->begin("gen_reduce");
  hipLaunchKernelGGL(k_gen_reduce, dim3((unsigned)((p.P + 256 / kRedSlices - 1) / (256 / kRedSlices)), G.n_members),
                     dim3(256), 0, st, r);
  if (tm) tm->end();
  return hipGetLastError();
}

hipError_t launch_ensemble(const sagips_gen& G, const float* noise, int64_t k, const float* p_true, float* p_hat,
                           float* sigma, float* r_hat, void* ws, int n_cu, hipStream_t st, Timer* tm) {
  const int out = G.width[G.n_layers];
  float* theta = static_cast<float*>(ws);
  const size_t th = (sizeof(float) * (size_t)G.n_members * k * out + 255) & ~(size_t)255;
  float* rowstat = reinterpret_cast<float*>(static_cast<char*>(ws) + th);
  hipError_t e = launch_gen_forward(G, noise, k, theta, n_cu, st, tm);
  if (e != hipSuccess) return e;
  if (tm) tm->begin("ensemble_rows");
  hipLaunchKernelGGL(k_ens_rows, dim3((unsigned)((k * out * kEnsLanes + 255) / 256)), dim3(256), 0, st, theta,
                     G.n_members, k, out, rowstat);
  if (tm) tm->end();
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (tm) tm->begin("ensemble_final");
  hipLaunchKernelGGL(k_ens_final, dim3(1), dim3(256), 0, st, rowstat, k, out, p_true, p_hat, sigma, r_hat);
  if (tm) tm->end();
  return hipGetLastError();
}

}  // namespace sagips
