// Fused fp32 discriminator step on gfx950: forward on fake and real events,
// BCE loss, backward to the weights (dL_D) and to the fake events (dL_G),
// and, when the fake events come from a source, the sampler and the
// per-parameter reduction as well -- one persistent kernel per call.
//
// Network: F -> H -> (H -> H) x NH -> 1, LeakyReLU on the hidden layers
// (paper Sec. V-A), weights in torch.nn.Linear layout.  Events have DX
// coordinates; the network sees F features of them: the coordinates
// themselves (F = DX), or the two observables y0 = x1 + x3, y1 = x2 + x3 of
// the six-parameter, two-observable pipeline (DX = 3, F = 2; Sec. V).
//
// Work decomposition
//   * One persistent workgroup of 8 waves (two per SIMD, so one hides the
//     other's load latency) per CU loops over tiles of T = 64 events; a tile
//     is all fake or all real.  The tile's activations
//     A_1..A_{NH+1} and one spare buffer live in LDS as [T][H+4] fp32
//     (event-major, padded so that the 16-byte fragment reads below are
//     bank-conflict free).  Where the spare buffer would not fit (H = 128
//     with three hidden-to-hidden layers), each backward signal overwrites
//     the activation it replaces, behind one more barrier per layer.
//   * Sampled fake events: event i takes parameter row i / E, so a tile may
//     straddle two rows (E >= T); its per-parameter partials keep one slot
//     per row it touches.
//   * The H x H products run on the fp32 matrix cores
//     (v_mfma_f32_16x16x4_f32).  Forward and backward-data products compute
//     out^T = W' * in^T with M = output feature, N = event, K = input
//     feature; each wave owns 16 output features (and, for H = 64, half of
//     the tile's events).  The W'
//     fragment of lane l is 4 consecutive K values of one row, a 16-byte
//     load from global memory (L2-resident); the activation fragment is the
//     matching 16 bytes of one event's row in LDS.  Because the K order of a
//     product is free, this one mapping serves all four K steps of a load.
//     Backward-data products use a transposed copy of W made per call.
//   * Weight gradients dW = sum_events e * delta^T A (K = events) accumulate
//     in registers across all of the workgroup's tiles: each wave owns 16 rows
//     of every hidden dW (for its events).  They are written once per
//     workgroup and summed over workgroups in a fixed order afterwards.
//   * One backward chain with a unit seed per event serves both losses: the
//     signals are linear in the seed, so dL_D terms are scaled by
//     e_D = dL_D/dz and the fake-input gradient by e_G = dL_G/dz.
//   * The first layer (K = F) and the logit layer (N = 1) are plain VALU work.
#include "device_math.hpp"
#include "kernels.hpp"

#include <string.h>

namespace sagips {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 512;  // 8 waves, two per SIMD
constexpr int kT = 64;         // events per tile
constexpr int kWGPerCU = 1;    // resident workgroups per CU (LDS-limited)
constexpr int kMaxNH = 4;

struct F32Params {
  // network
  const float* W1;             // [H][F]
  const float* b1;             // [H]
  const float* Wh[kMaxNH];     // [H][H]
  const float* WhT[kMaxNH];    // [H][H] transposed copies
  const float* bh[kMaxNH];     // [H]
  const float* Wo;             // [H]
  const float* bo;             // [1]
  float slope;
  // inputs
  const float* fake_x;         // [n_fake][DX] or NULL (then sampled)
  const float* real_x;         // [n_real][DX]
  SourceArgs src;              // valid when fake_x == NULL
  int64_t n_fake, n_real;
  int n_fake_tiles, n_tiles;
  int64_t E;                   // events per parameter row (source path)
  float inv_nf, inv_nr;
  // outputs
  float* logits_fake;
  float* logits_real;
  float* dLg_dx;               // [n_fake][DX] or NULL
  // workspace
  float* wg_part;              // [gridDim.x][P]
  float* loss_part;            // [n_tiles][2]
  float* theta_part;           // [n_fake_tiles][2][2 DX] (source path): slot 0 = row of the
                               // tile's first event, slot 1 = the next row
};

__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float leaky(float v, float s) { return v > 0.0f ? v : s * v; }
__device__ __forceinline__ float leaky_grad(float h, float s) { return h > 0.0f ? 1.0f : s; }

// softplus(t) = max(t, 0) + ln(1 + e^-|t|) on the hardware units (exp2 and
// log2 within 1 ulp; Kahan's log1p keeps the small-argument accuracy).  Only
// one lane in eight evaluates the seeds of an event, so their latency shows.
__device__ __forceinline__ float softplus(float t) { return fmaxf(t, 0.0f) + log1p_k(fast_exp(-fabsf(t))); }

template <int H, int NH, int DX, int F, int FEAT>
struct Fused {
  static_assert(FEAT == SAGIPS_FEAT_IDENTITY ? DX == F : (FEAT == SAGIPS_FEAT_PROXY2 && DX == 3 && F == 2),
                "feature map");
  static constexpr int LD = H + 4;             // LDS row stride in floats
  // Backward signals overwrite the activations they replace when a spare
  // buffer would not fit next to the others in 160 KB of LDS.
  static constexpr bool kInPlace = (NH + 2) * kT * LD * 4 + 8192 > 160 * 1024;
  static constexpr int NB = kInPlace ? NH + 1 : NH + 2;   // activation (+ spare) buffers
  // Products load the next product's first weight fragments during their tail,
  // except in the in-place networks, whose registers are already all in use.
  static constexpr bool kPF = !kInPlace;
  static constexpr int WAVES = kThreads / 64;
  static constexpr int WR = H / 16;            // waves along the output rows (16 rows each)
  static constexpr int WE = WAVES / WR;        // waves along the events
  static constexpr int TE = kT / WE;           // events per wave
  static constexpr int CB = TE / 16;           // 16-event column blocks per wave
  static constexpr int KB = H / 16;            // 16-wide K blocks
  static constexpr int PPO = kThreads / H;     // threads per output feature in VALU loops
  static constexpr int PARTS = kThreads / kT;  // threads per event in the per-event dot products
  static constexpr int PD = 2;                 // weight-fragment prefetch distance (K blocks)
  // The logit pass also forms dW_o and delta_{NH+1} from the activations it
  // already holds (no second pass over the tile, one barrier less), keeping
  // dW_o partials of H / PARTS features per thread; not in the in-place
  // networks, whose registers are all in use.
  static constexpr bool kTopInLogit = !kInPlace;
  static_assert(WR * WE == WAVES && CB >= 1 && TE % 16 == 0, "wave decomposition");
  // per-workgroup partial layout (floats)
  static constexpr int P_DWH = H * H + H;      // dW + db of one hidden layer
  static constexpr int OFF_W1 = NH * P_DWH;    // dW1 [H][F], then db1 [H]
  static constexpr int OFF_WO = OFF_W1 + H * F + H;  // dWo [H], then dbo
  static constexpr int P = OFF_WO + H + 1;

  struct Smem {
    float act[NB][kT][LD];
    float X[kT][F];          // the network's input features
    float xs[FEAT == SAGIPS_FEAT_IDENTITY ? 1 : kT][DX];   // raw coordinates (feature maps only)
    float dxd[kT][DX][2];
    float eD[kT];
    float eG[kT];
    float w1[H][F];          // first-layer weights (the dL/dx products)
    float red[2 * kT * 4];   // >= 2 T DX and >= 2 * waves
  };

  // Index of the buffer that holds delta_l (l = 1 .. NH+1).
  static constexpr __device__ int dbuf(int l) { return kInPlace ? l - 1 : NH + ((NH + 1 - l) & 1); }

  // out^T (this wave's 16 rows x CB event blocks) = Wg * in^T, K = H.  The
  // weight fragments are loaded PD K blocks ahead of their use.
  static __device__ __forceinline__ void gemm(const float* __restrict__ Wg, const float* in, f32x4 (&acc)[CB],
                                              int o0, int e0, int lr, int lg) {
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    const float* wrow = Wg + (o0 + lr) * H + 4 * lg;
    f32x4 a[PD + 1];
#pragma unroll
    for (int q = 0; q < PD; ++q) a[q] = *reinterpret_cast<const f32x4*>(wrow + 16 * q);
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      if (kb + PD < KB) a[(kb + PD) % (PD + 1)] = *reinterpret_cast<const f32x4*>(wrow + 16 * (kb + PD));
      f32x4 b[CB];
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        b[cb] = *reinterpret_cast<const f32x4*>(in + (e0 + 16 * cb + lr) * LD + 16 * kb + 4 * lg);
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) acc[cb] = mfma4(a[kb % (PD + 1)][s], b[cb][s], acc[cb]);
    }
  }

  // The same product where pf holds the first PD weight fragments of Wg on
  // entry and, loaded during the last PD K blocks, those of Wnext (the next
  // product's weights) on exit, so that no product starts by waiting for its
  // weights.
  static __device__ __forceinline__ void gemm_pf(const float* __restrict__ Wg, const float* __restrict__ Wnext,
                                                 f32x4 (&pf)[PD], const float* in, f32x4 (&acc)[CB], int o0,
                                                 int e0, int lr, int lg) {
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    const float* wrow = Wg + (o0 + lr) * H + 4 * lg;
    const float* nrow = Wnext + (o0 + lr) * H + 4 * lg;
    f32x4 a[PD + 1];
#pragma unroll
    for (int q = 0; q < PD; ++q) a[q] = pf[q];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      if (kb + PD < KB) a[(kb + PD) % (PD + 1)] = *reinterpret_cast<const f32x4*>(wrow + 16 * (kb + PD));
      else pf[kb + PD - KB] = *reinterpret_cast<const f32x4*>(nrow + 16 * (kb + PD - KB));
      f32x4 b[CB];
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        b[cb] = *reinterpret_cast<const f32x4*>(in + (e0 + 16 * cb + lr) * LD + 16 * kb + 4 * lg);
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) acc[cb] = mfma4(a[kb % (PD + 1)][s], b[cb][s], acc[cb]);
    }
  }

  // Weight-gradient tiles use a permuted row / column order against LDS bank
  // conflicts.  LDS serves a 64-lane 4-byte read as two passes of 32 lanes over
  // 32 banks; a pass here covers 2 event rows (4 banks apart, row stride H+4
  // floats) x 16 columns, so the 16 columns of a block sit at 8 (i/4) + (i%4)
  // and the neighbouring block fills the gaps (+4).  Row i of wave-row wr is
  // rowmap(wr, i), column j of block kb is colmap(kb, j); both are bijections
  // onto [0, H).
  static constexpr __device__ int rowmap(int wr, int i) {
    return 32 * (wr >> 1) + 8 * (i >> 2) + 4 * (wr & 1) + (i & 3);
  }
  static constexpr __device__ int colmap(int kb, int j) {
    return 32 * (kb >> 1) + 8 * (j >> 2) + 4 * (kb & 1) + (j & 3);
  }

  // accW += sum over this wave's events of e[ev] delta[ev][o] A[ev][k] for the
  // wave's rows o = rowmap(wr, .); dbacc += the e-scaled delta values this lane loaded.
  static __device__ __forceinline__ void wgrad(const float* dlt, const float* A, const float* e,
                                               f32x4 (&accW)[KB], float& dbacc, int wr, int e0, int lr, int lg) {
    const int orow = rowmap(wr, lr);
    int kcol[KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) kcol[kb] = colmap(kb, lr);
#pragma unroll 4
    for (int q = 0; q < TE / 4; ++q) {
      const int ev = e0 + 4 * q + lg;
      const float a = e[ev] * dlt[ev * LD + orow];
      dbacc += a;
      float b[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) b[kb] = A[ev * LD + kcol[kb]];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) accW[kb] = mfma4(a, b[kb], accW[kb]);
    }
  }

  // Per-event dot products over the H features: thread part dp (of PARTS)
  // takes the float4 chunks at 4 dp + 32 c, c < H / (4 PARTS), so that the
  // eight parts of one event read one contiguous 128-byte row segment.
  static constexpr int NCH = H / (4 * PARTS);
  static constexpr __device__ int chunk_off(int dp, int c) { return 4 * dp + 32 * c; }

  static __device__ void run(const F32Params& p) {
    __shared__ Smem sm;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int lr = lane & 15, lg = lane >> 4;
    const int o0 = (wave % WR) * 16;             // this wave's output rows
    const int ew = wave / WR;
    const int e0 = ew * TE;                      // this wave's events
    const float slope = p.slope;

    f32x4 accW[NH][KB];
    float dbacc[NH];
#pragma unroll
    for (int l = 0; l < NH; ++l) {
      dbacc[l] = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) accW[l][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    // VALU accumulators: thread (o = tid % H, part = tid / H) over events ev = part (mod PPO)
    const int vo = tid % H, vpart = tid / H;
    float acc_dW1[F];
#pragma unroll
    for (int j = 0; j < F; ++j) acc_dW1[j] = 0.f;
    float acc_db1 = 0.f, acc_dWo = 0.f, acc_dbo = 0.f;
    // kTopInLogit: dW_o of features chunk_off(dpart, c) + q over this thread's events
    f32x4 dwo[kTopInLogit ? NCH : 1];
#pragma unroll
    for (int c = 0; c < (kTopInLogit ? NCH : 1); ++c) dwo[c] = f32x4{0.f, 0.f, 0.f, 0.f};
    float w1r[F];
#pragma unroll
    for (int j = 0; j < F; ++j) w1r[j] = p.W1[vo * F + j];
    const float b1r = p.b1[vo];
    const float wor = p.Wo[vo];
    // per-event dot products: thread (ev = tid / PARTS, part = tid % PARTS) covers H / PARTS features
    const int dev_ = tid / PARTS, dpart = tid % PARTS;
    for (int i = tid; i < H * F; i += kThreads) sm.w1[i / F][i % F] = p.W1[i];
    // the first weight fragments of the first product (a tile's first hidden layer)
    f32x4 pf[kPF ? PD : 1];
    if constexpr (kPF) {
#pragma unroll
      for (int q = 0; q < PD; ++q) pf[q] = *reinterpret_cast<const f32x4*>(p.Wh[0] + (o0 + lr) * H + 4 * lg + 16 * q);
    }

    for (int tile = blockIdx.x; tile < p.n_tiles; tile += gridDim.x) {
      const bool fake = tile < p.n_fake_tiles;
      const int64_t ev0 = (int64_t)(fake ? tile : tile - p.n_fake_tiles) * kT;
      const int64_t n_here = fake ? p.n_fake : p.n_real;
      const bool sampled = fake && p.fake_x == nullptr;
      // Sampled tiles: the parameter row of the tile's first event, and the
      // tile-local index of the first event of the next row (E >= T, so a
      // tile touches at most these two rows).  n_fake < 2^30 keeps this in 32 bits.
      const uint32_t row_lo = sampled ? (uint32_t)ev0 / (uint32_t)p.E : 0u;
      const int split = sampled ? (int)min<int64_t>((int64_t)(row_lo + 1) * p.E - ev0, kT) : kT;

      // ---- 1. tile inputs: thread (event, coordinate) ---------------------------
      if (tid < kT * DX) {
        const int ev = tid / DX, j = tid % DX;
        const int64_t i = ev0 + ev;
        float xv = 0.5f;
        if (sampled) {
          float da = 0.f, db = 0.f;
          if (i < n_here) {
            const int row = (int)row_lo + (ev >= split ? 1 : 0);
            const Words w = event_words(p.src.base + (uint64_t)i, p.src.stream, p.src.k0, p.src.k1);
            const Shape sh = make_shape(p.src.theta[row * 2 * DX + 2 * j], p.src.theta[row * 2 * DX + 2 * j + 1]);
            const Quantile q = kumaraswamy_w(w.w[j], sh);
            pathwise(q, sh, da, db);
            xv = q.x;
          }
          sm.dxd[ev][j][0] = da;
          sm.dxd[ev][j][1] = db;
        } else {
          const float* src = fake ? p.fake_x : p.real_x;
          if (i < n_here) xv = src[i * DX + j];
        }
        if constexpr (FEAT == SAGIPS_FEAT_IDENTITY) sm.X[ev][j] = xv;
        else sm.xs[ev][j] = xv;
      }
      __syncthreads();
      if constexpr (FEAT == SAGIPS_FEAT_PROXY2) {
        if (tid < kT) {
          sm.X[tid][0] = sm.xs[tid][0] + sm.xs[tid][2];
          sm.X[tid][1] = sm.xs[tid][1] + sm.xs[tid][2];
        }
        __syncthreads();
      }

      // ---- 2. first layer (VALU): A_1 = leaky(X W1^T + b1) -------------------
#pragma unroll 4
      for (int ev = vpart; ev < kT; ev += PPO) {
        float v = b1r;
#pragma unroll
        for (int j = 0; j < F; ++j) v = fmaf(w1r[j], sm.X[ev][j], v);
        sm.act[0][ev][vo] = leaky(v, slope);
      }
      __syncthreads();

      // ---- 3. hidden layers on the matrix cores -----------------------------
#pragma unroll
      for (int l = 0; l < NH; ++l) {
        f32x4 acc[CB];
        if constexpr (kPF) gemm_pf(p.Wh[l], l + 1 < NH ? p.Wh[l + 1] : p.WhT[NH - 1], pf, &sm.act[l][0][0], acc, o0, e0, lr, lg);
        else gemm(p.Wh[l], &sm.act[l][0][0], acc, o0, e0, lr, lg);
        const int o = o0 + 4 * lg;
        const f32x4 bias = *reinterpret_cast<const f32x4*>(p.bh[l] + o);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
          f32x4 v = acc[cb] + bias;
          v.x = leaky(v.x, slope); v.y = leaky(v.y, slope);
          v.z = leaky(v.z, slope); v.w = leaky(v.w, slope);
          *reinterpret_cast<f32x4*>(&sm.act[l + 1][e0 + 16 * cb + lr][o]) = v;
        }
        __syncthreads();
      }

      // ---- 4. logits and BCE seeds (with kTopInLogit also 5, below) ------------
      {
        float* hrow = &sm.act[NH][dev_][0];
        f32x4 hv[NCH], wv[NCH];
        float z = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          const int f = chunk_off(dpart, c);
          hv[c] = *reinterpret_cast<const f32x4*>(hrow + f);
          wv[c] = *reinterpret_cast<const f32x4*>(p.Wo + f);
          z = fmaf(hv[c].x, wv[c].x, z); z = fmaf(hv[c].y, wv[c].y, z);
          z = fmaf(hv[c].z, wv[c].z, z); z = fmaf(hv[c].w, wv[c].w, z);
        }
#pragma unroll
        for (int m = 1; m < PARTS; m <<= 1) z += __shfl_xor(z, m, 64);
        z += p.bo[0];
        const int64_t i = ev0 + dev_;
        const bool valid = i < n_here;
        float l0 = 0.f, l1 = 0.f;
        // kTopInLogit: every lane of the event forms the seeds (the same values),
        // otherwise only part 0
        if (kTopInLogit || dpart == 0) {
          float eD = 0.f, eG = 0.f;
          if (valid) {
            const float sig_neg = fast_rcp(1.0f + fast_exp(z));   // sigmoid(-z)
            if (fake) {
              eD = (1.0f - sig_neg) * p.inv_nf;                // dL_D/dz = sigmoid(z)/N_f
              eG = -sig_neg * p.inv_nf;                        // dL_G/dz = (sigmoid(z)-1)/N_f
              if (dpart == 0) {
                l0 = softplus(z);
                l1 = softplus(-z);
                if (p.logits_fake) p.logits_fake[i] = z;
              }
            } else {
              eD = -sig_neg * p.inv_nr;                        // (sigmoid(z)-1)/N_r
              if (dpart == 0) {
                l0 = softplus(-z);
                if (p.logits_real) p.logits_real[i] = z;
              }
            }
          }
          if (dpart == 0) {
            sm.eD[dev_] = eD;
            sm.eG[dev_] = eG;
          }
          if constexpr (kTopInLogit) {
            // ---- 5. logit-layer gradients and delta_{NH+1} in place --------------
            // dW_o += e_D h, db_o += e_D, h -> w_o LeakyReLU'(h) for this lane's features
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
              dwo[c].x = fmaf(eD, hv[c].x, dwo[c].x); dwo[c].y = fmaf(eD, hv[c].y, dwo[c].y);
              dwo[c].z = fmaf(eD, hv[c].z, dwo[c].z); dwo[c].w = fmaf(eD, hv[c].w, dwo[c].w);
              f32x4 d;
              d.x = wv[c].x * leaky_grad(hv[c].x, slope); d.y = wv[c].y * leaky_grad(hv[c].y, slope);
              d.z = wv[c].z * leaky_grad(hv[c].z, slope); d.w = wv[c].w * leaky_grad(hv[c].w, slope);
              *reinterpret_cast<f32x4*>(hrow + chunk_off(dpart, c)) = d;
            }
            if (dpart == 0) acc_dbo += eD;
          }
        }
        l0 = wave_sum(l0);
        l1 = wave_sum(l1);
        if (lane == 0) { sm.red[2 * wave] = l0; sm.red[2 * wave + 1] = l1; }
      }
      __syncthreads();
      if (tid < 2) {
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) s += sm.red[2 * w + tid];
        p.loss_part[(int64_t)tile * 2 + tid] = s;
      }

      if constexpr (!kTopInLogit) {
        // ---- 5. logit-layer gradients and delta_{NH+1} in place, one pass --------
#pragma unroll 4
        for (int ev = vpart; ev < kT; ev += PPO) {
          const float e = sm.eD[ev];
          float& h = sm.act[NH][ev][vo];
          const float hv = h;
          acc_dWo = fmaf(e, hv, acc_dWo);
          if (vo == 0) acc_dbo += e;
          h = wor * leaky_grad(hv, slope);
        }
        __syncthreads();
      }

      // ---- 6. hidden layers backward ------------------------------------------
#pragma unroll
      for (int l = NH - 1; l >= 0; --l) {
        // layer l maps A_{l+1} (act[l]) -> A_{l+2}; its output signal is delta_{l+2}
        const float* dout = &sm.act[dbuf(l + 2)][0][0];
        float* din = &sm.act[dbuf(l + 1)][0][0];
        const float* Ain = &sm.act[l][0][0];
        wgrad(dout, Ain, sm.eD, accW[l], dbacc[l], wave % WR, e0, lr, lg);
        if constexpr (kInPlace) __syncthreads();   // din overwrites Ain, which every wave's wgrad read
        f32x4 acc[CB];
        if constexpr (kPF) gemm_pf(p.WhT[l], l > 0 ? p.WhT[l - 1] : p.Wh[0], pf, dout, acc, o0, e0, lr, lg);
        else gemm(p.WhT[l], dout, acc, o0, e0, lr, lg);
        const int k = o0 + 4 * lg;
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
          const int ev = e0 + 16 * cb + lr;
          const f32x4 h = *reinterpret_cast<const f32x4*>(Ain + ev * LD + k);
          f32x4 v = acc[cb];
          v.x *= leaky_grad(h.x, slope); v.y *= leaky_grad(h.y, slope);
          v.z *= leaky_grad(h.z, slope); v.w *= leaky_grad(h.w, slope);
          *reinterpret_cast<f32x4*>(din + ev * LD + k) = v;
        }
        __syncthreads();
      }

      // ---- 7. first-layer gradients --------------------------------------------
      const float* d1 = &sm.act[dbuf(1)][0][0];
#pragma unroll 4
      for (int ev = vpart; ev < kT; ev += PPO) {
        const float ed = sm.eD[ev] * d1[ev * LD + vo];
        acc_db1 += ed;
#pragma unroll
        for (int j = 0; j < F; ++j) acc_dW1[j] = fmaf(ed, sm.X[ev][j], acc_dW1[j]);
      }

      // ---- 8. fake events: dL_G/dx and the per-parameter partial ---------------
      if (fake) {
        // thread (dev_, dpart) sums its H / PARTS first-layer rows for every input j
        float g[F];
#pragma unroll
        for (int j = 0; j < F; ++j) g[j] = 0.f;
        const float* drow = d1 + dev_ * LD;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          const f32x4 dv = *reinterpret_cast<const f32x4*>(drow + chunk_off(dpart, c));
          const int f = chunk_off(dpart, c);
#pragma unroll
          for (int j = 0; j < F; ++j) {
            g[j] = fmaf(dv.x, sm.w1[f][j], g[j]);
            g[j] = fmaf(dv.y, sm.w1[f + 1][j], g[j]);
            g[j] = fmaf(dv.z, sm.w1[f + 2][j], g[j]);
            g[j] = fmaf(dv.w, sm.w1[f + 3][j], g[j]);
          }
        }
#pragma unroll
        for (int j = 0; j < F; ++j) {
#pragma unroll
          for (int m = 1; m < PARTS; m <<= 1) g[j] += __shfl_xor(g[j], m, 64);
        }
        if (dpart == 0) {
          const float eg = sm.eG[dev_];
          const int64_t i = ev0 + dev_;
          // dL_G/dx: the features' gradient through the feature map's Jacobian
          float gx[DX];
          if constexpr (FEAT == SAGIPS_FEAT_IDENTITY) {
#pragma unroll
            for (int j = 0; j < DX; ++j) gx[j] = g[j] * eg;
          } else {
            gx[0] = g[0] * eg;
            gx[1] = g[1] * eg;
            gx[2] = gx[0] + gx[1];
          }
#pragma unroll
          for (int j = 0; j < DX; ++j) {
            if (p.dLg_dx && i < n_here) p.dLg_dx[i * DX + j] = gx[j];
            if (sampled) {
              sm.red[2 * (dev_ * DX + j)] = gx[j] * sm.dxd[dev_][j][0];
              sm.red[2 * (dev_ * DX + j) + 1] = gx[j] * sm.dxd[dev_][j][1];
            }
          }
        }
        if (sampled) {
          __syncthreads();
          if (tid < 8 * 2 * DX) {
            // lane (component c = 2 j + (a|b), part q) sums events q, q + 8, ...;
            // the terms sit at red[2 (ev DX + j) + ab].  Slot 0 takes the events of
            // the tile's first row, slot 1 those of the next; the 8 parts of a
            // component are then added across lanes.
            const int c = tid >> 3, q = tid & 7;
            const int j = c >> 1, ab = c & 1;
            float s0 = 0.f, s1 = 0.f;
#pragma unroll
            for (int k = 0; k < kT / 8; ++k) {
              const int ev = q + 8 * k;
              const float t = sm.red[2 * (ev * DX + j) + ab];
              s0 += ev < split ? t : 0.f;
              s1 += ev < split ? 0.f : t;
            }
#pragma unroll
            for (int m = 1; m < 8; m <<= 1) {
              s0 += __shfl_xor(s0, m, 64);
              s1 += __shfl_xor(s1, m, 64);
            }
            if (q == 0) {
              p.theta_part[((int64_t)tile * 2) * 2 * DX + c] = s0;
              p.theta_part[((int64_t)tile * 2 + 1) * 2 * DX + c] = s1;
            }
          }
        }
      }
      __syncthreads();
    }

    // ---- per-workgroup partials ------------------------------------------------
    float* out = p.wg_part + (int64_t)blockIdx.x * P;
    // hidden dW: waves with equal rows and different event groups are added in ew order
    float* stage = &sm.act[0][0][0];           // WE > 1: [NH][16][H] per event group
#pragma unroll
    for (int g = 0; g < WE; ++g) {
      if (ew == g) {
#pragma unroll
        for (int l = 0; l < NH; ++l)
#pragma unroll
          for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int o = rowmap(wave % WR, 4 * lg + r), k = colmap(kb, lr);
              float v = accW[l][kb][r];
              if (WE > 1) {
                float& st = stage[(l * H + o) * H + k];
                v = (g == 0) ? v : st + v;
                if (g < WE - 1) st = v;
              }
              if (g == WE - 1) out[l * P_DWH + o * H + k] = v;
            }
      }
      if (WE > 1) __syncthreads();
    }
    // hidden-layer db: lanes lg = 0..3 hold four event classes of row rowmap(wr, lr)
    float* dbst = &sm.red[0];
#pragma unroll
    for (int g = 0; g < WE; ++g) {
      if (ew == g) {
#pragma unroll
        for (int l = 0; l < NH; ++l) {
          float v = dbacc[l];
          v += __shfl_xor(v, 16, 64);
          v += __shfl_xor(v, 32, 64);
          if (lg == 0) {
            const int o = rowmap(wave % WR, lr);
            if (WE > 1) {
              float& st = dbst[l * H + o];
              v = (g == 0) ? v : st + v;
              if (g < WE - 1) st = v;
            }
            if (g == WE - 1) out[l * P_DWH + H * H + o] = v;
          }
        }
      }
      if (WE > 1) __syncthreads();
    }
    // VALU partials: combine the PPO parts of each feature in a fixed order
    float* red = &sm.act[0][0][0];
    constexpr int NV = F + 2;  // dW1[F], db1, dWo per feature
    __syncthreads();
    if constexpr (kTopInLogit) {
      // dW_o: the 8 events of a wave (lanes dpart + 8 m), then the waves in order
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int m = 8; m < 64; m <<= 1) {
          dwo[c].x += __shfl_xor(dwo[c].x, m, 64); dwo[c].y += __shfl_xor(dwo[c].y, m, 64);
          dwo[c].z += __shfl_xor(dwo[c].z, m, 64); dwo[c].w += __shfl_xor(dwo[c].w, m, 64);
        }
      float* wst = red + (NV + 1) * kThreads;   // [WAVES][H]
      if (lane < PARTS) {
#pragma unroll
        for (int c = 0; c < NCH; ++c)
          *reinterpret_cast<f32x4*>(wst + wave * H + chunk_off(lane, c)) = dwo[c];
      }
    }
#pragma unroll
    for (int j = 0; j < F; ++j) red[j * kThreads + tid] = acc_dW1[j];
    red[F * kThreads + tid] = acc_db1;
    red[(F + 1) * kThreads + tid] = acc_dWo;
    red[NV * kThreads + tid] = acc_dbo;
    __syncthreads();
    if (tid < H) {
      float v[NV];
#pragma unroll
      for (int c = 0; c < NV; ++c) {
        float s = 0.f;
        for (int q = 0; q < PPO; ++q) s += red[c * kThreads + q * H + tid];
        v[c] = s;
      }
#pragma unroll
      for (int j = 0; j < F; ++j) out[OFF_W1 + tid * F + j] = v[j];
      out[OFF_W1 + H * F + tid] = v[F];
      if constexpr (kTopInLogit) {
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) s += red[(NV + 1) * kThreads + w * H + tid];
        out[OFF_WO + tid] = s;
      } else {
        out[OFF_WO + tid] = v[F + 1];
      }
    }
    if (tid == 0) {
      float s = 0.f;
      for (int q = 0; q < kThreads; ++q) s += red[NV * kThreads + q];
      out[OFF_WO + H] = s;
    }
  }
};

template <int H, int NH, int DX, int F, int FEAT>
__global__ __launch_bounds__(kThreads, 1) void k_disc_f32(F32Params p) {
  Fused<H, NH, DX, F, FEAT>::run(p);
}

// WT[k][o] = W[o][k] for the H x H hidden layers (blockIdx.z = layer).
struct TransposeArgs {
  const float* W[kMaxNH];
  float* WT[kMaxNH];
};

__global__ __launch_bounds__(256) void k_transpose(TransposeArgs t_, int H) {
  __shared__ float t[32][33];
  const float* W = t_.W[blockIdx.z];
  float* WT = t_.WT[blockIdx.z];
  const int bx = blockIdx.x * 32, by = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int r = ty; r < 32; r += 8) t[r][tx] = W[(by + r) * H + bx + tx];
  __syncthreads();
  for (int r = ty; r < 32; r += 8) WT[(bx + r) * H + by + tx] = t[tx][r];
}

// All fixed-order reductions after the fused kernel, in one launch:
//   blocks [0, wg_blocks)        sum over workgroups of every gradient partial,
//                                scattered to the caller's arrays (segment table);
//   block  wg_blocks             the two losses from the per-tile sums;
//   blocks wg_blocks + 1 + row   dL_G/dtheta of one parameter row from the slots of
//                                the tiles that hold its events.
struct Segments {
  int n;
  int off[2 * kMaxNH + 4];
  int len[2 * kMaxNH + 4];
  float* dst[2 * kMaxNH + 4];
};

struct ReduceArgs {
  const float* wg_part;
  int n_wg, P, wg_blocks;
  Segments sg;
  const float* loss_part;
  int n_fake_tiles, n_tiles;
  float inv_nf, inv_nr;
  float* loss_d;
  float* loss_g;
  const float* theta_part;
  int64_t E;
  int C;
  float* dLg_dtheta;
};

constexpr int kRedElems = 32;   // elements per block
constexpr int kRedSlices = 8;   // workgroup ranges summed side by side, then combined in order

__global__ __launch_bounds__(256) void k_reduce_all(ReduceArgs r) {
  __shared__ float red[256];
  const int tid = threadIdx.x;
  if ((int)blockIdx.x < r.wg_blocks) {
    const int le = tid % kRedElems, sl = tid / kRedElems;
    const int e = blockIdx.x * kRedElems + le;
    const int per = (r.n_wg + kRedSlices - 1) / kRedSlices;
    const int g0 = sl * per, g1 = min(r.n_wg, g0 + per);
    float s = 0.f;
    if (e < r.P)
      for (int g = g0; g < g1; ++g) s += r.wg_part[(int64_t)g * r.P + e];
    red[sl * kRedElems + le] = s;
    __syncthreads();
    if (sl != 0 || e >= r.P) return;
    float t = 0.f;
#pragma unroll
    for (int q = 0; q < kRedSlices; ++q) t += red[q * kRedElems + le];
    for (int i = 0; i < r.sg.n; ++i)
      if (e >= r.sg.off[i] && e < r.sg.off[i] + r.sg.len[i]) {
        if (r.sg.dst[i]) r.sg.dst[i][e - r.sg.off[i]] = t;
        break;
      }
    return;
  }
  if ((int)blockIdx.x == r.wg_blocks) {
    float sf = 0.f, sgg = 0.f, sr = 0.f;
    for (int t = tid; t < r.n_tiles; t += 256) {
      if (t < r.n_fake_tiles) { sf += r.loss_part[2 * t]; sgg += r.loss_part[2 * t + 1]; }
      else sr += r.loss_part[2 * t];
    }
    sf = wave_sum(sf); sgg = wave_sum(sgg); sr = wave_sum(sr);
    if ((tid & 63) == 0) { red[3 * (tid >> 6)] = sf; red[3 * (tid >> 6) + 1] = sgg; red[3 * (tid >> 6) + 2] = sr; }
    __syncthreads();
    if (tid == 0) {
      float a = 0.f, b = 0.f, c = 0.f;
      for (int w = 0; w < 4; ++w) { a += red[3 * w]; b += red[3 * w + 1]; c += red[3 * w + 2]; }
      if (r.loss_d) *r.loss_d = c * r.inv_nr + a * r.inv_nf;
      if (r.loss_g) *r.loss_g = b * r.inv_nf;
    }
    return;
  }
  // one parameter row: its events fill tiles t0..t1; a tile holds the row in
  // slot 0 if the row starts at or before the tile, else in slot 1.  Thread
  // (component c, slice s) sums tiles t0 + s, t0 + s + S, ...; slices combined in order.
  const int row = blockIdx.x - r.wg_blocks - 1;
  const int S = 256 / r.C;
  const int c = tid % r.C, sl = tid / r.C;
  const int64_t t0 = (int64_t)row * r.E / kT, t1 = ((int64_t)row * r.E + r.E - 1) / kT;
  float s = 0.f;
  if (sl < S)
    for (int64_t t = t0 + sl; t <= t1; t += S) {
      const int slot = (t * kT) / r.E == row ? 0 : 1;
      s += r.theta_part[(t * 2 + slot) * r.C + c];
    }
  red[tid] = s;
  __syncthreads();
  if (tid < r.C) {
    float t = 0.f;
    for (int q = 0; q < S; ++q) t += red[q * r.C + tid];
    r.dLg_dtheta[row * r.C + tid] = t;
  }
}

inline size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

struct Layout {
  int H, NH, DX, F, P;
  size_t off_wt, off_wg, off_loss, off_theta, total;
};

template <int H, int NH, int DX, int F, int FEAT>
Layout layout_for(const DiscArgs& a, int n_wg) {
  using K = Fused<H, NH, DX, F, FEAT>;
  Layout L;
  L.H = H; L.NH = NH; L.DX = DX; L.F = F; L.P = K::P;
  const int64_t nft = (a.n_fake + kT - 1) / kT, nrt = (a.n_real + kT - 1) / kT;
  size_t o = 0;
  L.off_wt = o; o += align256(sizeof(float) * NH * H * H);
  L.off_wg = o; o += align256(sizeof(float) * (size_t)n_wg * kWGPerCU * K::P);
  L.off_loss = o; o += align256(sizeof(float) * 2 * (size_t)(nft + nrt));
  L.off_theta = o; o += align256(sizeof(float) * 2 * 2 * DX * (size_t)nft);
  L.total = o;
  return L;
}

typedef void (*KernelFn)(F32Params);

struct Variant {
  int H, NH, DX, F, FEAT;
  KernelFn fn;
  Layout (*layout)(const DiscArgs&, int);
  int P;
};

#define SAGIPS_F32_VARIANT(H_, NH_, DX_, F_, FEAT_)                                          \
  { H_, NH_, DX_, F_, FEAT_, k_disc_f32<H_, NH_, DX_, F_, FEAT_>, layout_for<H_, NH_, DX_, F_, FEAT_>, \
    Fused<H_, NH_, DX_, F_, FEAT_>::P }
#define SAGIPS_F32_ID(H_, NH_, D_) SAGIPS_F32_VARIANT(H_, NH_, D_, D_, SAGIPS_FEAT_IDENTITY)

const Variant kVariants[] = {
    SAGIPS_F32_ID(64, 1, 2),  SAGIPS_F32_ID(64, 2, 2),  SAGIPS_F32_ID(64, 3, 2),
    SAGIPS_F32_ID(128, 1, 2), SAGIPS_F32_ID(128, 2, 2),
    SAGIPS_F32_ID(64, 1, 3),  SAGIPS_F32_ID(64, 2, 3),  SAGIPS_F32_ID(128, 2, 3),
    // the paper's discriminator, 2 -> 128 -> 128 -> 128 -> 128 -> 1, on the two observables
    SAGIPS_F32_VARIANT(128, 3, 3, 2, SAGIPS_FEAT_PROXY2),
};

const Variant* find_variant(const sagips_mlp& D, int d) {
  const int H = D.width[1];
  const int NH = D.n_layers - 2;
  const int F = D.width[0];
  for (const Variant& v : kVariants)
    if (v.H == H && v.NH == NH && v.DX == d && v.F == F && v.FEAT == D.features) return &v;
  return nullptr;
}

}  // namespace

int disc_f32_tile() { return kT; }

bool disc_f32_supported(const sagips_mlp& D, int d, const char** why) {
  if (D.features == SAGIPS_FEAT_HD8) { *why = "fp32 discriminator supports IDENTITY and PROXY2 features"; return false; }
  if (D.features == SAGIPS_FEAT_IDENTITY && D.width[0] != d) { *why = "width[0] must equal d for IDENTITY features"; return false; }
  if (D.n_layers < 3) { *why = "fp32 discriminator needs at least one hidden-to-hidden layer"; return false; }
  for (int l = 1; l < D.n_layers; ++l)
    if (D.width[l] != D.width[1]) { *why = "all hidden widths must be equal"; return false; }
  if (D.width[D.n_layers] != 1) { *why = "last layer must have width 1"; return false; }
  if (!find_variant(D, d)) {
    *why = "unsupported fp32 shape (IDENTITY: hidden width 64 with 1-3 or 128 with 1-2 hidden-to-hidden layers, "
           "d 2, or 3 with fewer layers; PROXY2: hidden width 128 with 3 hidden-to-hidden layers)";
    return false;
  }
  return true;
}

size_t disc_f32_workspace(const DiscArgs& a, int n_cu) {
  const Variant* v = find_variant(*a.D, a.d);
  return v ? v->layout(a, n_cu).total : 0;
}

hipError_t launch_disc_f32(const DiscArgs& a, void* ws, int n_cu, hipStream_t st, Timer* tm) {
  const Variant* v = find_variant(*a.D, a.d);
  const sagips_mlp& D = *a.D;
  const Layout L = v->layout(a, n_cu);
  char* base = static_cast<char*>(ws);
  float* WT = reinterpret_cast<float*>(base + L.off_wt);
  const int H = v->H, NH = v->NH, F = v->F, DX = v->DX;

  F32Params p;
  memset(&p, 0, sizeof(p));
  p.W1 = D.W[0];
  p.b1 = D.b[0];
  for (int l = 0; l < NH; ++l) {
    p.Wh[l] = D.W[1 + l];
    p.bh[l] = D.b[1 + l];
    p.WhT[l] = WT + (size_t)l * H * H;
  }
  p.Wo = D.W[NH + 1];
  p.bo = D.b[NH + 1];
  p.slope = D.leaky_slope;
  p.fake_x = a.fake_x;
  p.real_x = a.real_x;
  if (a.fake_src) p.src = *a.fake_src;
  p.n_fake = a.n_fake;
  p.n_real = a.n_real;
  p.n_fake_tiles = (int)((a.n_fake + kT - 1) / kT);
  p.n_tiles = p.n_fake_tiles + (int)((a.n_real + kT - 1) / kT);
  p.E = a.fake_src ? a.fake_src->E : 1;
  p.inv_nf = 1.0f / (float)a.n_fake;
  p.inv_nr = 1.0f / (float)a.n_real;
  p.logits_fake = a.out->logits_fake;
  p.logits_real = a.out->logits_real;
  p.dLg_dx = a.out->dLg_dx;
  p.wg_part = reinterpret_cast<float*>(base + L.off_wg);
  p.loss_part = reinterpret_cast<float*>(base + L.off_loss);
  p.theta_part = reinterpret_cast<float*>(base + L.off_theta);

  if (tm) tm->begin("disc_f32_transpose");
  {
    TransposeArgs ta;
    memset(&ta, 0, sizeof(ta));
    for (int l = 0; l < NH; ++l) { ta.W[l] = p.Wh[l]; ta.WT[l] = const_cast<float*>(p.WhT[l]); }
    hipLaunchKernelGGL(k_transpose, dim3(H / 32, H / 32, NH), dim3(256), 0, st, ta, H);
  }
  if (tm) tm->end();
  if (tm) tm->begin("disc_f32_fused");
  hipLaunchKernelGGL(v->fn, dim3(n_cu * kWGPerCU), dim3(kThreads), 0, st, p);
  if (tm) tm->end();
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;

  ReduceArgs r;
  memset(&r, 0, sizeof(r));
  r.wg_part = p.wg_part;
  r.n_wg = n_cu * kWGPerCU;
  r.P = L.P;
  if (a.out->dW[0]) {
    Segments& sg = r.sg;
    int n = 0;
    for (int l = 0; l < NH; ++l) {
      sg.off[n] = l * (H * H + H); sg.len[n] = H * H; sg.dst[n++] = a.out->dW[1 + l];
      sg.off[n] = l * (H * H + H) + H * H; sg.len[n] = H; sg.dst[n++] = a.out->db[1 + l];
    }
    const int offw1 = NH * (H * H + H);
    sg.off[n] = offw1; sg.len[n] = H * F; sg.dst[n++] = a.out->dW[0];
    sg.off[n] = offw1 + H * F; sg.len[n] = H; sg.dst[n++] = a.out->db[0];
    const int offwo = offw1 + H * F + H;
    sg.off[n] = offwo; sg.len[n] = H; sg.dst[n++] = a.out->dW[NH + 1];
    sg.off[n] = offwo + H; sg.len[n] = 1; sg.dst[n++] = a.out->db[NH + 1];
    sg.n = n;
    r.wg_blocks = (L.P + kRedElems - 1) / kRedElems;
  }
  r.loss_part = p.loss_part;
  r.n_fake_tiles = p.n_fake_tiles;
  r.n_tiles = p.n_tiles;
  r.inv_nf = p.inv_nf;
  r.inv_nr = p.inv_nr;
  r.loss_d = a.out->loss_d;
  r.loss_g = a.out->loss_g;
  r.theta_part = p.theta_part;
  r.E = p.E;
  r.C = 2 * DX;
  r.dLg_dtheta = a.out->dLg_dtheta;
  const int theta_blocks = (a.fake_src && a.out->dLg_dtheta) ? a.fake_src->n_theta : 0;
  if (tm) tm->begin("disc_f32_reduce");
  hipLaunchKernelGGL(k_reduce_all, dim3(r.wg_blocks + 1 + theta_blocks), dim3(256), 0, st, r);
  if (tm) tm->end();
  return hipGetLastError();
}

}  // namespace sagips
