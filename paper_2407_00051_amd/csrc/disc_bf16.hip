// bf16-operand / fp32-accumulate discriminator step on gfx950 for wide
// networks (hidden width 256 or 512), where weight gradients cannot stay in
// registers across tiles.  The step is processed in chunks of event rows
// (all fake or all real); each chunk goes through these kernels:
//
//   k_prep      features of every row (sampling fake events in place, HD8 map)
//   k_first_fwd A_1 = bf16(LeakyReLU(feat W1^T + b1))          (VALU, K <= 8)
//   k_gemm<FWD> A_{l+1} = bf16(LeakyReLU(A_l W^T + b))         (bf16 MFMA)
//   k_logit     z = A_L w_o + b_o, BCE seeds, delta_L = bf16(w_o * leaky'(A_L))
//   k_wgrad     dW partials = sum_rows (e_D delta) (x) A        (bf16 MFMA, K = rows)
//   k_gemm<BWD> delta_l = bf16((delta_{l+1} W) * leaky'(A_l))  (bf16 MFMA)
//   k_first_bwd dW1, db1 partials and dL_G/dx (through the HD8 Jacobian)
//
// Activations and signals are stored event-major [rows][H] bf16.  Forward
// and backward-data products compute out^T = W' in^T (M = output feature,
// N = event, K = input feature): both operands then have K contiguous in
// memory and the accumulator fragment of a lane is 4 consecutive features of
// one event, an 8-byte event-major store.  The weight-gradient product has
// K = events; its operands are read from event-major LDS tiles with the
// gfx950 transpose load ds_read_b64_tr_b16, which hands every lane 4
// consecutive rows of one column.
//
// Backward signals carry a unit seed per event; the weight gradients scale
// them by e_D = dL_D/dz while staging (and round to bf16 again), dL_G/dx
// scales the first-layer signal by e_G = dL_G/dz.  All sums are fixed-order:
// chunk partials are added to fp32 accumulators chunk by chunk.
#include "device_math.hpp"
#include "kernels.hpp"

#include <string.h>

#include <algorithm>

namespace sagips {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

constexpr int kMaxNH = 4;
constexpr int kChunkRows = 1 << 20;   // rows per chunk (fake or real), multiple of 128

// fp32 -> bf16, round to nearest even (finite inputs).
__device__ __forceinline__ u16 bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (u16)(u >> 16);
}
__device__ __forceinline__ float bf16_to_f32(u16 h) { return __uint_as_float(((uint32_t)h) << 16); }

// PER consecutive bf16 values (PER = 4 or 8, 8- or 16-byte aligned) <-> fp32.
template <int PER>
__device__ __forceinline__ void load_bf16(const u16* p, float (&v)[PER]) {
  uint32_t w[PER / 2];
  if constexpr (PER == 4) {
    const uint2 t = *reinterpret_cast<const uint2*>(p);
    w[0] = t.x; w[1] = t.y;
  } else {
    const uint4 t = *reinterpret_cast<const uint4*>(p);
    w[0] = t.x; w[1] = t.y; w[2] = t.z; w[3] = t.w;
  }
#pragma unroll
  for (int q = 0; q < PER / 2; ++q) {
    v[2 * q] = __uint_as_float(w[q] << 16);
    v[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
  }
}
template <int PER>
__device__ __forceinline__ void store_bf16(u16* p, const float (&v)[PER]) {
  uint32_t w[PER / 2];
#pragma unroll
  for (int q = 0; q < PER / 2; ++q) w[q] = (uint32_t)bf16_bits(v[2 * q]) | ((uint32_t)bf16_bits(v[2 * q + 1]) << 16);
  if constexpr (PER == 4) *reinterpret_cast<uint2*>(p) = make_uint2(w[0], w[1]);
  else *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ __forceinline__ float leaky(float v, float s) { return v > 0.0f ? v : s * v; }
__device__ __forceinline__ float leaky_grad(float h, float s) { return h > 0.0f ? 1.0f : s; }
__device__ __forceinline__ float softplus(float t) { return fmaxf(t, 0.0f) + log1pf(expf(-fabsf(t))); }

__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Weights: bf16 copies of the hidden layers, plain and transposed.
__global__ __launch_bounds__(256) void k_weights_bf16(const float* __restrict__ W, u16* __restrict__ Wb,
                                                      u16* __restrict__ WTb, int H) {
  __shared__ u16 t[32][33];
  const int bx = blockIdx.x * 32, by = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int r = ty; r < 32; r += 8) {
    const u16 v = bf16_bits(W[(by + r) * H + bx + tx]);
    Wb[(by + r) * H + bx + tx] = v;
    t[r][tx] = v;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) WTb[(bx + r) * H + by + tx] = t[tx][r];
}

// ---------------------------------------------------------------------------
// Rows of one chunk: features (and x for fake rows).  Rows past `valid` are
// padding: features 0.5, never stored anywhere visible.
struct ChunkArgs {
  int64_t row0;       // first event index (within the fake or the real batch)
  int rows;           // padded row count (multiple of 128)
  int valid;          // real rows in this chunk
  int fake;
};

// The two log features come from the quantile's log domain for sampled
// events: ln x1 = lam1 / a1 and ln(1 - x3) = log1mexp(lam3 / a3), which stay
// accurate (and finite) where fp32 x3 has rounded to within ulps of 1.  Buffer
// events only have their fp32 values: ln x1 and log1p(-x3) of those.
template <int D, bool kHD8>
__global__ __launch_bounds__(256) void k_prep(ChunkArgs c, const float* __restrict__ xin, SourceArgs src, int sampled,
                                              float* __restrict__ feat, float* __restrict__ xs) {
  constexpr int F = kHD8 ? 8 : D;
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r >= c.rows) return;
  float x[D];
  float lnx1 = 0.f, ln1mx3 = 0.f;
  if (r < c.valid) {
    const int64_t i = c.row0 + r;
    if (sampled) {
      const int row = (int)(i / src.E);
      const Words w = event_words(src.base + (uint64_t)i, src.stream, src.k0, src.k1);
#pragma unroll
      for (int j = 0; j < D; ++j) {
        const Shape sh = make_shape(src.theta[row * 2 * D + 2 * j], src.theta[row * 2 * D + 2 * j + 1]);
        const Quantile q = kumaraswamy_w(w.w[j], sh);
        x[j] = q.x;
        if constexpr (kHD8) {
          if (j == 0) lnx1 = log_x(q, sh);
          if (j == D - 1) ln1mx3 = log1mexp(log_x(q, sh));
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < D; ++j) x[j] = xin[i * D + j];
      lnx1 = logf(x[0]);
      ln1mx3 = log1pf(-x[D - 1]);
    }
  } else {
#pragma unroll
    for (int j = 0; j < D; ++j) x[j] = 0.5f;
    lnx1 = logf(0.5f);
    ln1mx3 = logf(0.5f);
  }
  if (c.fake) {
#pragma unroll
    for (int j = 0; j < D; ++j) xs[(int64_t)r * D + j] = x[j];
  }
  float f[F];
  if constexpr (kHD8) {
    f[0] = x[0]; f[1] = x[1]; f[2] = x[2];
    f[3] = x[0] * x[1]; f[4] = x[1] * x[2]; f[5] = x[0] * x[2];
    f[6] = lnx1;
    f[7] = ln1mx3;
  } else {
#pragma unroll
    for (int j = 0; j < D; ++j) f[j] = x[j];
  }
#pragma unroll
  for (int j = 0; j < F; ++j) feat[(int64_t)r * F + j] = f[j];
}

// A_1[r][o] for 8 consecutive o per thread.
template <int F>
__global__ __launch_bounds__(256) void k_first_fwd(const float* __restrict__ feat, const float* __restrict__ W1,
                                                   const float* __restrict__ b1, int H, int rows, float slope,
                                                   u16* __restrict__ A1) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int per_row = H / 8;
  const int64_t r = t / per_row;
  const int o0 = (int)(t % per_row) * 8;
  if (r >= rows) return;
  float f[F];
#pragma unroll
  for (int j = 0; j < F; ++j) f[j] = feat[r * F + j];
  uint32_t packed[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float v2[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int o = o0 + 2 * q + h;
      float v = b1[o];
#pragma unroll
      for (int j = 0; j < F; ++j) v = fmaf(W1[o * F + j], f[j], v);
      v2[h] = leaky(v, slope);
    }
    packed[q] = (uint32_t)bf16_bits(v2[0]) | ((uint32_t)bf16_bits(v2[1]) << 16);
  }
  *reinterpret_cast<uint4*>(A1 + r * H + o0) = make_uint4(packed[0], packed[1], packed[2], packed[3]);
}

// ---------------------------------------------------------------------------
// out[r][n] = epilogue(sum_k in[r][k] Wm[n][k]) for a 128 (n) x 128 (r) tile.
// Four waves in 2 x 2, each 64 x 64 = 4 x 4 MFMA tiles; K in steps of 32
// staged through LDS (double-buffered).
enum { kEpiFwd = 0, kEpiBwd = 1 };

constexpr int kGT = 128;            // tile edge
constexpr int kGK = 32;             // K step
constexpr int kGLD = kGK + 8;       // LDS row stride (bf16) of a staged [128][32] tile

template <int kEpi>
__global__ __launch_bounds__(256) void k_gemm(const u16* __restrict__ in, const u16* __restrict__ Wm,
                                              const float* __restrict__ bias, const u16* __restrict__ hmask,
                                              u16* __restrict__ out, int K, int Nf, float slope) {
  __shared__ __attribute__((aligned(16))) u16 sA[2][kGT * kGLD];   // weights [n][k]
  __shared__ __attribute__((aligned(16))) u16 sB[2][kGT * kGLD];   // activations [r][k]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int n0 = blockIdx.x * kGT;             // output-feature tile
  const int64_t r0 = (int64_t)blockIdx.y * kGT;  // row tile
  const int wn = (wave >> 1) * 64, wr = (wave & 1) * 64;

  // staging map: 128 rows x 32 k = 512 16-byte pieces per operand, 2 per thread
  auto stage = [&](int buf, int k0) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int piece = tid + 256 * p;
      const int row = piece >> 2, col = (piece & 3) * 8;
      const uint4 a = *reinterpret_cast<const uint4*>(Wm + (int64_t)(n0 + row) * K + k0 + col);
      const uint4 b = *reinterpret_cast<const uint4*>(in + (r0 + row) * K + k0 + col);
      *reinterpret_cast<uint4*>(&sA[buf][row * kGLD + col]) = a;
      *reinterpret_cast<uint4*>(&sB[buf][row * kGLD + col]) = b;
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = K / kGK;
  stage(0, 0);
  __syncthreads();
  for (int kk = 0; kk < nk; ++kk) {
    const int buf = kk & 1;
    if (kk + 1 < nk) stage(buf ^ 1, (kk + 1) * kGK);
    bf16x8 a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      a[i] = *reinterpret_cast<const bf16x8*>(&sA[buf][(wn + 16 * i + lr) * kGLD + 8 * lg]);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      b[j] = *reinterpret_cast<const bf16x8*>(&sB[buf][(wr + 16 * j + lr) * kGLD + 8 * lg]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma_bf16(a[i], b[j], acc[i][j]);
    __syncthreads();
  }

  // epilogue: lane holds features n0+wn+16i+4lg+q, row r0+wr+16j+lr
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int n = n0 + wn + 16 * i + 4 * lg;
    f32x4 bv = f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (kEpi == kEpiFwd) bv = *reinterpret_cast<const f32x4*>(bias + n);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t r = r0 + wr + 16 * j + lr;
      float v[4];
      if constexpr (kEpi == kEpiFwd) {
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = leaky(acc[i][j][q] + bv[q], slope);
      } else {
        const uint2 hm = *reinterpret_cast<const uint2*>(hmask + r * Nf + n);
        const float h[4] = {bf16_to_f32((u16)(hm.x & 0xffff)), bf16_to_f32((u16)(hm.x >> 16)),
                            bf16_to_f32((u16)(hm.y & 0xffff)), bf16_to_f32((u16)(hm.y >> 16))};
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = acc[i][j][q] * leaky_grad(h[q], slope);
      }
      uint2 o;
      o.x = (uint32_t)bf16_bits(v[0]) | ((uint32_t)bf16_bits(v[1]) << 16);
      o.y = (uint32_t)bf16_bits(v[2]) | ((uint32_t)bf16_bits(v[3]) << 16);
      *reinterpret_cast<uint2*>(out + r * Nf + n) = o;
    }
  }
}

// ---------------------------------------------------------------------------
// Logit layer and BCE seeds for one chunk.  One wave per row: lanes split H.
// Writes e_D[r] (0 on padding), e_G[r], delta_L (unit seed, bf16), logits,
// and per-block partials of the loss sums, dW_o and db_o.
constexpr int kRowBlocks = 2048;  // blocks of the row-reduction kernels (fixed partial count)

inline int row_blocks(int rows) { return std::max(1, std::min(kRowBlocks, (rows + 63) / 64)); }
inline int rows_per_block(int rows, int blocks) { return (rows + blocks - 1) / blocks; }

template <int PER>
__global__ __launch_bounds__(256) void k_logit(const u16* __restrict__ AL, const float* __restrict__ Wo,
                                               const float* __restrict__ bo, int H, ChunkArgs c, float inv_n,
                                               float slope, float* __restrict__ eD, float* __restrict__ eG,
                                               u16* __restrict__ dL, float* __restrict__ logits,
                                               float* __restrict__ part /*[blocks][H + 3]*/, int rpb) {
  extern __shared__ float sh_dwo[];   // [4 waves][H]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int per = PER;            // features per lane, H / 64
  float wo[PER];
#pragma unroll
  for (int q = 0; q < per; ++q) wo[q] = Wo[lane * per + q];
  float acc_dwo[PER];
#pragma unroll
  for (int q = 0; q < per; ++q) acc_dwo[q] = 0.f;
  float l0 = 0.f, l1 = 0.f, sum_e = 0.f;
  const int rbase = blockIdx.x * rpb;
  constexpr int R = 4;                 // rows per wave per iteration (independent loads in flight)
  for (int rr0 = wave * R; rr0 < rpb; rr0 += 4 * R) {
    float h[R][PER];
    float z[R];
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const int r = rbase + rr0 + k;
      if (rr0 + k < rpb && r < c.rows) load_bf16<PER>(AL + (int64_t)r * H + lane * per, h[k]);
      else {
#pragma unroll
        for (int q = 0; q < per; ++q) h[k][q] = 0.f;
      }
      float zz = 0.f;
#pragma unroll
      for (int q = 0; q < per; ++q) zz = fmaf(h[k][q], wo[q], zz);
      z[k] = zz;
    }
#pragma unroll
    for (int k = 0; k < R; ++k) z[k] = wave_sum(z[k]) + bo[0];
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const int r = rbase + rr0 + k;
      if (rr0 + k >= rpb || r >= c.rows) break;
      const bool valid = r < c.valid;
      float e = 0.f, g = 0.f;
      if (valid) {
        const float sig_neg = 1.0f / (1.0f + expf(z[k]));
        if (c.fake) {
          e = (1.0f - sig_neg) * inv_n;
          g = -sig_neg * inv_n;
          l0 += softplus(z[k]);
          l1 += softplus(-z[k]);
        } else {
          e = -sig_neg * inv_n;
          l0 += softplus(-z[k]);
        }
        if (lane == 0 && logits) logits[c.row0 + r] = z[k];
      }
      if (lane == 0) { eD[r] = e; eG[r] = g; }
      sum_e += e;
      float d[PER];
#pragma unroll
      for (int q = 0; q < per; ++q) {
        acc_dwo[q] = fmaf(e, h[k][q], acc_dwo[q]);
        d[q] = wo[q] * leaky_grad(h[k][q], slope);
      }
      store_bf16<PER>(dL + (int64_t)r * H + lane * per, d);
    }
  }
#pragma unroll
  for (int q = 0; q < per; ++q) sh_dwo[wave * H + lane * per + q] = acc_dwo[q];
  __syncthreads();
  float* p = part + (int64_t)blockIdx.x * (H + 3);
  for (int o = threadIdx.x; o < H; o += 256)
    p[o] = sh_dwo[o] + sh_dwo[H + o] + sh_dwo[2 * H + o] + sh_dwo[3 * H + o];
  __syncthreads();
  // the scalars: lane 0 of each wave holds its sums
  if (lane == 0) { sh_dwo[4 * wave] = l0; sh_dwo[4 * wave + 1] = l1; sh_dwo[4 * wave + 2] = sum_e; }
  __syncthreads();
  if (threadIdx.x < 3) {
    float s = 0.f;
    for (int w = 0; w < 4; ++w) s += sh_dwo[4 * w + threadIdx.x];
    p[H + threadIdx.x] = s;   // [H] = loss0, [H+1] = loss1, [H+2] = sum e_D (db_o)
  }
}

// ---------------------------------------------------------------------------
// Weight-gradient partial of one layer over a slice of rows:
//   P[o][i] = sum_r bf16(e_D[r] * delta[r][o]) * A[r][i],  db part = sum_r e_D[r] * delta[r][o]
// 128 (o) x 128 (i) tile per block; rows in steps of 32, staged through LDS
// event-major and read back transposed.
constexpr int kWK = 32;           // rows per step
constexpr int kWLD = kGT + 8;     // LDS row stride (bf16) of a staged [32][128] tile

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

__device__ __forceinline__ bf16x8 tr_fragment(const u16* tile, int row0, int col0, int lane) {
  // lane (g = lane/16, j = lane%16) points at row row0 + 8g + j/4 (+4), columns col0 + 4 (j%4) .. +3;
  // the transpose load then gives lane i of each 16-lane group rows 8g..8g+7 of column col0 + i.
  const int g = lane >> 4, j = lane & 15;
  const u16* p0 = tile + (row0 + 8 * g + (j >> 2)) * kWLD + col0 + 4 * (j & 3);
  const u16* p1 = p0 + 4 * kWLD;
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p0));
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p1));
  return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

// Global loads run two steps ahead of their LDS writes (two register sets),
// so a step's HBM latency is covered by the matrix work of the two before it.
__global__ __launch_bounds__(256, 2) void k_wgrad(const u16* __restrict__ dlt, const u16* __restrict__ A,
                                               const float* __restrict__ eD, int H, int rows_per_slice,
                                               int rows, float* __restrict__ P /*[slices][H][H]*/,
                                               float* __restrict__ Pdb /*[slices][H]*/) {
  __shared__ __attribute__((aligned(16))) u16 sD[2][kWK * kWLD];
  __shared__ __attribute__((aligned(16))) u16 sA[2][kWK * kWLD];
  __shared__ float sdb[256][8];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tiles = H / kGT;
  const int o0 = (blockIdx.x / tiles) * kGT, i0 = (blockIdx.x % tiles) * kGT;
  const int slice = blockIdx.y;
  const int rbeg = slice * rows_per_slice;
  const int rend = min(rows, rbeg + rows_per_slice);
  const int wo = (wave >> 1) * 64, wi = (wave & 1) * 64;
  const bool do_db = (i0 == 0);

  // staging map: 32 rows x 128 cols = 512 pieces of 8 bf16, 2 per thread (same columns every step)
  const int srow = tid >> 4, scol = (tid & 15) * 8;   // piece p: row srow + 16 p
  float db[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  struct Regs { uint4 d0, d1, a0, a1; float e0, e1; };
  auto load = [&](Regs& R, int r0) __attribute__((always_inline)) {
    const int64_t ra = r0 + srow, rb = ra + 16;
    R.e0 = eD[ra];
    R.e1 = eD[rb];
    R.d0 = *reinterpret_cast<const uint4*>(dlt + ra * H + o0 + scol);
    R.d1 = *reinterpret_cast<const uint4*>(dlt + rb * H + o0 + scol);
    R.a0 = *reinterpret_cast<const uint4*>(A + ra * H + i0 + scol);
    R.a1 = *reinterpret_cast<const uint4*>(A + rb * H + i0 + scol);
  };
  auto write = [&](const Regs& R, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int row = srow + 16 * p;
      const uint4 dv = p ? R.d1 : R.d0;
      const float ev = p ? R.e1 : R.e0;
      const uint32_t w[4] = {dv.x, dv.y, dv.z, dv.w};
      uint32_t o[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float a0 = ev * __uint_as_float(w[q] << 16);
        const float a1 = ev * __uint_as_float(w[q] & 0xffff0000u);
        db[2 * q] += a0;
        db[2 * q + 1] += a1;
        o[q] = (uint32_t)bf16_bits(a0) | ((uint32_t)bf16_bits(a1) << 16);
      }
      *reinterpret_cast<uint4*>(&sD[buf][row * kWLD + scol]) = make_uint4(o[0], o[1], o[2], o[3]);
      *reinterpret_cast<uint4*>(&sA[buf][row * kWLD + scol]) = p ? R.a1 : R.a0;
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int buf) __attribute__((always_inline)) {
    bf16x8 a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = tr_fragment(sD[buf], 0, wo + 16 * i, lane);
#pragma unroll
    for (int j = 0; j < 4; ++j) b[j] = tr_fragment(sA[buf], 0, wi + 16 * j, lane);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = mfma_bf16(a[i], b[j], acc[i][j]);
  };
  const int nsteps = (rend - rbeg) / kWK;   // rows are multiples of 128, slices multiples of 32
  // invariant at the top of step s (parity ph): R[ph ^ 1] holds step s+1, R[ph] holds step s+2
  Regs R[2];
  if (nsteps > 0) load(R[0], rbeg);
  if (nsteps > 1) load(R[1], rbeg + kWK);
  if (nsteps > 0) write(R[0], 0);
  if (nsteps > 2) load(R[0], rbeg + 2 * kWK);
  __syncthreads();
  for (int s0 = 0; s0 < nsteps; s0 += 2) {
#pragma unroll
    for (int ph = 0; ph < 2; ++ph) {
      const int s = s0 + ph;
      if (s < nsteps) {
        compute(ph);
        if (s + 1 < nsteps) write(R[ph ^ 1], ph ^ 1);
        if (s + 3 < nsteps) load(R[ph ^ 1], rbeg + (s + 3) * kWK);
      }
      __syncthreads();
    }
  }
  float* out = P + (int64_t)slice * H * H;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int o = o0 + wo + 16 * i + 4 * (lane >> 4) + q, ii = i0 + wi + 16 * j + (lane & 15);
        out[(int64_t)o * H + ii] = acc[i][j][q];
      }
  if (do_db) {
#pragma unroll
    for (int q = 0; q < 8; ++q) sdb[tid][q] = db[q];
    __syncthreads();
    if (tid < kGT) {
      // threads t with equal t & 15 stage the same 8 columns 8 (t & 15) .. + 7
      const int piece = tid >> 3, q = tid & 7;   // column = 8 * piece + q
      float sum = 0.f;
      for (int t = piece; t < 256; t += 16) sum += sdb[t][q];
      Pdb[(int64_t)slice * H + o0 + 8 * piece + q] = sum;
    }
  }
}

// ---------------------------------------------------------------------------
// First layer backward for one chunk: per-block partials of dW1 [H][F] and
// db1 [H]; for fake rows dL_G/dx (through the HD8 Jacobian when used).

template <int D, bool kHD8, int PER>
__global__ __launch_bounds__(256) void k_first_bwd(const u16* __restrict__ d1, const float* __restrict__ feat,
                                                   const float* __restrict__ xs, const float* __restrict__ W1,
                                                   const float* __restrict__ eD, const float* __restrict__ eG,
                                                   int H, ChunkArgs c, float* __restrict__ dLg_dx,
                                                   float* __restrict__ part /*[blocks][H*F + H]*/, int rpb) {
  constexpr int F = kHD8 ? 8 : D;
  extern __shared__ float smem[];          // W1 [H][F], then the block's accumulators [H][F+1]
  float* sW1 = smem;
  float* sacc = smem + H * F;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int k = threadIdx.x; k < H * F; k += 256) sW1[k] = W1[k];
  constexpr int per = PER;   // features per lane, H / 64
  float adw[PER][F + 1];
#pragma unroll
  for (int q = 0; q < PER; ++q)
#pragma unroll
    for (int j = 0; j <= F; ++j) adw[q][j] = 0.f;
  __syncthreads();
  const bool want_dx = c.fake && dLg_dx != nullptr;
  const int rbase = blockIdx.x * rpb;
  for (int rr = wave; rr < rpb; rr += 4) {
    const int r = rbase + rr;
    if (r >= c.rows) break;
    const float e = eD[r];
    float f[F];
#pragma unroll
    for (int j = 0; j < F; ++j) f[j] = feat[(int64_t)r * F + j];
    float g[F];
#pragma unroll
    for (int j = 0; j < F; ++j) g[j] = 0.f;
    float dvs[PER];
    load_bf16<PER>(d1 + (int64_t)r * H + lane * per, dvs);
#pragma unroll
    for (int q = 0; q < per; ++q) {
      const float dv = dvs[q];
      const float ed = e * dv;
      const int o = lane * per + q;
#pragma unroll
      for (int j = 0; j < F; ++j) adw[q][j] = fmaf(ed, f[j], adw[q][j]);
      adw[q][F] += ed;
      if (want_dx) {
#pragma unroll
        for (int j = 0; j < F; ++j) g[j] = fmaf(dv, sW1[o * F + j], g[j]);
      }
    }
    if (want_dx && r < c.valid) {
#pragma unroll
      for (int j = 0; j < F; ++j) g[j] = wave_sum(g[j]) * eG[r];
      if (lane == 0) {
        float dx[D];
        if constexpr (kHD8) {
          // d features / d x of [x1, x2, x3, x1x2, x2x3, x1x3, ln x1, ln(1 - x3)]
          // 1/x1 and 1/(1 - x3) from the log features, accurate where fp32 x3 is within ulps of 1
          const float x1 = xs[(int64_t)r * 3], x2 = xs[(int64_t)r * 3 + 1], x3 = xs[(int64_t)r * 3 + 2];
          const float inv_x1 = expf(-f[6]), inv_1mx3 = expf(-f[7]);
          dx[0] = g[0] + g[3] * x2 + g[5] * x3 + g[6] * inv_x1;
          dx[1] = g[1] + g[3] * x1 + g[4] * x3;
          dx[2] = g[2] + g[4] * x2 + g[5] * x1 - g[7] * inv_1mx3;
        } else {
#pragma unroll
          for (int j = 0; j < D; ++j) dx[j] = g[j];
        }
#pragma unroll
        for (int j = 0; j < D; ++j) dLg_dx[(c.row0 + r) * D + j] = dx[j];
      }
    }
  }
  // combine the four waves in a fixed order
  for (int w = 0; w < 4; ++w) {
    if (wave == w)
#pragma unroll
      for (int q = 0; q < per; ++q)
#pragma unroll
        for (int j = 0; j <= F; ++j) {
          float& dst = sacc[(lane * per + q) * (F + 1) + j];
          dst = (w == 0) ? adw[q][j] : dst + adw[q][j];
        }
    __syncthreads();
  }
  float* p = part + (int64_t)blockIdx.x * (H * F + H);
  for (int k = threadIdx.x; k < H * (F + 1); k += 256) {
    const int o = k / (F + 1), j = k % (F + 1);
    if (j < F) p[o * F + j] = sacc[k];
    else p[H * F + o] = sacc[k];
  }
}

// acc[e] (+)= sum_k part[k][e], k = 0..n-1, in a fixed order (S contiguous
// row ranges summed side by side, then combined in order); the first chunk
// overwrites.  C columns per block, S = 256 / C row slices.
template <int C>
__global__ __launch_bounds__(256) void k_accumulate(const float* __restrict__ part, int n, int64_t stride,
                                                    int64_t len, float* __restrict__ acc, int first) {
  constexpr int S = 256 / C;
  __shared__ float red[S][C];
  const int lc = threadIdx.x % C, sl = threadIdx.x / C;
  const int64_t e = (int64_t)blockIdx.x * C + lc;
  const int per = (n + S - 1) / S;
  const int k0 = sl * per, k1 = min(n, k0 + per);
  float s = 0.f;
  if (e < len) {
#pragma unroll 8
    for (int k = k0; k < k1; ++k) s += part[(int64_t)k * stride + e];
  }
  red[sl][lc] = s;
  __syncthreads();
  if (sl != 0 || e >= len) return;
  float t = 0.f;
#pragma unroll
  for (int q = 0; q < S; ++q) t += red[q][lc];
  acc[e] = first ? t : acc[e] + t;
}

void accumulate(const float* part, int n, int64_t stride, int64_t len, float* acc, int first, hipStream_t st) {
  if (len >= 16384)
    hipLaunchKernelGGL(k_accumulate<64>, dim3((unsigned)((len + 63) / 64)), dim3(256), 0, st, part, n, stride, len, acc, first);
  else
    hipLaunchKernelGGL(k_accumulate<16>, dim3((unsigned)((len + 15) / 16)), dim3(256), 0, st, part, n, stride, len, acc, first);
}

// Logit-layer scalars of one chunk: sum e_D -> db_o, loss sums -> lacc
// ([0] fake softplus(z), [1] fake softplus(-z), [2] real softplus(-z)).
__global__ __launch_bounds__(256) void k_logit_scalars(const float* __restrict__ plog, int nb, int H,
                                                       float* __restrict__ dbo, float* __restrict__ lacc, int fake,
                                                       int first_all, int first_batch) {
  __shared__ float red[3][4];
  float a = 0.f, b = 0.f, e = 0.f;
  for (int t = threadIdx.x; t < nb; t += 256) {
    const float* q = plog + (int64_t)t * (H + 3) + H;
    a += q[0]; b += q[1]; e += q[2];
  }
  a = wave_sum(a); b = wave_sum(b); e = wave_sum(e);
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = a; red[1][threadIdx.x >> 6] = b; red[2][threadIdx.x >> 6] = e;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float sa = 0.f, sb = 0.f, se = 0.f;
    for (int w = 0; w < 4; ++w) { sa += red[0][w]; sb += red[1][w]; se += red[2][w]; }
    if (dbo) *dbo = first_all ? se : *dbo + se;
    if (fake) {
      lacc[0] = first_batch ? sa : lacc[0] + sa;
      lacc[1] = first_batch ? sb : lacc[1] + sb;
    } else {
      lacc[2] = first_batch ? sa : lacc[2] + sa;
    }
  }
}

__global__ void k_losses(const float* __restrict__ lacc, float inv_nf, float inv_nr, float* loss_d, float* loss_g) {
  if (loss_d) *loss_d = lacc[2] * inv_nr + lacc[0] * inv_nf;
  if (loss_g) *loss_g = lacc[1] * inv_nf;
}

// ---------------------------------------------------------------------------
inline size_t al(size_t b) { return (b + 255) & ~(size_t)255; }

struct Plan {
  int H, NH, F, D;
  bool hd8;
  int rows_max;          // padded rows of the largest chunk
  int logit_blocks, fb_blocks;
  int slices;            // weight-gradient slices per chunk
  size_t off_wb, off_wtb, off_feat, off_xs, off_act, off_dlt0, off_dlt1, off_eD, off_eG, off_plog, off_pfb,
      off_pw, off_pdb, off_accl, total;
};

int pad128(int64_t n) { return (int)((n + 127) / 128 * 128); }



Plan make_plan(const DiscArgs& a) {
  const sagips_mlp& D = *a.D;
  Plan p;
  p.H = D.width[1];
  p.NH = D.n_layers - 2;
  p.F = D.width[0];
  p.hd8 = D.features == SAGIPS_FEAT_HD8;
  p.D = a.d;
  const int64_t biggest = std::min<int64_t>(std::max(a.n_fake, a.n_real), kChunkRows);
  p.rows_max = pad128(biggest);
  p.logit_blocks = kRowBlocks;
  p.fb_blocks = kRowBlocks;
  const int tiles = (p.H / kGT) * (p.H / kGT);
  p.slices = std::max(1, 768 / tiles);   // three weight-gradient blocks per CU
  const size_t H = p.H, R = p.rows_max;
  size_t o = 0;
  p.off_wb = o; o += al(2 * H * H * p.NH);
  p.off_wtb = o; o += al(2 * H * H * p.NH);
  p.off_feat = o; o += al(4 * R * p.F);
  p.off_xs = o; o += al(4 * R * p.D);
  p.off_act = o; o += al(2 * R * H * (p.NH + 1));
  p.off_dlt0 = o; o += al(2 * R * H);
  p.off_dlt1 = o; o += al(2 * R * H);
  p.off_eD = o; o += al(4 * R);
  p.off_eG = o; o += al(4 * R);
  p.off_plog = o; o += al(4 * (size_t)p.logit_blocks * (H + 3));
  p.off_pfb = o; o += al(4 * (size_t)p.fb_blocks * (H * p.F + H));
  p.off_pw = o; o += al(4 * (size_t)p.slices * H * H);
  p.off_pdb = o; o += al(4 * (size_t)p.slices * H);
  p.off_accl = o; o += al(4 * 4);
  p.total = o;
  return p;
}

}  // namespace

bool disc_bf16_supported(const sagips_mlp& D, int d, const char** why) {
  const int H = D.width[1];
  if (H != 256 && H != 512) { *why = "bf16 discriminator supports hidden width 256 or 512"; return false; }
  if (D.n_layers < 3 || D.n_layers - 2 > kMaxNH) { *why = "bf16 discriminator needs 1-4 hidden-to-hidden layers"; return false; }
  for (int l = 1; l < D.n_layers; ++l)
    if (D.width[l] != H) { *why = "all hidden widths must be equal"; return false; }
  if (D.features == SAGIPS_FEAT_HD8) {
    if (d != 3 || D.width[0] != 8) { *why = "HD8 features need d = 3 and width[0] = 8"; return false; }
  } else if (D.width[0] != d || (d != 2 && d != 3)) {
    *why = "IDENTITY features need width[0] == d in {2, 3}";
    return false;
  }
  return true;
}

size_t disc_bf16_workspace(const DiscArgs& a) { return make_plan(a).total; }

hipError_t launch_disc_bf16(const DiscArgs& a, void* ws, int n_cu, hipStream_t st, Timer* tm) {
  const sagips_mlp& Dm = *a.D;
  const Plan p = make_plan(a);
  char* base = static_cast<char*>(ws);
  auto F32 = [&](size_t off) { return reinterpret_cast<float*>(base + off); };
  auto B16 = [&](size_t off) { return reinterpret_cast<u16*>(base + off); };
  const int H = p.H, NH = p.NH;
  const float slope = Dm.leaky_slope;
  u16* Wb = B16(p.off_wb);
  u16* WTb = B16(p.off_wtb);
  float* feat = F32(p.off_feat);
  float* xs = F32(p.off_xs);
  u16* act = B16(p.off_act);          // A_1 .. A_{NH+1}
  u16* dl[2] = {B16(p.off_dlt0), B16(p.off_dlt1)};
  float* eD = F32(p.off_eD);
  float* eG = F32(p.off_eG);
  const sagips_disc_out& out = *a.out;
  const bool want_grads = out.dW[0] != nullptr;
  const float inv_nf = 1.0f / (float)a.n_fake, inv_nr = 1.0f / (float)a.n_real;

  if (tm) tm->begin("disc_bf16_weights");
  for (int l = 0; l < NH; ++l)
    hipLaunchKernelGGL(k_weights_bf16, dim3(H / 32, H / 32), dim3(256), 0, st, Dm.W[1 + l], Wb + (size_t)l * H * H,
                       WTb + (size_t)l * H * H, H);
  if (tm) tm->end();

  SourceArgs src{};
  const bool sampled = a.fake_src != nullptr;
  if (sampled) src = *a.fake_src;

  int chunk_index = 0;
  float* lacc = F32(p.off_accl);
  for (int pass = 0; pass < 2; ++pass) {
    const bool fake = pass == 0;
    const int64_t n = fake ? a.n_fake : a.n_real;
    for (int64_t row0 = 0; row0 < n; row0 += kChunkRows, ++chunk_index) {
      ChunkArgs c;
      c.row0 = row0;
      c.valid = (int)std::min<int64_t>(kChunkRows, n - row0);
      c.rows = pad128(c.valid);
      c.fake = fake ? 1 : 0;
      const int first = chunk_index == 0 ? 1 : 0;
      const int first_batch = row0 == 0 ? 1 : 0;
      const dim3 g1((c.rows + 255) / 256);
      const float* xin = fake ? a.fake_x : a.real_x;
      const int samp = (fake && sampled) ? 1 : 0;
      if (p.hd8) hipLaunchKernelGGL((k_prep<3, true>), g1, dim3(256), 0, st, c, xin, src, samp, feat, xs);
      else if (p.D == 2) hipLaunchKernelGGL((k_prep<2, false>), g1, dim3(256), 0, st, c, xin, src, samp, feat, xs);
      else hipLaunchKernelGGL((k_prep<3, false>), g1, dim3(256), 0, st, c, xin, src, samp, feat, xs);
      const int64_t nthr = (int64_t)c.rows * (H / 8);
      const dim3 gf((unsigned)((nthr + 255) / 256));
      if (p.F == 8) hipLaunchKernelGGL(k_first_fwd<8>, gf, dim3(256), 0, st, feat, Dm.W[0], Dm.b[0], H, c.rows, slope, act);
      else if (p.F == 3) hipLaunchKernelGGL(k_first_fwd<3>, gf, dim3(256), 0, st, feat, Dm.W[0], Dm.b[0], H, c.rows, slope, act);
      else hipLaunchKernelGGL(k_first_fwd<2>, gf, dim3(256), 0, st, feat, Dm.W[0], Dm.b[0], H, c.rows, slope, act);
      const size_t ast = (size_t)c.rows * H;     // stride between this chunk's activation buffers
      for (int l = 0; l < NH; ++l) {
        if (tm) tm->begin("bf16_gemm");
        hipLaunchKernelGGL(k_gemm<kEpiFwd>, dim3(H / kGT, c.rows / kGT), dim3(256), 0, st, act + l * ast,
                           Wb + (size_t)l * H * H, Dm.b[1 + l], (const u16*)nullptr, act + (l + 1) * ast, H, H, slope);
        if (tm) tm->end();
      }

      const int lb = row_blocks(c.rows), lrpb = rows_per_block(c.rows, lb);
      float* plog = F32(p.off_plog);
      if (H == 256)
        hipLaunchKernelGGL(k_logit<4>, dim3(lb), dim3(256), 4 * H * sizeof(float), st, act + NH * ast, Dm.W[NH + 1],
                           Dm.b[NH + 1], H, c, fake ? inv_nf : inv_nr, slope, eD, eG, dl[0],
                           fake ? out.logits_fake : out.logits_real, plog, lrpb);
      else
        hipLaunchKernelGGL(k_logit<8>, dim3(lb), dim3(256), 4 * H * sizeof(float), st, act + NH * ast, Dm.W[NH + 1],
                           Dm.b[NH + 1], H, c, fake ? inv_nf : inv_nr, slope, eD, eG, dl[0],
                           fake ? out.logits_fake : out.logits_real, plog, lrpb);
      if (want_grads)
        accumulate(plog, lb, (int64_t)(H + 3), (int64_t)H, out.dW[NH + 1], first, st);
      hipLaunchKernelGGL(k_logit_scalars, dim3(1), dim3(256), 0, st, plog, lb, H, want_grads ? out.db[NH + 1] : nullptr,
                         lacc, c.fake, first, first_batch);

      const int tiles = (H / kGT) * (H / kGT);
      const int rows_per_slice = ((c.rows / p.slices + kWK - 1) / kWK) * kWK;
      int cur = 0;
      for (int l = NH - 1; l >= 0; --l) {
        // hidden layer l maps A_{l+1} (act + l*ast) -> A_{l+2}; its output signal is in dl[cur]
        if (want_grads) {
          if (tm) tm->begin("bf16_wgrad");
          hipLaunchKernelGGL(k_wgrad, dim3(tiles, p.slices), dim3(256), 0, st, dl[cur], act + l * ast, eD, H,
                             rows_per_slice, c.rows, F32(p.off_pw), F32(p.off_pdb));
          if (tm) tm->end();
          accumulate(F32(p.off_pw), p.slices, (int64_t)H * H, (int64_t)H * H, out.dW[1 + l], first, st);
          accumulate(F32(p.off_pdb), p.slices, (int64_t)H, (int64_t)H, out.db[1 + l], first, st);
        }
        if (tm) tm->begin("bf16_gemm");
        hipLaunchKernelGGL(k_gemm<kEpiBwd>, dim3(H / kGT, c.rows / kGT), dim3(256), 0, st, dl[cur],
                           WTb + (size_t)l * H * H, (const float*)nullptr, act + l * ast, dl[cur ^ 1], H, H, slope);
        if (tm) tm->end();
        cur ^= 1;
      }
      const int fbb = row_blocks(c.rows), frpb = rows_per_block(c.rows, fbb);
      const size_t fb_smem = sizeof(float) * ((size_t)H * p.F + (size_t)H * (p.F + 1));
      float* pfb = F32(p.off_pfb);
      float* gx = fake ? out.dLg_dx : nullptr;
#define SAGIPS_FIRST_BWD(D_, HD8_, PER_)                                                                   \
  hipLaunchKernelGGL((k_first_bwd<D_, HD8_, PER_>), dim3(fbb), dim3(256), fb_smem, st, dl[cur], feat, xs, Dm.W[0], \
                     eD, eG, H, c, gx, pfb, frpb)
      if (p.hd8) { if (H == 256) SAGIPS_FIRST_BWD(3, true, 4); else SAGIPS_FIRST_BWD(3, true, 8); }
      else if (p.D == 2) { if (H == 256) SAGIPS_FIRST_BWD(2, false, 4); else SAGIPS_FIRST_BWD(2, false, 8); }
      else { if (H == 256) SAGIPS_FIRST_BWD(3, false, 4); else SAGIPS_FIRST_BWD(3, false, 8); }
#undef SAGIPS_FIRST_BWD
      if (want_grads) {
        accumulate(pfb, fbb, (int64_t)(H * p.F + H), (int64_t)(H * p.F), out.dW[0], first, st);
        accumulate(pfb + (size_t)H * p.F, fbb, (int64_t)(H * p.F + H), (int64_t)H, out.db[0], first, st);
      }
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  if (out.loss_d || out.loss_g)
    hipLaunchKernelGGL(k_losses, dim3(1), dim3(1), 0, st, lacc, inv_nf, inv_nr, out.loss_d, out.loss_g);
  return hipGetLastError();
}

}  // namespace sagips
