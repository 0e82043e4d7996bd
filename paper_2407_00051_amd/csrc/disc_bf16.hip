// bf16-operand / fp32-accumulate discriminator step on gfx950 for wide
// networks (hidden width 256 or 512), where the hidden weight gradients do not
// fit in registers across tiles.  The step is processed in chunks of event
// rows (all fake or all real); each chunk goes through these kernels:
//
//   k_fwd_chain  per tile of rows, in LDS: the tile's events (fake events
//                sampled there from their Philox words, real ones read), their
//                features, A_1 = bf16(LeakyReLU(feat W1^T + b1))
//                (bf16 matrix cores on exact split terms), then every hidden
//                layer on the bf16 matrix cores, then the logit z and the BCE
//                seeds e_D, e_G; stores A_1 .. A_NH, the activation sign
//                masks and the top layer's sign bits
//   k_bwd_chain  per tile, in LDS: the events again, the unit-seed signal from the logit layer
//                down to A_1 (matrix cores, LeakyReLU' from the masks); stores
//                the signals the weight gradients need; first-layer dW_1, db_1
//                and dL_G/dx (through the HD8 Jacobian), also on the matrix
//                cores with the fp32 operand split into exact bf16 terms
//   k_wgrad_shared  dW partials = sum_rows bf16(e_D delta) (x) A  (K = rows)
//
// Forward and backward products compute outT = W' inT (M = output feature,
// N = event, K = input feature): both operands then have K contiguous in
// memory and the accumulator fragment of a lane is 4 consecutive features of
// one event.  The weight-gradient product has K = events; its operands are
// read from event-major LDS tiles with the gfx950 transpose load
// ds_read_b64_tr_b16, which hands every lane 4 consecutive rows of one column.
//
// Backward signals carry a unit seed per event; the weight gradients scale
// them by e_D = dL_D/dz while staging (and round to bf16 again), dL_G/dx
// scales the first-layer signal by e_G = dL_G/dz.  All sums are fixed-order:
// per-workgroup partials are added to fp32 accumulators chunk by chunk.
#include "device_math.hpp"
#include "kernels.hpp"

#include <string.h>

#include <algorithm>
#include <type_traits>

namespace sagips {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

constexpr int kMaxNH = 4;
constexpr int kChunkRows = 1 << 22;   // default and largest rows per chunk (fake or real), multiple of 128

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



// ---------------------------------------------------------------------------
// Weights: bf16 copies of one hidden layer in the order the chain kernels
// consume them as MFMA A fragments.  Piece (rb, ks, lane) of a copy holds rows
// 32 rb + lane % 32, columns 16 ks + 8 (lane / 32) .. + 7, so the 64 lanes of
// a wave read one contiguous kilobyte per fragment.  The forward copy (of W,
// [out][in]) has KS + 1 pieces per 32-row block: the extra step KS carries the
// bias as three bf16 terms hi + mid + lo in columns 0..2 of lane half 0 (zeros
// elsewhere), and the forward products multiply it by a constant fragment of
// ones.  The terms sum to the fp32 bias exactly for magnitudes between about
// 1e-33 and 3.3e38 (below, lo is subnormal; above, hi overflows).  The
// backward copy (of W^T) has KS pieces per row block.
__device__ __forceinline__ uint32_t bias_terms(float x, uint32_t& lo) {
  const u16 hi = bf16_bits(x);
  const float r = x - bf16_to_f32(hi);       // exact
  const u16 mid = bf16_bits(r);
  lo = bf16_bits(r - bf16_to_f32(mid));      // the last 8 bits (exact unless subnormal)
  return (uint32_t)hi | ((uint32_t)mid << 16);
}

__global__ __launch_bounds__(256) void k_weights_frag(const float* __restrict__ W, const float* __restrict__ b,
                                                      u16* __restrict__ Wf, u16* __restrict__ WTf, int H) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int KS = H / 16;
  if (t >= (H / 32) * (KS + 1) * 64) return;
  const int rb = t / ((KS + 1) * 64), rem = t % ((KS + 1) * 64), ks = rem / 64, lane = rem % 64;
  const int row = 32 * rb + (lane & 31), col0 = 16 * ks + 8 * (lane >> 5);
  uint32_t wp[4] = {0u, 0u, 0u, 0u};
  if (ks < KS) {
    uint32_t wt[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      wp[u] = (uint32_t)bf16_bits(W[row * H + col0 + 2 * u]) | ((uint32_t)bf16_bits(W[row * H + col0 + 2 * u + 1]) << 16);
      wt[u] = (uint32_t)bf16_bits(W[(col0 + 2 * u) * H + row]) | ((uint32_t)bf16_bits(W[(col0 + 2 * u + 1) * H + row]) << 16);
    }
    *reinterpret_cast<uint4*>(WTf + ((size_t)(rb * KS + ks) * 64 + lane) * 8) = make_uint4(wt[0], wt[1], wt[2], wt[3]);
  } else if (lane < 32) {
    wp[0] = bias_terms(b[row], wp[1]);
  }
  *reinterpret_cast<uint4*>(Wf + (size_t)t * 8) = make_uint4(wp[0], wp[1], wp[2], wp[3]);
}

// a b rounded once to fp32: never fused with a later subtraction.
__device__ __forceinline__ float mul_rounded(float a, float b) {
#pragma clang fp contract(off)
  return a * b;
}

// Term t (0 = hi, 1 = mid, 2 = lo) of the exact three-term bf16 split above.
__device__ __forceinline__ u16 bf16_term(float x, int t) {
  uint32_t lo;
  const uint32_t hm = bias_terms(x, lo);
  return (u16)(t == 0 ? (hm & 0xffffu) : t == 1 ? (hm >> 16) : lo);
}

// The first-layer products of the backward chain (dW_1, db_1 and dL/dx, with
// K <= 8 first-layer inputs) run on the bf16 matrix cores with the fp32
// operand (W_1, or e_D times an input) split into its three bf16 terms: the
// terms sum to the operand exactly and every product of the bf16 signal with
// a term is exact in fp32, so only the fp32 accumulation rounds.
// Their 32-row operand puts term t of input j (j = 4 h + p < 8) in row
// R = 8 t + 4 h + p: in the accumulator fragment of a lane in half h, register
// 4 t + p then holds term t of input 4 h + p, and the three terms add up
// within the lane.  Rows 24..26 carry the terms of the db_1 column (all-ones
// input) where it is used; other rows are zero.
//
// k_w0_frag: W_1 ([H][F] fp32) in that arrangement as the A operand of the
// dL/dx product (M = 32 rows, K = hidden features): piece (ks, lane) holds
// row R = lane % 32 for hidden features 16 ks + 8 (lane / 32) .. + 7.
__global__ __launch_bounds__(256) void k_w0_frag(const float* __restrict__ W0, int F, int H, u16* __restrict__ out) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= (H / 16) * 64) return;
  const int ks = t / 64, lane = t % 64, R = lane & 31, term = R >> 3, j = R & 7;
  uint32_t w[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    uint32_t h2[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int o = 16 * ks + 8 * (lane >> 5) + 2 * u + e;
      h2[e] = (term < 3 && j < F) ? bf16_term(W0[o * F + j], term) : 0u;
    }
    w[u] = h2[0] | (h2[1] << 16);
  }
  *reinterpret_cast<uint4*>(out + (size_t)t * 8) = make_uint4(w[0], w[1], w[2], w[3]);
}

// ---------------------------------------------------------------------------
// The forward chain's first layer, z = W_1 x + b_1 with K = F inputs, on the
// bf16 matrix cores: every fp32 weight, bias and input is split into its three
// exact bf16 terms hi + mid + lo (bias_terms), and the K dimension holds the
// term products that reach fp32 accuracy.  Slot k < 6 F pairs term a(p) of
// W_1[f][j] with term b(p) of x[e][j], p = k / F, j = k % F, for the pairs
// p = (hi,hi), (hi,mid), (mid,hi), (hi,lo), (mid,mid), (lo,hi); the three
// pairs left out are each below 2^-25 of |W_1[f][j] x[e][j]|, under fp32
// rounding.  Slots 6 F .. 6 F + 2 hold the bias terms against 1, the rest 0.
// Every product of two bf16 terms is exact in fp32, so z carries only the
// fp32 accumulation's rounding and the dropped pairs.
template <int F>
struct FirstLayer {
  static constexpr int KS = (6 * F + 3 + 15) / 16;   // K steps of 16
  static constexpr int KP = 16 * KS;                 // slots
  static constexpr int LDB = KP + 8;                 // LDS row stride (bf16) of the input slots
};

__host__ __device__ constexpr int pair_a(int p) { return (p == 2 || p == 4) ? 1 : (p == 5 ? 2 : 0); }
__host__ __device__ constexpr int pair_b(int p) { return (p == 1 || p == 4) ? 1 : (p == 3 ? 2 : 0); }

// k_w1_frag: the weight side as MFMA A fragments, piece (rb, s, lane) =
// row 32 rb + lane % 32, slots 16 s + 8 (lane / 32) .. + 7.
template <int F>
__global__ __launch_bounds__(256) void k_w1_frag(const float* __restrict__ W0, const float* __restrict__ b0, int H,
                                                 u16* __restrict__ out) {
  using L = FirstLayer<F>;
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= (H / 32) * L::KS * 64) return;
  const int rb = t / (L::KS * 64), sidx = (t / 64) % L::KS, lane = t % 64;
  const int f = 32 * rb + (lane & 31);
  uint32_t w[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    uint32_t h2[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int k = 16 * sidx + 8 * (lane >> 5) + 2 * u + e;
      u16 v = 0;
      if (k < 6 * F) v = bf16_term(W0[f * F + k % F], pair_a(k / F));
      else if (k < 6 * F + 3) v = bf16_term(b0[f], k - 6 * F);
      h2[e] = v;
    }
    w[u] = h2[0] | (h2[1] << 16);
  }
  *reinterpret_cast<uint4*>(out + (size_t)t * 8) = make_uint4(w[0], w[1], w[2], w[3]);
}

// The input side of one event: its KP slots (row e of the [T][LDB] array the
// B fragments are read from), from its F inputs.
template <int F>
__device__ __forceinline__ void first_layer_row(const float (&x)[F], u16* row) {
  using L = FirstLayer<F>;
  u16 t[F][3];
#pragma unroll
  for (int j = 0; j < F; ++j) {
    uint32_t lo;
    const uint32_t hm = bias_terms(x[j], lo);
    t[j][0] = (u16)(hm & 0xffffu);
    t[j][1] = (u16)(hm >> 16);
    t[j][2] = (u16)lo;
  }
  constexpr u16 one = 0x3f80;
#pragma unroll
  for (int q = 0; q < L::KP / 8; ++q) {
    uint32_t w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      uint32_t h2[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int k = 8 * q + 2 * u + e;
        h2[e] = k < 6 * F ? t[k % F][pair_b(k / F)] : (k < 6 * F + 3 ? one : 0);
      }
      w[u] = h2[0] | (h2[1] << 16);
    }
    *reinterpret_cast<uint4*>(row + 8 * q) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// ---------------------------------------------------------------------------
// Rows of one chunk.  Rows past `valid` are padding: coordinates 0.5, never
// stored anywhere visible (their e_D and e_G are 0).
struct ChunkArgs {
  int64_t row0;       // first event index (within the fake or the real batch)
  int rows;           // padded row count (multiple of 128)
  int valid;          // real rows in this chunk
  int fake;
};

// Where a chunk's events come from: sampled from the source (fake events of a
// source call) or read from a buffer (the real batch, or fake events passed as
// a buffer).
struct EventArgs {
  SourceArgs src;
  const float* xin;   // [n][D] when not sampled
  int sampled;
};

// Parameter row of event i (32-bit division when both fit).
__device__ __forceinline__ int64_t row_of(int64_t i, int64_t E) {
  if (((uint64_t)i | (uint64_t)E) >> 32) return i / E;
  return (int64_t)((uint32_t)i / (uint32_t)E);
}

// The chains stage their tile's events in LDS themselves: coordinate j of
// event i is computed by one thread, in two halves.  event_fetch (a tile
// ahead) loads what it needs from memory into two registers: theta (a, b) of
// the event's parameter row for sampled events, the coordinate itself for
// buffer events.  event_coord then forms the coordinate, from the event's
// Philox words and the quantile, and for HD8 its log feature (j = 0: ln x1,
// j = D - 1: ln(1 - x_D)).  The log features of sampled events come from the
// quantile's log domain, ln x1 = lam1 / a1 and ln(1 - x3) = log1mexp(lam3 / a3),
// which stay accurate (and finite) where fp32 x3 has rounded to within ulps
// of 1; buffer events only have their fp32 values: ln x1 and log1p(-x3) of
// those.
template <int D>
__device__ __forceinline__ void event_fetch(const EventArgs& ev, int64_t i, bool valid, int j, float& a, float& b) {
  a = b = 0.5f;
  if (!valid) return;
  if (ev.sampled) {
    const float* th = ev.src.theta + row_of(i, ev.src.E) * (2 * D) + 2 * j;
    a = th[0];
    b = th[1];
  } else {
    a = ev.xin[i * D + j];
  }
}

template <int D, bool kHD8>
__device__ __forceinline__ float event_coord(const EventArgs& ev, int64_t i, bool valid, int j, float a, float b,
                                             float& lg) {
  lg = 0.f;
  if (!valid) {
    if (kHD8) lg = logf(0.5f);
    return 0.5f;
  }
  if (ev.sampled) {
    const Words w = event_words(ev.src.base + (uint64_t)i, ev.src.stream, ev.src.k0, ev.src.k1);
    const uint32_t wj = j == 0 ? w.w[0] : (j == 1 ? w.w[1] : w.w[2]);
    const Shape sh = make_shape(a, b);
    const Quantile q = kumaraswamy_w(wj, sh);
    if (kHD8) {
      const float lx = log_x(q, sh);
      if (j == 0) lg = lx;
      else if (j == D - 1) lg = log1mexp(lx);
    }
    return q.x;
  }
  if (kHD8) {
    if (j == 0) lg = logf(a);
    else if (j == D - 1) lg = log1pf(-a);
  }
  return a;
}

// A tile's events in LDS: thread t < T D computes coordinate j = t / T of
// event e = t % T (j is wave-uniform) into sx[e][j] and, for HD8, the log
// feature into slg[e][0 or 1].  EU pieces per thread; the fetched registers
// hold the next tile's inputs.
template <int T, int D, int NTH>
struct TileEvents {
  static constexpr int EU = (T * D + NTH - 1) / NTH;
  float a[EU], b[EU];

  __device__ __forceinline__ void fetch(const EventArgs& ev, const ChunkArgs& c, int tile, int tid) {
#pragma unroll
    for (int u = 0; u < EU; ++u) {
      const int q = tid + NTH * u, e = q % T, j = q / T, r = tile * T + e;
      if (q < T * D) event_fetch<D>(ev, c.row0 + r, r < c.valid, j, a[u], b[u]);
    }
  }
  // With xg the coordinates also go to xg[row][D] (chunk rows, padding included).
  template <bool kHD8>
  __device__ __forceinline__ void form(const EventArgs& ev, const ChunkArgs& c, int tile, int tid, float* sx,
                                       float* slg, float* xg = nullptr) {
#pragma unroll
    for (int u = 0; u < EU; ++u) {
      const int q = tid + NTH * u, e = q % T, j = q / T, r = tile * T + e;
      if (q < T * D) {
        float lg;
        const float x = event_coord<D, kHD8>(ev, c.row0 + r, r < c.valid, j, a[u], b[u], lg);
        sx[e * D + j] = x;
        if (xg) xg[(size_t)r * D + j] = x;
        if (kHD8 && j != 1) slg[2 * e + (j == 0 ? 0 : 1)] = lg;
      }
    }
  }
};

// Hidden width 256 with two identity features: the first hidden layer's weight
// gradient rebuilds A_1 from the events' coordinates (8 bytes a row) instead
// of reading a stored copy (512 bytes a row, written by the forward chain),
// when that layer is not also the top one (whose kernel rebuilds its signal
// from sign bytes instead): NH >= 2, checked at run time.
template <int H, int F, bool kHD8>
constexpr bool kRebuildA1 = H == 256 && F == 2 && !kHD8;

// HD8 features of event e from its coordinates and log features:
// [x1, x2, x3, x1 x2, x2 x3, x1 x3, ln x1, ln(1 - x3)].
__device__ __forceinline__ void hd8_features(const float* sx, const float* slg, int e, float* f) {
  const float x1 = sx[3 * e], x2 = sx[3 * e + 1], x3 = sx[3 * e + 2];
  f[0] = x1; f[1] = x2; f[2] = x3;
  f[3] = x1 * x2; f[4] = x2 * x3; f[5] = x1 * x3;
  f[6] = slg[2 * e];
  f[7] = slg[2 * e + 1];
}

// ---------------------------------------------------------------------------
// Per-tile layer chains.  Persistent workgroups of H / 64 waves (eight waves
// per CU: two workgroups for H = 256, so that one workgroup's VALU epilogues
// and barriers overlap the other's matrix products; one for H = 512) loop
// over tiles of T = 128 event rows; the tile's activations (forward) or
// unit-seed signals (backward) live in LDS as [T][H + 8] bf16 and are
// overwritten layer by layer, so between layers nothing goes through HBM
// except what the weight-gradient products need later.  Wave w owns output
// features [64 w, 64 w + 64) of every product outT = W' inT for all T events,
// as 2 x 4 tiles of v_mfma_f32_32x32x16_bf16: each 16-byte weight fragment
// feeds four products and each 16-byte LDS fragment two, so that with the
// matrix cores at full rate a CU's weight loads and LDS reads stay near half
// of what its L1 and LDS can deliver.  Each K step of 16 takes two weight
// loads (L2-resident fragment-ordered copies, issued PD steps ahead) and four
// LDS reads (one step ahead).  The 16-byte row pad makes each 8-lane group of
// an LDS fragment read hit distinct banks.
//
// The HBM copies of each product's input for the weight gradients are written
// after the product: each wave copies the feature columns it owns, which only
// its own epilogue overwrites.
//
// The VALU work per output is kept to the LeakyReLU (two operations), the
// bf16 rounding (half of a v_cvt_pk_bf16_f32) and a quarter of the sign-mask
// packing: biases enter the forward products as one more K step, and the
// first layer (exact bf16 split terms, with the bias) and the logit (bf16 activations
// against the fp32 w_o split into three bf16 terms) also run on the matrix
// cores.
//
// Global streams inside the products use one per-lane 32-bit offset register
// each, with every per-step offset a scalar constant: buffer loads for the
// weights, global stores with a scalar base for the HBM copies.  That keeps
// the 128 accumulators and the rings within the 256 registers a wave has at
// two waves per SIMD.
//
// Lane l holds, in register 4 g + q of tile (mt, nt), the output of feature
// ow + 32 mt + 8 g + 4 (l / 32) + q for event 32 nt + (l % 32): each group g
// is 4 consecutive features of one event (one 8-byte bf16 store).
//
// Signs of the hidden activations are kept as lane-local bit masks, 4 words
// per lane and layer: the sign bit of output (mt, nt, g, q) is bit
// 8 q + g + 4 (t % 2) of word t / 2, t = mt NT + nt, set where the bf16
// activation is negative (or -0).  Each lane stores its words as one vector,
// [layer][tile][wave][lane]; the backward chain has the same lane arrangement
// and reads them back, so LeakyReLU' costs one bit per output.

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t Rsrc;

template <int H>
struct Chain {
  static constexpr int MT = 2;                  // 32-feature MFMA tiles per wave
  static constexpr int NT = 4;                  // 32-event MFMA tiles per wave
  static constexpr int WAVES = H / (32 * MT);   // waves per workgroup
  static constexpr int THREADS = 64 * WAVES;    // = H
  static constexpr int T = 32 * NT;             // events per tile
  static constexpr int LDA = H + 8;             // LDS row stride (bf16)
  static constexpr int KS = H / 16;             // K steps of a product's input
  static constexpr int PD = 2;                  // weight prefetch distance (K steps)
  static constexpr int MW = MT * NT / 2;        // mask words per lane and layer
  static constexpr int BPC = 512 / H;           // workgroups per CU
  static constexpr int COPIES = T * H / 512 / WAVES;   // copy kilobytes per wave and product
  static_assert(MW == 4 && COPIES == 16 && THREADS == H, "chain decomposition");
};

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 values -> a packed bf16 pair, round to nearest even
// (v_cvt_pk_bf16_f32, identical to bf16_bits on every non-NaN input).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{lo, hi}), bf16x2_t));
}

// Raw buffer resource over [base, base + bytes): accesses past the end read 0
// and write nothing.
__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ bf16x8 load_frag(Rsrc r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0));
}
__device__ __forceinline__ float load_f32(Rsrc r, uint32_t voff) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, 0, 0));
}

// K steps per 32-row block of a weight copy: KS + 1 forward (with the bias
// step), KS backward.
template <int H, bool kFwd>
struct WSteps {
  static constexpr int N = H / 16 + (kFwd ? 1 : 0);
};

// Weight copy of one hidden layer, and the per-lane offset of fragment (0, 0)
// of wave w: fragment (m, ks) is piece ((2 w + m) N + ks) 64 + lane, i.e.
// byte woff + (m N + ks) 1024.
template <int H, bool kFwd>
__device__ __forceinline__ Rsrc weight_rsrc(const u16* Wb, int layer) {
  constexpr uint32_t bytes = (H / 32) * WSteps<H, kFwd>::N * 1024;
  return make_rsrc(Wb + (size_t)layer * (bytes / 2), bytes);
}
template <int H, bool kFwd>
__device__ __forceinline__ uint32_t weight_offset(int wave, int lane) {
  return (uint32_t)(2 * wave * WSteps<H, kFwd>::N * 64 + lane) * 16;
}

// The first PD weight-fragment steps of the next product, loaded during the
// tail of the current one.
template <int H>
struct WeightPrefetch {
  bf16x8 a[Chain<H>::PD][Chain<H>::MT];
};

template <int H, bool kFwd>
__device__ __forceinline__ void prefetch_weights(Rsrc W, WeightPrefetch<H>& pf, uint32_t woff) {
  using C = Chain<H>;
  constexpr int N = WSteps<H, kFwd>::N;
#pragma unroll
  for (int q = 0; q < C::PD; ++q)
#pragma unroll
    for (int m = 0; m < C::MT; ++m) pf.a[q][m] = load_frag(W, woff, (uint32_t)(m * N + q) * 1024);
}

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// K-fragment order of the weight-gradient operands ([rows][H] matrices with
// K = rows): piece (kb, cb, lane) holds column 32 cb + lane % 32, rows
// 16 kb + 8 (lane / 32) .. + 7, at bf16 offset ((kb H / 32 + cb) 64 + lane) 8,
// so each 32-column, 16-row block is one contiguous kilobyte: an MFMA
// fragment of v_mfma_f32_32x32x16_bf16 with K = rows.
//
// Wave w writes the column blocks cb = 2 w + u (u = 0, 1) of every 16-row
// block of the tile: copy kilobyte j is (kb, u) = (j / 2, j % 2).  It turns a
// block of the LDS tile into its kilobyte with two ds_read_b64_tr_b16: lane i
// of each 16-lane group g addresses row 16 kb + 8 (g / 2) + i / 4 (+ 4) and
// columns 32 cb + 16 (g % 2) + 4 (i % 4) .. + 3; the transpose then hands
// lane i of the group rows +0..3 (+4..7) of column 32 cb + 16 (g % 2) + i.
// copy_lds_base is that address for (kb, u) = (0, 0); block (kb, u) adds
// 16 kb LDA + 32 u.
template <int LDA>
__device__ __forceinline__ int copy_lds_base(int lane, int wave) {
  const int g = lane >> 4, i = lane & 15;
  return (8 * (g >> 1) + (i >> 2)) * LDA + 64 * wave + 16 * (g & 1) + 4 * (i & 3);
}
template <int LDA>
__device__ __forceinline__ bf16x8 copy_read(const u16* p0) {
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p0));
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p0 + 4 * LDA));
  return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

// acc[mt][nt] = sum_k W[feature][k] act[event][k] (+ the bias with kFwd; see
// above for the arrangement).  pf holds the first PD weight steps of W on
// entry and those of Wnext (the next product) on exit.
//
// With `copy` (wave-uniform) the product's input goes to HBM meanwhile, as the
// weight-gradient operand: the wave's own columns of act, copy kilobyte j (the
// K-fragment order above; dst at per-lane byte offset coff) read with the
// operands of step CS j and stored after its products.  Spread over the product, the stores drain while the matrix cores
// run, and a weight load waits behind at most a few of them (loads and stores
// share one completion counter).
template <int H, bool kFwd>
__device__ __forceinline__ void chain_gemm(Rsrc W, Rsrc Wnext, uint32_t woff, WeightPrefetch<H>& pf, const u16* act,
                                           f32x16 (&acc)[Chain<H>::MT][Chain<H>::NT], int lane, int wave, u16* dst,
                                           uint32_t coff, bool copy) {
  using C = Chain<H>;
  constexpr int KS = C::KS, PD = C::PD, LDA = C::LDA, MT = C::MT, NT = C::NT;
  constexpr int N = WSteps<H, kFwd>::N;          // K steps, the bias step last
  constexpr int CS = KS / C::COPIES;             // K steps per copy kilobyte
  static_assert(CS >= 1 && KS % C::COPIES == 0, "copy spread");
  const u16* cbase = act + copy_lds_base<LDA>(lane, wave);
  char* cdst = reinterpret_cast<char*>(dst) + coff;
  const int lr = lane & 31, lh = lane >> 5;
  const u16* brow = act + lr * LDA + 8 * lh;
  // B fragment of the bias step: ones against the three bias terms (lane
  // half 1 meets zero weights)
  const bf16x8 ones = __builtin_bit_cast(bf16x8, make_uint4(0x3f803f80u, 0x00003f80u, 0u, 0u));
  bf16x8 a[PD + 1][MT];
  bf16x8 b[2][NT];
#pragma unroll
  for (int q = 0; q < PD; ++q)
#pragma unroll
    for (int m = 0; m < MT; ++m) a[q][m] = pf.a[q][m];
#pragma unroll
  for (int n = 0; n < NT; ++n) b[0][n] = *reinterpret_cast<const bf16x8*>(brow + 32 * n * LDA);
  const f32x16 zero = {};
#pragma unroll
  for (int ks = 0; ks < N; ++ks) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      if (ks + PD < N)
        a[(ks + PD) % (PD + 1)][m] = load_frag(W, woff, (uint32_t)(m * N + ks + PD) * 1024);
      else
        pf.a[ks + PD - N][m] = load_frag(Wnext, woff, (uint32_t)(m * N + ks + PD - N) * 1024);
    }
    const int j = ks / CS;                       // copy kilobyte of this step, if ks % CS == 0
    const bool cp = ks % CS == 0 && j < C::COPIES && copy;
    bf16x8 cv;
    if (cp) cv = copy_read<LDA>(cbase + 16 * (j >> 1) * LDA + 32 * (j & 1));
    if (ks + 1 < KS) {
#pragma unroll
      for (int n = 0; n < NT; ++n)
        b[(ks + 1) & 1][n] = *reinterpret_cast<const bf16x8*>(brow + 32 * n * LDA + 16 * (ks + 1));
    }
    // keep the prefetches above the products of this step (the scheduler
    // would otherwise sink each load next to its first use)
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int m = 0; m < MT; ++m)
        acc[m][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ks % (PD + 1)][m], ks < KS ? b[ks & 1][n] : ones,
                                                           ks == 0 ? zero : acc[m][n], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    if (cp)
      *reinterpret_cast<uint4*>(cdst + ((j >> 1) * (H / 32) + (j & 1)) * 1024) = __builtin_bit_cast(uint4, cv);
    __builtin_amdgcn_sched_barrier(0);
  }
}

// max(a, b) of two finite values as one v_max_f32: written out so that the
// compiler adds no NaN-quieting operation on the matrix-core results.
__device__ __forceinline__ float vmax(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// LeakyReLU (slope in [0, 1]: max(v, s v)), bf16 rounding and the lane's sign
// mask words of one layer's outputs.  pk[mt][nt][g] = packed bf16 of q = 0,1
// and 2,3.  The sign bits are gathered with one byte permute per group (the
// sign of a packed bf16 is bit 7 of its high byte) and a shift-and-or.
template <int MT, int NT>
__device__ __forceinline__ void activate(const f32x16 (&v)[MT][NT], float slope, uint2 (&pk)[MT][NT][4],
                                         uint32_t (&m)[MT * NT / 2]) {
#pragma unroll
  for (int k = 0; k < MT * NT / 2; ++k) m[k] = 0u;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int t = mt * NT + nt;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x16& x = v[mt][nt];
        const uint32_t p01 = pack_bf16(vmax(x[4 * g], slope * x[4 * g]), vmax(x[4 * g + 1], slope * x[4 * g + 1]));
        const uint32_t p23 = pack_bf16(vmax(x[4 * g + 2], slope * x[4 * g + 2]), vmax(x[4 * g + 3], slope * x[4 * g + 3]));
        pk[mt][nt][g] = make_uint2(p01, p23);
        // bytes: high byte of q0, q1, q2, q3 -> sign of q at bit 8 q + 7
        const uint32_t r = __builtin_amdgcn_perm(p23, p01, 0x07050301u);
        const int pos = g + 4 * (t & 1);
        m[t >> 1] |= (r >> (7 - pos)) & (0x01010101u << pos);
      }
    }
}

// Sign bits of eight bf16 values (an MFMA operand fragment): bit t is set
// where value t is negative (or -0).  A byte permute with the sign-replicating
// selectors turns each value's sign bit into a byte 0x00 or 0xff (-1), and a
// signed 4-way byte dot product against -1, -2, -4, -8 (-16 .. -128 for
// values 4..7) sums them into the byte.
__device__ __forceinline__ uint32_t sign_byte(bf16x8 v) {
  const uint4 w = __builtin_bit_cast(uint4, v);
  const int lo = (int)__builtin_amdgcn_perm(w.y, w.x, 0x0B0A0908u);   // values 0..3
  const int hi = (int)__builtin_amdgcn_perm(w.w, w.z, 0x0B0A0908u);   // values 4..7
  return (uint32_t)__builtin_amdgcn_sdot4(lo, (int)0xF8FCFEFFu, __builtin_amdgcn_sdot4(hi, (int)0x80C0E0F0u, 0, false),
                                          false);
}

// All-ones where output (t, g, q) of a lane's mask words is negative.
template <int MW>
__device__ __forceinline__ uint32_t neg_mask(const uint32_t (&m)[MW], int t, int g, int q) {
  return (uint32_t)__builtin_amdgcn_sbfe((int)m[t >> 1], 8 * q + g + 4 * (t & 1), 1);
}

// v times LeakyReLU' (1, or the slope where the mask is set): a bitwise
// select, neg ? slope v : v.
__device__ __forceinline__ float leaky_grad(float v, float slope, uint32_t neg) {
  return __uint_as_float(__builtin_amdgcn_bitop3_b32(neg, __float_as_uint(slope * v), __float_as_uint(v), 0xCA));
}

// A lane's mask words of one layer: store and load as one vector.
__device__ __forceinline__ void store_mask(uint32_t* dst, const uint32_t (&m)[4]) {
  *reinterpret_cast<uint4*>(dst) = make_uint4(m[0], m[1], m[2], m[3]);
}
__device__ __forceinline__ void load_mask(const uint32_t* src, uint32_t (&m)[4]) {
  const uint4 v = *reinterpret_cast<const uint4*>(src);
  m[0] = v.x; m[1] = v.y; m[2] = v.z; m[3] = v.w;
}
__device__ __forceinline__ void load_mask(Rsrc r, uint32_t voff, uint32_t (&m)[4]) {
  const uint4 v = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, 0, 0));
  m[0] = v.x; m[1] = v.y; m[2] = v.z; m[3] = v.w;
}

// Writes a layer's packed outputs into the LDS tile.
template <int MT, int NT, int LDA>
__device__ __forceinline__ void store_tile(u16* act, const uint2 (&pk)[MT][NT][4], int ow, int lane) {
  const int lr = lane & 31, lh = lane >> 5;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<uint2*>(act + (32 * nt + lr) * LDA + ow + 32 * mt + 8 * g + 4 * lh) = pk[mt][nt][g];
}

struct ChainArgs {
  const float* W0;           // first layer [H][F] fp32
  const u16* W0f;            // the same as split-term fragments (k_w0_frag)
  const u16* W1f;            // W_1 and b_1 as first-layer slot fragments (k_w1_frag)
  const float* b0;           // [H]
  const u16* Wb;             // hidden layers, bf16, forward fragment order with the bias step
  const u16* WTb;            // the same, transposed ([in][out]), backward fragment order
  const float* wo;           // logit layer [H]
  const float* bo;           // [1]
  float slope;
  int NH;
  ChunkArgs c;
  float inv_n;               // 1 / (events of this batch)
  EventArgs ev;              // this chunk's events (sampled or from a buffer)
  u16* act;                  // [NH][rows H]: A_1 .. A_NH, K-fragment order (A_1 not stored with kRebuildA1)
  float* xs;                 // [rows][2]: the events' coordinates, with kRebuildA1
  u16* dlt;                  // [NH][rows H]: unit-seed signal at A_2 .. A_{NH+1}, K-fragment order
  uint32_t* mask;            // [NH + 1][rows / T][WAVES][64 lanes][4]: signs of A_1 .. A_{NH+1}
  uint8_t* maskT;            // [rows / T][H / 32][64 lanes][T / 16]: signs of A_{NH+1}, K-fragment order
  float* eD;                 // [rows] dL_D/dz (0 on padding)
  float* eG;                 // [rows] dL_G/dz (fake; 0 otherwise)
  float* logits;             // caller's array (indexed from c.row0) or NULL
  float* dLg_dx;             // caller's array (indexed from c.row0) or NULL
  float* plog;               // [gridDim.x][H + 3]: dW_o, then sum softplus(+-z), sum e_D
  float* pfb;                // [gridDim.x][H F + H]: dW_1, then db_1
};

// softplus(t) = max(t, 0) + ln(1 + e^-|t|), on the hardware units.
__device__ __forceinline__ float softplus_fast(float t) { return fmaxf(t, 0.0f) + log1p_k(fast_exp(-fabsf(t))); }

// Forward chain of one chunk: the tile's events sampled (or read) into LDS,
// A_1 (bf16 matrix cores on split terms) -> hidden layers -> logit z, BCE seeds
// e_D and e_G, and per-workgroup partials of dW_o, db_o and the loss sums.
// Stores A_1 .. A_NH, the masks and the top layer's sign bytes for later
// kernels.
template <int H, int F, int D, bool kHD8>
__global__ __launch_bounds__(Chain<H>::THREADS, Chain<H>::BPC) void k_fwd_chain(ChainArgs p) {
  using C = Chain<H>;
  constexpr int T = C::T, LDA = C::LDA, WAVES = C::WAVES, MT = C::MT, NT = C::NT, MW = C::MW, NTH = C::THREADS;
  using L1 = FirstLayer<F>;
  static_assert(kHD8 ? (F == 8 && D == 3) : F == D, "features");
  // The first layer's input slots ([T][L1::LDB] bf16) live in the activation
  // tile where a separate array would not fit two workgroups per CU (or one)
  // into the 160 KB of LDS; they are consumed before A_1 is written there.
  constexpr size_t kLds = 2 * T * LDA + 4 * T * D + (kHD8 ? 8 * T : 4) + 4 * WAVES * T + 4 * T + 6 * T;
  constexpr bool kAliasB = (kLds + 2 * T * L1::LDB) * C::BPC > 163840;
  __shared__ __attribute__((aligned(16))) u16 act[T * LDA];
  __shared__ __attribute__((aligned(16))) u16 sBbuf[kAliasB ? 8 : T * L1::LDB];
  __shared__ float sx[T * D];                   // coordinates (and HD8 log features), before the feature map
  __shared__ float slg[kHD8 ? T * 2 : 1];
  __shared__ float zpart[WAVES][T];
  __shared__ float se_s[T];
  __shared__ __attribute__((aligned(16))) u16 sterm[3][T];   // e_D of each event as bf16 terms hi, mid, lo
  u16* const sB = kAliasB ? act : sBbuf;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lh = lane >> 5;
  const int ow = 32 * MT * wave;
  const uint32_t woff = weight_offset<H, true>(wave, lane);
  const uint32_t coff = ((uint32_t)(2 * wave * 64 + lane)) * 16;
  const ChunkArgs c = p.c;
  const int64_t rstride = (int64_t)c.rows;
  const int ntiles = c.rows / T;
  const float slope = p.slope;
  // the wave's first-layer weight fragments (k_w1_frag), loaded per tile
  const Rsrc rs_w1 = make_rsrc(p.W1f, (uint32_t)(H / 32) * L1::KS * 1024u);
  const uint32_t w1off = ((uint32_t)MT * wave * L1::KS * 64u + lane) * 16u;
  // logit A fragments: rows 0..2 are the bf16 terms hi, mid, lo of w_o (their
  // sum is w_o exactly), other rows zero; the K order matches the lane's
  // activations (see the logit below)
  bf16x8 wof[MT][2];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      uint32_t w[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        uint32_t h2[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int i = 2 * u + e;
          const int f = ow + 32 * mt + 16 * s + (i < 4 ? 4 * lh + i : 8 + 4 * lh + i - 4);
          uint32_t lo;
          const uint32_t hm = bias_terms(p.wo[f], lo);
          h2[e] = lr == 0 ? (hm & 0xffffu) : lr == 1 ? (hm >> 16) : lr == 2 ? lo : 0u;
        }
        w[u] = h2[0] | (h2[1] << 16);
      }
      wof[mt][s] = __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
    }
  float dwo[MT] = {0.f, 0.f};                   // dW_o partial of feature ow + 32 nb + lr (lane half 0)
  const float bo = p.bo[0];
  float l0 = 0.f, l1 = 0.f, se = 0.f;           // loss and e_D sums of event tid (tid < T)
  WeightPrefetch<H> pf;
  prefetch_weights<H, true>(weight_rsrc<H, true>(p.Wb, 0), pf, woff);
  // the tile's events are formed in LDS from inputs fetched one tile ahead
  TileEvents<T, D, NTH> te;
  if ((int)blockIdx.x < ntiles) te.fetch(p.ev, c, blockIdx.x, tid);
  const f32x16 zero = {};

  for (int tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int r0 = tile * T;
    te.template form<kHD8>(p.ev, c, tile, tid, sx, slg, kRebuildA1<H, F, kHD8> ? p.xs : nullptr);
    if (tile + (int)gridDim.x < ntiles) te.fetch(p.ev, c, tile + gridDim.x, tid);
    bf16x8 a1[MT][L1::KS];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int s = 0; s < L1::KS; ++s) a1[mt][s] = load_frag(rs_w1, w1off, (uint32_t)(mt * L1::KS + s) * 1024u);
    auto mask_at = [&](int layer) __attribute__((always_inline)) {
      return p.mask + ((((int64_t)layer * ntiles + tile) * WAVES + wave) * 64 + lane) * MW;
    };
    __syncthreads();                              // coordinates staged; last tile's readers of act are done
    if (tid < T) {
      float f[F];
      if constexpr (kHD8) {
        hd8_features(sx, slg, tid, f);
      } else {
#pragma unroll
        for (int j = 0; j < F; ++j) f[j] = sx[tid * D + j];
      }
      first_layer_row<F>(f, sB + tid * L1::LDB);
    }
    __syncthreads();                              // input slots staged

    // ---- first layer on the bf16 matrix cores (split terms) ----------------
    {
      f32x16 v[MT][NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        bf16x8 bfr[L1::KS];                       // slots 16 s + 8 (l / 32) .. + 7 of event 32 nt + l % 32
#pragma unroll
        for (int s = 0; s < L1::KS; ++s)
          bfr[s] = *reinterpret_cast<const bf16x8*>(sB + (32 * nt + lr) * L1::LDB + 16 * s + 8 * lh);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          v[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[mt][0], bfr[0], zero, 0, 0, 0);
#pragma unroll
          for (int s = 1; s < L1::KS; ++s)
            v[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[mt][s], bfr[s], v[mt][nt], 0, 0, 0);
        }
      }
      if constexpr (kAliasB) __syncthreads();     // every wave has read the slots before A_1 overwrites them
      uint2 pk[MT][NT][4];
      uint32_t m[MW];
      activate<MT, NT>(v, slope, pk, m);
      store_mask(mask_at(0), m);
      store_tile<MT, NT, LDA>(act, pk, ow, lane);
    }
    __syncthreads();

    // ---- hidden layers -----------------------------------------------------
    for (int l = 0; l < p.NH; ++l) {
      const bool last = l == p.NH - 1;
      f32x16 acc[MT][NT];
      // the next product is layer l + 1, or the first hidden layer of the next
      // tile; then the product's input A_{l+1} goes to HBM
      chain_gemm<H, true>(weight_rsrc<H, true>(p.Wb, l), weight_rsrc<H, true>(p.Wb, last ? 0 : l + 1), woff, pf,
                          act, acc, lane, wave, p.act + ((int64_t)l * rstride + r0) * H, coff,
                          !(kRebuildA1<H, F, kHD8> && l == 0 && p.NH > 1));
      uint2 pk[MT][NT][4];
      uint32_t m[MW];
      activate<MT, NT>(acc, slope, pk, m);
      store_mask(mask_at(l + 1), m);
      if (!last) {
        __syncthreads();                             // every wave is done reading this layer's input
        store_tile<MT, NT, LDA>(act, pk, ow, lane);
        __syncthreads();
        continue;
      }
      // ---- logit layer: z = w_o . A_{NH+1} + b_o on the matrix cores -------
      // The lane's activations of tile (mt, nt), groups 2 s and 2 s + 1, are a
      // B fragment (K = 16 features 32 mt + 16 s .. + 15 of the wave, in the
      // order 4 h + 0..3, 8 + 4 h + 0..3 for lane half h) of event 32 nt + l % 32;
      // row m < 3 of the product is the event's dot with term m of w_o.
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        f32x16 zacc = zero;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int s = 0; s < 2; ++s) {
            const bf16x8 bfr = __builtin_bit_cast(
                bf16x8, make_uint4(pk[mt][nt][2 * s].x, pk[mt][nt][2 * s].y, pk[mt][nt][2 * s + 1].x,
                                   pk[mt][nt][2 * s + 1].y));
            zacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wof[mt][s], bfr, zacc, 0, 0, 0);
          }
        // rows 0, 1, 2 of column l % 32 sit in registers 0, 1, 2 of lane half 0
        if (lh == 0) zpart[wave][32 * nt + lr] = (zacc[0] + zacc[1]) + zacc[2];
      }
      __syncthreads();                               // zpart complete; every wave is done reading act
      store_tile<MT, NT, LDA>(act, pk, ow, lane);    // A_{NH+1}, for dW_o
      if (tid < T) {
        const int r = r0 + tid;
        float z = bo;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) z += zpart[w][tid];
        const bool valid = r < c.valid;
        float e = 0.f, g = 0.f;
        if (valid) {
          const float sig_neg = fast_rcp(1.0f + fast_exp(z));
          if (c.fake) {
            e = (1.0f - sig_neg) * p.inv_n;
            g = -sig_neg * p.inv_n;
          } else {
            e = -sig_neg * p.inv_n;
          }
        }
        se_s[tid] = e;
        {
          uint32_t lo;
          const uint32_t hm = bias_terms(e, lo);
          sterm[0][tid] = (u16)(hm & 0xffffu);
          sterm[1][tid] = (u16)(hm >> 16);
          sterm[2][tid] = (u16)lo;
        }
        p.eD[r] = e;
        p.eG[r] = g;
        se += e;
        if (valid) {
          if (p.logits) p.logits[c.row0 + r] = z;
          if (c.fake) {
            l0 += softplus_fast(z);
            l1 += softplus_fast(-z);
          } else {
            l0 += softplus_fast(-z);
          }
        }
      }
      __syncthreads();                               // A_{NH+1} and the seeds staged
      // dW_o partial = sum_events e_D A_{NH+1} on the matrix cores: rows 0..2
      // of the A operand are the bf16 terms of e_D (their sum is e_D exactly),
      // the B operand the wave's own columns of the tile (K = events); rows
      // 0..2 of the product sit in registers 0..2 of lane half 0
      {
        // the transposed-read base, formed here (an opaque copy keeps the
        // compiler from hoisting sixteen far-offset addresses out of the tile
        // loop into spilled registers)
        int ci = copy_lds_base<LDA>(lane, wave);
        asm volatile("" : "+v"(ci));
        const u16* cbase = act + ci;
        f32x16 cz[MT];
        // the same fragments' sign bits, for the top layer's weight gradient:
        // byte kb of (nb, lane) covers rows 16 kb + 8 (lane / 32) .. + 7 of
        // column ow + 32 nb + lane % 32
        uint32_t sb[MT][2];
#pragma unroll
        for (int kb = 0; kb < T / 16; ++kb) {
          const uint4 tv = *reinterpret_cast<const uint4*>(&sterm[lr < 3 ? lr : 0][16 * kb + 8 * lh]);
          const bf16x8 af = __builtin_bit_cast(bf16x8, lr < 3 ? tv : make_uint4(0u, 0u, 0u, 0u));
#pragma unroll
          for (int nb = 0; nb < MT; ++nb) {
            const bf16x8 bv = copy_read<LDA>(cbase + 16 * kb * LDA + 32 * nb);
            cz[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bv, kb == 0 ? zero : cz[nb], 0, 0, 0);
            const uint32_t byte = sign_byte(bv) << (8 * (kb & 3));
            sb[nb][kb >> 2] = (kb & 3) == 0 ? byte : (sb[nb][kb >> 2] | byte);
          }
        }
#pragma unroll
        for (int nb = 0; nb < MT; ++nb) {
          dwo[nb] += (cz[nb][0] + cz[nb][1]) + cz[nb][2];
          *reinterpret_cast<uint2*>(p.maskT + ((size_t)(tile * (H / 32) + MT * wave + nb) * 64 + lane) * (T / 16)) =
              make_uint2(sb[nb][0], sb[nb][1]);
        }
      }
      // act, zpart, se_s and sterm are next written after the next tile's
      // first barrier, which every thread reaches only after this point.
    }
  }

  // ---- per-workgroup partials, fixed order ---------------------------------
  float* dst = p.plog + (int64_t)blockIdx.x * (H + 3);
  if (lh == 0) {
#pragma unroll
    for (int nb = 0; nb < MT; ++nb) dst[ow + 32 * nb + lr] = dwo[nb];
  }
  float s3[3] = {l0, l1, se};
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    float v = s3[k];
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) zpart[wave][k] = v;
  }
  __syncthreads();
  if (tid < 3) {
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) v += zpart[w][tid];
    dst[H + tid] = v;
  }
}

// Backward chain of one chunk: the unit-seed signal from the logit layer down
// through the hidden layers (MFMA, LeakyReLU' from the masks), storing the
// signals at A_2 .. A_{NH+1} for the weight-gradient products; then the first
// layer on the matrix cores: dW_1 and db_1 (signal times e_D times the
// features, accumulated across tiles into per-workgroup partials) and, for
// fake chunks, dL_G/dx (signal times W_1, scaled by e_G, through the HD8
// Jacobian when used).  Each tile's events are formed in LDS again (sampled
// or read, as in the forward chain), and its seeds and masks loaded one tile
// ahead.
template <int H, int F, int D, bool kHD8>
__global__ __launch_bounds__(Chain<H>::THREADS, Chain<H>::BPC) void k_bwd_chain(ChainArgs p) {
  using C = Chain<H>;
  constexpr int T = C::T, LDA = C::LDA, WAVES = C::WAVES, MT = C::MT, NT = C::NT, MW = C::MW, NTH = C::THREADS;
  constexpr int SU = (2 * T + NTH - 1) / NTH;   // staged seed values per thread
  constexpr int KB = T / 16;                    // K steps of the dW_1 product (events)
  constexpr int NB = T / 32;                    // 32-event blocks of the dL/dx product
  constexpr int WPB = WAVES / NB;               // waves per event block (K split over hidden features)
  constexpr int KSW = C::KS / WPB;              // dL/dx K steps per wave
  static_assert(F <= 8 && D <= F && (WPB == 1 || WPB == 2) && (KB * 64) % NTH == 0, "first-layer layout");
  static_assert(kHD8 ? (F == 8 && D == 3) : F == D, "features");
  __shared__ __attribute__((aligned(16))) u16 act[T * LDA];
  __shared__ float srow[T * (2 + F + D)];       // per event: e_D, e_G | features | x
  __shared__ float slg[kHD8 ? T * 2 : 1];       // HD8: log features, before the map
  __shared__ __attribute__((aligned(16))) float swo[H];
  __shared__ __attribute__((aligned(16))) u16 sfp[KB * 64 * 8];   // dW_1 A operand of the tile
  __shared__ float sgx[WPB == 2 ? T * 8 : 1];   // dL/dx partials of the second K half
  float* se = srow;                             // [T][2]
  float* sfeat = srow + 2 * T;                  // [T][F]
  float* sx = sfeat + T * F;                    // [T][D]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lh = lane >> 5;
  const int ow = 32 * MT * wave;
  const uint32_t woff = weight_offset<H, false>(wave, lane);
  const uint32_t coff = ((uint32_t)(2 * wave * 64 + lane)) * 16;
  const ChunkArgs c = p.c;
  const int64_t rstride = (int64_t)c.rows;
  const int ntiles = c.rows / T;
  for (int k = tid; k < H; k += NTH) swo[k] = p.wo[k];
  // dW_1 partial of features ow + 32 nb + lr, inputs 4 lh + 0..3, then db_1
  // (lane half 0)
  float adw[MT][5];
#pragma unroll
  for (int nb = 0; nb < MT; ++nb)
#pragma unroll
    for (int k = 0; k < 5; ++k) adw[nb][k] = 0.f;
  const bool want_dx = c.fake && p.dLg_dx != nullptr;
  const float slope = p.slope;
  const int NH = p.NH;
  WeightPrefetch<H> pf;
  prefetch_weights<H, false>(weight_rsrc<H, false>(p.WTb, NH - 1), pf, woff);
  // Loads through buffer resources with 32-bit per-lane offsets, so that no
  // 64-bit per-lane pointer stays live across the tile loop (the compiler would
  // hoist and spill it, and each reload waits for every outstanding store).
  const Rsrc rs_mask = make_rsrc(p.mask, (uint32_t)(NH + 1) * ntiles * WAVES * 64u * MW * 4u);
  const uint32_t mlane = ((uint32_t)wave * 64u + lane) * MW * 4u;
  auto mask_off = [&](int layer, int tile) __attribute__((always_inline)) {
    return ((uint32_t)(layer * ntiles + tile) * WAVES * 64u) * MW * 4u + mlane;
  };
  const Rsrc rs_eD = make_rsrc(p.eD, (uint32_t)c.rows * 4u), rs_eG = make_rsrc(p.eG, (uint32_t)c.rows * 4u);
  // the tile's seeds (value k of srow: e_D of event k / 2 for even k, e_G for
  // odd k), loaded one tile ahead; its events formed in LDS from inputs
  // fetched one tile ahead
  float sv[SU];
  auto load_seeds = [&](int tile) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < SU; ++u) {
      const int k = tid + NTH * u;
      if (k < 2 * T) sv[u] = load_f32((k & 1) ? rs_eG : rs_eD, (uint32_t)(tile * T + (k >> 1)) * 4u);
    }
  };
  TileEvents<T, D, NTH> te;
  // With kRebuildA1 the forward chain has stored the chunk's coordinates:
  // read them back (8 bytes a row) instead of sampling the events again.
  EventArgs evb = p.ev;
  ChunkArgs cb = c;
  if (kRebuildA1<H, F, kHD8> && p.xs) {
    evb.sampled = 0;
    evb.xin = p.xs;
    cb.row0 = 0;
  }
  uint32_t mtop[MW];
  if ((int)blockIdx.x < ntiles) {
    load_seeds(blockIdx.x);
    te.fetch(evb, cb, blockIdx.x, tid);
    load_mask(rs_mask, mask_off(NH, blockIdx.x), mtop);
  }
  __syncthreads();                              // swo staged

  for (int tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int r0 = tile * T;
    const int next = tile + gridDim.x;
#pragma unroll
    for (int u = 0; u < SU; ++u) {
      const int k = tid + NTH * u;
      if (k < 2 * T) se[k] = sv[u];
    }
    te.template form<kHD8>(evb, cb, tile, tid, kHD8 ? sx : sfeat, slg);
    if (next < ntiles) {
      load_seeds(next);
      te.fetch(evb, cb, next, tid);
    }
    // ---- unit-seed signal at A_{NH+1}: w_o * LeakyReLU'(A_{NH+1}) ----------
    {
      uint2 pk[MT][NT][4];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 w4 = *reinterpret_cast<const f32x4*>(&swo[ow + 32 * mt + 8 * g + 4 * lh]);
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            const int t = mt * NT + nt;
            float d[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) d[q] = leaky_grad(w4[q], slope, neg_mask(mtop, t, g, q));
            pk[mt][nt][g] = make_uint2(pack_bf16(d[0], d[1]), pack_bf16(d[2], d[3]));
          }
        }
      store_tile<MT, NT, LDA>(act, pk, ow, lane);
    }
    if constexpr (kHD8) {
      __syncthreads();                           // coordinates staged
      if (tid < T) {
        float f[8];
        hd8_features(sx, slg, tid, f);
#pragma unroll
        for (int j = 0; j < 8; ++j) sfeat[tid * 8 + j] = f[j];
      }
    }
    __syncthreads();                             // the staged rows too
    // ---- dW_1 A operand: the split terms of e_D times each input ------------
    // piece (kb, l) holds row R = l % 32 for events 16 kb + 8 (l / 32) .. + 7
    // (the row arrangement is described at k_w0_frag; rows 24..26 are the
    // terms of e_D itself, for db_1).  Read after the hidden layers' barriers.
#pragma unroll
    for (int q = 0; q < KB * 64 / NTH; ++q) {
      const int slot = tid + NTH * q, l = slot & 63, R = l & 31, term = R >> 3, j = R & 7;
      const int ev0 = 16 * (slot >> 6) + 8 * (l >> 5);
      // row R = 8 term + j holds term `term` of e_D times input j (term < 3,
      // j < F); the db_1 rows 24 + p (p < 3) hold term p of e_D itself; the
      // other rows are zero
      const bool is_in = term < 3 && j < F, is_db = term == 3 && j < 3;
      const int jj = is_in ? j : 0, ts = term < 3 ? term : (j < 3 ? j : 0);
      const uint32_t keep = is_in ? 0xffffffffu : 0u;
      const float* frow = sfeat + ev0 * F + jj;
      uint32_t w[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        uint32_t h2[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int i = 2 * u + e;
          const float fv = __uint_as_float(__float_as_uint(frow[i * F]) & keep);   // input j, or +0
          // the product rounded once (not fused into the split), so the
          // three terms sum to it exactly
          h2[e] = bf16_term(mul_rounded(se[2 * (ev0 + i)], is_db ? 1.0f : fv), ts);
        }
        w[u] = h2[0] | (h2[1] << 16);
      }
      *reinterpret_cast<uint4*>(sfp + slot * 8) = make_uint4(w[0], w[1], w[2], w[3]);
    }
    // ---- hidden layers, top down ---------------------------------------------
    for (int l = NH - 1; l >= 0; --l) {
      uint32_t m[MW];
      load_mask(rs_mask, mask_off(l, tile), m);
      if (l == 0 && next < ntiles) load_mask(rs_mask, mask_off(NH, next), mtop);
      f32x16 acc[MT][NT];
      // the next product is layer l - 1, or the top layer of the next tile;
      // the product's input (the signal at A_{l+2}) goes to HBM meanwhile,
      // except at the top: the top layer's weight gradient rebuilds that
      // signal from w_o and the forward chain's sign bytes
      chain_gemm<H, false>(weight_rsrc<H, false>(p.WTb, l), weight_rsrc<H, false>(p.WTb, l > 0 ? l - 1 : NH - 1), woff,
                           pf, act, acc, lane, wave, p.dlt + ((int64_t)(l < NH - 1 ? l : 0) * rstride + r0) * H, coff,
                           l < NH - 1);
      uint2 pk[MT][NT][4];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int t = mt * NT + nt;
            float d[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) d[q] = leaky_grad(acc[mt][nt][4 * g + q], slope, neg_mask(m, t, g, q));
            pk[mt][nt][g] = make_uint2(pack_bf16(d[0], d[1]), pack_bf16(d[2], d[3]));
          }
      __syncthreads();                               // every wave is done reading this layer's input
      store_tile<MT, NT, LDA>(act, pk, ow, lane);
      __syncthreads();
    }
    // ---- first layer: act holds the signal at A_1 ---------------------------
    // dW_1 / db_1: rows R of sfp against the wave's own feature columns of the
    // signal (K = the tile's events), the terms added within the lane
    {
      int ci = copy_lds_base<LDA>(lane, wave);   // formed here, as in the forward chain's dW_o
      asm volatile("" : "+v"(ci));
      const u16* cbase = act + ci;
      f32x16 cw[MT];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const bf16x8 af = *reinterpret_cast<const bf16x8*>(sfp + (kb * 64 + lane) * 8);
#pragma unroll
        for (int nb = 0; nb < MT; ++nb) {
          const bf16x8 bf = copy_read<LDA>(cbase + 16 * kb * LDA + 32 * nb);
          cw[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bf, kb == 0 ? f32x16{} : cw[nb], 0, 0, 0);
        }
      }
#pragma unroll
      for (int nb = 0; nb < MT; ++nb) {
#pragma unroll
        for (int q = 0; q < 4; ++q) adw[nb][q] += (cw[nb][q] + cw[nb][4 + q]) + cw[nb][8 + q];
        adw[nb][4] += (cw[nb][12] + cw[nb][13]) + cw[nb][14];
      }
    }
    if (want_dx) {
      // g[event][j] = sum_o signal[event][o] W_1[o][j]: rows R of W0f against
      // the signal rows of event block nb (K = hidden features, split over
      // WPB waves); lane (lh, lr) gets inputs 4 lh + 0..3 of event 32 nb + lr
      const int nb = wave % NB, kh = wave / NB;
      const u16* grow = act + (32 * nb + lr) * LDA + 8 * lh;
      const Rsrc w0r = make_rsrc(p.W0f, (uint32_t)C::KS * 1024);
      bf16x8 af[KSW];
#pragma unroll
      for (int s = 0; s < KSW; ++s) af[s] = load_frag(w0r, (uint32_t)lane * 16, (uint32_t)(kh * KSW + s) * 1024);
      f32x16 cg = {};
#pragma unroll
      for (int s = 0; s < KSW; ++s)
        cg = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s], *reinterpret_cast<const bf16x8*>(grow + 16 * (kh * KSW + s)),
                                                     cg, 0, 0, 0);
      float g4[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) g4[q] = (cg[q] + cg[4 + q]) + cg[8 + q];
      const int ev = 32 * nb + lr;
      if constexpr (WPB == 2) {
        if (kh == 1) {
#pragma unroll
          for (int q = 0; q < 4; ++q) sgx[ev * 8 + 4 * lh + q] = g4[q];
        }
        __syncthreads();
        if (kh == 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q) g4[q] += sgx[ev * 8 + 4 * lh + q];
        }
      }
      if (kh == 0) {
        // inputs 4..7 from the other lane half
        float o4[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) o4[q] = __shfl_xor(g4[q], 32, 64);
        const int r = r0 + ev;
        if (lh == 0 && r < c.valid) {
          const float eg = se[2 * ev + 1];
          float g[F];
#pragma unroll
          for (int j = 0; j < F; ++j) g[j] = (j < 4 ? g4[j & 3] : o4[j & 3]) * eg;
          float dx[D];
          if constexpr (kHD8) {
            // d features / d x of [x1, x2, x3, x1x2, x2x3, x1x3, ln x1, ln(1 - x3)];
            // 1/x1 and 1/(1 - x3) from the log features, accurate where fp32 x3 is within ulps of 1
            const float* xe = sx + ev * D;
            const float* fe = sfeat + ev * F;
            const float x1 = xe[0], x2 = xe[1], x3 = xe[2];
            const float inv_x1 = expf(-fe[6]), inv_1mx3 = expf(-fe[7]);
            dx[0] = g[0] + g[3] * x2 + g[5] * x3 + g[6] * inv_x1;
            dx[1] = g[1] + g[3] * x1 + g[4] * x3;
            dx[2] = g[2] + g[4] * x2 + g[5] * x1 - g[7] * inv_1mx3;
          } else {
#pragma unroll
            for (int j = 0; j < D; ++j) dx[j] = g[j];
          }
#pragma unroll
          for (int j = 0; j < D; ++j) p.dLg_dx[(c.row0 + r) * D + j] = dx[j];
        }
      }
    }
    __syncthreads();                                 // before the next tile overwrites act and the staged rows
  }

  // ---- per-workgroup partials of dW_1 and db_1 ------------------------------
  float* dst = p.pfb + (int64_t)blockIdx.x * (H * F + H);
#pragma unroll
  for (int nb = 0; nb < MT; ++nb) {
    const int o = ow + 32 * nb + lr;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (4 * lh + q < F) dst[o * F + 4 * lh + q] = adw[nb][q];
    if (lh == 0) dst[H * F + o] = adw[nb][4];
  }
}

// ---------------------------------------------------------------------------
// Weight-gradient partial of one hidden layer over a slice of rows:
//   P[slice][o][i] = sum_rows bf16(e_D delta)[r][o] A[r][i]
// for one 256 x 256 tile (o0, i0) of the H x H gradient, and in the tiles with
// i0 = 0 the hidden-layer db partial Pdb[slice][o] = sum_rows (e_D delta)[r][o]
// (fp32, before the rounding).  delta (the unit-seed signal) and A come in
// K-fragment order, so every fragment is a contiguous kilobyte read from
// global memory straight into registers; each delta fragment is scaled by the
// e_D of its 8 rows and rounded to bf16 in registers.  One workgroup of four
// waves (one per SIMD) per CU, each wave holding 16 accumulators of 32 x 32 in
// the accumulation registers.
constexpr int kWT = 256;     // weight-gradient tile edge
constexpr int kWThreads = 256;

// The top hidden layer's signal is not stored: its unit-seed value at
// A_{NH+1} is w_o times LeakyReLU' of A_{NH+1}, rounded to bf16, i.e. one of
// two values per output feature, chosen by the sign of the activation.  With
// kTop the weight-gradient kernels rebuild the delta fragments from the sign
// bytes the forward chain stores (byte kb % 8 of piece (kb / 8, column block,
// lane) covers the lane's 8 rows of K block kb) and the two bf16 values of
// the lane's feature, exactly the values the backward chain forms.
struct TopSignal {
  const uint8_t* maskT;    // [K blocks / 8][H / 32][64 lanes][8]
  const float* wo;         // [H]
  float slope;
};

// Unit-seed signal of feature o where the activation is positive (1) or
// negative (slope), as bf16 values in fp32.
__device__ __forceinline__ void top_values(const TopSignal& ts, int o, uint32_t& dpos, uint32_t& dneg) {
  const float w = ts.wo[o];
  dpos = (uint32_t)bf16_bits(w) << 16;
  dneg = (uint32_t)bf16_bits(ts.slope * w) << 16;
}

// One sign byte (per-lane offset voff, scalar offset soff).
__device__ __forceinline__ uint32_t top_byte(Rsrc r, uint32_t voff, uint32_t soff) {
  return (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(r, (int)voff, (int)soff, 0);
}

// Byte offset of the sign byte of K block kb in the lane's column block.
__device__ __forceinline__ uint32_t top_koff(int kb, int CB) { return (uint32_t)(kb >> 3) * CB * 512u + (kb & 7); }

// The 8 rows' signal values of a lane (bit t of `bits` selects row t's value).
__device__ __forceinline__ float top_delta(uint32_t bits, int t, uint32_t dpos, uint32_t dneg) {
  return __uint_as_float(__builtin_amdgcn_bitop3_b32((uint32_t)__builtin_amdgcn_sbfe((int)bits, t, 1), dneg, dpos, 0xCA));
}

// The value of lane N of x's 16-lane row (DPP row_newbcast).
template <int N>
__device__ __forceinline__ float row_bcast(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x150 + N, 0xF, 0xF, true));
}

// kA1 (kRebuildA1, k_wgrad_shared): the input-side operand A_1 is rebuilt
// from the events' coordinates, A_1 = bf16(LeakyReLU(W_1 x + b_1)) with the
// two products and the bias added in fp32 (fmaf), instead of being read.  It
// is the same function as the forward chain's split-term product, evaluated
// in another fp32 order, so an activation can differ from the forward chain's
// by one bf16 step where its fp32 value falls on a rounding boundary.
struct A1Source {
  const float* xs;    // [rows][2]
  const float* W1;    // [H][2]
  const float* b1;    // [H]
  float slope;
};

// The kernel (k_wgrad_shared): each wave owns 64 output rows x all 256
// columns of the tile, so the four waves all need the same eight A fragments
// (256 columns) of every K step.  Instead of each wave streaming all eight,
// wave w fetches fragments 2w and 2w + 1 into registers kWLG steps ahead (kA1:
// rebuilds them from the coordinates, fetched kWXD steps ahead, during the
// products of the step three before), writes them into LDS slot k mod kWNS
// three steps ahead, and every wave reads the eight from there one step ahead,
// so the reads of step k + 1 overlap the products of step k.  This brings one
// copy of each operand into the CU and lets the register prefetch run far
// enough ahead to cover HBM latency.  A barrier after every second K step
// publishes the slots written since the last one (three steps ahead, every
// slot is published before it is read and read by every wave before it is
// written again); the loads in flight are not waited for at the barrier.
// (Staging the fragments through LDS with direct global-to-LDS loads measured
// slower.)
constexpr int kWLG = 5;      // register prefetch distance (K steps) of k_wgrad_shared
constexpr int kWNS = 6;      // register and LDS ring slots: kWLG + 1, even so that step parity is a constant
constexpr int kWXD = 8;      // kA1: the coordinates' prefetch distance (five steps ahead of the rebuild)

// Steps Q = 0 .. N-1 of one pass of the register ring, as a compile-time
// sequence: run() with every step prefetching, tail() with the bounds checked.
template <int N>
struct WRing {
  template <class F>
  __device__ __forceinline__ static void run(F& f, int k0) {
    WRing<N - 1>::run(f, k0);
    f(std::integral_constant<int, N - 1>{}, k0 + N - 1, true, true, true, true);
  }
  template <class F>
  __device__ __forceinline__ static void tail(F& f, int k0, int nk) {
    WRing<N - 1>::tail(f, k0, nk);
    const int k = k0 + N - 1;
    if (k < nk) f(std::integral_constant<int, N - 1>{}, k, k + 1 < nk, k + 3 < nk, k + kWLG < nk, k + kWXD < nk);
  }
};
template <>
struct WRing<0> {
  template <class F>
  __device__ __forceinline__ static void run(F&, int) {}
  template <class F>
  __device__ __forceinline__ static void tail(F&, int, int) {}
};

__device__ __forceinline__ void lds_barrier() {
  // LDS writes complete, then the workgroup barrier; global loads stay in flight
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int H, bool kTop, bool kA1 = false>
__global__ __launch_bounds__(kWThreads, 1) void k_wgrad_shared(const u16* __restrict__ dsc, const u16* __restrict__ A,
                                                               const float* __restrict__ eD, int kb_per_slice,
                                                               int kb_total, float* __restrict__ P,
                                                               float* __restrict__ Pdb, int xcd_map, TopSignal ts,
                                                               A1Source a1s) {
  constexpr int TI = H / kWT;     // tiles per dimension: 1 or 2
  constexpr int CB = H / 32;      // 32-column blocks
  constexpr int FM = 2, FN = 8;   // a wave owns 64 output rows x all 256 columns of the tile
  constexpr int NS = kWNS;
  static_assert(NS == kWLG + 1 && NS % 2 == 0, "ring slots: step parity must be a constant");
  static_assert(!kA1 || (H == 256 && !kTop), "A_1 is rebuilt for the first hidden layer at H = 256");
  constexpr size_t KSTRIDE = (size_t)CB * 512;
  __shared__ __attribute__((aligned(16))) u16 sb[NS][FN][512];
  int tile, slice;
  if (xcd_map) {
    const int x = blockIdx.x % 8, r = blockIdx.x / 8;
    tile = r % (TI * TI);
    slice = (r / (TI * TI)) * 8 + x;
  } else {
    tile = blockIdx.x % (TI * TI);
    slice = blockIdx.x / (TI * TI);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 31, lh = lane >> 5;
  const int ob = (tile / TI) * (kWT / 32) + FM * wave;
  const int ib = (tile % TI) * (kWT / 32);
  const int kb0 = slice * kb_per_slice;
  const int nk = max(0, min(kb_total, kb0 + kb_per_slice) - kb0);
  const u16* pa = dsc + (((size_t)kb0 * CB + ob) * 64 + lane) * 8;
  const u16* pb = A + (((size_t)kb0 * CB + ib + 2 * wave) * 64 + lane) * 8;   // this wave's two A fragments
  const float* pe = eD + (size_t)kb0 * 16 + 8 * lh;
  // kTop: sign bytes through a buffer resource (per-lane offset of column
  // block ob, the K block's offset a scalar)
  const Rsrc rm_top = make_rsrc(ts.maskT, (uint32_t)kb_total * CB * 64u);
  const uint32_t moff = ((uint32_t)ob * 64u + lane) * 8u;
  // kA1: W_1 and b_1 at this wave's two column blocks, and its coordinates
  // pointer: lane l reads row 8 (l / 32) + l % 8 of each K block, so that lane
  // t of every 16-lane row holds row 8 (l / 32) + t of the lane's half
  float w0[2], w1[2], bb[2];
  const float* px = a1s.xs + ((size_t)kb0 * 16 + 8 * lh + (lane & 7)) * 2;
  if constexpr (kA1) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = 32 * (ib + 2 * wave + j) + lr;
      w0[j] = a1s.W1[2 * col];
      w1[j] = a1s.W1[2 * col + 1];
      bb[j] = a1s.b1[col];
    }
  }
  uint32_t dpos[FM], dneg[FM];
  if constexpr (kTop) {
#pragma unroll
    for (int m = 0; m < FM; ++m) top_values(ts, 32 * (ob + m) + lr, dpos[m], dneg[m]);
  }
  f32x16 acc[FM][FN];
#pragma unroll
  for (int m = 0; m < FM; ++m)
#pragma unroll
    for (int n = 0; n < FN; ++n)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[m][n][r] = 0.f;
  float dbs[FM] = {0.f, 0.f};
  bf16x8 ra[kA1 ? 1 : NS][2], rd[NS][FM];
  float2 fx[kA1 ? NS : 1];        // kA1: coordinates of step k in slot k mod NS
  bf16x8 rb[2];                   // kA1: the two rebuilt A_1 fragments of step k + 3
  uint32_t rm[NS][FM];            // kTop: sign bytes instead of rd
  f32x4 re[NS][2];
  bf16x8 fb[2][FN];               // the A fragments of the current and the next step
  auto load = [&](int slot, int k) __attribute__((always_inline)) {
    if constexpr (!kA1) {
#pragma unroll
      for (int j = 0; j < 2; ++j) ra[slot][j] = *reinterpret_cast<const bf16x8*>(pb + k * KSTRIDE + j * 512);
    }
#pragma unroll
    for (int m = 0; m < FM; ++m) {
      if constexpr (kTop) rm[slot][m] = top_byte(rm_top, moff, top_koff(kb0 + k, CB) + m * 512);
      else rd[slot][m] = *reinterpret_cast<const bf16x8*>(pa + k * KSTRIDE + m * 512);
    }
    re[slot][0] = *reinterpret_cast<const f32x4*>(pe + (size_t)k * 16);
    re[slot][1] = *reinterpret_cast<const f32x4*>(pe + (size_t)k * 16 + 4);
  };
  // this wave's two fragments (loaded, or rebuilt with kA1) into LDS slot buf
  auto put = [&](int slot, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
      *reinterpret_cast<bf16x8*>(&sb[buf][2 * wave + j][lane * 8]) = kA1 ? rb[j] : ra[kA1 ? 0 : slot][j];
  };
  auto load_x = [&](int slot, int k) __attribute__((always_inline)) {
    fx[slot] = *reinterpret_cast<const float2*>(px + (size_t)k * 32);
  };
  // kA1: the wave's two A_1 fragments of the step whose coordinates sit in
  // `slot`, bf16(LeakyReLU(fmaf(w1, x1, fmaf(w0, x0, b)))), each row's
  // coordinates broadcast from the lane that loaded them
  auto rebuild = [&](int slot) __attribute__((always_inline)) {
    const float x0 = fx[slot].x, x1 = fx[slot].y;
    const float c0[8] = {row_bcast<0>(x0), row_bcast<1>(x0), row_bcast<2>(x0), row_bcast<3>(x0),
                         row_bcast<4>(x0), row_bcast<5>(x0), row_bcast<6>(x0), row_bcast<7>(x0)};
    const float c1[8] = {row_bcast<0>(x1), row_bcast<1>(x1), row_bcast<2>(x1), row_bcast<3>(x1),
                         row_bcast<4>(x1), row_bcast<5>(x1), row_bcast<6>(x1), row_bcast<7>(x1)};
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      float y[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const float z = fmaf(w1[j], c1[t], fmaf(w0[j], c0[t], bb[j]));
        y[t] = vmax(z, a1s.slope * z);
      }
      rb[j] = __builtin_bit_cast(bf16x8, make_uint4(pack_bf16(y[0], y[1]), pack_bf16(y[2], y[3]),
                                                    pack_bf16(y[4], y[5]), pack_bf16(y[6], y[7])));
    }
  };
  auto get = [&](int buf, int into) __attribute__((always_inline)) {
#pragma unroll
    for (int n = 0; n < FN; ++n) fb[into][n] = *reinterpret_cast<const bf16x8*>(&sb[buf][n][lane * 8]);
  };
  // The delta fragments of one step scaled by e_D and rounded (the A operand
  // of its products), and their fp32 sums for db.
  bf16x8 sa[2][FM];
  auto scale = [&](int slot, int into) __attribute__((always_inline)) {
#pragma unroll
    for (int m = 0; m < FM; ++m) {
      float v[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        float d;
        if constexpr (kTop) d = top_delta(rm[slot][m], t, dpos[m], dneg[m]);
        else d = (float)rd[slot][m][t];
        v[t] = d * re[slot][t >> 2][t & 3];
      }
      dbs[m] += ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
      sa[into][m] = __builtin_bit_cast(bf16x8, make_uint4(pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3]),
                                                          pack_bf16(v[4], v[5]), pack_bf16(v[6], v[7])));
    }
  };
  // Step k (q = k mod NS, so k mod 2 = q mod 2 and k mod 3 = q mod 3): read
  // the fragments of step k + 1 (written during step k - 2, published by the
  // barrier since), write this wave's two of step k + 3 (with kA1 rebuilt
  // during the products and written after them), prefetch step k + kWLG,
  // then the products of step k from the fragments read and scaled one step
  // earlier, with the scaling of step k + 1 interleaved between them (one
  // wave per SIMD: the vector ALU work would otherwise wait for the
  // products' issue).
  auto step = [&](auto qc, int k, bool get_next, bool put_ahead, bool load_ahead, bool x_ahead)
                  __attribute__((always_inline)) {
    constexpr int q = decltype(qc)::value;
    if (get_next) get((q + 1) % NS, (q + 1) & 1);
    if (!kA1 && put_ahead) put((q + 3) % NS, (q + 3) % NS);
    if (load_ahead) load((q + kWLG) % NS, k + kWLG);
    if (kA1 && x_ahead) load_x((q + kWXD) % NS, k + kWXD);
    // keep each step's work inside the step: the scheduler would otherwise
    // hoist later steps' scaling above their loads' waits
    __builtin_amdgcn_sched_barrier(0);
    if (get_next) scale((q + 1) % NS, (q + 1) & 1);
    if (kA1 && put_ahead) rebuild((q + 3) % NS);   // step k + 3, written to LDS after the products
#pragma unroll
    for (int n = 0; n < FN; ++n)
#pragma unroll
      for (int m = 0; m < FM; ++m)
        acc[m][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(sa[q & 1][m], fb[q & 1][n], acc[m][n], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < FM * FN; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one product
      // four vector ALU instructions (five with the sign-bit selects of kTop,
      // ten with the rebuild of A_1)
      __builtin_amdgcn_sched_group_barrier(0x002, kA1 ? 10 : (kTop ? 5 : 4), 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (kA1 && put_ahead) put(0, (q + 3) % NS);
    if (q & 1) lds_barrier();
  };
  if (nk > 0) {
    // prologue without branches (a step past the slice reloads its last step,
    // never used), so that the waits on the loads stay exact in the loop below
    if constexpr (kA1) {
      // coordinates of steps 0..5 into slots 0..5; steps 0..2 rebuilt and
      // published; then steps 6, 7 into the slots 0, 1 they leave
#pragma unroll
      for (int q = 0; q < NS; ++q) load_x(q, min(q, nk - 1));
    }
#pragma unroll
    for (int q = 0; q < kWLG; ++q) load(q, min(q, nk - 1));
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      if constexpr (kA1) rebuild(q);
      put(q, q);
    }
    if constexpr (kA1) {
#pragma unroll
      for (int q = NS; q < kWXD; ++q) load_x(q % NS, min(q, nk - 1));
    }
    lds_barrier();
    get(0, 0);
    scale(0, 0);
  }
  // steady state: NS steps per pass, every step reading, publishing and
  // prefetching (no branches, so the waits on the loads stay exact)
  constexpr int kAhead = kA1 ? kWXD : kWLG;
  int k0 = 0;
  for (; k0 + NS - 1 + kAhead < nk; k0 += NS) WRing<NS>::run(step, k0);
  // tail: the last steps, with the bounds checked
  for (; k0 < nk; k0 += NS) WRing<NS>::tail(step, k0, nk);
  float* out = P + (size_t)slice * H * H;
#pragma unroll
  for (int m = 0; m < FM; ++m)
#pragma unroll
    for (int n = 0; n < FN; ++n)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int o = (ob + m) * 32 + 8 * (r / 4) + 4 * lh + (r % 4), i = (ib + n) * 32 + lr;
        out[(size_t)o * H + i] = acc[m][n][r];
      }
  if (tile % TI == 0) {
#pragma unroll
    for (int m = 0; m < FM; ++m) {
      const float v = dbs[m] + __shfl_xor(dbs[m], 32, 64);
      if (lh == 0) Pdb[(size_t)slice * H + 32 * (ob + m) + lr] = v;
    }
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
  bool a1;               // kRebuildA1: the coordinates are stored instead of A_1
  int chunk;             // rows per chunk
  int rows_max;          // padded rows of the largest chunk
  int blocks;            // workgroups of the chain kernels
  int slices;            // weight-gradient slices per chunk
  size_t off_wb, off_wtb, off_w0f, off_w1f, off_act, off_dlt, off_mask, off_maskT, off_xs, off_eD, off_eG, off_plog,
      off_pfb, off_pw, off_pwdb, off_accl, total;
};

int pad128(int64_t n) { return (int)((n + 127) / 128 * 128); }

int chunk_rows_of(const DiscArgs& a) { return a.chunk_rows > 0 ? a.chunk_rows : kChunkRows; }

Plan make_plan(const DiscArgs& a, int n_cu) {
  const sagips_mlp& D = *a.D;
  Plan p;
  p.H = D.width[1];
  p.NH = D.n_layers - 2;
  p.F = D.width[0];
  p.hd8 = D.features == SAGIPS_FEAT_HD8;
  p.D = a.d;
  p.a1 = p.H == 256 && !p.hd8 && p.F == 2 && p.NH > 1;   // kRebuildA1<H, F, kHD8>, and layer 0 is not the top one
  p.chunk = chunk_rows_of(a);
  const int64_t biggest = std::min<int64_t>(std::max(a.n_fake, a.n_real), p.chunk);
  p.rows_max = pad128(biggest);
  p.blocks = std::max(1, n_cu * (p.H <= 256 ? Chain<256>::BPC : Chain<512>::BPC));
  const int tiles = (p.H / kWT) * (p.H / kWT);
  p.slices = std::max(1, n_cu / tiles);  // one weight-gradient workgroup per CU
  const size_t H = p.H, R = p.rows_max, NH = p.NH;
  size_t o = 0;
  p.off_wb = o; o += al(2 * H * (H + 16) * NH);     // forward copies carry one bias step per 32 rows
  p.off_wtb = o; o += al(2 * H * H * NH);
  p.off_w0f = o; o += al(64 * H);                 // H / 16 pieces of 1 KB
  p.off_w1f = o; o += al(32 * H * 4);             // (H / 32) x at most 4 pieces of 1 KB
  p.off_act = o; o += al(2 * R * H * NH);        // (slot 0, A_1, unused with a1)
  p.off_dlt = o; o += al(2 * R * H * (NH - 1));   // the top layer's signal is rebuilt from signs
  p.off_mask = o; o += al(8 * R * (H / 64) * (NH + 1));
  p.off_maskT = o; o += al(R * H / 8);
  p.off_xs = o; o += p.a1 ? al(8 * R) : 0;
  p.off_eD = o; o += al(4 * R);
  p.off_eG = o; o += al(4 * R);
  p.off_plog = o; o += al(4 * (size_t)p.blocks * (H + 3));
  p.off_pfb = o; o += al(4 * (size_t)p.blocks * (H * p.F + H));
  p.off_pw = o; o += al(4 * (size_t)p.slices * H * H);
  p.off_pwdb = o; o += al(4 * (size_t)p.slices * H);
  p.off_accl = o; o += al(4 * 4);
  p.total = o;
  return p;
}

template <int H, int F, int D, bool kHD8>
void launch_chains(const ChainArgs& ca, int blocks, bool bwd, hipStream_t st) {
  if (!bwd) hipLaunchKernelGGL((k_fwd_chain<H, F, D, kHD8>), dim3(blocks), dim3(Chain<H>::THREADS), 0, st, ca);
  else hipLaunchKernelGGL((k_bwd_chain<H, F, D, kHD8>), dim3(blocks), dim3(Chain<H>::THREADS), 0, st, ca);
}

void launch_chain(const Plan& p, const ChainArgs& ca, bool bwd, hipStream_t st) {
  const int blocks = std::min(p.blocks, ca.c.rows / (p.H == 256 ? Chain<256>::T : Chain<512>::T));
  if (p.H == 256) {
    if (p.hd8) launch_chains<256, 8, 3, true>(ca, blocks, bwd, st);
    else if (p.D == 2) launch_chains<256, 2, 2, false>(ca, blocks, bwd, st);
    else launch_chains<256, 3, 3, false>(ca, blocks, bwd, st);
  } else {
    if (p.hd8) launch_chains<512, 8, 3, true>(ca, blocks, bwd, st);
    else if (p.D == 2) launch_chains<512, 2, 2, false>(ca, blocks, bwd, st);
    else launch_chains<512, 3, 3, false>(ca, blocks, bwd, st);
  }
}

}  // namespace

bool disc_bf16_supported(const sagips_mlp& D, int d, const char** why) {
  const int H = D.width[1];
  if (H != 256 && H != 512) { *why = "bf16 discriminator supports hidden width 256 or 512"; return false; }
  if (!(D.leaky_slope >= 0.0f && D.leaky_slope <= 1.0f)) { *why = "bf16 discriminator needs leaky_slope in [0, 1]"; return false; }
  if (D.n_layers < 3 || D.n_layers - 2 > kMaxNH) { *why = "bf16 discriminator needs 1-4 hidden-to-hidden layers"; return false; }
  for (int l = 1; l < D.n_layers; ++l)
    if (D.width[l] != H) { *why = "all hidden widths must be equal"; return false; }
  if (D.features == SAGIPS_FEAT_PROXY2) { *why = "PROXY2 features are supported by the fp32 discriminator only"; return false; }
  if (D.features == SAGIPS_FEAT_HD8) {
    if (d != 3 || D.width[0] != 8) { *why = "HD8 features need d = 3 and width[0] = 8"; return false; }
  } else if (D.width[0] != d || (d != 2 && d != 3)) {
    *why = "IDENTITY features need width[0] == d in {2, 3}";
    return false;
  }
  return true;
}

size_t disc_bf16_workspace(const DiscArgs& a, int n_cu) { return make_plan(a, n_cu).total; }

int disc_bf16_max_chunk_rows() { return kChunkRows; }

hipError_t launch_disc_bf16(const DiscArgs& a, void* ws, int n_cu, hipStream_t st, Timer* tm) {
  const sagips_mlp& Dm = *a.D;
  const Plan p = make_plan(a, n_cu);
  char* base = static_cast<char*>(ws);
  auto F32 = [&](size_t off) { return reinterpret_cast<float*>(base + off); };
  auto B16 = [&](size_t off) { return reinterpret_cast<u16*>(base + off); };
  const int H = p.H, NH = p.NH;
  u16* Wb = B16(p.off_wb);
  u16* WTb = B16(p.off_wtb);
  const sagips_disc_out& out = *a.out;
  const bool want_grads = out.dW[0] != nullptr;
  const float inv_nf = 1.0f / (float)a.n_fake, inv_nr = 1.0f / (float)a.n_real;

  if (tm) tm->begin("disc_bf16_weights");
  for (int l = 0; l < NH; ++l)
    hipLaunchKernelGGL(k_weights_frag, dim3(((H / 32) * (H / 16 + 1) * 64 + 255) / 256), dim3(256), 0, st, Dm.W[1 + l],
                       Dm.b[1 + l], Wb + (size_t)l * H * (H + 16), WTb + (size_t)l * H * H, H);
  hipLaunchKernelGGL(k_w0_frag, dim3((H / 16) * 64 / 256), dim3(256), 0, st, Dm.W[0], p.F, H, B16(p.off_w0f));
  {
    const int F = p.F, pieces = (H / 32) * ((6 * F + 3 + 15) / 16) * 64;
    const dim3 g((pieces + 255) / 256);
    if (F == 2) hipLaunchKernelGGL(k_w1_frag<2>, g, dim3(256), 0, st, Dm.W[0], Dm.b[0], H, B16(p.off_w1f));
    else if (F == 3) hipLaunchKernelGGL(k_w1_frag<3>, g, dim3(256), 0, st, Dm.W[0], Dm.b[0], H, B16(p.off_w1f));
    else hipLaunchKernelGGL(k_w1_frag<8>, g, dim3(256), 0, st, Dm.W[0], Dm.b[0], H, B16(p.off_w1f));
  }
  if (tm) tm->end();

  SourceArgs src{};
  const bool sampled = a.fake_src != nullptr;
  if (sampled) src = *a.fake_src;

  ChainArgs ca{};
  ca.W0 = Dm.W[0];
  ca.W0f = B16(p.off_w0f);
  ca.W1f = B16(p.off_w1f);
  ca.b0 = Dm.b[0];
  ca.Wb = Wb;
  ca.WTb = WTb;
  ca.wo = Dm.W[NH + 1];
  ca.bo = Dm.b[NH + 1];
  ca.slope = Dm.leaky_slope;
  ca.NH = NH;
  ca.act = B16(p.off_act);
  ca.xs = p.a1 ? F32(p.off_xs) : nullptr;
  ca.dlt = B16(p.off_dlt);
  ca.mask = reinterpret_cast<uint32_t*>(base + p.off_mask);
  ca.maskT = reinterpret_cast<uint8_t*>(base + p.off_maskT);
  const TopSignal top{ca.maskT, ca.wo, ca.slope};
  const A1Source a1s{ca.xs, Dm.W[0], Dm.b[0], ca.slope};
  ca.eD = F32(p.off_eD);
  ca.eG = F32(p.off_eG);
  ca.plog = F32(p.off_plog);
  ca.pfb = F32(p.off_pfb);

  int chunk_index = 0;
  float* lacc = F32(p.off_accl);
  for (int pass = 0; pass < 2; ++pass) {
    const bool fake = pass == 0;
    const int64_t n = fake ? a.n_fake : a.n_real;
    for (int64_t row0 = 0; row0 < n; row0 += p.chunk, ++chunk_index) {
      ChunkArgs c;
      c.row0 = row0;
      c.valid = (int)std::min<int64_t>(p.chunk, n - row0);
      c.rows = pad128(c.valid);
      c.fake = fake ? 1 : 0;
      const int first = chunk_index == 0 ? 1 : 0;
      const int first_batch = row0 == 0 ? 1 : 0;
      ca.ev.src = src;
      ca.ev.xin = fake ? a.fake_x : a.real_x;
      ca.ev.sampled = (fake && sampled) ? 1 : 0;
      ca.c = c;
      ca.inv_n = fake ? inv_nf : inv_nr;
      ca.logits = fake ? out.logits_fake : out.logits_real;
      ca.dLg_dx = fake ? out.dLg_dx : nullptr;
      const int nb = std::min(p.blocks, c.rows / (H == 256 ? Chain<256>::T : Chain<512>::T));
      if (tm) tm->begin("bf16_fwd_chain");
      launch_chain(p, ca, false, st);
      if (tm) tm->end();
      if (want_grads) accumulate(ca.plog, nb, (int64_t)(H + 3), (int64_t)H, out.dW[NH + 1], first, st);
      hipLaunchKernelGGL(k_logit_scalars, dim3(1), dim3(256), 0, st, ca.plog, nb, H, want_grads ? out.db[NH + 1] : nullptr,
                         lacc, c.fake, first, first_batch);

      if (tm) tm->begin("bf16_bwd_chain");
      launch_chain(p, ca, true, st);
      if (tm) tm->end();
      if (want_grads) {
        accumulate(ca.pfb, nb, (int64_t)(H * p.F + H), (int64_t)(H * p.F), out.dW[0], first, st);
        accumulate(ca.pfb + (size_t)H * p.F, nb, (int64_t)(H * p.F + H), (int64_t)H, out.db[0], first, st);
        const int tiles = (H / kWT) * (H / kWT);
        const int xcd_map = p.slices % 8 == 0 ? 1 : 0;
        const int kb_total = c.rows / 16;                           // 16-row K blocks of the chunk
        const int kb_per_slice = (kb_total + p.slices - 1) / p.slices;
        const size_t bst = (size_t)c.rows * H;   // stride between this chunk's per-layer buffers
        for (int l = 0; l < NH; ++l) {
          // hidden layer l maps A_{l+1} -> A_{l+2}: operands A_{l+1} and the signal at A_{l+2}
          // (the top layer's signal rebuilt from the sign bytes)
          const bool top_layer = l == NH - 1;
          const u16* dsc = top_layer ? nullptr : ca.dlt + l * bst;
          const dim3 grid(tiles * p.slices);
          if (tm) tm->begin("bf16_wgrad");
          if (H == 256) {
            if (top_layer)
              hipLaunchKernelGGL((k_wgrad_shared<256, true>), grid, dim3(kWThreads), 0, st, dsc, ca.act + l * bst, ca.eD,
                                 kb_per_slice, kb_total, F32(p.off_pw), F32(p.off_pwdb), xcd_map, top, a1s);
            else if (l == 0 && p.a1)
              hipLaunchKernelGGL((k_wgrad_shared<256, false, true>), grid, dim3(kWThreads), 0, st, dsc, nullptr, ca.eD,
                                 kb_per_slice, kb_total, F32(p.off_pw), F32(p.off_pwdb), xcd_map, top, a1s);
            else
              hipLaunchKernelGGL((k_wgrad_shared<256, false>), grid, dim3(kWThreads), 0, st, dsc, ca.act + l * bst, ca.eD,
                                 kb_per_slice, kb_total, F32(p.off_pw), F32(p.off_pwdb), xcd_map, top, a1s);
          } else {
            if (top_layer)
              hipLaunchKernelGGL((k_wgrad_shared<512, true>), grid, dim3(kWThreads), 0, st, dsc, ca.act + l * bst, ca.eD,
                                 kb_per_slice, kb_total, F32(p.off_pw), F32(p.off_pwdb), xcd_map, top, a1s);
            else
              hipLaunchKernelGGL((k_wgrad_shared<512, false>), grid, dim3(kWThreads), 0, st, dsc, ca.act + l * bst, ca.eD,
                                 kb_per_slice, kb_total, F32(p.off_pw), F32(p.off_pwdb), xcd_map, top, a1s);
          }
          if (tm) tm->end();
          accumulate(F32(p.off_pw), p.slices, (int64_t)H * H, (int64_t)H * H, out.dW[1 + l], first, st);
          accumulate(F32(p.off_pwdb), p.slices, (int64_t)H, (int64_t)H, out.db[1 + l], first, st);
        }
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
