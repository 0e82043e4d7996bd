// Device-side building blocks of the SAGIPS step on gfx950: the
// Philox4x32-10 counter-based generator, the word -> uniform map and a
// numerically stable fp32 Kumaraswamy quantile with its pathwise
// (reparameterisation) derivatives.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sagips {

struct Words {
  uint32_t w[4];
};

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11).  Each round takes two
// 32x32->64 products of counter lanes 0 and 2 with the published multipliers
// and mixes their halves with lanes 1, 3 and the key; the key is advanced by
// the published Weyl increments between rounds.  The key is wave-uniform, so
// its schedule stays in scalar registers.
__device__ __forceinline__ Words philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                               uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    // three-input xor in one v_bitop3_b32 (truth table 0x96)
    const uint32_t n0 = __builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), c1, k0, 0x96);
    const uint32_t n2 = __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), c3, k1, 0x96);
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  Words o;
  o.w[0] = c0; o.w[1] = c1; o.w[2] = c2; o.w[3] = c3;
  return o;
}

// One Philox block per event: counter = (id lo, id hi, stream, 0).
__device__ __forceinline__ Words event_words(uint64_t id, uint32_t stream, uint32_t k0, uint32_t k1) {
  return philox4x32_10((uint32_t)id, (uint32_t)(id >> 32), stream, 0u, k0, k1);
}

// u = ((w >> 9) + 1/2) * 2^-23 and v = 1 - u, both exact in fp32: the
// products and sums below involve at most 24 significant bits.
__device__ __forceinline__ float uniform_u(uint32_t w) {
  return fmaf((float)(w >> 9), 0x1p-23f, 0x1p-24f);
}
__device__ __forceinline__ float uniform_1mu(uint32_t w) {
  return fmaf((float)(w >> 9), -0x1p-23f, 1.0f - 0x1p-24f);
}

// Per-observable constants of one parameter row.
struct Shape {
  float ra;   // 1/a
  float rb;   // 1/b
  float cda;  // -ln2 / a^2:      dx/da = cda * x * log2(g)
  float cdb;  // ln2 / (a b^2):   dx/db = cdb * x * s * log2(1-u) / g
};

// Elementary functions on the hardware transcendental units (v_log_f32 = log2,
// v_exp_f32 = 2^x, v_rcp_f32; each within 1 ulp over the ranges used here).
constexpr float kLn2 = 0.693147180559945309f;
constexpr float kLog2e = 1.442695040888963407f;

__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log(float x) { return __builtin_amdgcn_logf(x) * kLn2; }
__device__ __forceinline__ float fast_exp(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

__device__ __forceinline__ Shape make_shape(float a, float b) {
  Shape s;
  s.ra = 1.0f / a;
  s.rb = 1.0f / b;
  s.cda = -kLn2 * s.ra * s.ra;
  s.cdb = kLn2 * s.ra * s.rb * s.rb;
  return s;
}

// e^t - 1 by Kahan's method: with w = fl(e^t), (w - 1) t / ln w cancels the
// rounding error of w, so the result keeps its relative accuracy as t -> 0.
__device__ __forceinline__ float expm1_k(float t, float w) {
  if (w == 1.0f) return t;
  const float wm1 = w - 1.0f;
  if (wm1 == -1.0f) return -1.0f;       // e^t below half an ulp of 1 (or flushed to 0)
  return wm1 * t * fast_rcp(fast_log(w));
}

// ln(1 + y) by Kahan's method: with v = fl(1 + y), ln(v) y / (v - 1).
__device__ __forceinline__ float log1p_k(float y) {
  const float v = 1.0f + y;
  if (v == 1.0f) return y;
  return fast_log(v) * y * fast_rcp(v - 1.0f);
}

// Kumaraswamy quantile x = (1 - (1-u)^(1/b))^(1/a), written through base-2
// logs so that no step cancels: with L = log2(1-u) (1-u is exact),
// s = 2^(L/b) = (1-u)^(1/b), g = 1 - s, lam2 = log2 g = a log2 x and
// x = 2^(lam2/a).  g and ln g come from Kahan's two tricks:
//   s >= 1/2:  g = -expm1(t) = (s - 1) log2(s_exact) / -log2(s)   (s - 1 exact),
//              lam2 = log2 g;
//   s <  1/2:  g = fl(1 - s) (no cancellation), lam2 = log2(1 - s) =
//              log2(g) (-s) / (g - 1)                              (g - 1 exact).
// Each case needs g, 1/g (for dx/db) and one more reciprocal; the two
// reciprocals 1/X and 1/Y come from one: R = 1/(XY), 1/X = Y R, 1/Y = X R.
// Six transcendental instructions per coordinate in all.
struct Quantile {
  float x;
  float l2;    // log2(1-u)
  float s;     // (1-u)^(1/b)
  float lam2;  // log2(1-s) = a log2 x
  float rg;    // 1/(1-s)
};

__device__ __forceinline__ Quantile kumaraswamy_v(float v /* = 1 - u, exact */, Shape sh) {
  Quantile q;
  q.l2 = fast_log2(v);
  const float t2 = q.l2 * sh.rb;                 // log2 s
  const float s = fast_exp2(t2);
  q.s = s;
  const bool hi = s >= 0.5f;
  const float gb = 1.0f - s;
  float X, Y;
  if (hi) {
    if (s == 1.0f) {                             // |t| below half an ulp of 1: g = -t
      X = -t2 * kLn2;
      Y = 1.0f;
    } else {
      X = (s - 1.0f) * t2;
      Y = -fast_log2(s);
    }
  } else {
    X = gb;
    Y = fminf(gb - 1.0f, -0x1p-25f);             // g == 1 (s below 2^-25) is handled below
  }
  const float R = fast_rcp(X * Y);
  const float rX = Y * R, rY = X * R;
  const float G = hi ? X * rY : X;
  q.rg = hi ? Y * rX : rX;
  const float LG = fast_log2(G);
  q.lam2 = hi ? LG : (gb == 1.0f ? -s * kLog2e : LG * (-s) * rY);
  q.x = fast_exp2(q.lam2 * sh.ra);
  return q;
}

// The event's quantile from its Philox word.
__device__ __forceinline__ Quantile kumaraswamy_w(uint32_t w, Shape sh) { return kumaraswamy_v(uniform_1mu(w), sh); }

// ln x = lam / a.
__device__ __forceinline__ float log_x(const Quantile& q, Shape sh) { return q.lam2 * sh.ra * kLn2; }

// Pathwise derivatives by the chain rule through the quantile:
//   dx/da = -x lam / a^2                     (>= 0)
//   dx/db = x s l / (a b^2 g)                (<= 0)
// with lam = ln g = lam2 ln 2 and l = ln(1-u) = L ln 2 folded into cda, cdb.
__device__ __forceinline__ void pathwise(const Quantile& q, Shape sh, float& dxda, float& dxdb) {
  dxda = sh.cda * q.x * q.lam2;
  dxdb = sh.cdb * q.x * q.s * q.l2 * q.rg;
}

// ln(1 - e^m) for m < 0 without cancellation (Maechler 2012, "Accurately
// computing log(1 - exp(-|a|))"): ln(-expm1(m)) near 0, log1p(-e^m) below -ln 2.
__device__ __forceinline__ float log1mexp(float m) {
  const float w = fast_exp(m);
  return (m > -kLn2) ? fast_log(-expm1_k(m, w)) : log1p_k(-w);
}

// Wave-wide sum (64 lanes), same order on every call.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace sagips
