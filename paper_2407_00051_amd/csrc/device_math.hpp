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
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
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
  float ra;  // 1/a
  float rb;  // 1/b
};

__device__ __forceinline__ Shape make_shape(float a, float b) {
  Shape s;
  s.ra = 1.0f / a;
  s.rb = 1.0f / b;
  return s;
}

// Elementary functions on the hardware transcendental units (v_log_f32 = log2,
// v_exp_f32 = 2^x, v_rcp_f32; each within 1 ulp over the ranges used here).
constexpr float kLn2 = 0.693147180559945309f;
constexpr float kLog2e = 1.442695040888963407f;

__device__ __forceinline__ float fast_log(float x) { return __builtin_amdgcn_logf(x) * kLn2; }
__device__ __forceinline__ float fast_exp(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

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

// Kumaraswamy quantile x = (1 - (1-u)^(1/b))^(1/a), written through logs so
// that no step cancels: with l = ln(1-u) (1-u is exact), t = l/b,
// s = e^t = (1-u)^(1/b), g = 1 - s = -expm1(t) and lam = ln g, x = e^(lam/a).
// ln g is taken as log1p(-s) while s < 1/2, where g is close to 1.
struct Quantile {
  float x;
  float l;    // ln(1-u)
  float s;    // (1-u)^(1/b)
  float g;    // 1 - s
  float lam;  // ln g = a ln x
};

__device__ __forceinline__ Quantile kumaraswamy_v(float v /* = 1 - u, exact */, Shape sh) {
  Quantile q;
  q.l = fast_log(v);
  const float t = q.l * sh.rb;
  q.s = fast_exp(t);
  q.g = -expm1_k(t, q.s);
  q.lam = (q.s < 0.5f) ? log1p_k(-q.s) : fast_log(q.g);
  q.x = fast_exp(q.lam * sh.ra);
  return q;
}

__device__ __forceinline__ Quantile kumaraswamy(float u, Shape sh) { return kumaraswamy_v(1.0f - u, sh); }

// Pathwise derivatives by the chain rule through the quantile:
//   dx/da = -x lam / a^2                     (>= 0)
//   dx/db = x s l / (a b^2 g)                (<= 0)
__device__ __forceinline__ void pathwise(const Quantile& q, Shape sh, float& dxda, float& dxdb) {
  dxda = -q.x * q.lam * (sh.ra * sh.ra);
  dxdb = q.x * q.s * q.l * (sh.ra * sh.rb * sh.rb) * fast_rcp(q.g);
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
