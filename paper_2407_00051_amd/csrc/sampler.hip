// Event sampler and per-parameter gradient reduction on gfx950.
//
// Both kernels run on a 2D grid: blockIdx.y is the parameter row (so theta
// and its reciprocals are wave-uniform scalars) and blockIdx.x a chunk of
// kEPB consecutive events of that row.  Thread t of a chunk handles events
// chunk*kEPB + t + j*256, j < kEPT, so every store is coalesced.
#include "device_math.hpp"
#include "kernels.hpp"

#include <algorithm>

namespace sagips {
namespace {

constexpr int kThreads = 256;
constexpr int kEPT = 8;
constexpr int kEPB = kThreads * kEPT;

template <int D>
__global__ __launch_bounds__(kThreads) void k_sample(SourceArgs s, float* __restrict__ x,
                                                     uint32_t* __restrict__ words) {
  const int row = blockIdx.y;
  Shape sh[D];
#pragma unroll
  for (int j = 0; j < D; ++j) sh[j] = make_shape(s.theta[row * 2 * D + 2 * j], s.theta[row * 2 * D + 2 * j + 1]);
  const int64_t k_first = (int64_t)blockIdx.x * kEPB + threadIdx.x;
  const int64_t row_base = (int64_t)row * s.E;
#pragma unroll 2
  for (int e = 0; e < kEPT; ++e) {
    const int64_t k = k_first + e * kThreads;
    if (k >= s.E) break;
    const int64_t i = row_base + k;
    const Words w = event_words(s.base + (uint64_t)i, s.stream, s.k0, s.k1);
    if (words) {
      uint4 v;
      v.x = w.w[0]; v.y = w.w[1]; v.z = w.w[2]; v.w = w.w[3];
      reinterpret_cast<uint4*>(words)[i] = v;
    }
    if (x) {
      float xv[D];
#pragma unroll
      for (int j = 0; j < D; ++j) xv[j] = kumaraswamy_w(w.w[j], sh[j]).x;
      if constexpr (D == 2) {
        reinterpret_cast<float2*>(x)[i] = make_float2(xv[0], xv[1]);
      } else {
#pragma unroll
        for (int j = 0; j < D; ++j) x[i * D + j] = xv[j];
      }
    }
  }
}

// Per-chunk partial sums of dL/dtheta (2D values) and, for the quadratic
// critic, of the loss: partial[(row * chunks + chunk) * (2D+1) + c].
template <int D, bool kQuadratic>
__global__ __launch_bounds__(kThreads) void k_param_grad(SourceArgs s, const float* __restrict__ dLdx,
                                                         float* __restrict__ partial) {
  constexpr int C = 2 * D + 1;
  __shared__ float red[kThreads / 64][C];
  const int row = blockIdx.y;
  Shape sh[D];
#pragma unroll
  for (int j = 0; j < D; ++j) sh[j] = make_shape(s.theta[row * 2 * D + 2 * j], s.theta[row * 2 * D + 2 * j + 1]);
  float acc[C];
#pragma unroll
  for (int c = 0; c < C; ++c) acc[c] = 0.0f;
  const int64_t k_first = (int64_t)blockIdx.x * kEPB + threadIdx.x;
  const int64_t row_base = (int64_t)row * s.E;
#pragma unroll 2
  for (int e = 0; e < kEPT; ++e) {
    const int64_t k = k_first + e * kThreads;
    if (k >= s.E) break;
    const int64_t i = row_base + k;
    const Words w = event_words(s.base + (uint64_t)i, s.stream, s.k0, s.k1);
    float gx[D];
    if constexpr (!kQuadratic) {
      if constexpr (D == 2) {
        const float2 v = reinterpret_cast<const float2*>(dLdx)[i];
        gx[0] = v.x; gx[1] = v.y;
      } else {
#pragma unroll
        for (int j = 0; j < D; ++j) gx[j] = dLdx[i * D + j];
      }
    }
#pragma unroll
    for (int j = 0; j < D; ++j) {
      const Quantile q = kumaraswamy_w(w.w[j], sh[j]);
      float da, db;
      pathwise(q, sh[j], da, db);
      float g;
      if constexpr (kQuadratic) {
        const float r = q.x - 0.5f;
        g = 2.0f * r;
        acc[2 * D] = fmaf(r, r, acc[2 * D]);
      } else {
        g = gx[j];
      }
      acc[2 * j] = fmaf(g, da, acc[2 * j]);
      acc[2 * j + 1] = fmaf(g, db, acc[2 * j + 1]);
    }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const float v = wave_sum(acc[c]);
    if (lane == 0) red[wave][c] = v;
  }
  __syncthreads();
  if (threadIdx.x < C) {
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) v += red[w][threadIdx.x];
    partial[((int64_t)row * gridDim.x + blockIdx.x) * C + threadIdx.x] = v;
  }
}

// One block per row: fixed-order sum of the row's chunk partials.
__global__ __launch_bounds__(kThreads) void k_reduce_rows(const float* __restrict__ partial, int chunks, int C,
                                                          float* __restrict__ dLdtheta, float* __restrict__ row_loss,
                                                          int has_loss) {
  __shared__ float red[kThreads / 64];
  const int row = blockIdx.x;
  const float* p = partial + (int64_t)row * chunks * C;
  for (int c = 0; c < C; ++c) {
    if (c == C - 1 && !has_loss) break;
    float v = 0.0f;
    for (int k = threadIdx.x; k < chunks; k += kThreads) v += p[(int64_t)k * C + c];
    v = wave_sum(v);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
      float t = 0.0f;
      for (int w = 0; w < kThreads / 64; ++w) t += red[w];
      if (c < C - 1) dLdtheta[row * (C - 1) + c] = t;
      else row_loss[row] = t;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(kThreads) void k_reduce_loss(const float* __restrict__ row_loss, int n,
                                                          float* __restrict__ loss) {
  __shared__ float red[kThreads / 64];
  float v = 0.0f;
  for (int k = threadIdx.x; k < n; k += kThreads) v += row_loss[k];
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.0f;
    for (int w = 0; w < kThreads / 64; ++w) t += red[w];
    *loss = t;
  }
}

inline int chunks_per_row(const SourceArgs& s) { return (int)((s.E + kEPB - 1) / kEPB); }

// Bootstrap draws, one per thread (grid-stride): draw i takes row
// floor(w0 * n_data / 2^32), w0 the first Philox word of counter
// (i lo, i hi, stream, step).  The rows are gathered (8 or 12 bytes each) and
// written back contiguously.
template <int D>
__global__ __launch_bounds__(kThreads) void k_bootstrap(const float* __restrict__ data, uint64_t n_data, uint32_t k0,
                                                        uint32_t k1, uint32_t step, int64_t n_out,
                                                        float* __restrict__ out, int64_t* __restrict__ idx_out) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n_out; i += stride) {
    const Words w = philox4x32_10((uint32_t)i, (uint32_t)((uint64_t)i >> 32), SAGIPS_STREAM_BOOTSTRAP, step, k0, k1);
    const uint64_t r = ((uint64_t)w.w[0] * n_data) >> 32;    // < n_data <= 2^32: the product fits in 64 bits
    if (idx_out) idx_out[i] = (int64_t)r;
    if constexpr (D == 2) {
      reinterpret_cast<float2*>(out)[i] = reinterpret_cast<const float2*>(data)[r];
    } else {
#pragma unroll
      for (int j = 0; j < D; ++j) out[i * D + j] = data[r * D + j];
    }
  }
}

// The same draws listed in ascending row order, by a counting sort over
// slabs of 2^kSlabBits consecutive rows of the reference data:
//   k_boot_count    each chunk of draws: its rows (kept for the scatter) and a
//                   per-slab count, [slab][chunk]
//   k_boot_scan     per slab, the exclusive scan of its chunk counts, and the
//                   slab's total
//   k_boot_base     the exclusive scan of the slab totals (one workgroup)
//   k_boot_scatter  each draw's row offset within its slab (16 bits) into the
//                   slab's segment, at the chunk's place
//   k_boot_expand   per slab: a histogram of the offsets in LDS, its scan, then
//                   output position p takes row upper_bound(scan, p) - 1 of the
//                   slab; rows are read nearly in order and written in order.
// Placement within a (slab, chunk) segment follows LDS atomics, but the final
// output is the unique ascending listing of the drawn rows.
constexpr int kSlabBits = 14;
constexpr int kSlabRows = 1 << kSlabBits;
constexpr int kBootBig = 1024;     // threads of the count, scatter and expand kernels

__global__ __launch_bounds__(kBootBig) void k_boot_count(uint64_t n_data, uint32_t k0, uint32_t k1, uint32_t step,
                                                         int64_t n_out, int64_t per_chunk, int n_slabs, int n_chunks,
                                                         uint32_t* __restrict__ rows, uint32_t* __restrict__ cnt) {
  extern __shared__ uint32_t hist[];   // [n_slabs]
  for (int s = threadIdx.x; s < n_slabs; s += kBootBig) hist[s] = 0u;
  __syncthreads();
  const int64_t i0 = (int64_t)blockIdx.x * per_chunk, i1 = min(n_out, i0 + per_chunk);
  for (int64_t i = i0 + threadIdx.x; i < i1; i += kBootBig) {
    const Words w = philox4x32_10((uint32_t)i, (uint32_t)((uint64_t)i >> 32), SAGIPS_STREAM_BOOTSTRAP, step, k0, k1);
    const uint32_t r = (uint32_t)(((uint64_t)w.w[0] * n_data) >> 32);
    rows[i] = r;
    atomicAdd(&hist[r >> kSlabBits], 1u);
  }
  __syncthreads();
  for (int s = threadIdx.x; s < n_slabs; s += kBootBig) cnt[(int64_t)s * n_chunks + blockIdx.x] = hist[s];
}

// One wave per slab: exclusive scan of cnt[slab][0 .. n_chunks) in place, and
// the slab's total.
__global__ __launch_bounds__(64) void k_boot_scan(uint32_t* __restrict__ cnt, int n_chunks,
                                                  uint32_t* __restrict__ total) {
  uint32_t* c = cnt + (int64_t)blockIdx.x * n_chunks;
  const int lane = threadIdx.x;
  uint32_t carry = 0u;
  for (int b = 0; b < n_chunks; b += 64) {
    const int j = b + lane;
    const uint32_t v = j < n_chunks ? c[j] : 0u;
    uint32_t incl = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t t = __shfl_up(incl, o, 64);
      if (lane >= o) incl += t;
    }
    if (j < n_chunks) c[j] = carry + incl - v;
    carry += __shfl(incl, 63, 64);
  }
  if (lane == 0) total[blockIdx.x] = carry;
}

// One workgroup: base[s] = sum of total[0 .. s), base[n_slabs] = n_out.
__global__ __launch_bounds__(kBootBig) void k_boot_base(const uint32_t* __restrict__ total, int n_slabs,
                                                        uint32_t* __restrict__ base) {
  __shared__ uint32_t part[kBootBig];
  const int t = threadIdx.x;
  const int per = (n_slabs + kBootBig - 1) / kBootBig;
  uint32_t s = 0u;
  for (int j = 0; j < per; ++j) {
    const int q = t * per + j;
    if (q < n_slabs) s += total[q];
  }
  part[t] = s;
  __syncthreads();
  for (int o = 1; o < kBootBig; o <<= 1) {     // inclusive scan of the thread sums (Hillis-Steele)
    const uint32_t v = t >= o ? part[t - o] : 0u;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  uint32_t run = t > 0 ? part[t - 1] : 0u;
  for (int j = 0; j < per; ++j) {
    const int q = t * per + j;
    if (q < n_slabs) {
      base[q] = run;
      run += total[q];
    }
  }
  if (t == kBootBig - 1) base[n_slabs] = part[kBootBig - 1];
}

__global__ __launch_bounds__(kBootBig) void k_boot_scatter(const uint32_t* __restrict__ rows, int64_t n_out,
                                                           int64_t per_chunk, int n_slabs, int n_chunks,
                                                           const uint32_t* __restrict__ cnt,
                                                           const uint32_t* __restrict__ base, uint16_t* __restrict__ keys) {
  extern __shared__ uint32_t cursor[];   // [n_slabs]
  for (int s = threadIdx.x; s < n_slabs; s += kBootBig) cursor[s] = base[s] + cnt[(int64_t)s * n_chunks + blockIdx.x];
  __syncthreads();
  const int64_t i0 = (int64_t)blockIdx.x * per_chunk, i1 = min(n_out, i0 + per_chunk);
  for (int64_t i = i0 + threadIdx.x; i < i1; i += kBootBig) {
    const uint32_t r = rows[i];
    const uint32_t pos = atomicAdd(&cursor[r >> kSlabBits], 1u);
    keys[pos] = (uint16_t)(r & (kSlabRows - 1));
  }
}

template <int D>
__global__ __launch_bounds__(kBootBig) void k_boot_expand(const float* __restrict__ data, const uint16_t* __restrict__ keys,
                                                          const uint32_t* __restrict__ base, float* __restrict__ out,
                                                          int64_t* __restrict__ idx_out) {
  __shared__ uint32_t h[kSlabRows];
  __shared__ uint32_t part[kBootBig];
  constexpr int PER = kSlabRows / kBootBig;   // 16 histogram entries per thread
  const int t = threadIdx.x;
  const uint32_t b0 = base[blockIdx.x], b1 = base[blockIdx.x + 1];
  for (int j = t; j < kSlabRows; j += kBootBig) h[j] = 0u;
  __syncthreads();
  for (uint32_t p = b0 + t; p < b1; p += kBootBig) atomicAdd(&h[keys[p]], 1u);
  __syncthreads();
  // exclusive scan of h: each thread its 16 entries, then the thread sums
  uint32_t loc[PER];
  uint32_t s = 0u;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    loc[j] = s;
    s += h[t * PER + j];
  }
  part[t] = s;
  __syncthreads();
  for (int o = 1; o < kBootBig; o <<= 1) {
    const uint32_t v = t >= o ? part[t - o] : 0u;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  const uint32_t off = t > 0 ? part[t - 1] : 0u;
#pragma unroll
  for (int j = 0; j < PER; ++j) h[t * PER + j] = off + loc[j];
  __syncthreads();
  // output q of the slab takes the last row j with h[j] <= q (rows drawn zero
  // times share their start with the next row and are passed over)
  const uint64_t row0 = (uint64_t)blockIdx.x << kSlabBits;
  for (uint32_t p = b0 + t; p < b1; p += kBootBig) {
    const uint32_t q = p - b0;
    int lo = 0, n = kSlabRows;                 // upper_bound over h[0 .. kSlabRows)
    while (n > 0) {
      const int half = n >> 1;
      if (h[lo + half] <= q) {
        lo += half + 1;
        n -= half + 1;
      } else {
        n = half;
      }
    }
    const uint64_t r = row0 + (uint64_t)(lo - 1);
    if (idx_out) idx_out[p] = (int64_t)r;
#pragma unroll
    for (int j = 0; j < D; ++j) out[(int64_t)p * D + j] = data[r * D + j];
  }
}

}  // namespace

hipError_t launch_bootstrap(const float* data, uint64_t n_data, int d, uint32_t k0, uint32_t k1, uint32_t step,
                            int64_t n_out, float* out, int64_t* idx_out, int n_cu, hipStream_t st, Timer* tm) {
  const int64_t want = (n_out + kThreads - 1) / kThreads;
  const int blocks = (int)std::min<int64_t>(want, (int64_t)n_cu * 32);
  if (tm) tm->begin("bootstrap");
  if (d == 2) hipLaunchKernelGGL(k_bootstrap<2>, dim3(blocks), dim3(kThreads), 0, st, data, n_data, k0, k1, step, n_out, out, idx_out);
  else hipLaunchKernelGGL(k_bootstrap<3>, dim3(blocks), dim3(kThreads), 0, st, data, n_data, k0, k1, step, n_out, out, idx_out);
  if (tm) tm->end();
  return hipGetLastError();
}

size_t bootstrap_rows_workspace(uint64_t n_data, int64_t n_out, int* n_slabs_out, int* n_chunks_out,
                                int64_t* per_chunk_out) {
  const int n_slabs = (int)((n_data + kSlabRows - 1) / kSlabRows);
  int n_chunks = (int)std::min<int64_t>(256, std::max<int64_t>(1, (n_out + 16383) / 16384));
  const int64_t per_chunk = (n_out + n_chunks - 1) / n_chunks;
  if (n_slabs_out) *n_slabs_out = n_slabs;
  if (n_chunks_out) *n_chunks_out = n_chunks;
  if (per_chunk_out) *per_chunk_out = per_chunk;
  auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
  return al(4 * (size_t)n_out) + al(2 * (size_t)n_out) + al(4 * (size_t)n_slabs * n_chunks) + al(4 * (size_t)n_slabs) +
         al(4 * ((size_t)n_slabs + 1));
}

hipError_t launch_bootstrap_rows(const float* data, uint64_t n_data, int d, uint32_t k0, uint32_t k1, uint32_t step,
                                 int64_t n_out, float* out, int64_t* idx_out, void* ws, hipStream_t st, Timer* tm) {
  int n_slabs, n_chunks;
  int64_t per_chunk;
  bootstrap_rows_workspace(n_data, n_out, &n_slabs, &n_chunks, &per_chunk);
  auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
  char* w = static_cast<char*>(ws);
  uint32_t* rows = reinterpret_cast<uint32_t*>(w);
  w += al(4 * (size_t)n_out);
  uint16_t* keys = reinterpret_cast<uint16_t*>(w);
  w += al(2 * (size_t)n_out);
  uint32_t* cnt = reinterpret_cast<uint32_t*>(w);
  w += al(4 * (size_t)n_slabs * n_chunks);
  uint32_t* total = reinterpret_cast<uint32_t*>(w);
  w += al(4 * (size_t)n_slabs);
  uint32_t* base = reinterpret_cast<uint32_t*>(w);
  const size_t lds = sizeof(uint32_t) * (size_t)n_slabs;
  if (tm) tm->begin("bootstrap_rows");
  hipLaunchKernelGGL(k_boot_count, dim3(n_chunks), dim3(kBootBig), lds, st, n_data, k0, k1, step, n_out, per_chunk,
                     n_slabs, n_chunks, rows, cnt);
  hipLaunchKernelGGL(k_boot_scan, dim3(n_slabs), dim3(64), 0, st, cnt, n_chunks, total);
  hipLaunchKernelGGL(k_boot_base, dim3(1), dim3(kBootBig), 0, st, total, n_slabs, base);
  hipLaunchKernelGGL(k_boot_scatter, dim3(n_chunks), dim3(kBootBig), lds, st, rows, n_out, per_chunk, n_slabs, n_chunks,
                     cnt, base, keys);
  if (d == 2) hipLaunchKernelGGL(k_boot_expand<2>, dim3(n_slabs), dim3(kBootBig), 0, st, data, keys, base, out, idx_out);
  else hipLaunchKernelGGL(k_boot_expand<3>, dim3(n_slabs), dim3(kBootBig), 0, st, data, keys, base, out, idx_out);
  if (tm) tm->end();
  return hipGetLastError();
}

hipError_t launch_sample(const SourceArgs& s, float* x, uint32_t* words, hipStream_t st, Timer* tm) {
  const dim3 grid(chunks_per_row(s), s.n_theta);
  if (tm) tm->begin("sample_events");
  if (s.d == 2) hipLaunchKernelGGL(k_sample<2>, grid, dim3(kThreads), 0, st, s, x, words);
  else hipLaunchKernelGGL(k_sample<3>, grid, dim3(kThreads), 0, st, s, x, words);
  if (tm) tm->end();
  return hipGetLastError();
}

size_t param_grad_workspace(const SourceArgs& s) {
  const size_t C = 2 * s.d + 1;
  return ((size_t)s.n_theta * chunks_per_row(s) * C + s.n_theta) * sizeof(float);
}

hipError_t launch_param_grad(const SourceArgs& s, const float* dLdx, float* dLdtheta, float* loss, void* ws,
                             hipStream_t st, Timer* tm) {
  const int chunks = chunks_per_row(s);
  const int C = 2 * s.d + 1;
  float* partial = static_cast<float*>(ws);
  float* row_loss = partial + (size_t)s.n_theta * chunks * C;
  const dim3 grid(chunks, s.n_theta);
  const bool quad = (dLdx == nullptr);
  if (tm) tm->begin("param_grad");
  if (s.d == 2) {
    if (quad) hipLaunchKernelGGL((k_param_grad<2, true>), grid, dim3(kThreads), 0, st, s, dLdx, partial);
    else hipLaunchKernelGGL((k_param_grad<2, false>), grid, dim3(kThreads), 0, st, s, dLdx, partial);
  } else {
    if (quad) hipLaunchKernelGGL((k_param_grad<3, true>), grid, dim3(kThreads), 0, st, s, dLdx, partial);
    else hipLaunchKernelGGL((k_param_grad<3, false>), grid, dim3(kThreads), 0, st, s, dLdx, partial);
  }
  if (tm) tm->end();
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (tm) tm->begin("param_grad_reduce");
  hipLaunchKernelGGL(k_reduce_rows, dim3(s.n_theta), dim3(kThreads), 0, st, partial, chunks, C, dLdtheta, row_loss,
                     quad ? 1 : 0);
  if (quad && loss) hipLaunchKernelGGL(k_reduce_loss, dim3(1), dim3(kThreads), 0, st, row_loss, s.n_theta, loss);
  if (tm) tm->end();
  return hipGetLastError();
}

}  // namespace sagips
