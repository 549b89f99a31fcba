// Bandwidth-bound kernels of the Kraken layer:
//  * LN1: the LayerNorm in front of each sub-layer's attention (Algorithm 1);
//  * combine + LN2: the element-wise sum of the previous layer's N sub-layer
//    outputs (the paper's AllReduce, done on-device; Section 3.1), added to the
//    sub-layer's residual and normalised in front of its FFN (Algorithm 1),
//    in one pass over HBM;
//  * conversions and the one-time weight transpose used at load.
//
// One workgroup owns one token: it reads the token's row of every sub-layer,
// so each HBM byte is touched once.  Rows are read as float4, statistics are
// kept in fp32 with a two-pass (mean, then centred variance) reduction.
#include <algorithm>

#include "kraken_internal.hpp"

namespace kraken {
namespace {

constexpr int NORM_THREADS = 256;
constexpr int MAX_VEC = 16;  // float4 per thread -> d <= 16384

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Sum over the workgroup; every thread gets the result.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();                     // red[] may still be read by a previous call
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < NORM_THREADS / 64; ++w) s += red[w];
  return s;
}

template <typename S>
__device__ __forceinline__ void store4(S* dst, float a, float b, float c, float d);

template <>
__device__ __forceinline__ void store4<float>(float* dst, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(dst) = make_float4(a, b, c, d);
}

template <>
__device__ __forceinline__ void store4<bf16>(bf16* dst, float a, float b, float c, float d) {
  bf16x4 v;
  v[0] = (bf16)a; v[1] = (bf16)b; v[2] = (bf16)c; v[3] = (bf16)d;
  *reinterpret_cast<bf16x4*>(dst) = v;
}

template <>
__device__ __forceinline__ void store4<f16>(f16* dst, float a, float b, float c, float d) {
  f16x4 v;
  v[0] = (f16)a; v[1] = (f16)b; v[2] = (f16)c; v[3] = (f16)d;
  *reinterpret_cast<f16x4*>(dst) = v;
}

// Largest magnitude that rounds to a finite fp16 value: |v| >= 65520 rounds (to nearest
// even) to infinity.
constexpr float F16_OVERFLOW = 65520.0f;

// Normalise v (this thread's float4s of one row, at most V) and write the row to dst.
// Returns the largest output magnitude written (for the fp16 overflow check).
template <typename S, int V>
__device__ __forceinline__ float ln_write(const float4* v, int nv, float mean, float rstd,
                                          const float* gamma, const float* beta, S* dst) {
  const int tid = threadIdx.x;
  float amax = 0.f;
#pragma unroll
  for (int u = 0; u < V; ++u) {
    if (u >= nv) break;
    const int c = (tid + u * NORM_THREADS) * 4;
    const float4 g = *reinterpret_cast<const float4*>(gamma + c);
    const float4 b = *reinterpret_cast<const float4*>(beta + c);
    const float o0 = (v[u].x - mean) * rstd * g.x + b.x, o1 = (v[u].y - mean) * rstd * g.y + b.y;
    const float o2 = (v[u].z - mean) * rstd * g.z + b.z, o3 = (v[u].w - mean) * rstd * g.w + b.w;
    if constexpr (__is_same(S, f16))
      amax = fmaxf(amax, fmaxf(fmaxf(fabsf(o0), fabsf(o1)), fmaxf(fabsf(o2), fabsf(o3))));
    store4(dst + c, o0, o1, o2, o3);
  }
  return amax;
}

// fp16 outputs: one lane of each wave whose outputs overflowed sets *ovf (a vector store).
template <typename S>
__device__ __forceinline__ void flag_overflow(float amax, int* ovf) {
  if constexpr (__is_same(S, f16)) {
    if (ovf && __ballot(!(amax < F16_OVERFLOW)) && (threadIdx.x & 63) == 0) *ovf = 1;
  }
}

// Statistics of a row over its first dl (logical) elements, dl a multiple of 4: a row
// stored with padding columns past dl (a width rounded up for the kernels) keeps them out
// of the mean and the variance.
template <int V>
__device__ __forceinline__ void row_stats(const float4* v, int nv, int dl, float eps,
                                          float* red, float& mean, float& rstd) {
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < V; ++u)
    if (u < nv && (threadIdx.x + u * NORM_THREADS) * 4 < dl)
      s += (v[u].x + v[u].y) + (v[u].z + v[u].w);
  mean = block_sum(s, red) / (float)dl;
  float q = 0.f;
#pragma unroll
  for (int u = 0; u < V; ++u)
    if (u < nv && (threadIdx.x + u * NORM_THREADS) * 4 < dl) {
      const float a = v[u].x - mean, b = v[u].y - mean, c = v[u].z - mean, e = v[u].w - mean;
      q += (a * a + b * b) + (c * c + e * e);
    }
  const float var = block_sum(q, red) / (float)dl;
  rstd = rsqrtf(var + eps);
}

// Float4s per thread a row of d floats needs at most (1, 2, 4, 8 or MAX_VEC): the kernels'
// register arrays are sized by it, so a short row keeps occupancy high.
inline int vecs_for(int d) {
  const int v = (d / 4 + NORM_THREADS - 1) / NORM_THREADS;
  return v <= 1 ? 1 : v <= 2 ? 2 : v <= 4 ? 4 : v <= 8 ? 8 : MAX_VEC;
}

// Number of float4s this thread owns in a row of d floats.
__device__ __forceinline__ int my_vecs(int d) {
  const int nv4 = d / 4;
  const int tid = threadIdx.x;
  return tid < nv4 ? (nv4 - tid + NORM_THREADS - 1) / NORM_THREADS : 0;
}

// V: float4s per thread that the launch's d needs at most (registers are sized by it).
template <typename S, int V>
__global__ __launch_bounds__(NORM_THREADS) void layernorm_kernel(
    const float* __restrict__ x, int64_t xs, const float* __restrict__ gamma,
    const float* __restrict__ beta, S* __restrict__ out, int n, int T, int d, int dl, float eps,
    int* __restrict__ ovf) {
  __shared__ float red[NORM_THREADS / 64];
  const int t = blockIdx.x;
  const int nv = my_vecs(d);
  float amax = 0.f;
  // sub-layers [i0, i1) of this block (gridDim.y blocks share the n sub-layers)
  const int i0 = (int)((int64_t)n * blockIdx.y / gridDim.y);
  const int i1 = (int)((int64_t)n * (blockIdx.y + 1) / gridDim.y);
  float4 v[V];
  float mean = 0.f, rstd = 0.f;
  for (int i = i0; i < i1; ++i) {
    if (i == i0 || xs != 0) {
      const float* row = x + i * xs + (int64_t)t * d;
#pragma unroll
      for (int u = 0; u < V; ++u)
        if (u < nv) v[u] = *reinterpret_cast<const float4*>(row + (threadIdx.x + u * NORM_THREADS) * 4);
      row_stats<V>(v, nv, dl, eps, red, mean, rstd);
    }
    amax = fmaxf(amax, ln_write<S, V>(v, nv, mean, rstd, gamma + (int64_t)i * d,
                                      beta + (int64_t)i * d, out + ((int64_t)i * T + t) * d));
  }
  flag_overflow<S>(amax, ovf);
}

template <typename S, int V>
__global__ __launch_bounds__(NORM_THREADS) void combine_ln2_kernel(
    const float* __restrict__ x, const float* __restrict__ shared, const float* __restrict__ h,
    const float* __restrict__ gamma, const float* __restrict__ beta, S* __restrict__ out, int n,
    int T, int d, int dl, float eps, int* __restrict__ ovf) {
  __shared__ float red[NORM_THREADS / 64];
  float amax = 0.f;
  const int t = blockIdx.x;
  const int nv = my_vecs(d);
  const int64_t plane = (int64_t)T * d;
  float4 y[V];
  // y = X (first layer) or the N-way sum of the previous layer's outputs
#pragma unroll
  for (int u = 0; u < V; ++u) {
    if (u >= nv) break;
    const int c = (threadIdx.x + u * NORM_THREADS) * 4;
    if (shared) {
      y[u] = *reinterpret_cast<const float4*>(shared + (int64_t)t * d + c);
    } else {
      float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int k = 0; k < n; ++k) {
        const float4 b = *reinterpret_cast<const float4*>(x + k * plane + (int64_t)t * d + c);
        a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
      }
      y[u] = a;
    }
  }
  const int i0 = (int)((int64_t)n * blockIdx.y / gridDim.y);
  const int i1 = (int)((int64_t)n * (blockIdx.y + 1) / gridDim.y);
  for (int i = i0; i < i1; ++i) {
    float4 v[V];
    const float* hrow = h + i * plane + (int64_t)t * d;
#pragma unroll
    for (int u = 0; u < V; ++u) {
      if (u >= nv) break;
      const float4 a = *reinterpret_cast<const float4*>(hrow + (threadIdx.x + u * NORM_THREADS) * 4);
      v[u] = make_float4(a.x + y[u].x, a.y + y[u].y, a.z + y[u].z, a.w + y[u].w);
    }
    float mean, rstd;
    row_stats<V>(v, nv, dl, eps, red, mean, rstd);
    amax = fmaxf(amax, ln_write<S, V>(v, nv, mean, rstd, gamma + (int64_t)i * d,
                                      beta + (int64_t)i * d, out + (i * plane + (int64_t)t * d)));
  }
  flag_overflow<S>(amax, ovf);
}

template <typename S>
__global__ void to_f32_kernel(const S* __restrict__ src, float* __restrict__ dst, int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < count; k += stride)
    dst[k] = (float)src[k];
}

template <typename S>
__global__ void scale_kernel(S* __restrict__ p, int64_t count, float c) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < count; k += stride)
    p[k] = (S)((float)p[k] * c);
}

template <typename S>
__global__ void split16_kernel(const float* __restrict__ src, S* __restrict__ dst, int64_t count,
                               int* __restrict__ ovf) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  float amax = 0.f;
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < count; k += stride) {
    const float v = src[k];
    const S hi = (S)v;
    dst[k] = hi;
    dst[k + count] = (S)(v - (float)hi);
    amax = fmaxf(amax, fabsf(v));
  }
  flag_overflow<S>(amax, ovf);
}

// Index of logical element x in a padded layout: x's group of g elements (a head of hd
// features, or a sub-layer's d features) starts at (x / g) * gp.  g = gp: the identity.
__device__ __forceinline__ int64_t pad_index(int64_t x, int g, int gp) {
  return g == gp ? x : (x / g) * gp + x % g;
}

template <typename Src, typename Dst>
__global__ __launch_bounds__(256) void transpose_kernel(const Src* __restrict__ src, int64_t sld,
                                                        Dst* __restrict__ dst, int64_t dld, int R,
                                                        int C, int* __restrict__ overflow,
                                                        int gr, int grp, int gc, int gcp) {
  __shared__ float tile[64][65];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int k = ty; k < 64; k += 4) {
    const int r = r0 + k, c = c0 + tx;
    if (r < R && c < C) tile[k][tx] = (float)src[(int64_t)r * sld + c];
  }
  __syncthreads();
  bool over = false;
  for (int k = ty; k < 64; k += 4) {
    const int c = c0 + k, r = r0 + tx;
    if (r < R && c < C) {
      const float v = tile[tx][k];
      const Dst o = (Dst)v;
      if constexpr (__is_same(Dst, f16)) over |= (__builtin_isinf((float)o) && !__builtin_isinf(v));
      dst[pad_index(c, gc, gcp) * dld + pad_index(r, gr, grp)] = o;
    }
  }
  if (over && overflow) *overflow = 1;
}

// dst[r * dld + pad_index(c)] = float(src[r * sld + c]) for r < R, c < C.
template <typename S>
__global__ void to_f32_2d_kernel(const S* __restrict__ src, int64_t sld, float* __restrict__ dst,
                                 int64_t dld, int R, int C, int g, int gp) {
  const int64_t total = (int64_t)R * C;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < total; k += stride) {
    const int64_t r = k / C, c = k % C;
    dst[r * dld + pad_index(c, g, gp)] = (float)src[r * sld + c];
  }
}

// dst[r * dld + c] = Dst(src[r * sld + c]) for r < R, c < C (rows converted in place, no
// transpose); a finite value that overflows an fp16 destination sets *overflow.
template <typename Src, typename Dst>
__global__ void convert_2d_kernel(const Src* __restrict__ src, int64_t sld, Dst* __restrict__ dst,
                                  int64_t dld, int R, int C, int* __restrict__ overflow) {
  const int64_t total = (int64_t)R * C;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  bool over = false;
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < total; k += stride) {
    const int64_t r = k / C, c = k % C;
    const float v = (float)src[r * sld + c];
    const Dst o = (Dst)v;
    if constexpr (__is_same(Dst, f16)) over |= (__builtin_isinf((float)o) && !__builtin_isinf(v));
    dst[r * dld + c] = o;
  }
  if (over && overflow) *overflow = 1;
}

// First-layer input of a token sequence: X[t] = tok[ids[t]] + pos[pos_ids[t]] over the
// (padded) row width dp.  Token rows in the MFMA operand type (the table the tied
// unembedding multiplies), position rows in fp32.  ids[] were checked against the table
// size on the host.
template <typename S>
__global__ __launch_bounds__(256) void embed_kernel(const int* __restrict__ ids,
                                                    const int* __restrict__ pos_ids,
                                                    const S* __restrict__ tok,
                                                    const float* __restrict__ pos,
                                                    float* __restrict__ X, int dp) {
  const int t = blockIdx.x;
  const S* trow = tok + (int64_t)ids[t] * dp;
  const float* prow = pos + (int64_t)pos_ids[t] * dp;
  float* xrow = X + (int64_t)t * dp;
  for (int c = threadIdx.x; c < dp; c += 256) xrow[c] = (float)trow[c] + prow[c];
}

// dst[b] = src[rows[b]] (fp32 rows of width dp).
__global__ __launch_bounds__(256) void gather_rows_kernel(const float* __restrict__ src,
                                                          const int* __restrict__ rows,
                                                          float* __restrict__ dst, int dp) {
  const int b = blockIdx.x;
  const float4* srow = reinterpret_cast<const float4*>(src + (int64_t)rows[b] * dp);
  float4* drow = reinterpret_cast<float4*>(dst + (int64_t)b * dp);
  for (int c = threadIdx.x; c < dp / 4; c += 256) drow[c] = srow[c];
}

template <typename S>
__global__ void zero_cols_kernel(S* __restrict__ base, int64_t rows, int64_t ld, int c0, int w) {
  const int64_t total = rows * w;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < total; k += stride)
    base[(k / w) * ld + c0 + (k % w)] = S(0.f);
}

unsigned grid_for(int64_t count) {
  int64_t b = (count + 255) / 256;
  if (b > 65536) b = 65536;
  if (b < 1) b = 1;
  return (unsigned)b;
}

template <class Fn>
hipError_t by_type(DType dt, Fn&& fn) {
  switch (dt) {
    case DType::BF16: return fn(bf16{});
    case DType::F16: return fn(f16{});
    case DType::F32: return fn(float{});
  }
  return hipErrorInvalidValue;
}

// Blocks per token row: one block loops over all n sub-layers when there are enough
// rows to fill the chip (the shared-input statistics and the N-way sum are then computed
// once per row); few rows (a decode step) spread the sub-layers over up to n blocks.
unsigned sub_groups(int n, int T) {
  if (T >= 512) return 1;
  return (unsigned)std::min(n, (512 + T - 1) / T);
}

}  // namespace

hipError_t launch_layernorm(DType dt, const float* x, int64_t xs, const float* gamma,
                            const float* beta, void* out, int n, int T, int d, int dl, float eps,
                            int* ovf, hipStream_t s) {
  if (T <= 0 || n <= 0) return hipSuccess;
  if (d % 4 != 0 || d > NORM_THREADS * MAX_VEC * 4 || dl % 4 != 0 || dl < 4 || dl > d)
    return hipErrorInvalidValue;
  return by_type(dt, [&](auto tag) {
    using S = decltype(tag);
    // one workgroup per (token, sub-layer) row when the rows differ (more rows in flight);
    // a shared input row keeps its statistics in one workgroup per token
    const dim3 grid(T, xs != 0 ? (unsigned)n : sub_groups(n, T)), block(NORM_THREADS);
    S* o = static_cast<S*>(out);
    switch (vecs_for(d)) {
      case 1: hipLaunchKernelGGL((layernorm_kernel<S, 1>), grid, block, 0, s, x, xs, gamma, beta, o, n, T, d, dl, eps, ovf); break;
      case 2: hipLaunchKernelGGL((layernorm_kernel<S, 2>), grid, block, 0, s, x, xs, gamma, beta, o, n, T, d, dl, eps, ovf); break;
      case 4: hipLaunchKernelGGL((layernorm_kernel<S, 4>), grid, block, 0, s, x, xs, gamma, beta, o, n, T, d, dl, eps, ovf); break;
      case 8: hipLaunchKernelGGL((layernorm_kernel<S, 8>), grid, block, 0, s, x, xs, gamma, beta, o, n, T, d, dl, eps, ovf); break;
      default: hipLaunchKernelGGL((layernorm_kernel<S, MAX_VEC>), grid, block, 0, s, x, xs, gamma, beta, o, n, T, d, dl, eps, ovf); break;
    }
    return hipGetLastError();
  });
}

hipError_t launch_combine_ln2(DType dt, const float* x, const float* shared, const float* h,
                              const float* gamma, const float* beta, void* out, int n, int T,
                              int d, int dl, float eps, int* ovf, hipStream_t s) {
  if (T <= 0 || n <= 0) return hipSuccess;
  if (d % 4 != 0 || d > NORM_THREADS * MAX_VEC * 4 || dl % 4 != 0 || dl < 4 || dl > d)
    return hipErrorInvalidValue;
  return by_type(dt, [&](auto tag) {
    using S = decltype(tag);
    const dim3 grid(T, sub_groups(n, T)), block(NORM_THREADS);
    S* o = static_cast<S*>(out);
    switch (vecs_for(d)) {
      case 1: hipLaunchKernelGGL((combine_ln2_kernel<S, 1>), grid, block, 0, s, x, shared, h, gamma, beta, o, n, T, d, dl, eps, ovf); break;
      case 2: hipLaunchKernelGGL((combine_ln2_kernel<S, 2>), grid, block, 0, s, x, shared, h, gamma, beta, o, n, T, d, dl, eps, ovf); break;
      case 4: hipLaunchKernelGGL((combine_ln2_kernel<S, 4>), grid, block, 0, s, x, shared, h, gamma, beta, o, n, T, d, dl, eps, ovf); break;
      case 8: hipLaunchKernelGGL((combine_ln2_kernel<S, 8>), grid, block, 0, s, x, shared, h, gamma, beta, o, n, T, d, dl, eps, ovf); break;
      default: hipLaunchKernelGGL((combine_ln2_kernel<S, MAX_VEC>), grid, block, 0, s, x, shared, h, gamma, beta, o, n, T, d, dl, eps, ovf); break;
    }
    return hipGetLastError();
  });
}

hipError_t launch_scale(DType dt, void* p, int64_t count, float c, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  return by_type(dt, [&](auto tag) {
    using S = decltype(tag);
    hipLaunchKernelGGL(scale_kernel<S>, dim3(grid_for(count)), dim3(256), 0, s,
                       static_cast<S*>(p), count, c);
    return hipGetLastError();
  });
}

hipError_t launch_to_f32(DType dt, const void* src, float* dst, int64_t count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  return by_type(dt, [&](auto tag) {
    using S = decltype(tag);
    hipLaunchKernelGGL(to_f32_kernel<S>, dim3(grid_for(count)), dim3(256), 0, s,
                       static_cast<const S*>(src), dst, count);
    return hipGetLastError();
  });
}

hipError_t launch_zero_cols(DType dt, void* base, int64_t rows, int64_t ld, int c0, int c1,
                            hipStream_t s) {
  if (rows <= 0 || c1 <= c0) return hipSuccess;
  const int w = c1 - c0;
  return by_type(dt, [&](auto tag) {
    using S = decltype(tag);
    hipLaunchKernelGGL(zero_cols_kernel<S>, dim3(grid_for(rows * w)), dim3(256), 0, s,
                       static_cast<S*>(base), rows, ld, c0, w);
    return hipGetLastError();
  });
}

hipError_t launch_split16(DType dt, const float* src, void* dst, int64_t count, int* ovf,
                          hipStream_t s) {
  if (count <= 0) return hipSuccess;
  if (dt == DType::BF16)
    hipLaunchKernelGGL(split16_kernel<bf16>, dim3(grid_for(count)), dim3(256), 0, s, src,
                       static_cast<bf16*>(dst), count, ovf);
  else if (dt == DType::F16)
    hipLaunchKernelGGL(split16_kernel<f16>, dim3(grid_for(count)), dim3(256), 0, s, src,
                       static_cast<f16*>(dst), count, ovf);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_transpose(DType src_t, const void* src, int64_t src_ld, DType dst_t, void* dst,
                            int64_t dst_ld, int R, int C, int* overflow, hipStream_t s,
                            int gr, int grp, int gc, int gcp) {
  if (R <= 0 || C <= 0) return hipSuccess;
  if (gr < 1 || grp < gr || gc < 1 || gcp < gc) return hipErrorInvalidValue;
  dim3 grid((C + 63) / 64, (R + 63) / 64), block(256);
  return by_type(src_t, [&](auto stag) {
    using Src = decltype(stag);
    return by_type(dst_t, [&](auto dtag) {
      using Dst = decltype(dtag);
      hipLaunchKernelGGL((transpose_kernel<Src, Dst>), grid, block, 0, s,
                         static_cast<const Src*>(src), src_ld, static_cast<Dst*>(dst), dst_ld, R,
                         C, overflow, gr, grp, gc, gcp);
      return hipGetLastError();
    });
  });
}

hipError_t launch_to_f32_2d(DType st, const void* src, int64_t src_ld, float* dst,
                            int64_t dst_ld, int R, int C, int g, int gp, hipStream_t s) {
  if (R <= 0 || C <= 0) return hipSuccess;
  if (g < 1 || gp < g) return hipErrorInvalidValue;
  return by_type(st, [&](auto tag) {
    using S = decltype(tag);
    hipLaunchKernelGGL(to_f32_2d_kernel<S>, dim3(grid_for((int64_t)R * C)), dim3(256), 0, s,
                       static_cast<const S*>(src), src_ld, dst, dst_ld, R, C, g, gp);
    return hipGetLastError();
  });
}

hipError_t launch_embed(DType dt, const int* ids, const int* pos_ids, const void* tok,
                        const float* pos, float* X, int T, int dp, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  return by_type(dt, [&](auto tag) {
    using S = decltype(tag);
    hipLaunchKernelGGL(embed_kernel<S>, dim3(T), dim3(256), 0, s, ids, pos_ids,
                       static_cast<const S*>(tok), pos, X, dp);
    return hipGetLastError();
  });
}

hipError_t launch_gather_rows(const float* src, const int* rows, float* dst, int B, int dp,
                              hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if (dp % 4 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gather_rows_kernel, dim3(B), dim3(256), 0, s, src, rows, dst, dp);
  return hipGetLastError();
}

hipError_t launch_convert_2d(DType src_t, const void* src, int64_t src_ld, DType dst_t, void* dst,
                             int64_t dst_ld, int R, int C, int* overflow, hipStream_t s) {
  if (R <= 0 || C <= 0) return hipSuccess;
  return by_type(src_t, [&](auto stag) {
    using Src = decltype(stag);
    return by_type(dst_t, [&](auto dtag) {
      using Dst = decltype(dtag);
      hipLaunchKernelGGL((convert_2d_kernel<Src, Dst>), dim3(grid_for((int64_t)R * C)), dim3(256),
                         0, s, static_cast<const Src*>(src), src_ld, static_cast<Dst*>(dst),
                         dst_ld, R, C, overflow);
      return hipGetLastError();
    });
  });
}

}  // namespace kraken
