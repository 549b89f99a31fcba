// KV cache and one-token decode for the Kraken sub-layers.
//
// Section 2.1 (KV cache): the keys and values every token's attention produced are
// kept, so that a later token attends to them without recomputing them; a decode step
// appends the new token's own.  Each sub-layer of each layer has its own cache (the N
// sub-layers of a Kraken layer are independent Transformer sub-layers, Section 3.1).
//
// Cache layout (one layer): [N][2 (K, V)][max_seqs][H][capacity][hd], elements of the
// MFMA operand type; slot b holds sequence b, position p its p-th token.  A head's keys
// (and values) of one sequence are then contiguous rows of hd elements, which the decode
// attention streams.
//
// Kernels:
//   kv_store_kernel    after a prefill's Q,K and V projections: the K half of the Q|K
//                      rows and the transposed V (through an LDS tile) into the cache;
//   kv_append_kernel   a decode step's new keys and values at position lens[b];
//   decode_attn_kernel softmax(q K^T / sqrt(hd)) V of one new token per sequence over
//                      its lens[b] + 1 cached keys, split over key chunks (one workgroup
//                      per (sub-layer, sequence, head, chunk)), fp32 scores, online
//                      softmax across the chunk's 256-key pieces; writes (max, sum,
//                      unnormalised output) partials;
//   decode_combine_kernel merges a head's chunk partials into the attention output.
#include <math.h>

#include "kraken_internal.hpp"
#include "../../include/kraken.h"

namespace kraken {
namespace {

constexpr int KV_TILE = 64;       // tokens x features of one kv_store tile
constexpr int DEC_KEYS = 256;     // keys per piece of a decode-attention chunk

// Sequence of packed token t (largest b with cu[b] <= t).
__device__ __forceinline__ int seq_of(const int* cu, int num_seqs, int t) {
  int lo = 0, hi = num_seqs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

struct KvStoreParams {
  const void* qk;   // [n][T][2d], K half at columns d..2d-1
  const void* vt;   // [n][d][ldv]
  void* cache;      // one layer: [n][2][max_seqs][H][cap][hd]
  int n, T, d, hd, H, ldv, max_seqs, cap, num_seqs;
  int cu[KRAKEN_MAX_SEQS + 1];
};

// Element (i, kv, b, h, pos, e) of one layer's cache.
__device__ __forceinline__ int64_t cache_index(int i, int kv, int b, int h, int pos, int e,
                                               int max_seqs, int H, int cap, int hd) {
  return (((((int64_t)i * 2 + kv) * max_seqs + b) * H + h) * (int64_t)cap + pos) * hd + e;
}

// Block (token tile, feature tile, sub-layer); 256 threads.  K: each thread copies 16-byte
// chunks of its tokens' K rows.  V: the [feature][token] tile of V^T is staged in LDS and
// written back as token rows.
template <typename S>
__global__ __launch_bounds__(256) void kv_store_kernel(KvStoreParams p) {
  constexpr int EPC = 16 / sizeof(S);                  // elements per 16-byte chunk
  constexpr int CPR = KV_TILE / EPC;                   // chunks per 64-element row
  __shared__ S tile[KV_TILE][KV_TILE + EPC];           // [feature][token], padded rows
  const int i = blockIdx.z, t0 = blockIdx.x * KV_TILE, c0 = blockIdx.y * KV_TILE;
  const int tid = threadIdx.x;
  const S* qk = static_cast<const S*>(p.qk) + (int64_t)i * p.T * 2 * p.d;
  const S* vt = static_cast<const S*>(p.vt) + (int64_t)i * p.d * p.ldv;
  S* cache = static_cast<S*>(p.cache);
  // V^T rows c0 .. c0+63, tokens t0 .. t0+63 (the padded columns up to ldv are readable)
  for (int q = tid; q < KV_TILE * CPR; q += 256) {
    const int r = q / CPR, cc = q % CPR;
    const int t = t0 + cc * EPC;
    if (t < p.ldv) {
      const uint4 v = *reinterpret_cast<const uint4*>(vt + (int64_t)(c0 + r) * p.ldv + t);
      const S* e = reinterpret_cast<const S*>(&v);
#pragma unroll
      for (int k = 0; k < EPC; ++k) tile[r][cc * EPC + k] = e[k];
    }
  }
  __syncthreads();
  // token rows: chunk cc of features c0 + cc*EPC .. +EPC-1 (inside one head: hd % EPC == 0)
  for (int q = tid; q < KV_TILE * CPR; q += 256) {
    const int tt = q / CPR, cc = q % CPR;
    const int t = t0 + tt;
    if (t >= p.T) continue;
    const int b = seq_of(p.cu, p.num_seqs, t);
    const int pos = t - p.cu[b];
    const int c = c0 + cc * EPC;
    const int h = c / p.hd, e = c % p.hd;
    const uint4 kch = *reinterpret_cast<const uint4*>(qk + (int64_t)t * 2 * p.d + p.d + c);
    *reinterpret_cast<uint4*>(cache + cache_index(i, 0, b, h, pos, e, p.max_seqs, p.H, p.cap,
                                                  p.hd)) = kch;
    uint4 vch;
    S* ve = reinterpret_cast<S*>(&vch);
#pragma unroll
    for (int k = 0; k < EPC; ++k) ve[k] = tile[cc * EPC + k][tt];
    *reinterpret_cast<uint4*>(cache + cache_index(i, 1, b, h, pos, e, p.max_seqs, p.H, p.cap,
                                                  p.hd)) = vch;
  }
}

struct KvAppendParams {
  const void* qk;   // [n][B][2d]
  const void* v;    // [n][B][d]
  void* cache;
  int n, B, d, hd, H, max_seqs, cap;
  int lens[KRAKEN_MAX_SEQS];
};

// One thread per 16-byte chunk of a new token's K or V row.
template <typename S>
__global__ __launch_bounds__(256) void kv_append_kernel(KvAppendParams p) {
  constexpr int EPC = 16 / sizeof(S);
  const int per_row = p.d / EPC;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)p.n * p.B * 2 * per_row) return;
  const int cc = (int)(idx % per_row);
  int64_t r = idx / per_row;
  const int kv = (int)(r % 2);
  r /= 2;
  const int b = (int)(r % p.B);
  const int i = (int)(r / p.B);
  const int c = cc * EPC, h = c / p.hd, e = c % p.hd;
  const S* src = kv == 0
      ? static_cast<const S*>(p.qk) + ((int64_t)i * p.B + b) * 2 * p.d + p.d + c
      : static_cast<const S*>(p.v) + ((int64_t)i * p.B + b) * p.d + c;
  S* cache = static_cast<S*>(p.cache);
  *reinterpret_cast<uint4*>(cache + cache_index(i, kv, b, h, p.lens[b], e, p.max_seqs, p.H,
                                                p.cap, p.hd)) =
      *reinterpret_cast<const uint4*>(src);
}

struct DecAttnParams {
  const void* qk;   // [n][B][2d], Q half at columns 0..d-1
  const void* cache;
  float* part;      // [n][B][H][S][hd + 2]: max, sum, unnormalised output
  int n, B, d, H, max_seqs, cap, S, chunk;
  float scale;      // 1 / sqrt(hd)
  int lens[KRAKEN_MAX_SEQS];   // cached tokens of slot b, new token included at lens[b]
};

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <typename S>
__device__ __forceinline__ float to_f(S v) { return (float)v; }

// Workgroup (sub-layer i, sequence b, head h, chunk s) over keys [s*chunk, (s+1)*chunk)
// of the lens[b] + 1 keys.  Scores: thread t takes key kb + t of a 256-key piece (a dot
// product over its key row in 16-byte loads, the query from LDS).  Values: thread t
// accumulates two output features over every G-th key of the piece (G = 256 / (hd/2)),
// so that each value row is read as one contiguous segment by the group.
template <typename S, int HD>
__global__ __launch_bounds__(256) void decode_attn_kernel(DecAttnParams p) {
  constexpr int EPC = 16 / sizeof(S);
  constexpr int TPG = HD / 2;                 // threads per key group (two features each)
  constexpr int G = 256 / TPG;                // key groups
  __shared__ float qs[HD];
  __shared__ float pw[DEC_KEYS];
  __shared__ float red[2][4];
  __shared__ float2 osum[G][TPG];
  int r = blockIdx.x;
  const int s = r % p.S; r /= p.S;
  const int h = r % p.H; r /= p.H;
  const int b = r % p.B;
  const int i = r / p.B;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nkeys = p.lens[b] + 1;
  const int k_begin = s * p.chunk, k_end = min(k_begin + p.chunk, nkeys);

  const S* q = static_cast<const S*>(p.qk) + ((int64_t)i * p.B + b) * 2 * p.d + h * HD;
  if (tid < HD) qs[tid] = to_f(q[tid]) * p.scale;
  const S* cache = static_cast<const S*>(p.cache);
  const S* Kb = cache + cache_index(i, 0, b, h, 0, 0, p.max_seqs, p.H, p.cap, HD);
  const S* Vb = cache + cache_index(i, 1, b, h, 0, 0, p.max_seqs, p.H, p.cap, HD);
  __syncthreads();

  float m_run = -INFINITY, l_run = 0.f, o0 = 0.f, o1 = 0.f;
  const int g = tid / TPG, f = 2 * (tid % TPG);
  for (int kb = k_begin; kb < k_end; kb += DEC_KEYS) {
    const int k = kb + tid;
    float sv = -INFINITY;
    if (k < k_end) {
      const S* krow = Kb + (int64_t)k * HD;
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < HD; c += EPC) {
        const uint4 ch = *reinterpret_cast<const uint4*>(krow + c);
        const S* e = reinterpret_cast<const S*>(&ch);
#pragma unroll
        for (int u = 0; u < EPC; ++u) acc = fmaf(to_f(e[u]), qs[c + u], acc);
      }
      sv = acc;
    }
    // piece maximum and the running rescale (block-uniform values)
    float mx = wave_max(sv);
    if (lane == 0) red[0][wave] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = m_run == -INFINITY ? 0.f : __expf(m_run - m_new);
    const float pv = k < k_end ? __expf(sv - m_new) : 0.f;
    pw[tid] = pv;
    float ps = wave_sum(pv);
    if (lane == 0) red[1][wave] = ps;
    __syncthreads();
    ps = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
    l_run = l_run * alpha + ps;
    o0 *= alpha;
    o1 *= alpha;
    m_run = m_new;
    const int nk = min(DEC_KEYS, k_end - kb);
    for (int kk = g; kk < nk; kk += G) {
      const float w = pw[kk];
      const S* vrow = Vb + (int64_t)(kb + kk) * HD + f;
      o0 = fmaf(w, to_f(vrow[0]), o0);
      o1 = fmaf(w, to_f(vrow[1]), o1);
    }
    __syncthreads();    // pw and red are rewritten by the next piece
  }
  osum[g][tid % TPG] = make_float2(o0, o1);
  __syncthreads();
  float* out = p.part + ((((int64_t)i * p.B + b) * p.H + h) * p.S + s) * (HD + 2);
  if (tid < TPG) {
    float a0 = 0.f, a1 = 0.f;
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
      a0 += osum[gg][tid].x;
      a1 += osum[gg][tid].y;
    }
    out[2 + 2 * tid] = a0;
    out[3 + 2 * tid] = a1;
  }
  if (tid == 0) {
    out[0] = m_run;
    out[1] = l_run;
  }
}

struct DecCombineParams {
  const float* part;
  void* out;        // [n][B][d]
  int n, B, d, H, hd, S;
};

// Block (sub-layer, sequence, head), one thread per output feature: the chunk partials
// (m_s, l_s, o_s) merge as o = sum_s o_s e^(m_s - M) / sum_s l_s e^(m_s - M), M = max m_s.
template <typename S>
__global__ __launch_bounds__(128) void decode_combine_kernel(DecCombineParams p) {
  int r = blockIdx.x;
  const int h = r % p.H; r /= p.H;
  const int b = r % p.B;
  const int i = r / p.B;
  const float* part = p.part + (((int64_t)i * p.B + b) * p.H + h) * p.S * (p.hd + 2);
  const int t = threadIdx.x;
  if (t >= p.hd) return;
  float M = -INFINITY;
  for (int s = 0; s < p.S; ++s) M = fmaxf(M, part[s * (p.hd + 2)]);
  float L = 0.f, O = 0.f;
  for (int s = 0; s < p.S; ++s) {
    const float ms = part[s * (p.hd + 2)];
    if (ms == -INFINITY) continue;               // a chunk past the sequence's keys
    const float w = __expf(ms - M);
    L += part[s * (p.hd + 2) + 1] * w;
    O += part[s * (p.hd + 2) + 2 + t] * w;
  }
  static_cast<S*>(p.out)[((int64_t)i * p.B + b) * p.d + h * p.hd + t] = (S)(O / L);
}

template <typename S>
hipError_t kv_store_typed(const KvStoreParams& p, hipStream_t s) {
  dim3 grid((unsigned)((p.T + KV_TILE - 1) / KV_TILE), (unsigned)(p.d / KV_TILE), (unsigned)p.n);
  hipLaunchKernelGGL(kv_store_kernel<S>, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

template <typename S>
hipError_t decode_attn_typed(const DecAttnParams& p, int hd, hipStream_t s) {
  dim3 grid((unsigned)((int64_t)p.n * p.B * p.H * p.S));
  switch (hd) {
    case 32: hipLaunchKernelGGL((decode_attn_kernel<S, 32>), grid, dim3(256), 0, s, p); break;
    case 64: hipLaunchKernelGGL((decode_attn_kernel<S, 64>), grid, dim3(256), 0, s, p); break;
    case 128: hipLaunchKernelGGL((decode_attn_kernel<S, 128>), grid, dim3(256), 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_kv_store(DType dt, const void* qk, const void* vt, void* cache_layer, int n,
                           int T, int d, int n_heads, const int32_t* cu_host, int num_seqs,
                           int max_seqs, int capacity, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (d % KV_TILE != 0 || num_seqs <= 0 || num_seqs > KRAKEN_MAX_SEQS) return hipErrorInvalidValue;
  KvStoreParams p;
  p.qk = qk; p.vt = vt; p.cache = cache_layer;
  p.n = n; p.T = T; p.d = d; p.H = n_heads; p.hd = d / n_heads; p.ldv = vt_ld(T);
  p.max_seqs = max_seqs; p.cap = capacity; p.num_seqs = num_seqs;
  for (int b = 0; b <= num_seqs; ++b) p.cu[b] = cu_host[b];
  switch (dt) {
    case DType::BF16: return kv_store_typed<bf16>(p, s);
    case DType::F16: return kv_store_typed<f16>(p, s);
    default: return kv_store_typed<float>(p, s);
  }
}

hipError_t launch_kv_append(DType dt, const void* qk, const void* v, void* cache_layer, int n,
                            int B, int d, int n_heads, const int32_t* lens_host, int max_seqs,
                            int capacity, hipStream_t s) {
  if (B <= 0 || B > KRAKEN_MAX_SEQS) return hipErrorInvalidValue;
  KvAppendParams p;
  p.qk = qk; p.v = v; p.cache = cache_layer;
  p.n = n; p.B = B; p.d = d; p.H = n_heads; p.hd = d / n_heads;
  p.max_seqs = max_seqs; p.cap = capacity;
  for (int b = 0; b < B; ++b) p.lens[b] = lens_host[b];
  const int epc = 16 / (int)dtype_size(dt);
  const int64_t threads = (int64_t)n * B * 2 * (d / epc);
  dim3 grid((unsigned)((threads + 255) / 256));
  switch (dt) {
    case DType::BF16: hipLaunchKernelGGL(kv_append_kernel<bf16>, grid, dim3(256), 0, s, p); break;
    case DType::F16: hipLaunchKernelGGL(kv_append_kernel<f16>, grid, dim3(256), 0, s, p); break;
    default: hipLaunchKernelGGL(kv_append_kernel<float>, grid, dim3(256), 0, s, p); break;
  }
  return hipGetLastError();
}

int64_t decode_partial_floats(int n, int B, int n_heads, int hd, int splits) {
  return (int64_t)n * B * n_heads * splits * (hd + 2);
}

hipError_t launch_decode_attention(DType dt, const void* qk, const void* cache_layer,
                                   float* part, int64_t part_floats, void* out, int n, int B,
                                   int d, int n_heads, const int32_t* lens_host, int max_seqs,
                                   int capacity, hipStream_t s) {
  if (B <= 0 || B > KRAKEN_MAX_SEQS) return hipErrorInvalidValue;
  const int hd = d / n_heads;
  int max_keys = 1;
  for (int b = 0; b < B; ++b) max_keys = max(max_keys, lens_host[b] + 1);
  // splits of the key range: as many 256-key chunks as the partial buffer holds, and the
  // chunk grows (in whole 256-key pieces) when it cannot hold one per piece
  const int64_t per_split = decode_partial_floats(n, B, n_heads, hd, 1);
  const int64_t max_splits = part_floats / per_split;
  if (max_splits < 1) return hipErrorInvalidValue;
  int chunk = DEC_KEYS;
  while ((max_keys + chunk - 1) / chunk > max_splits) chunk += DEC_KEYS;
  DecAttnParams p;
  p.qk = qk; p.cache = cache_layer; p.part = part;
  p.n = n; p.B = B; p.d = d; p.H = n_heads; p.max_seqs = max_seqs; p.cap = capacity;
  p.chunk = chunk;
  p.S = (max_keys + chunk - 1) / chunk;
  p.scale = (float)(1.0 / sqrt((double)hd));
  for (int b = 0; b < B; ++b) p.lens[b] = lens_host[b];
  hipError_t e;
  switch (dt) {
    case DType::BF16: e = decode_attn_typed<bf16>(p, hd, s); break;
    case DType::F16: e = decode_attn_typed<f16>(p, hd, s); break;
    default: e = decode_attn_typed<float>(p, hd, s); break;
  }
  if (e != hipSuccess) return e;
  DecCombineParams c;
  c.part = part; c.out = out; c.n = n; c.B = B; c.d = d; c.H = n_heads; c.hd = hd; c.S = p.S;
  dim3 grid((unsigned)((int64_t)n * B * n_heads));
  switch (dt) {
    case DType::BF16: hipLaunchKernelGGL(decode_combine_kernel<bf16>, grid, dim3(128), 0, s, c); break;
    case DType::F16: hipLaunchKernelGGL(decode_combine_kernel<f16>, grid, dim3(128), 0, s, c); break;
    default: hipLaunchKernelGGL(decode_combine_kernel<float>, grid, dim3(128), 0, s, c); break;
  }
  return hipGetLastError();
}

}  // namespace kraken
