// KV cache and one-token decode for the Kraken sub-layers.
//
// Section 2.1 (KV cache): the keys and values every token's attention produced are
// kept, so that a later token attends to them without recomputing them; a decode step
// appends the new token's own.  Each sub-layer of each layer has its own cache (the N
// sub-layers of a Kraken layer are independent Transformer sub-layers, Section 3.1).
//
// Cache layout (one layer): [N][2 (K, V)][max_seqs][Hkv][capacity][hd], elements of the
// MFMA operand type (Hkv key/value heads; grouped-query attention shares each among
// n_heads / Hkv consecutive query heads).  Slot b holds sequence b, position p its p-th
// token.  A head's keys (and values) of one sequence are then contiguous rows of hd
// elements, which the decode attention streams.
//
// Kernels:
//   kv_store_kernel    after a prefill's Q,K and V projections: the K columns of the Q|K
//                      rows and the transposed V (through an LDS tile) into the cache;
//   kv_append_kernel   a decode step's new keys and values at position lens[b];
//   decode_attn_kernel softmax(q K^T / sqrt(hd)) V of one new token per sequence over
//                      its lens[b] + 1 cached keys, split over key chunks (one workgroup
//                      per (sub-layer, sequence, group of query heads sharing a key/value
//                      head, chunk)), fp32 scores, online softmax per wave; writes (max,
//                      sum, unnormalised output) partials per query head;
//   decode_combine_kernel merges a head's chunk partials into the attention output.
#include <math.h>

#include <algorithm>

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
  const void* qk;   // [n][T][d + dkv], K at columns d .. d+dkv-1
  const void* vt;   // [n][dkv][ldv]
  void* cache;      // one layer: [n][2][max_seqs][Hkv][cap][hd]
  int n, T, d, dkv, hd, Hkv, ldv, max_seqs, cap, num_seqs;
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
  const int64_t ld_qk = (int64_t)p.d + p.dkv;
  const S* qk = static_cast<const S*>(p.qk) + (int64_t)i * p.T * ld_qk;
  const S* vt = static_cast<const S*>(p.vt) + (int64_t)i * p.dkv * p.ldv;
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
    const uint4 kch = *reinterpret_cast<const uint4*>(qk + (int64_t)t * ld_qk + p.d + c);
    *reinterpret_cast<uint4*>(cache + cache_index(i, 0, b, h, pos, e, p.max_seqs, p.Hkv, p.cap,
                                                  p.hd)) = kch;
    uint4 vch;
    S* ve = reinterpret_cast<S*>(&vch);
#pragma unroll
    for (int k = 0; k < EPC; ++k) ve[k] = tile[cc * EPC + k][tt];
    *reinterpret_cast<uint4*>(cache + cache_index(i, 1, b, h, pos, e, p.max_seqs, p.Hkv, p.cap,
                                                  p.hd)) = vch;
  }
}

struct KvAppendParams {
  const void* qk;   // [n][B][d + dkv]
  const void* v;    // [n][B][dkv]
  void* cache;
  int n, B, d, dkv, hd, Hkv, max_seqs, cap;
  int lens[KRAKEN_MAX_SEQS];
};

// One thread per 16-byte chunk of a new token's K or V row.
template <typename S>
__global__ __launch_bounds__(256) void kv_append_kernel(KvAppendParams p) {
  constexpr int EPC = 16 / sizeof(S);
  const int per_row = p.dkv / EPC;
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
      ? static_cast<const S*>(p.qk) + ((int64_t)i * p.B + b) * (p.d + p.dkv) + p.d + c
      : static_cast<const S*>(p.v) + ((int64_t)i * p.B + b) * p.dkv + c;
  S* cache = static_cast<S*>(p.cache);
  *reinterpret_cast<uint4*>(cache + cache_index(i, kv, b, h, p.lens[b], e, p.max_seqs, p.Hkv,
                                                p.cap, p.hd)) =
      *reinterpret_cast<const uint4*>(src);
}

struct DecAttnParams {
  const void* qk;   // [n][B][d + dkv], Q at columns 0..d-1
  const void* cache;
  float* part;      // [n][B][H][S][hd + 2]: max, sum, unnormalised output
  int n, B, d, dkv, H, Hkv, group, max_seqs, cap, S, chunk;
  float scale;      // 1 / sqrt(hd); ln 2 when Q already carries log2(e) / sqrt(hd)
  int lens[KRAKEN_MAX_SEQS];   // cached tokens of slot b, new token included at lens[b]
};

template <typename S>
__device__ __forceinline__ float to_f(S v) { return (float)v; }

// Sum (max) over the lanes l ^ o for o = FROM, 2 FROM, .. < 64: lanes of one residue
// class mod FROM.
template <int FROM>
__device__ __forceinline__ float xor_sum_from(float v) {
#pragma unroll
  for (int o = FROM; o < 64; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}
template <int FROM>
__device__ __forceinline__ float xor_max_from(float v) {
#pragma unroll
  for (int o = FROM; o < 64; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
// Lane x of a DPP pattern (a VALU operand modifier: no LDS traffic).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                               CTRL, 0xf, 0xf, false));
}

// Sum over the lanes of one aligned group of UPTO lanes, in every lane of the group.  Up to
// 16 lanes with DPP adds: the quad permutations [1,0,3,2] and [2,3,0,1] pair lanes 1 and 2
// apart, the half-row mirror pairs each lane of a 4-lane quad with one of the other quad,
// and the row mirror each lane of an 8-lane half with one of the other half.
template <int UPTO>
__device__ __forceinline__ float group_sum(float v) {
  if constexpr (UPTO >= 2) v += dpp_f<0xB1>(v);    // quad_perm [1,0,3,2]
  if constexpr (UPTO >= 4) v += dpp_f<0x4E>(v);    // quad_perm [2,3,0,1]
  if constexpr (UPTO >= 8) v += dpp_f<0x141>(v);   // row_half_mirror
  if constexpr (UPTO >= 16) v += dpp_f<0x140>(v);  // row_mirror
  if constexpr (UPTO >= 32) v += __shfl_xor(v, 16, 64);
  if constexpr (UPTO >= 64) v += __shfl_xor(v, 32, 64);
  return v;
}

// Dot product of a 16-byte chunk of a key row with the matching query elements, fp32
// accumulation: v_dot2 on 16-bit pairs (exact products, fp32 sums), fp32 FMAs otherwise.
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
template <typename S>
__device__ __forceinline__ float chunk_dot(uint4 k, uint4 q) {
  if constexpr (__is_same(S, f16)) {
    float a = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, k.x), __builtin_bit_cast(f16x2, q.x), 0.f, false);
    a = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, k.y), __builtin_bit_cast(f16x2, q.y), a, false);
    a = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, k.z), __builtin_bit_cast(f16x2, q.z), a, false);
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, k.w), __builtin_bit_cast(f16x2, q.w), a, false);
  } else if constexpr (__is_same(S, bf16)) {
    float a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, k.x), __builtin_bit_cast(bf16x2, q.x), 0.f, false);
    a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, k.y), __builtin_bit_cast(bf16x2, q.y), a, false);
    a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, k.z), __builtin_bit_cast(bf16x2, q.z), a, false);
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, k.w), __builtin_bit_cast(bf16x2, q.w), a, false);
  } else {
    const float4 kf = __builtin_bit_cast(float4, k), qf = __builtin_bit_cast(float4, q);
    return fmaf(kf.w, qf.w, fmaf(kf.z, qf.z, fmaf(kf.y, qf.y, kf.x * qf.x)));
  }
}

// Workgroup (sub-layer i, sequence b, query heads h0 .. h0+QG-1, chunk s) over keys
// [s*chunk, (s+1)*chunk) of the lens[b] + 1 keys, 4 waves.  The QG query heads share one
// key/value head (grouped-query attention; QG = 1 for multi-head attention), so each key
// and value row is read once for all of them.  A key row of HD elements is read by LPR
// consecutive lanes, one 16-byte chunk each, so that every load instruction of the
// workgroup reads whole consecutive rows.  A piece of PIECE keys is R rows per lane; its
// keys and values are loaded before any arithmetic.  Each wave keeps, per query head, its
// own running max, sum and unnormalised output (online softmax over its rows, in fp32);
// the four waves merge at the end and write each head's chunk partial (max, sum, output).
template <typename S, int HD, int QG>
__global__ __launch_bounds__(256) void decode_attn_kernel(DecAttnParams p) {
  constexpr int EPC = 16 / sizeof(S);          // elements per 16-byte chunk
  constexpr int LPR = HD / EPC;                // lanes per key row
  constexpr int RPW = 64 / LPR;                // rows per wave per pass
  constexpr int RPP = 4 * RPW;                 // rows per workgroup per pass
  constexpr int RMAX = QG >= 4 ? 4 : 8;        // register budget of the row buffers
  constexpr int R = LPR < RMAX ? LPR : RMAX;   // passes per piece
  constexpr int PIECE = RPP * R;
  static_assert(DEC_KEYS % PIECE == 0, "a chunk is a whole number of pieces");
  __shared__ float wm[4][QG], wl[4][QG];
  __shared__ float wo[4][QG][HD];

  int r = blockIdx.x;
  const int s = r % p.S; r /= p.S;
  const int hgroups = p.H / QG;
  const int hg = r % hgroups; r /= hgroups;
  const int b = r % p.B;
  const int i = r / p.B;
  const int h0 = hg * QG, hkv = h0 / p.group;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane % LPR;                    // this lane's chunk of a row
  const int row0 = wave * RPW + lane / LPR;    // this lane's row within a pass
  const int nkeys = p.lens[b] + 1;
  const int k_begin = s * p.chunk, k_end = min(k_begin + p.chunk, nkeys);

  // this lane's chunk of each query, as stored (the scale applies to the fp32 score)
  uint4 q[QG];
#pragma unroll
  for (int g = 0; g < QG; ++g)
    q[g] = *reinterpret_cast<const uint4*>(static_cast<const S*>(p.qk) +
                                           ((int64_t)i * p.B + b) * (p.d + p.dkv) +
                                           (h0 + g) * HD + c * EPC);
  const S* cache = static_cast<const S*>(p.cache);
  const S* Kb = cache + cache_index(i, 0, b, hkv, 0, 0, p.max_seqs, p.Hkv, p.cap, HD) + c * EPC;
  const S* Vb = cache + cache_index(i, 1, b, hkv, 0, 0, p.max_seqs, p.Hkv, p.cap, HD) + c * EPC;

  float m_run[QG], l_run[QG], acc[QG][EPC];
#pragma unroll
  for (int g = 0; g < QG; ++g) {
    m_run[g] = -INFINITY;
    l_run[g] = 0.f;
#pragma unroll
    for (int u = 0; u < EPC; ++u) acc[g][u] = 0.f;
  }

  for (int kb = k_begin; kb < k_end; kb += PIECE) {
    uint4 kr[R], vr[R];
#pragma unroll
    for (int j = 0; j < R; ++j) {
      // rows past the chunk's end read its last row and get probability zero
      const int k = min(kb + j * RPP + row0, k_end - 1);
      kr[j] = *reinterpret_cast<const uint4*>(Kb + (int64_t)k * HD);
    }
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const int k = min(kb + j * RPP + row0, k_end - 1);
      vr[j] = *reinterpret_cast<const uint4*>(Vb + (int64_t)k * HD);
    }
#pragma unroll
    for (int g = 0; g < QG; ++g) {
      float sc[R];
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < R; ++j) {
        // the row's full dot product, in every lane of its group
        const float a = group_sum<LPR>(chunk_dot<S>(kr[j], q[g])) * p.scale;
        sc[j] = kb + j * RPP + row0 < k_end ? a : -INFINITY;
        mx = fmaxf(mx, sc[j]);
      }
      mx = xor_max_from<LPR>(mx);
      const float m_new = fmaxf(m_run[g], mx);
      const float mref = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __expf(m_run[g] - mref);
      float ps = 0.f;
#pragma unroll
      for (int u = 0; u < EPC; ++u) acc[g][u] *= alpha;
#pragma unroll
      for (int j = 0; j < R; ++j) {
        const float pj = __expf(sc[j] - mref);
        ps += pj;
        const S* e = reinterpret_cast<const S*>(&vr[j]);
#pragma unroll
        for (int u = 0; u < EPC; ++u) acc[g][u] = fmaf(pj, to_f(e[u]), acc[g][u]);
      }
      l_run[g] = l_run[g] * alpha + ps;        // this lane's rows (repeated in LPR lanes)
      m_run[g] = m_new;
    }
  }

  // wave totals: lanes of one chunk residue hold disjoint rows
#pragma unroll
  for (int g = 0; g < QG; ++g) {
#pragma unroll
    for (int u = 0; u < EPC; ++u) acc[g][u] = xor_sum_from<LPR>(acc[g][u]);
    l_run[g] = xor_sum_from<LPR>(l_run[g]);
    if (lane < LPR) {
#pragma unroll
      for (int u = 0; u < EPC; ++u) wo[wave][g][lane * EPC + u] = acc[g][u];
    }
    if (lane == 0) {
      wm[wave][g] = m_run[g];
      wl[wave][g] = l_run[g];
    }
  }
  __syncthreads();
#pragma unroll
  for (int g = 0; g < QG; ++g) {
    float* out = p.part + ((((int64_t)i * p.B + b) * p.H + h0 + g) * p.S + s) * (HD + 2);
    const float M = fmaxf(fmaxf(wm[0][g], wm[1][g]), fmaxf(wm[2][g], wm[3][g]));
    float sw[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) sw[w] = M == -INFINITY ? 0.f : __expf(wm[w][g] - M);
    for (int f = tid; f < HD; f += 256)
      out[2 + f] = (wo[0][g][f] * sw[0] + wo[1][g][f] * sw[1]) +
                   (wo[2][g][f] * sw[2] + wo[3][g][f] * sw[3]);
    if (tid == 0) {
      out[0] = M;
      out[1] = (wl[0][g] * sw[0] + wl[1][g] * sw[1]) + (wl[2][g] * sw[2] + wl[3][g] * sw[3]);
    }
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
  dim3 grid((unsigned)((p.T + KV_TILE - 1) / KV_TILE), (unsigned)(p.dkv / KV_TILE),
            (unsigned)p.n);
  hipLaunchKernelGGL(kv_store_kernel<S>, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

template <typename S, int QG>
hipError_t decode_attn_qg(const DecAttnParams& p, int hd, hipStream_t s) {
  dim3 grid((unsigned)((int64_t)p.n * p.B * (p.H / QG) * p.S));
  switch (hd) {
    case 32: hipLaunchKernelGGL((decode_attn_kernel<S, 32, QG>), grid, dim3(256), 0, s, p); break;
    case 64: hipLaunchKernelGGL((decode_attn_kernel<S, 64, QG>), grid, dim3(256), 0, s, p); break;
    case 128: hipLaunchKernelGGL((decode_attn_kernel<S, 128, QG>), grid, dim3(256), 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename S>
hipError_t decode_attn_typed(const DecAttnParams& p, int hd, int qg, hipStream_t s) {
  if (qg == 4) return decode_attn_qg<S, 4>(p, hd, s);
  if (qg == 2) return decode_attn_qg<S, 2>(p, hd, s);
  return decode_attn_qg<S, 1>(p, hd, s);
}

// Query heads one decode-attention workgroup serves: the largest of 4, 2, 1 that divides
// the group of query heads sharing a key/value head.
int heads_per_workgroup(int group) { return group % 4 == 0 ? 4 : group % 2 == 0 ? 2 : 1; }

}  // namespace

hipError_t launch_kv_store(DType dt, const void* qk, const void* vt, void* cache_layer, int n,
                           int T, int d, int n_heads, int n_kv_heads, const int32_t* cu_host,
                           int num_seqs, int max_seqs, int capacity, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const int hd = d / n_heads, kvh = n_kv_heads > 0 ? n_kv_heads : n_heads;
  if ((kvh * hd) % KV_TILE != 0 || n_heads % kvh != 0 || num_seqs <= 0 ||
      num_seqs > KRAKEN_MAX_SEQS)
    return hipErrorInvalidValue;
  KvStoreParams p;
  p.qk = qk; p.vt = vt; p.cache = cache_layer;
  p.n = n; p.T = T; p.d = d; p.dkv = kvh * hd; p.Hkv = kvh; p.hd = hd; p.ldv = vt_ld(T);
  p.max_seqs = max_seqs; p.cap = capacity; p.num_seqs = num_seqs;
  for (int b = 0; b <= num_seqs; ++b) p.cu[b] = cu_host[b];
  switch (dt) {
    case DType::BF16: return kv_store_typed<bf16>(p, s);
    case DType::F16: return kv_store_typed<f16>(p, s);
    default: return kv_store_typed<float>(p, s);
  }
}

hipError_t launch_kv_append(DType dt, const void* qk, const void* v, void* cache_layer, int n,
                            int B, int d, int n_heads, int n_kv_heads, const int32_t* lens_host,
                            int max_seqs, int capacity, hipStream_t s) {
  if (B <= 0 || B > KRAKEN_MAX_SEQS) return hipErrorInvalidValue;
  const int hd = d / n_heads, kvh = n_kv_heads > 0 ? n_kv_heads : n_heads;
  if (n_heads % kvh != 0) return hipErrorInvalidValue;
  KvAppendParams p;
  p.qk = qk; p.v = v; p.cache = cache_layer;
  p.n = n; p.B = B; p.d = d; p.dkv = kvh * hd; p.Hkv = kvh; p.hd = hd;
  p.max_seqs = max_seqs; p.cap = capacity;
  for (int b = 0; b < B; ++b) p.lens[b] = lens_host[b];
  const int epc = 16 / (int)dtype_size(dt);
  const int64_t threads = (int64_t)n * B * 2 * (p.dkv / epc);
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
                                   int d, int n_heads, int n_kv_heads, const int32_t* lens_host,
                                   int max_seqs, int capacity, int q_prescaled, hipStream_t s) {
  if (B <= 0 || B > KRAKEN_MAX_SEQS) return hipErrorInvalidValue;
  const int hd = d / n_heads, kvh = n_kv_heads > 0 ? n_kv_heads : n_heads;
  if (n_heads % kvh != 0) return hipErrorInvalidValue;
  const int group = n_heads / kvh, qg = heads_per_workgroup(group);
  int max_keys = 1;
  for (int b = 0; b < B; ++b) max_keys = max(max_keys, lens_host[b] + 1);
  // Chunks of 256 .. 1536 keys (whole 256-key units) sized for about 384 workgroups: long
  // chunks amortise each workgroup's query loads and final merge.  Measured at N=8, 16
  // query heads of 128, 8192 cached keys: 16 key/value heads, one sequence 1536-key chunks
  // 96 us against 119 us with 256; 4 key/value heads, one sequence 768-key chunks 38 us
  // against 48 us; eight sequences 1536 keys best in both.  The chunk grows further when
  // the partial buffer is too small.
  const int64_t per_split = decode_partial_floats(n, B, n_heads, hd, 1);
  const int64_t max_splits = part_floats / per_split;
  if (max_splits < 1) return hipErrorInvalidValue;
  const int64_t per_chunk_wgs = (int64_t)n * B * (n_heads / qg);
  const int64_t want =
      ((int64_t)max_keys * per_chunk_wgs / 384 + DEC_KEYS - 1) / DEC_KEYS * DEC_KEYS;
  int chunk = (int)std::min<int64_t>(std::max<int64_t>(want, DEC_KEYS), 6 * DEC_KEYS);
  while ((max_keys + chunk - 1) / chunk > max_splits) chunk += DEC_KEYS;
  DecAttnParams p;
  p.qk = qk; p.cache = cache_layer; p.part = part;
  p.n = n; p.B = B; p.d = d; p.dkv = kvh * hd; p.H = n_heads; p.Hkv = kvh; p.group = group;
  p.max_seqs = max_seqs; p.cap = capacity;
  p.chunk = chunk;
  p.S = (max_keys + chunk - 1) / chunk;
  // scores in natural units: a pre-scaled Q's dot products are in log2 units
  p.scale = q_prescaled ? 0.69314718055994531f : (float)(1.0 / sqrt((double)hd));
  for (int b = 0; b < B; ++b) p.lens[b] = lens_host[b];
  hipError_t e;
  switch (dt) {
    case DType::BF16: e = decode_attn_typed<bf16>(p, hd, qg, s); break;
    case DType::F16: e = decode_attn_typed<f16>(p, hd, qg, s); break;
    default: e = decode_attn_typed<float>(p, hd, qg, s); break;
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
