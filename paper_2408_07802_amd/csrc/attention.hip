// Causal flash attention for the Kraken sub-layers (Section 2.1: per head,
// softmax(Q K^T / sqrt(hd)) V; causal; packed sequences never attend across
// each other).  All N sub-layers and all heads of a layer run in one launch.
//
// Layout: qk [n][T][2d] holds Q then K per token (head h at columns h*hd of
// each half); vt [n][d][ldv] holds V transposed (feature-major), written that
// way by the V projection so that V^T tiles are contiguous rows.
//
// Formulation (one wave = 32 queries): the wave computes the score tile
// transposed, S^T = K Q^T, with 32x32 MFMA blocks.  In the MFMA result layout
// a lane then owns one query (one column) and half of the keys, so the running
// max / sum of the online softmax are per-lane values; only the max is
// exchanged once per tile with the partner lane (lane ^ 32).  The output is
// accumulated transposed, O^T = V^T P^T, whose columns are again the lane's
// query, so the rescale by exp(m_old - m_new) is lane-local too.  P^T goes from
// the S^T accumulator registers straight into the B operand of the second MFMA:
// the k-order of that operand is a permutation of the keys, and the V^T
// operand is read from LDS in the same permuted order.
//
// Workgroup: 4 waves = 128 queries of one (sub-layer, head, sequence); K and
// V^T tiles of 64 keys are staged in a double-buffered LDS ring shared by the
// four waves.  Tiles are ordered heaviest (longest causal prefix) first.
#include "kraken_internal.hpp"
#include "../../include/kraken.h"

namespace kraken {
namespace {

constexpr int BQ = 128;   // queries per workgroup
constexpr int BKV = 64;   // keys per tile
constexpr int ATT_THREADS = 256;

struct AttnParams {
  const void* qk;
  const void* vt;
  void* out;
  int T, d, n_heads, ldv, num_seqs;
  float scale_log2;       // log2(e) / sqrt(hd)
  int cu[KRAKEN_MAX_SEQS + 1];
  int tile_prefix[KRAKEN_MAX_SEQS + 1];
};

template <typename S>
__device__ __forceinline__ void store_out4(S* dst, float a, float b, float c, float e);

template <>
__device__ __forceinline__ void store_out4<bf16>(bf16* dst, float a, float b, float c, float e) {
  bf16x4 v;
  v[0] = (bf16)a; v[1] = (bf16)b; v[2] = (bf16)c; v[3] = (bf16)e;
  *reinterpret_cast<bf16x4*>(dst) = v;
}

template <>
__device__ __forceinline__ void store_out4<f16>(f16* dst, float a, float b, float c, float e) {
  f16x4 v;
  v[0] = (f16)a; v[1] = (f16)b; v[2] = (f16)c; v[3] = (f16)e;
  *reinterpret_cast<f16x4*>(dst) = v;
}

template <>
__device__ __forceinline__ void store_out4<float>(float* dst, float a, float b, float c, float e) {
  *reinterpret_cast<float4*>(dst) = make_float4(a, b, c, e);
}

template <typename S, int HD>
__global__ __launch_bounds__(ATT_THREADS) void attn_kernel(AttnParams p) {
  constexpr int ES = sizeof(S);
  constexpr int CHK = HD * ES / 16;           // 16-byte chunks per K row
  constexpr int KSW = (CHK < 8 ? CHK : 8) - 1;  // swizzle mask for K rows
  constexpr int VROWB = BKV * ES;             // bytes per V^T row (64 keys)
  constexpr int VCH = VROWB / 16;             // 16-byte chunks per V^T row
  constexpr int NQC = HD * ES / 32;           // chunk pairs per head row
  constexpr int OB = HD / 32;                 // 32-row blocks of O^T
  constexpr int KLOAD = BKV * CHK / ATT_THREADS;
  constexpr int VLOAD = HD * VCH / ATT_THREADS;
  constexpr int KBYTES = BKV * HD * ES;
  static_assert(KLOAD >= 1 && VLOAD >= 1, "tile too small for the workgroup");

  __shared__ __attribute__((aligned(16))) unsigned char smem[2][2 * KBYTES];

  // ---- which (sub-layer, head, sequence, query tile)
  const int i = blockIdx.x / p.n_heads;
  const int h = blockIdx.x - i * p.n_heads;
  const int rank = blockIdx.y;
  int lo = 0, hi = p.num_seqs - 1;           // last b with tile_prefix[b] <= rank
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.tile_prefix[mid] <= rank) lo = mid; else hi = mid - 1;
  }
  const int b = lo;
  const int ntiles_b = p.tile_prefix[b + 1] - p.tile_prefix[b];
  const int qt = ntiles_b - 1 - (rank - p.tile_prefix[b]);
  const int seq_start = p.cu[b], seq_end = p.cu[b + 1];
  const int q0 = seq_start + qt * BQ;
  const int q_hi = min(q0 + BQ, seq_end);
  const int kv_begin = seq_start & ~7;       // 16-byte aligned V^T rows

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int wq0 = q0 + wave * 32;
  const int wq_last = min(wq0 + 31, q_hi - 1);
  const int my_q = wq0 + lrow;

  const int64_t ld_qk = 2 * (int64_t)p.d;
  const S* qkz = static_cast<const S*>(p.qk) + (int64_t)i * p.T * ld_qk;
  const S* Kbase = qkz + p.d + h * HD;
  const S* Vbase = static_cast<const S*>(p.vt) + ((int64_t)i * p.d + h * HD) * p.ldv;

  // ---- Q fragments (B operand of S^T = K Q^T): lane's query, chunk 2*kc + lhalf
  uint4 qf[NQC];
  {
    const S* qrow = qkz + (int64_t)my_q * ld_qk + h * HD;
#pragma unroll
    for (int kc = 0; kc < NQC; ++kc)
      qf[kc] = (my_q < q_hi) ? *reinterpret_cast<const uint4*>(qrow + (2 * kc + lhalf) * (16 / ES))
                             : make_uint4(0, 0, 0, 0);
  }

  // ---- global -> register -> LDS staging of one K tile and one V^T tile
  uint4 rk[KLOAD], rv[VLOAD];
  auto gload = [&](int kt0) {
#pragma unroll
    for (int u = 0; u < KLOAD; ++u) {
      const int q = tid + u * ATT_THREADS, row = q / CHK, ch = q % CHK;
      const int key = kt0 + row;
      rk[u] = (key < q_hi) ? *reinterpret_cast<const uint4*>(Kbase + (int64_t)key * ld_qk + ch * (16 / ES))
                           : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < VLOAD; ++u) {
      const int q = tid + u * ATT_THREADS, row = q / VCH, ch = q % VCH;
      const int key = kt0 + ch * (16 / ES);
      const S* src = Vbase + (int64_t)row * p.ldv + key;
      if (key + 16 / ES <= q_hi) {
        rv[u] = *reinterpret_cast<const uint4*>(src);
      } else {
        S tmp[16 / ES];
#pragma unroll
        for (int e = 0; e < 16 / ES; ++e) tmp[e] = (key + e < q_hi) ? src[e] : S(0.f);
        rv[u] = __builtin_bit_cast(uint4, tmp);
      }
    }
  };
  auto lstore = [&](int buf) {
    uint4* Ks = reinterpret_cast<uint4*>(smem[buf]);
    unsigned char* Vs = smem[buf] + KBYTES;
#pragma unroll
    for (int u = 0; u < KLOAD; ++u) {
      const int q = tid + u * ATT_THREADS, row = q / CHK, ch = q % CHK;
      Ks[row * CHK + (ch ^ (row & KSW))] = rk[u];
    }
#pragma unroll
    for (int u = 0; u < VLOAD; ++u) {
      const int q = tid + u * ATT_THREADS, row = q / VCH, ch = q % VCH;
      if constexpr (ES == 2) {
        // 8-byte units, unit index XOR (row & 15)
        uint2* V8 = reinterpret_cast<uint2*>(Vs + row * VROWB);
        const int u0 = 2 * ch, sw = row & 15;
        V8[u0 ^ sw] = make_uint2(rv[u].x, rv[u].y);
        V8[(u0 + 1) ^ sw] = make_uint2(rv[u].z, rv[u].w);
      } else {
        uint4* V16 = reinterpret_cast<uint4*>(Vs + row * VROWB);
        V16[ch ^ (row & 7)] = rv[u];
      }
    }
  };

  f32x16 oacc[OB];
#pragma unroll
  for (int ob = 0; ob < OB; ++ob)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[ob][r] = 0.f;
  float m_run = -1e30f, l_run = 0.f;

  const int n_tiles = (q_hi - kv_begin + BKV - 1) / BKV;
  gload(kv_begin);
  lstore(0);
  __syncthreads();

  for (int it = 0; it < n_tiles; ++it) {
    const int buf = it & 1;
    const int kt0 = kv_begin + it * BKV;
    if (it + 1 < n_tiles) gload(kt0 + BKV);

    if (wq0 < q_hi && kt0 <= wq_last) {
      const uint4* Ks = reinterpret_cast<const uint4*>(smem[buf]);
      const unsigned char* Vs = smem[buf] + KBYTES;
      // S^T for keys [kt0, kt0+64): two 32x32 blocks
      f32x16 st[2];
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) st[sb][r] = 0.f;
        const int row = sb * 32 + lrow;
#pragma unroll
        for (int kc = 0; kc < NQC; ++kc)
          st[sb] = mfma_chunk<S>(Ks[row * CHK + ((2 * kc + lhalf) ^ (row & KSW))], qf[kc], st[sb]);
      }
      // scale, causal / sequence-start mask, online softmax (lane = one query)
      const bool need_mask = (kt0 < seq_start) || (kt0 + BKV - 1 > wq0);
      float mx = m_run;
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float s = st[sb][r] * p.scale_log2;
          if (need_mask) {
            const int key = kt0 + sb * 32 + (r >> 2) * 8 + lhalf * 4 + (r & 3);
            if (key > my_q || key < seq_start) s = -INFINITY;
          }
          st[sb][r] = s;
          mx = fmaxf(mx, s);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float alpha = exp2f(m_run - mx);
      m_run = mx;
      float lsum = 0.f;
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float e = exp2f(st[sb][r] - mx);
          st[sb][r] = e;
          lsum += e;
        }
      l_run = l_run * alpha + lsum;
#pragma unroll
      for (int ob = 0; ob < OB; ++ob)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[ob][r] *= alpha;

      // O^T += V^T P^T
      if constexpr (ES == 2) {
        typedef S s8 __attribute__((ext_vector_type(8)));
        uint4 pb[2][2];
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            s8 v;
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = (S)st[sb][8 * hh + j];
            pb[sb][hh] = __builtin_bit_cast(uint4, v);
          }
#pragma unroll
        for (int ob = 0; ob < OB; ++ob) {
          const int m = ob * 32 + lrow;
          const uint2* V8 = reinterpret_cast<const uint2*>(Vs + m * VROWB);
          const int sw = m & 15;
#pragma unroll
          for (int sb = 0; sb < 2; ++sb)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
              // k = 8*lhalf + j  <->  key = 32 sb + 16 hh + 8 (j / 4) + 4 lhalf + j % 4
              const int u1 = 8 * sb + 4 * hh + lhalf;
              const uint2 lo4 = V8[u1 ^ sw], hi4 = V8[(u1 + 2) ^ sw];
              oacc[ob] = mfma_chunk<S>(make_uint4(lo4.x, lo4.y, hi4.x, hi4.y), pb[sb][hh],
                                       oacc[ob]);
            }
        }
      } else {
#pragma unroll
        for (int ob = 0; ob < OB; ++ob) {
          const int m = ob * 32 + lrow;
          const uint4* V16 = reinterpret_cast<const uint4*>(Vs + m * VROWB);
#pragma unroll
          for (int sb = 0; sb < 2; ++sb)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              // registers r = 4g .. 4g+3 hold keys 32 sb + 8 g + 4 lhalf + (0..3)
              const int c = 8 * sb + 2 * g + lhalf;
              const f32x4 a4 = __builtin_bit_cast(f32x4, V16[c ^ (m & 7)]);
#pragma unroll
              for (int q = 0; q < 4; ++q)
                oacc[ob] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q], st[sb][4 * g + q],
                                                                 oacc[ob], 0, 0, 0);
            }
        }
      }
    }

    if (it + 1 < n_tiles) lstore(buf ^ 1);
    __syncthreads();
  }

  // ---- normalise and write O (lane: query my_q, features ob*32 + (r/4)*8 + 4*lhalf + r%4)
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (wq0 < q_hi && my_q < q_hi) {
    const float inv = 1.0f / l_tot;
    S* orow = static_cast<S*>(p.out) + ((int64_t)i * p.T + my_q) * p.d + h * HD;
#pragma unroll
    for (int ob = 0; ob < OB; ++ob)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int m = ob * 32 + g * 8 + lhalf * 4;
        store_out4(orow + m, oacc[ob][4 * g] * inv, oacc[ob][4 * g + 1] * inv,
                   oacc[ob][4 * g + 2] * inv, oacc[ob][4 * g + 3] * inv);
      }
  }
}

template <typename S>
hipError_t launch_typed(const AttnParams& p, int n, int hd, hipStream_t s) {
  const int total_tiles = p.tile_prefix[p.num_seqs];
  dim3 grid((unsigned)(n * p.n_heads), (unsigned)total_tiles), block(ATT_THREADS);
  switch (hd) {
    case 32: hipLaunchKernelGGL((attn_kernel<S, 32>), grid, block, 0, s, p); break;
    case 64: hipLaunchKernelGGL((attn_kernel<S, 64>), grid, block, 0, s, p); break;
    case 128: hipLaunchKernelGGL((attn_kernel<S, 128>), grid, block, 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnDesc& a, hipStream_t s) {
  if (a.num_seqs <= 0 || a.num_seqs > KRAKEN_MAX_SEQS || a.n <= 0) return hipErrorInvalidValue;
  AttnParams p;
  p.qk = a.qk; p.vt = a.vt; p.out = a.out;
  p.T = a.T; p.d = a.d; p.n_heads = a.n_heads; p.ldv = vt_ld(a.T); p.num_seqs = a.num_seqs;
  const int hd = a.d / a.n_heads;
  p.scale_log2 = (float)(1.4426950408889634 / __builtin_sqrt((double)hd));
  p.tile_prefix[0] = 0;
  for (int b = 0; b <= a.num_seqs; ++b) p.cu[b] = a.cu_host[b];
  for (int b = 0; b < a.num_seqs; ++b)
    p.tile_prefix[b + 1] = p.tile_prefix[b] + (a.cu_host[b + 1] - a.cu_host[b] + BQ - 1) / BQ;
  if (p.tile_prefix[a.num_seqs] == 0) return hipSuccess;
  switch (a.dt) {
    case DType::BF16: return launch_typed<bf16>(p, a.n, hd, s);
    case DType::F16: return launch_typed<f16>(p, a.n, hd, s);
    default: return launch_typed<float>(p, a.n, hd, s);
  }
}

}  // namespace kraken
