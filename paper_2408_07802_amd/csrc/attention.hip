// Causal flash attention for the Kraken sub-layers (Section 2.1: per head,
// softmax(Q K^T / sqrt(hd)) V; causal; packed sequences never attend across
// each other).  All N sub-layers and all heads of a layer run in one launch.
//
// Layout: qk [n][T][2d] holds Q then K per token (head h at columns h*hd of
// each half); vt [n][d][ldv] holds V transposed (feature-major), written that
// way by the V projection so that V^T tiles are contiguous rows.
//
// Formulation: a wave owns one or two 32-query MFMA blocks and computes the
// score tile transposed, S^T = K Q^T.  In the MFMA result layout a lane
// then owns one query (one column) and half of the keys, so the running max /
// sum of the online softmax are per-lane values; only the max is exchanged
// once per tile with the partner lane (lane ^ 32).  The output is accumulated
// transposed, O^T = V^T P^T, whose columns are again the lane's query, so the
// rescale by exp(m_old - m_new) is lane-local; the exponent base only moves when
// a maximum outgrows it by more than 2^8, so rescales are rare.  P^T goes from the S^T accumulator registers straight into
// the B operand of the second MFMA.  The K rows of each 32-row fragment are
// read in an order that swaps bits 2 and 3 of the row index; then result
// register r of lane half h holds key 16 (r / 8) + 8 h + r % 8, so the eight
// keys a lane feeds to one P V MFMA are contiguous and the V^T operand is a
// single 16-byte LDS read.
//
// Workgroup: 256 queries of one (sub-layer, head, sequence), as 8 waves of 32
// queries (two waves per SIMD, so one wave's softmax arithmetic runs while the
// other's MFMAs do) or, for tiles that do not split over 8 waves, 4 waves of 64.
// K and V^T tiles of 64 keys are copied from HBM straight into a 3-stage LDS
// ring (global_load_lds_dwordx4), two tiles ahead of the tile being computed.
// Workgroups are ordered heaviest (longest causal prefix) first.
#include "kraken_internal.hpp"
#include "../../include/kraken.h"

namespace kraken {
namespace {

constexpr int BQ = 256;              // queries per workgroup
constexpr int BKV = 64;              // keys per tile

struct AttnParams {
  const void* qk;
  const void* vt;
  void* out;
  int n, T, d, n_heads, ldv, num_seqs;
  int head_group;         // heads per XCD group of the workgroup order (0: plain order)
  float scale_log2;       // log2(e) / sqrt(hd)
  int cu[KRAKEN_MAX_SEQS + 1];
  int tile_prefix[KRAKEN_MAX_SEQS + 1];
};

typedef __attribute__((address_space(3))) void* lds_void_ptr;

// Workgroup order.  Workgroup b runs on XCD b % 8 (round-robin dispatch), and each XCD
// has its own L2.  With head_group G > 0 (the host sets it when the (sub-layer, head)
// pairs split evenly over the 8 XCDs and there are many rounds of workgroups), XCD k
// takes pairs k, k + 8, ... in groups of G, and inside a group goes through the query
// tiles heaviest first, interleaving the group's heads.  The ~32 workgroups an XCD runs
// at a time then cover a few heads at several query tiles each; they sweep the same K/V
// tiles at about the same time and share them in L2.  Otherwise (few rounds, where the
// tail of a heaviest-first order matters more) the order is heaviest tile first over all
// pairs.
constexpr int HEAD_GROUP = 4;
__device__ __forceinline__ void head_rank_of(int b, int pairs, int tiles, int G, int& x,
                                             int& rank) {
  if (G == 0) {
    x = b % pairs;
    rank = b / pairs;
    return;
  }
  const int k = b & 7, j = b >> 3;
  const int per_xcd = pairs >> 3;
  const int g = j / (G * tiles);
  const int gsize = min(G, per_xcd - g * G);
  const int r = j - g * G * tiles;
  rank = r / gsize;
  x = k + 8 * (g * G + r % gsize);
}

// 16 bytes per lane from global memory into LDS at `lds` + 16 * lane; ordered by the
// kernel's own s_waitcnt vmcnt + barrier (see the GEMM for why it is inline assembly).
__device__ __forceinline__ void dma16(const void* g, void* lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_ptr)lds);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(l), "v"(g) : "memory", "m0");
}

// Key row read by fragment row r: bits 2 and 3 of r swapped.
__device__ __forceinline__ int kperm(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}
// Chunk swizzle of a tile with NC 16-byte chunks per row: logical chunk c of row r sits at
// physical chunk c ^ row_key<NC>(r).  One ds_read_b128 serves 16 lanes per LDS cycle; the
// fragment reads here give those 16 lanes 16 distinct rows (of one aligned block of 16)
// and the same logical chunk, and the key makes their 16 (bank-group) positions
// (r * NC + physical chunk) mod 16 distinct, so the reads are free of bank conflicts.
template <int NC>
__device__ __forceinline__ int row_key(int r) {
  if constexpr (NC >= 16) return r & 15;
  else if constexpr (NC == 8) return (r >> 1) & 7;
  else return (r >> 2) & 3;
}

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

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  if constexpr (N == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if constexpr (N == 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
  else if constexpr (N == 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if constexpr (N == 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else if constexpr (N == 12) asm volatile("s_waitcnt vmcnt(12)" ::: "memory");
  else if constexpr (N == 16) asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// NQB 32-query blocks per wave: NQB = 1 runs 8 waves (two per SIMD, so one wave's
// softmax arithmetic overlaps the other's matrix work); NQB = 2 runs 4 waves.
template <typename S, int HD, int NQB>
__global__ __launch_bounds__(BQ / NQB / 32 * 64, 1) void attn_kernel(AttnParams p) {
  constexpr int QW = 32 * NQB;                // queries per wave
  constexpr int NW = BQ / QW;                 // waves per workgroup
  constexpr int ES = sizeof(S);
  constexpr int EPC = 16 / ES;                // elements per 16-byte chunk
  constexpr int CHK = HD * ES / 16;           // chunks per K row
  constexpr int VCH = BKV * ES / 16;          // chunks per V^T row
  constexpr int NQC = HD * ES / 32;           // chunk pairs per head row (MFMA k steps)
  constexpr int OB = HD / 32;                 // 32-row blocks of O^T
  constexpr int TILE = BKV * HD * ES;         // bytes of one K (or V^T) tile
  constexpr int STAGE = 2 * TILE;
  constexpr int STAGES = 3 * STAGE <= 144 * 1024 ? 3 : 2;
  constexpr int KI = CHK / NW;                // K DMA instructions per wave per tile
  constexpr int VI = HD * VCH / 64 / NW;      // V^T DMA instructions per wave per tile
  constexpr int NPT = KI + VI;                // DMA instructions per wave per tile
  static_assert(KI >= 1 && VI >= 1 && KI * NW == CHK && VI * NW * 64 == HD * VCH,
                "tile does not split evenly over the waves");

  __shared__ __attribute__((aligned(16))) unsigned char smem[STAGES * STAGE];

  // ---- which (sub-layer, head, sequence, query tile)
  int x, rank;
  head_rank_of(blockIdx.x, p.n * p.n_heads, p.tile_prefix[p.num_seqs], p.head_group, x, rank);
  const int i = x / p.n_heads;
  const int h = x - i * p.n_heads;
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
  const int kv_begin = seq_start & ~7;       // 16-byte aligned V^T chunks

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int wq0 = q0 + wave * QW;

  const int64_t ld_qk = 2 * (int64_t)p.d;
  const S* qkz = static_cast<const S*>(p.qk) + (int64_t)i * p.T * ld_qk;
  const S* Kbase = qkz + p.d + h * HD;
  const S* Vbase = static_cast<const S*>(p.vt) + ((int64_t)i * p.d + h * HD) * p.ldv;

  // ---- Q fragments (B operand of S^T = K Q^T): lane's query, chunk 2*kc + lhalf
  uint4 qf[NQB][NQC];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const int q = wq0 + qb * 32 + lrow;
    const S* qrow = qkz + (int64_t)min(q, p.T - 1) * ld_qk + h * HD;
#pragma unroll
    for (int kc = 0; kc < NQC; ++kc)
      qf[qb][kc] = (q < q_hi) ? *reinterpret_cast<const uint4*>(qrow + (2 * kc + lhalf) * EPC)
                              : make_uint4(0, 0, 0, 0);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  // ---- DMA of one K tile and one V^T tile into stage `st`.
  auto issue = [&](int kt0, int st) {
    unsigned char* base = smem + st * STAGE;
#pragma unroll
    for (int u = 0; u < KI; ++u) {
      const int ins = wave * KI + u;                       // 1 KB = 64 / CHK rows
      const int row = ins * (64 / CHK) + lane / CHK;
      const int pch = lane % CHK;
      const int lch = pch ^ row_key<CHK>(row);
      const int key = min(kt0 + row, p.T - 1);
      dma16(Kbase + (int64_t)key * ld_qk + lch * EPC, base + ins * 1024);
    }
#pragma unroll
    for (int u = 0; u < VI; ++u) {
      const int ins = wave * VI + u;                       // 1 KB = 64 / VCH rows
      const int row = ins * (64 / VCH) + lane / VCH;
      const int pch = lane % VCH;
      const int lch = pch ^ row_key<VCH>(row);
      const int key = min(kt0 + lch * EPC, p.ldv - EPC);
      dma16(Vbase + (int64_t)row * p.ldv + key, base + TILE + ins * 1024);
    }
  };

  f32x16 oacc[NQB][OB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
    for (int ob = 0; ob < OB; ++ob)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[qb][ob][r] = 0.f;
  float m_run[NQB], l_run[NQB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    m_run[qb] = -1e30f;
    l_run[qb] = 0.f;
  }

  const int n_tiles = (q_hi - kv_begin + BKV - 1) / BKV;
#pragma unroll
  for (int t = 0; t < STAGES - 1; ++t)
    if (t < n_tiles) issue(kv_begin + t * BKV, t);

  for (int t = 0; t < n_tiles; ++t) {
    // tile t is complete once at most the later prefetched tiles are outstanding
    if (STAGES == 3 && t + 1 < n_tiles) wait_vmcnt<NPT>();
    else wait_vmcnt<0>();
    __syncthreads();
    if (t + STAGES - 1 < n_tiles) issue(kv_begin + (t + STAGES - 1) * BKV, (t + STAGES - 1) % STAGES);

    const int kt0 = kv_begin + t * BKV;
    const unsigned char* base = smem + (t % STAGES) * STAGE;
    const uint4* Ks = reinterpret_cast<const uint4*>(base);
    const uint4* Vs = reinterpret_cast<const uint4*>(base + TILE);

    // skip the tile when none of this wave's queries sees any of its keys; inside a
    // processed tile both query blocks run (a block that sees none of the keys gets
    // all-masked scores, i.e. zero weights)
    if (wq0 >= q_hi || kt0 > min(wq0 + QW - 1, q_hi - 1)) continue;

    // S^T for keys [kt0, kt0 + 64): two 32-key blocks per query block
    f32x16 st[NQB][2];
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) st[qb][sb][r] = 0.f;
    // (k steps outer, key blocks inner: consecutive MFMAs feed independent accumulators)
#pragma unroll
    for (int kc = 0; kc < NQC; ++kc)
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        const int row = kperm(sb * 32 + lrow);
        const uint4 a = Ks[row * CHK + ((2 * kc + lhalf) ^ row_key<CHK>(row))];
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) st[qb][sb] = mfma_chunk<S>(a, qf[qb][kc], st[qb][sb]);
      }

#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      const int my_q = wq0 + qb * 32 + lrow;
      // scores stay unscaled here; the scale (positive) enters the running max and, fused,
      // the exponent argument
      if ((kt0 < seq_start) || (kt0 + BKV - 1 > wq0 + qb * 32)) {
        // keys outside [seq_start, my_q] get weight 0; register r holds key
        // kt0 + 8 lhalf + off(r) with off(r) = 32 sb + 16 (r / 8) + r % 8, so the test is
        // one unsigned range check per register
        const int base = kt0 + 8 * lhalf;
        const unsigned lo = (unsigned)(seq_start - base);
        const unsigned span = (unsigned)(my_q - seq_start);
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const unsigned off = (unsigned)(sb * 32 + (r >> 3) * 16 + (r & 7));
            st[qb][sb][r] = (off - lo <= span) ? st[qb][sb][r] : -INFINITY;
          }
      }
      float mraw = -INFINITY;
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mraw = fmaxf(mraw, st[qb][sb][r]);
      float mx = fmaxf(m_run[qb], mraw * p.scale_log2);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      // The exponent base m_run is only moved when some lane's maximum exceeds it by
      // more than 8 (log2 units): weights stay <= 2^8, exact in the fp32 sums and within
      // the range of the 16-bit P operand, and the O rescale is rare.
      if (__ballot(mx > m_run[qb] + 8.0f)) {
        const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - mx);
        l_run[qb] *= alpha;
#pragma unroll
        for (int ob = 0; ob < OB; ++ob)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[qb][ob][r] *= alpha;
        m_run[qb] = mx;
      }
      float lsum = 0.f;
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float e = __builtin_amdgcn_exp2f(fmaf(st[qb][sb][r], p.scale_log2, -m_run[qb]));
          st[qb][sb][r] = e;
          lsum += e;
        }
      l_run[qb] += lsum;
    }

    // O^T += V^T P^T
    if constexpr (ES == 2) {
      typedef S s8 __attribute__((ext_vector_type(8)));
      uint4 pb[NQB][2][2];
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            s8 v;
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = (S)st[qb][sb][8 * hh + j];
            pb[qb][sb][hh] = __builtin_bit_cast(uint4, v);
          }
      // (key chunks outer, output blocks inner: independent accumulators back to back)
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int ob = 0; ob < OB; ++ob) {
            const int m = ob * 32 + lrow;
            // k = 8 lhalf + j  <->  key 32 sb + 16 hh + 8 lhalf + j: one 16-byte chunk
            const uint4 a = Vs[m * VCH + ((4 * sb + 2 * hh + lhalf) ^ row_key<VCH>(m))];
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb)
              oacc[qb][ob] = mfma_chunk<S>(a, pb[qb][sb][hh], oacc[qb][ob]);
          }
    } else {
#pragma unroll
      for (int ob = 0; ob < OB; ++ob) {
        const int m = ob * 32 + lrow;
#pragma unroll
        for (int sb = 0; sb < 2; ++sb)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            // registers 4g .. 4g+3 hold keys 32 sb + 16 (g/2) + 8 lhalf + 4 (g%2) + (0..3)
            const int c = 8 * sb + 4 * (g >> 1) + 2 * lhalf + (g & 1);
            const f32x4 a4 = __builtin_bit_cast(f32x4, Vs[m * VCH + (c ^ row_key<VCH>(m))]);
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
              for (int qb = 0; qb < NQB; ++qb)
                oacc[qb][ob] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q], st[qb][sb][4 * g + q],
                                                                    oacc[qb][ob], 0, 0, 0);
          }
      }
    }
  }

  // ---- normalise and write O (lane: query, features ob*32 + (r/4)*8 + 4*lhalf + r%4)
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 32, 64);
    const int my_q = wq0 + qb * 32 + lrow;
    if (my_q < q_hi) {
      const float inv = 1.0f / l_tot;
      S* orow = static_cast<S*>(p.out) + ((int64_t)i * p.T + my_q) * p.d + h * HD;
#pragma unroll
      for (int ob = 0; ob < OB; ++ob)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int m = ob * 32 + g * 8 + lhalf * 4;
          store_out4(orow + m, oacc[qb][ob][4 * g] * inv, oacc[qb][ob][4 * g + 1] * inv,
                     oacc[qb][ob][4 * g + 2] * inv, oacc[qb][ob][4 * g + 3] * inv);
        }
    }
  }
}

// 8 waves of one query block each when the K and V^T tiles split evenly over 8 waves
// (all head sizes but 32 with 16-bit storage), else 4 waves of two.
template <typename S, int HD>
constexpr int nqb_for() {
  return ((HD * (int)sizeof(S) / 16) % 8 == 0) ? 1 : 2;
}

template <typename S, int HD>
void launch_hd(const AttnParams& p, dim3 grid, hipStream_t s) {
  constexpr int NQB = nqb_for<S, HD>();
  hipLaunchKernelGGL((attn_kernel<S, HD, NQB>), grid, dim3(BQ / NQB / 32 * 64), 0, s, p);
}

template <typename S>
hipError_t launch_typed(const AttnParams& p, int n, int hd, hipStream_t s) {
  const int total_tiles = p.tile_prefix[p.num_seqs];
  dim3 grid((unsigned)(n * p.n_heads * total_tiles));
  switch (hd) {
    case 32: launch_hd<S, 32>(p, grid, s); break;
    case 64: launch_hd<S, 64>(p, grid, s); break;
    case 128: launch_hd<S, 128>(p, grid, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnDesc& a, hipStream_t s) {
  if (a.num_seqs <= 0 || a.num_seqs > KRAKEN_MAX_SEQS || a.n <= 0) return hipErrorInvalidValue;
  AttnParams p;
  p.qk = a.qk; p.vt = a.vt; p.out = a.out;
  p.n = a.n; p.T = a.T; p.d = a.d; p.n_heads = a.n_heads; p.ldv = vt_ld(a.T); p.num_seqs = a.num_seqs;
  const int hd = a.d / a.n_heads;
  p.scale_log2 = (float)(1.4426950408889634 / __builtin_sqrt((double)hd));
  p.tile_prefix[0] = 0;
  for (int b = 0; b <= a.num_seqs; ++b) p.cu[b] = a.cu_host[b];
  for (int b = 0; b < a.num_seqs; ++b)
    p.tile_prefix[b + 1] = p.tile_prefix[b] + (a.cu_host[b + 1] - a.cu_host[b] + BQ - 1) / BQ;
  if (p.tile_prefix[a.num_seqs] == 0) return hipSuccess;
  const int64_t pairs = (int64_t)a.n * a.n_heads, wgs = pairs * p.tile_prefix[a.num_seqs];
  p.head_group = (pairs % 8 == 0 && wgs >= 2048) ? HEAD_GROUP : 0;
  switch (a.dt) {
    case DType::BF16: return launch_typed<bf16>(p, a.n, hd, s);
    case DType::F16: return launch_typed<f16>(p, a.n, hd, s);
    default: return launch_typed<float>(p, a.n, hd, s);
  }
}

}  // namespace kraken
