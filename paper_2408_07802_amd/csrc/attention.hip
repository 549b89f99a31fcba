// Causal flash attention for the Kraken sub-layers (Section 2.1: per head,
// softmax(Q K^T / sqrt(hd)) V; causal; packed sequences never attend across
// each other).  All N sub-layers and all heads of a layer run in one launch.
//
// Layout: qk [n][T][d + dkv] holds Q then K per token (query head h at columns
// h*hd, key head g at columns d + g*hd); vt [n][dkv][ldv] holds V transposed
// (feature-major), written that way by the V projection so that V^T tiles are
// contiguous rows.  With grouped-query attention (dkv = n_kv_heads * hd < d) query
// head h reads key/value head h / group, group = n_heads / n_kv_heads.
//
// Formulation: a wave owns one or two 32-query MFMA blocks and computes the
// score tile transposed, S^T = K Q^T.  In the MFMA result layout a lane
// then owns one query (one column) and half of the keys, so the running max /
// sum of the online softmax are per-lane values; only the max is exchanged
// once per tile with the partner lane (lane ^ 32).  The output is accumulated
// transposed, O^T = V^T P^T, whose columns are again the lane's query, so the
// rescale by exp(m_old - m_new) is lane-local; the exponent base only moves when
// a maximum exceeds it by more than 8 in base-2 log units (a weight would pass 2^8),
// so rescales are rare.  P^T goes from the
// S^T accumulator registers straight into the B operand of the second MFMA.  The K
// rows of each 32-row fragment are read in an order that swaps bits 2 and 3 of the
// row index; then result
// register r of lane half h holds key 16 (r / 8) + 8 h + r % 8, so the eight
// keys a lane feeds to one P V MFMA are contiguous and the V^T operand is a
// single 16-byte LDS read.
//
// Workgroup: 256 queries of one (sub-layer, head, sequence), as 8 waves of 32
// queries (two waves per SIMD, so one wave's softmax arithmetic runs while the
// other's MFMAs do) or, for tiles that do not split over 8 waves, 4 waves of 64.
// K and V^T tiles of 64 keys are copied from HBM straight into a 3-stage LDS
// ring (global_load_lds_dwordx4), two tiles ahead of the tile being computed.
// 16-bit operands with head size 128 take the ping-pong form further down (a 4-stage
// ring of range-checked buffer loads, the two waves of a SIMD in opposite phases).
// Workgroups are ordered heaviest (longest causal prefix) first.
#include <type_traits>

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
  int dkv, group;         // key/value width, query heads per key/value head
  int head_group;         // heads per XCD group of the workgroup order (0: plain order)
  float scale_log2;       // log2(e) / sqrt(hd), or 1 when Q already carries that factor
  int q_prescaled;        // Q columns were multiplied by log2(e) / sqrt(hd) upstream
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

// The same DMA with a wave-uniform base address (SGPR pair) and a per-lane 32-bit byte
// offset, so that per-tile address arithmetic stays on the scalar unit.
// (The base goes through readfirstlane so that it is an SGPR pair whatever the compiler
// concludes about its uniformity.)
__device__ __forceinline__ void dma16_off(uint32_t lds_addr, const void* base, uint32_t off) {
  // (readfirstlane returns a signed int: each half is taken as unsigned before widening,
  // or a low half with bit 31 set would sign-extend over the high half)
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint64_t bu = ((uint64_t)hi << 32) | (uint64_t)lo;
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
               :: "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(off),
                  "s"(reinterpret_cast<const void*>(bu)) : "memory", "m0");
}

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// Buffer resource for raw (unstructured) access to the part from byte `off` on of the
// `bytes` bytes at `base` (nothing when off >= bytes): no stride, no swizzle, 32-bit data
// format.  A buffer access whose byte offset lies beyond the part reads zero and never
// faults.  All of it is scalar arithmetic.
__device__ __forceinline__ i32x4 raw_rsrc(const void* base, uint32_t bytes, uint32_t off) {
  const uint64_t b = reinterpret_cast<uint64_t>(base) + off;
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((uint32_t)b);
  r[1] = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32) & 0xffffu);
  r[2] = __builtin_amdgcn_readfirstlane(off < bytes ? bytes - off : 0u);
  r[3] = 0x00020000;
  return r;
}

// dma16 through a buffer resource: lane i's 16 bytes at byte offset `off` (range checked)
// land at LDS address lds_addr + 16 i; ordered like dma16.
__device__ __forceinline__ void dma16_buf(uint32_t lds_addr, i32x4 rsrc, uint32_t off) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(off), "s"(rsrc)
               : "memory", "m0");
}

// A pointer that is the same for every lane, moved to scalar registers (each half taken
// as unsigned before widening, like dma16_off's base).
template <typename T>
__device__ __forceinline__ const T* uniform_ptr(const T* ptr) {
  const uint64_t v = reinterpret_cast<uint64_t>(ptr);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)v);
  return reinterpret_cast<const T*>(((uint64_t)hi << 32) | (uint64_t)lo);
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

// s_waitcnt immediate for vmcnt(0) alone (expcnt and lgkmcnt at their maximum).
constexpr int VMCNT0 = 0x0f70;

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

  // ---- which (sub-layer, head, sequence, query tile): the same for every lane (kept in
  // scalar registers, see attn_pp_kernel)
  int x, rank;
  head_rank_of(blockIdx.x, p.n * p.n_heads, p.tile_prefix[p.num_seqs], p.head_group, x, rank);
  x = __builtin_amdgcn_readfirstlane(x);
  rank = __builtin_amdgcn_readfirstlane(rank);
  const int i = x / p.n_heads;
  const int h = x - i * p.n_heads;
  int lo = 0, hi = p.num_seqs - 1;           // last b with tile_prefix[b] <= rank
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.tile_prefix[mid] <= rank) lo = mid; else hi = mid - 1;
  }
  const int b = __builtin_amdgcn_readfirstlane(lo);
  const int ntiles_b = p.tile_prefix[b + 1] - p.tile_prefix[b];
  const int qt = ntiles_b - 1 - (rank - p.tile_prefix[b]);
  const int seq_start = p.cu[b], seq_end = p.cu[b + 1];
  const int q0 = seq_start + qt * BQ;
  const int q_hi = min(q0 + BQ, seq_end);
  const int kv_begin = seq_start & ~7;       // 16-byte aligned V^T chunks

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int wq0 = q0 + wave * QW;

  const int64_t ld_qk = (int64_t)p.d + p.dkv;
  const S* qkz = static_cast<const S*>(p.qk) + (int64_t)i * p.T * ld_qk;
  const int hkv = h / p.group;              // the key/value head this head reads
  const S* Kbase = uniform_ptr(qkz + p.d + hkv * HD);
  const S* Vbase =
      uniform_ptr(static_cast<const S*>(p.vt) + ((int64_t)i * p.dkv + hkv * HD) * p.ldv);

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
  // The Q loads are complete before any DMA is issued.  (The compiler's own wait, which
  // it can see, not inline assembly: an opaque wait here would leave the loads pending in
  // its bookkeeping, and it would then wait for every outstanding vector-memory operation,
  // the K/V prefetches included, before the first use of Q in every tile.)
  __builtin_amdgcn_s_waitcnt(VMCNT0);

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
    if (t + STAGES - 1 < n_tiles)
      issue(kv_begin + (t + STAGES - 1) * BKV, (t + STAGES - 1) % STAGES);

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

// ---------------------------------------------------------------------------------------
// Ping-pong form for 16-bit operands: 8 waves of 32 queries, two waves per SIMD.  Each
// wave alternates a matrix phase M(t) = { O^T += V(t-1)^T P(t-1)^T, S(t) = K(t) Q^T } and a
// vector phase V(t) = { online softmax of S(t): mask, running max, exponentials, row sums,
// 16-bit P(t) }, with a workgroup barrier after every phase.  One group of four waves starts
// one barrier later than the other, so the two waves sharing a SIMD are in opposite phases
// and one wave's softmax arithmetic runs while the other's MFMAs do.  K/V^T tiles go
// through a 4-stage LDS ring.  Numbering the intervals between barriers (interval k ends
// at barrier k), the leading group runs M(t) in interval 2t+1 and V(t) in 2t+2, the
// trailing group one interval later; so K(u) is read in intervals 2u+1 and 2u+2, V(u) in
// 2u+3 and 2u+4.  Every wave issues its share of tile u right after its M(u-2) (interval
// 2u-3 for the leading group, 2u-2 for the trailing one), when tile u-4, the stage's
// previous tile, is no longer read (its last reader ends in interval 2u-4), and waits for
// that share just before barrier 2u (leading group in V(u-1), trailing group in M(u-1)),
// so the tile is complete before its first reader.  The K/V^T loads are buffer loads
// straight into LDS whose range check zero-fills rows past the key range: no branch and
// no per-lane clamping; tiles past the end are loaded too (they read nothing).
constexpr int PP_STAGES = 4;

template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int N>
using IC = std::integral_constant<int, N>;

template <int B, int E, typename F>
__device__ __forceinline__ void sfor(F&& f) {
  if constexpr (B < E) {
    f(IC<B>{});
    sfor<B + 1, E>(f);
  }
}

// Sum of the eight 16-bit values packed in v, added to acc in fp32 (v_dot2 with (1, 1)).
template <typename S>
__device__ __forceinline__ float sum8(uint4 v, float acc);
template <>
__device__ __forceinline__ float sum8<f16>(uint4 v, float acc) {
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  const h2 one = {(_Float16)1.0f, (_Float16)1.0f};
  acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, v.x), one, acc, false);
  acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, v.y), one, acc, false);
  acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, v.z), one, acc, false);
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, v.w), one, acc, false);
}
template <>
__device__ __forceinline__ float sum8<bf16>(uint4 v, float acc) {
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  const b2 one = {(__bf16)1.0f, (__bf16)1.0f};
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(b2, v.x), one, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(b2, v.y), one, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(b2, v.z), one, acc, false);
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(b2, v.w), one, acc, false);
}

// PRE: Q already carries log2(e) / sqrt(hd), so the scores come out of the MFMAs in log2
// units.  Then the first S MFMAs of a tile accumulate onto -c0 (a per-lane constant: in the
// transposed layout a lane's 16 score registers all belong to its query), c0 being the
// running maximum, and a weight is a bare exp2 of its accumulator; only a rescale (rare)
// shifts the tile's scores by the growth of the maximum.
template <typename S, int HD, bool PRE>
__global__ __launch_bounds__(512, 1) void attn_pp_kernel(AttnParams p) {
  constexpr int NW = 8, QW = 32;
  constexpr int EPC = 8;                      // 16-bit elements per 16-byte chunk
  constexpr int CHK = HD * 2 / 16;            // chunks per K row
  constexpr int VCH = BKV * 2 / 16;           // chunks per V^T row
  constexpr int NQC = HD * 2 / 32;            // 16-deep k steps of S
  constexpr int OB = HD / 32;                 // 32-row blocks of O^T
  constexpr int TILE = BKV * HD * 2;
  constexpr int STAGE = 2 * TILE;
  constexpr int KI = CHK / NW;
  constexpr int VI = HD * VCH / 64 / NW;
  constexpr int NPT = KI + VI;                // DMA instructions per wave per tile
  constexpr int NS = 2 * NQC;                 // S MFMAs per tile
  constexpr int NP = 4 * OB;                  // PV MFMAs per tile
  constexpr int RING = 4;                     // fragment register ring depth
  static_assert(KI >= 1 && VI >= 1 && KI * NW == CHK && VI * NW * 64 == HD * VCH,
                "tile does not split evenly over the waves");
  static_assert(PP_STAGES * STAGE <= 160 * 1024, "LDS ring too large");
  static_assert(NS == NP && NS >= RING, "S and PV MFMAs alternate one for one");

  __shared__ __attribute__((aligned(16))) uint4 smem[PP_STAGES * STAGE / 16];

  // The workgroup's (sub-layer, head, sequence, query tile) is the same for every lane.
  // readfirstlane tells the compiler so (it cannot see it through the search loop): the
  // per-tile DMA addresses and branches then run on the scalar unit instead of as 64-bit
  // vector multiplies and exec-mask branches that compete with the other wave's softmax.
  int x, rank;
  head_rank_of(blockIdx.x, p.n * p.n_heads, p.tile_prefix[p.num_seqs], p.head_group, x, rank);
  x = __builtin_amdgcn_readfirstlane(x);
  rank = __builtin_amdgcn_readfirstlane(rank);
  const int i = x / p.n_heads;
  const int h = x - i * p.n_heads;
  int lo = 0, hi = p.num_seqs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.tile_prefix[mid] <= rank) lo = mid; else hi = mid - 1;
  }
  const int b = __builtin_amdgcn_readfirstlane(lo);
  const int ntiles_b = p.tile_prefix[b + 1] - p.tile_prefix[b];
  const int qt = ntiles_b - 1 - (rank - p.tile_prefix[b]);
  const int seq_start = p.cu[b], seq_end = p.cu[b + 1];
  const int q0 = seq_start + qt * BQ;
  const int q_hi = min(q0 + BQ, seq_end);
  const int kv_begin = seq_start & ~7;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // group B (one barrier behind group A): waves 1, 3, 4, 6.  Whether the hardware puts waves
  // w and w + 4 or waves 2k and 2k + 1 on one SIMD, each SIMD gets one wave of each group.
  const bool trail = ((wave & 1) ^ (wave >> 2)) != 0;
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int wq0 = q0 + wave * QW;
  const int my_q = wq0 + lrow;
  // last key tile this wave's queries see (-1: the wave has no queries)
  const int wlast = (wq0 >= q_hi) ? -1 : (min(wq0 + QW - 1, q_hi - 1) - kv_begin) / BKV;
  const int n_tiles = (q_hi - kv_begin + BKV - 1) / BKV;

  const int64_t ld_qk = (int64_t)p.d + p.dkv;
  const S* qkz = static_cast<const S*>(p.qk) + (int64_t)i * p.T * ld_qk;
  const int hkv = h / p.group;              // the key/value head this head reads
  const S* Kbase = uniform_ptr(qkz + p.d + hkv * HD);
  const S* Vbase =
      uniform_ptr(static_cast<const S*>(p.vt) + ((int64_t)i * p.dkv + hkv * HD) * p.ldv);

  uint4 qf[NQC];
  {
    const S* qrow = qkz + (int64_t)min(my_q, p.T - 1) * ld_qk + h * HD;
#pragma unroll
    for (int kc = 0; kc < NQC; ++kc)
      qf[kc] = (my_q < q_hi) ? *reinterpret_cast<const uint4*>(qrow + (2 * kc + lhalf) * EPC)
                             : make_uint4(0, 0, 0, 0);
  }
  __builtin_amdgcn_s_waitcnt(VMCNT0);        // (visible to the compiler: see attn_kernel)

  // this wave's share of the DMA of key tile u (K and V^T) into stage u % PP_STAGES, as
  // buffer loads.  Lane offsets within a tile are computed once; a tile moves the buffer
  // resource (scalar arithmetic), whose range check replaces any clamping: K rows from T
  // on (the sequence's last tile) and V^T bytes past the head's rows read as zeros, and no
  // key they hold is ever unmasked.  The tiles past the end that the pipeline loads
  // without a branch get an empty range and read nothing.  Any 32-bit tile offset is
  // safe: out of range reads nothing.  (The host sends only key ranges whose byte offsets
  // fit in 32 bits here.)
  const uint32_t smem_base =
      __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_ptr)smem);
  const uint32_t kbytes = (uint32_t)(((int64_t)p.T * ld_qk - p.d - hkv * HD) * 2);
  const uint32_t vbytes = (uint32_t)((int64_t)HD * p.ldv * 2);
  uint32_t koff[KI], voff[VI];
#pragma unroll
  for (int k = 0; k < KI; ++k) {
    const int row = (wave * KI + k) * (64 / CHK) + lane / CHK;
    const int lch = (lane % CHK) ^ row_key<CHK>(row);
    koff[k] = (uint32_t)((row * ld_qk + lch * EPC) * 2);
  }
#pragma unroll
  for (int k = 0; k < VI; ++k) {
    const int row = (wave * VI + k) * (64 / VCH) + lane / VCH;
    const int lch = (lane % VCH) ^ row_key<VCH>(row);
    voff[k] = (uint32_t)((row * (int64_t)p.ldv + lch * EPC) * 2);
  }
  auto issue = [&](int u) {
    const int kt0 = kv_begin + u * BKV;
    const uint32_t st = smem_base + (uint32_t)((u % PP_STAGES) * STAGE);
    const i32x4 kr = raw_rsrc(Kbase, kbytes, (uint32_t)((int64_t)kt0 * ld_qk * 2));
    const i32x4 vr = raw_rsrc(Vbase, u < n_tiles ? vbytes : 0u, (uint32_t)(kt0 * 2));
#pragma unroll
    for (int k = 0; k < KI; ++k) dma16_buf(st + (uint32_t)((wave * KI + k) * 1024), kr, koff[k]);
#pragma unroll
    for (int k = 0; k < VI; ++k)
      dma16_buf(st + (uint32_t)(TILE + (wave * VI + k) * 1024), vr, voff[k]);
  };
  // Every wave issues each tile, real or past the end, so before the barrier that makes
  // tile u readable only tile u + 1 may still be in flight; the last tile's wait drains
  // everything.  (The branch matters to the compiler: with a loop body of one basic block
  // its register allocation spills.)
  auto wait_tile = [&](int u) {
    if (u + 1 < n_tiles) wait_vm<NPT>();
    else wait_vm<0>();
  };

  // Fragment addresses.  A fragment's physical chunk is (logical chunk) ^ key(row); the
  // lane's own bits (lhalf and the key) are folded into a per-lane base once, so a read is
  // (base + stage offset, a multiple of the row size) XOR a compile-time chunk offset,
  // plus a compile-time row-block offset.
  uint32_t kbase[2];
#pragma unroll
  for (int sb = 0; sb < 2; ++sb) {
    const int row = kperm(sb * 32 + lrow);
    kbase[sb] = smem_base + (uint32_t)(row * CHK * 16 + ((lhalf ^ row_key<CHK>(row)) * 16));
  }
  // (ob * 32 + lrow) has the same key for every ob
  const uint32_t vbase =
      smem_base + TILE + (uint32_t)(lrow * VCH * 16 + ((lhalf ^ row_key<VCH>(lrow)) * 16));
  // 16-byte LDS read at byte address addr + 16 idx (typed indexing keeps the 16-byte
  // alignment visible to the compiler, so every read is one ds_read_b128)
  auto lds16 = [](uint32_t addr, int idx = 0) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    __builtin_assume((addr & 15u) == 0);
    const __attribute__((address_space(3))) u32x4* ptr =
        reinterpret_cast<const __attribute__((address_space(3))) u32x4*>((size_t)addr);
    return __builtin_bit_cast(uint4, ptr[idx]);
  };
  auto stage_off = [](int u) { return (uint32_t)((u % PP_STAGES) * STAGE); };
  // operand of S MFMA j (k step j/2, key block j%2) of the tile at stage offset st
  auto k_frag = [&](uint32_t st, int j) {
    const int kc = j >> 1, sb = j & 1;
    return lds16((kbase[sb] + st) ^ (uint32_t)(2 * kc * 16));
  };
  // operand of PV MFMA j = (key block sb, half hh, output block ob)
  auto v_frag = [&](uint32_t st, int j) {
    const int sb = j / (2 * OB), hh = (j / OB) & 1, ob = j % OB;
    return lds16((vbase + st) ^ (uint32_t)((4 * sb + 2 * hh) * 16), ob * 32 * VCH);
  };

  f32x16 oacc[OB];
#pragma unroll
  for (int ob = 0; ob < OB; ++ob)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[ob][r] = 0.f;
  float m_run = -1e30f, l_run = 0.f;
  const float scale = p.scale_log2;
  float c0 = 0.f;                             // (PRE) the S accumulators start from -c0
  f32x16 cneg = {};
  f32x16 sacc[2];                             // S(t), key blocks 0 and 1
  uint4 pb[2][2];                             // 16-bit P(t-1): [key block][half]
#pragma unroll
  for (int sb = 0; sb < 2; ++sb)
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) pb[sb][hh] = make_uint4(0, 0, 0, 0);
  const f32x16 zero16 = {};
  uint4 vpre[RING];                           // first V^T fragments of the next M phase

  // M(t): PV(t-1) and S(t), alternating.  At t = 0 P is zero and V is read from tile 0's
  // stage (real data), so the PV MFMAs add exactly zero; for t > wlast the scores are never
  // used.  The wave's last step only needs PV.  The phase runs at raised wave priority:
  // when the matrix pipe takes a new MFMA, this wave's is issued before the other wave's
  // softmax instructions (measured: attention 8% faster in the full pass).
  auto mphase = [&](int t) {
    __builtin_amdgcn_s_setprio(1);
    const uint32_t kst = stage_off(t);
    const uint32_t vst = stage_off(t >= 1 ? t - 1 : 0);
    uint4 kf[RING], vf[RING];
    sfor<0, RING>([&](auto J) {
      kf[J()] = k_frag(kst, J());
      vf[J()] = vpre[J()];
    });
    // slot order PV0, PV1, S0, PV2, S1, ..., PV15, S14, S15: the V^T fragments of the
    // first PV MFMAs are already in registers, and the K fragment reads issued at the
    // start of the phase land under them
    sfor<0, 2 * NS>([&](auto Sl) {
      constexpr int sl = decltype(Sl)::value;
      constexpr bool pv = sl < 2 || (sl < 2 * NS - 2 && (sl & 1));
      constexpr int j = sl < 2 ? sl
                        : pv ? (sl - 3) / 2 + 2
                        : sl < 2 * NS - 2 ? (sl - 2) / 2 : sl - NS;
      if constexpr (pv) {
        constexpr int sb = j / (2 * OB), hh = (j / OB) & 1, ob = j % OB;
        oacc[ob] = mfma_chunk<S>(vf[j % RING], pb[sb][hh], oacc[ob]);
        if constexpr (j + RING < NP) vf[j % RING] = v_frag(vst, j + RING);
      } else {
        sacc[j & 1] = mfma_chunk<S>(kf[j % RING], qf[j >> 1],
                                    j < 2 ? (PRE ? cneg : zero16) : sacc[j & 1]);
        if constexpr (j + RING < NS) kf[j % RING] = k_frag(kst, j + RING);
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    __builtin_amdgcn_s_setprio(0);
  };

  // V(t): online softmax of S(t) into P(t)
  auto vphase = [&](int t) {
    // the next matrix phase's first V^T fragments (tile t: complete since M(t)), read
    // here so that their latency passes under the softmax
    sfor<0, RING>([&](auto J) { vpre[J()] = v_frag(stage_off(t), J()); });
    const int kt0 = kv_begin + t * BKV;
    // keys outside [seq_start, my_q] get weight 0 (only tiles crossing the diagonal or the
    // sequence start): register r of key block sb holds key kt0 + 8 lhalf + off(r)
    if ((kt0 < seq_start) || (kt0 + BKV - 1 > wq0)) {
      const int base = kt0 + 8 * lhalf;
      const unsigned lo_ = (unsigned)(seq_start - base);
      const unsigned span = (unsigned)(my_q - seq_start);
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const unsigned off = (unsigned)(sb * 32 + (r >> 3) * 16 + (r & 7));
          sacc[sb][r] = (off - lo_ <= span) ? sacc[sb][r] : -INFINITY;
        }
    }
    // Weights, packed to 16 bits for the PV MFMAs; the row sums add the packed (rounded)
    // weights, i.e. exactly the ones the MFMAs multiply (four independent partial sums).
    // The scores stay in sacc, so that the exact path below can start over from them.
    float lsum[4];
    auto weights = [&]() {
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        typedef S s8 __attribute__((ext_vector_type(8)));
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          s8 v;
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            const float x = sacc[sb][8 * hh + k];
            v[k] = (S)(PRE ? __builtin_amdgcn_exp2f(x)
                           : __builtin_amdgcn_exp2f(fmaf(x, scale, -m_run)));
          }
          pb[sb][hh] = __builtin_bit_cast(uint4, v);
          lsum[2 * sb + hh] = sum8<S>(pb[sb][hh], 0.f);
        }
      }
    };
    // The exponent base moves only when a maximum outgrows it by more than 8 (log2):
    // weights stay <= 2^8 and rescales of O are rare.  After the first tile the weights
    // are taken against the current base straight away, and the row maximum is computed
    // only if some lane's packed row sum reaches 2^8: a weight above 2^8 rounds to at
    // least 2^8 in 16 bits and no sum of non-negative weights is smaller than any of
    // them, so every tile that needs a new base takes the exact path, which decides as
    // if there were no shortcut (the results are the same bit for bit).
    bool exact = t == 0;
    if (!exact) {
      weights();
      exact = __ballot((lsum[0] + lsum[1]) + (lsum[2] + lsum[3]) >= 256.0f) != 0;
    }
    if (exact) {
      // (four independent chains of three-input maxima, not one chain of 16)
      float mq[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x16& sq = sacc[q >> 1];
        const int o = 8 * (q & 1);
        mq[q] = fmaxf(sq[o], sq[o + 1]);
#pragma unroll
        for (int r = 2; r < 8; r += 2) mq[q] = fmaxf(fmaxf(mq[q], sq[o + r]), sq[o + r + 1]);
      }
      const float mraw = fmaxf(fmaxf(mq[0], mq[1]), fmaxf(mq[2], mq[3]));
      float mx = fmaxf(m_run, PRE ? mraw + c0 : mraw * scale);
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                       false, false);
      mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
      if (__ballot(mx > m_run + 8.0f)) {
        const float alpha = __builtin_amdgcn_exp2f(m_run - mx);
        l_run *= alpha;
#pragma unroll
        for (int ob = 0; ob < OB; ++ob)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[ob][r] *= alpha;
        if constexpr (PRE) {
          const float shift = mx - c0;
#pragma unroll
          for (int sb = 0; sb < 2; ++sb)
#pragma unroll
            for (int r = 0; r < 16; ++r) sacc[sb][r] -= shift;
          c0 = mx;
#pragma unroll
          for (int r = 0; r < 16; ++r) cneg[r] = -mx;
        }
        m_run = mx;
      }
      weights();
    }
    l_run += (lsum[0] + lsum[1]) + (lsum[2] + lsum[3]);
  };

  // ---- prologue.  The ring starts at zero: LDS holds whatever the previous workgroup
  // left, a range-checked load need not write the bytes of its out-of-range lanes, and a
  // zero weight times a stale NaN would not be zero.  Then every wave loads its share of
  // tiles 0 and 1 (later tiles are issued after M(t)); tile 0 complete at barrier 0.
  for (int k = tid; k < PP_STAGES * STAGE / 16; k += NW * 64) smem[k] = make_uint4(0, 0, 0, 0);
  __syncthreads();
  issue(0);
  issue(1);
  wait_tile(0);
  __syncthreads();
  sfor<0, RING>([&](auto J) { vpre[J()] = v_frag(stage_off(0), J()); });
  if (trail) __syncthreads();                 // group B: one interval behind

  for (int t = 0; t < n_tiles; ++t) {
    // ---- M(t), then this wave's share of tile t + 2
    if (t <= wlast + 1) mphase(t);
    issue(t + 2);
    if (trail) wait_tile(t + 1);
    __syncthreads();
    // ---- V(t)
    if (t <= wlast) vphase(t);
    if (!trail) wait_tile(t + 1);
    __syncthreads();
  }
  // ---- M(n): the last PV
  if (n_tiles <= wlast + 1) mphase(n_tiles);
  __syncthreads();
  if (!trail) __syncthreads();                // group A: matches group B's extra barrier
  wait_vm<0>();                               // no DMA into this LDS after the workgroup

  // ---- normalise and write O (lane: query, features ob*32 + (r/4)*8 + 4*lhalf + r%4)
  {
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l_run),
                                                     __float_as_uint(l_run), false, false);
    const float l_tot = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
    if (my_q < q_hi) {
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
  // (the ping-pong form needs enough MFMA work per tile to cover the softmax: head size 128;
  // its buffer loads address one layer's Q|K rows with 32-bit byte offsets)
  if constexpr (sizeof(S) == 2 && HD == 128) {
    if ((int64_t)p.T * (p.d + p.dkv) * (int64_t)sizeof(S) < (int64_t)UINT32_MAX) {
      if (p.q_prescaled)
        hipLaunchKernelGGL((attn_pp_kernel<S, HD, true>), grid, dim3(512), 0, s, p);
      else
        hipLaunchKernelGGL((attn_pp_kernel<S, HD, false>), grid, dim3(512), 0, s, p);
      return;
    }
  }
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
  p.n = a.n; p.T = a.T; p.d = a.d; p.n_heads = a.n_heads; p.ldv = vt_ld(a.T);
  p.num_seqs = a.num_seqs;
  const int hd = a.d / a.n_heads;
  const int kvh = a.n_kv_heads > 0 ? a.n_kv_heads : a.n_heads;
  if (a.n_heads % kvh != 0) return hipErrorInvalidValue;
  p.dkv = kvh * hd;
  p.group = a.n_heads / kvh;
  p.q_prescaled = a.q_prescaled ? 1 : 0;
  p.scale_log2 =
      a.q_prescaled ? 1.0f : (float)(1.4426950408889634 / __builtin_sqrt((double)hd));
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
