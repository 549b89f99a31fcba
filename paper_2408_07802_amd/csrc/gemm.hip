// Batched MFMA GEMM with fused epilogues for the Kraken projections
// (QKV, output projection, FFN up/down, W_concat).
//
//   C[z][m][n] = epi( sum_g sum_k A[z][g][m][k] * B[z][g mod gBmod][n][k] )
//
// Both operands are K-contiguous ("A B^T"): activations are [tokens][features]
// and weights are stored [out][in] after the one-time repack at load, so every
// MFMA operand fragment is one 16-byte LDS read.  The batch index z runs over
// the N sub-layers of a Kraken layer (Section 3.1: N independent sub-layers of
// width d), so one launch covers a whole layer's projection.
//
// Tiling (gfx950): a workgroup of 4 waves (2 x 2) computes a BM x BN tile
// (256 x 256, 128 x 128 or 128 x 64); each wave owns a (BM/2) x (BN/2) sub-tile of 32x32
// MFMA blocks (v_mfma_f32_32x32x16_{bf16,f16} for 16-bit operands,
// v_mfma_f32_32x32x2_f32 for fp32).  K advances in 128-byte slices (64 16-bit or
// 32 fp32 elements).  Operand tiles go from HBM straight into LDS with
// global_load_lds_dwordx4 (no register staging) into a ring of five operand-tile slots
// (the whole 160 KB LDS at 256 x 256): while the MFMAs consume slice s, the B tile of
// slice s+1 and the A tile of slice s+2 are loading, so A tiles get two slices of
// MFMAs to arrive and B tiles one.  Tile rows are 128 bytes; 16-byte chunk c of row r
// is stored at chunk c ^ swz_key(r), which keeps fragment reads free of bank conflicts.
// The swizzle is applied on the load side: each lane of a DMA load writes the next 16
// bytes of LDS, so it fetches the logical chunk that belongs there.  The main loop's
// instruction order is fixed by hand (fragment reads and DMAs interleaved one per MFMA,
// one barrier per slice) so that the single wave per SIMD keeps the matrix pipe busy.
// Rows past M (or N) load a clamped in-bounds row; they only feed outputs that
// are never stored.
#include <type_traits>

#include "kraken_internal.hpp"

namespace kraken {
namespace {

struct GemmParams {
  const void* A;
  const void* B;
  void* C;
  const float* bias;
  const float* R;
  int M, N, K;
  int lda, ldb, ldc;
  int64_t sA, sB, sC, sR, sBias;
  int kgroups;
  int64_t gA, gB;
  int gBmod;
  int tiles_m, tiles_n, batch;
  int xshare;              // XCDs that work through the same tile groups together (1, 2, 4, 8)
  int* ovf;                // fp16 outputs: overflow flag (NULL: not checked)
};

// GELU(v) = v Phi(v) with Phi the standard normal CDF.  With h = Phi(-|v|) this is
// max(v, 0) - |v| h for either sign of v (v >= 0: v (1 - h); v < 0: v h).  h =
// erfc(x) / 2 at x = |v| / sqrt 2, from Abramowitz & Stegun, Handbook of Mathematical
// Functions, formula 7.1.26: for x >= 0,
//   erfc(x) = (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-x^2),  t = 1 / (1 + p x),
// within 1.5e-7 absolute, so the GELU error is below 1e-7 |v|.  The halving is folded
// into the coefficients and exp(-x^2) = exp2(-v^2 log2(e) / 2): eleven VALU operations
// and two transcendentals per value.
__device__ __forceinline__ float gelu_erf(float v) {
  const float a = fabsf(v);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f * 0.70710678118654752f, a, 1.0f));
  float poly = 0.5f * 1.061405429f;
  poly = fmaf(poly, t, 0.5f * -1.453152027f);
  poly = fmaf(poly, t, 0.5f * 1.421413741f);
  poly = fmaf(poly, t, 0.5f * -0.284496736f);
  poly = fmaf(poly, t, 0.5f * 0.254829592f);
  poly *= t;
  const float e = __builtin_amdgcn_exp2f(v * (v * -0.72134752044448170f));
  return fmaf(-a, poly * e, fmaxf(v, 0.0f));
}

template <typename S>
__device__ __forceinline__ void store_val(S* p, float v) {
  *p = static_cast<S>(v);
}

// fp16 overflow check of the epilogues: a value of magnitude >= 65520 rounds (to nearest
// even) to an fp16 infinity.  amax tracks the largest magnitude a thread stores; at the end
// one lane of each wave that saw an overflow sets the flag with a vector store.
constexpr float F16_OVERFLOW = 65520.0f;
template <typename OutT>
__device__ __forceinline__ void track4(float& amax, float4 v) {
  if constexpr (__is_same(OutT, f16))
    amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v.x), fabsf(v.y)), fmaxf(fabsf(v.z), fabsf(v.w))));
}
template <typename OutT>
__device__ __forceinline__ void flag_overflow(float amax, int* ovf) {
  if constexpr (__is_same(OutT, f16)) {
    if (ovf && __ballot(!(amax < F16_OVERFLOW)) && (threadIdx.x & 63) == 0) *ovf = 1;
  }
}

// Four consecutive outputs of a row segment, stored non-temporally: a tile's outputs are
// written once and read by a later kernel, and streaming stores keep the burst of every
// workgroup's epilogue from evicting the operands the other tiles are still reading
// (measured: Q,K projection -8%, output projection -6% of kernel time).
typedef float f32v4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32v2 __attribute__((ext_vector_type(2)));
template <typename S>
__device__ __forceinline__ void store4(S* p, float4 v);
template <>
__device__ __forceinline__ void store4<float>(float* p, float4 v) {
  const f32v4 w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, reinterpret_cast<f32v4*>(p));
}
template <>
__device__ __forceinline__ void store4<bf16>(bf16* p, float4 v) {
  bf16x4 o;
  o[0] = (bf16)v.x; o[1] = (bf16)v.y; o[2] = (bf16)v.z; o[3] = (bf16)v.w;
  __builtin_nontemporal_store(__builtin_bit_cast(u32v2, o), reinterpret_cast<u32v2*>(p));
}
template <>
__device__ __forceinline__ void store4<f16>(f16* p, float4 v) {
  f16x4 o;
  o[0] = (f16)v.x; o[1] = (f16)v.y; o[2] = (f16)v.z; o[3] = (f16)v.w;
  __builtin_nontemporal_store(__builtin_bit_cast(u32v2, o), reinterpret_cast<u32v2*>(p));
}

// Swizzle of 16-byte chunks inside a 128-byte tile row: logical chunk k of row r sits at
// physical chunk k ^ swz_key(r).  The key mixes bit 3 of the row into bits 0-2 so that the
// 16 rows one ds_read_b128 serves per LDS cycle cover all 64 banks exactly once (rows r and
// r + 8 would collide under the plain r & 7).
__device__ __forceinline__ int swz_key(int row) { return (row ^ (row >> 3)) & 7; }

template <int N>
using I = std::integral_constant<int, N>;

// Compile-time loop: f(I<B>{}), f(I<B+1>{}), ..., f(I<E-1>{}).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(I<B>{});
    static_for<B + 1, E>(f);
  }
}

// MFMA slot (in [lo, hi)) that item k of n evenly spread items issues after.
__host__ __device__ constexpr int spread_slot(int k, int n, int lo, int hi) {
  return lo + (k * (hi - lo)) / n;
}

typedef __attribute__((address_space(3))) void* lds_void_ptr;

// One 16-byte-per-lane DMA from global memory into LDS: global_load_lds_dwordx4 with a
// wave-uniform base address (SGPR pair), a per-lane 32-bit byte offset, and the
// wave-uniform LDS destination in M0; lane i's 16 bytes land at M0 + 16 i.  It is issued
// from inline assembly so that the compiler does not order later LDS reads of *other*
// ring slots behind it; the kernel orders it explicitly (s_waitcnt vmcnt + barrier before
// the slot is read).
__device__ __forceinline__ void dma16(uint32_t lds_addr, const void* base, uint32_t off) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
               :: "s"(lds_addr), "v"(off), "s"(base) : "memory", "m0");
}

// Raster groups of the tiled GEMM: GEMM_GROUP_M M-tiles x all N-tiles, walked M-fastest
// (measured against 8, with the XCD sharing below, on each GEMM of the N = 8, width 2048,
// 8192-token prefill alone: 1-5% faster; 16: 3% slower over the whole prefill).  The
// kernel's tile map and the host's choice of XCD sharing both use it.
constexpr int GEMM_GROUP_M = 4;

template <typename S, int BM, int BN, int EPI>
__global__ __launch_bounds__(256, 1) void gemm_kernel(GemmParams p) {
  constexpr int NT = 256;
  constexpr int CH = 8;                        // 16-byte chunks per 128-byte row
  constexpr int EPC = 16 / sizeof(S);          // elements per chunk
  constexpr int BK = CH * EPC;                 // K elements per slice
  constexpr int TM = BM / 2, TN = BN / 2;      // wave tile
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int AI = BM / 32, BI = BN / 32;    // DMA instructions per wave per slice
  constexpr int SLOT = (BM > BN ? BM : BN) * CH;  // uint4 per ring slot (one operand tile)
  constexpr int NSLOT = 5;                     // ring slots: 2.5 slices of A and B tiles
  constexpr int NCH = CH / 2;                  // 16-byte-per-lane K chunks per slice
  constexpr int NM = FM * FN;                  // MFMA blocks per chunk
  constexpr int NR = FM + FN;                  // fragment reads per chunk
  constexpr int BAR = NM * 3 / 4;              // last-chunk MFMA slot of the barrier
  static_assert(NCH == 4 && BAR < NM, "schedule slots out of range");
  static_assert(AI == 4 || AI == 8, "vmcnt immediates below cover 4 or 8 A DMAs");

  __shared__ uint4 lds[NSLOT * SLOT];

  // ---- tile scheduling: XCD-aware remap, then grouped raster inside a batch entry
  constexpr int GROUP_M = GEMM_GROUP_M;
  const int tiles_per_batch = p.tiles_m * p.tiles_n;
  const int total = tiles_per_batch * p.batch;
  const int group_sz = GROUP_M * p.tiles_n;
  // Workgroup b runs on XCD b % 8.  Each XCD takes 1/8 of the tiles: with xshare = 1 a
  // contiguous range; with xshare = S > 1 the XCDs form groups of S that share S
  // contiguous ranges, the members taking consecutive raster groups in turn, so that S
  // XCDs stream the same B panels (a batch entry's weights) at the same time and all but
  // one of them find them in the chip's shared cache.  (The host picks S > 1 only when an
  // XCD's share is a whole number of raster groups, which keeps the map a permutation.)
  int pid = blockIdx.x;
  if ((total & 7) == 0) {
    const int x = pid & 7, l = pid >> 3, per_xcd = total >> 3;
    if (p.xshare > 1) {
      const int q = x / p.xshare, h = x - q * p.xshare;
      const int u = l / group_sz, o = l - u * group_sz;
      pid = q * p.xshare * per_xcd + (u * p.xshare + h) * group_sz + o;
    } else {
      pid = x * per_xcd + l;
    }
  }
  pid = __builtin_amdgcn_readfirstlane(pid);   // (uniform: keeps the tile's bases scalar)
  const int z = pid / tiles_per_batch;
  const int t = pid - z * tiles_per_batch;
  const int gid = t / group_sz;
  const int first_m = gid * GROUP_M;
  const int gm = min(p.tiles_m - first_m, GROUP_M);
  const int tm = first_m + (t % group_sz) % gm;
  const int tn = (t % group_sz) / gm;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int lrow = lane & 31, lhalf = lane >> 5;

  // The epilogue's bias: one value per thread (tile column n0 + tid, or tile row m0 + tid
  // for the row bias), loaded before the main loop so that its latency is hidden there,
  // and parked in LDS once the loop is done.  (Loaded inside the epilogue, every load
  // would wait for the memory pipe, including the stores already issued.)
  constexpr int NB = (EPI == EPI_BIAS_M) ? BM : BN;
  float bias_v = 0.f;
  {
    const int idx = (EPI == EPI_BIAS_M ? m0 : n0) + tid;
    const int lim = EPI == EPI_BIAS_M ? p.M : p.N;
    if (p.bias && tid < NB && idx < lim) bias_v = p.bias[z * p.sBias + idx];
  }

  const S* Az = static_cast<const S*>(p.A) + z * p.sA;
  const S* Bz = static_cast<const S*>(p.B) + z * p.sB;

  // DMA: wave loads rows [wave*BM/4, +BM/4) of the A tile (and likewise of B) in
  // instructions of 8 rows; lane writes row 8u + lane/8 of that block at physical chunk
  // lane%8, so it fetches the logical chunk that the swizzle puts there.  Byte offsets
  // from the slice's base pointer fit 32 bits (the host rejects larger operands).
  uint32_t aoff[AI], boff[BI];
#pragma unroll
  for (int u = 0; u < AI; ++u) {
    const int rl = wave * (BM / 4) + u * 8 + (lane >> 3);
    const int m = min(m0 + rl, p.M - 1);
    aoff[u] = ((uint32_t)m * (uint32_t)p.lda + (uint32_t)(((lane & 7) ^ swz_key(rl)) * EPC)) *
              (uint32_t)sizeof(S);
  }
#pragma unroll
  for (int u = 0; u < BI; ++u) {
    const int rl = wave * (BN / 4) + u * 8 + (lane >> 3);
    const int n = min(n0 + rl, p.N - 1);
    boff[u] = ((uint32_t)n * (uint32_t)p.ldb + (uint32_t)(((lane & 7) ^ swz_key(rl)) * EPC)) *
              (uint32_t)sizeof(S);
  }
  const uint32_t lds_base =
      __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_ptr)lds);
  const uint32_t a_dst = lds_base + (uint32_t)(wave * (BM / 4)) * 128u;
  const uint32_t b_dst = lds_base + (uint32_t)(wave * (BN / 4)) * 128u;

  // Sources of the next A and B slices to load, each a (K group, k offset) pair advanced
  // one slice at a time: A runs two slices ahead of the MFMAs, B one.
  const int ksl = p.K / BK;                // slices per K group
  const int nsl = ksl * p.kgroups;         // total slices
  const char* a_src = reinterpret_cast<const char*>(Az);
  const char* b_src = reinterpret_cast<const char*>(Bz);
  int a_k = 0, a_g = 0, b_k = 0, b_bg = 0;
  auto advance_a = [&]() {
    if (++a_k < ksl) {
      a_src += BK * sizeof(S);
    } else {
      a_k = 0;
      ++a_g;
      a_src = reinterpret_cast<const char*>(Az + a_g * p.gA);
    }
  };
  auto advance_b = [&]() {
    if (++b_k < ksl) {
      b_src += BK * sizeof(S);
    } else {
      b_k = 0;
      if (++b_bg == p.gBmod) b_bg = 0;
      b_src = reinterpret_cast<const char*>(Bz + b_bg * p.gB);
    }
  };
  // DMA instruction u of the current A (or B) source slice into the ring slot at byte
  // offset `slot`.
  auto dma_a = [&](uint32_t slot, auto U) {
    constexpr int u = decltype(U)::value;
    dma16(a_dst + slot + u * 1024u, a_src, aoff[u]);
  };
  auto dma_b = [&](uint32_t slot, auto U) {
    constexpr int u = decltype(U)::value;
    dma16(b_dst + slot + u * 1024u, b_src, boff[u]);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Fragment reads (uint4 index inside the ring).  Row r of an operand tile holds its
  // logical chunk k at physical chunk k ^ swz_key(r); for fragment row base + 32i + lrow
  // (base = wm*TM for A, wn*TN for B, multiples of 32) that key is
  // swz_key(lrow) ^ 4((base/32 + i) & 1).
  static_assert(TM % 32 == 0 && TN % 32 == 0, "fragment row bases");
  const int arow = (wm * TM + lrow) * CH, brow = (wn * TN + lrow) * CH;
  const int sw = swz_key(lrow);
  const int apar = (wm * (TM / 32)) & 1, bpar = (wn * (TN / 32)) & 1;
  uint4 af[2][FM], bfr[2][FN];
  // Read k of a chunk from the A tile at a_base and the B tile at b_base: 0 -> A block 0,
  // 1..FN -> B blocks, then A blocks 1..FM-1, the order in which the chunk's MFMAs (i
  // outer, j inner) first need them.
  auto read_item = [&](int a_base, int b_base, auto Cc, auto Slot, auto K) {
    constexpr int c = decltype(Cc)::value, slot = decltype(Slot)::value;
    constexpr int k = decltype(K)::value;
    constexpr bool is_a = k == 0 || k > FN;
    constexpr int idx = k == 0 ? 0 : (k <= FN ? k - 1 : k - FN);
    const int ch = ((2 * c + lhalf) ^ sw) ^ (((idx + (is_a ? apar : bpar)) & 1) * 4);
    if constexpr (is_a)
      af[slot][idx] = lds[a_base + arow + idx * 32 * CH + ch];
    else
      bfr[slot][idx] = lds[b_base + brow + idx * 32 * CH + ch];
  };
  auto wrap = [](int x) { return x >= NSLOT ? x - NSLOT : x; };

  // Ring: the A tile of slice s sits in slot 2s mod 5 and its B tile in slot 2s+1 mod 5.
  // While slice s is multiplied, slices s+1 (A loaded, B loading) and the A tile of s+2
  // (loading) occupy three more slots; the two slots of slice s-1 were freed by the
  // barrier that ended it.  So an A tile has two slices of MFMAs to arrive, a B tile
  // one; the B DMAs go out first in the slice.
  // Prologue: A0, B0 and A1 into slots 0, 1, 2, then the fragments of slice 0's first
  // chunk (loads complete in issue order, so vmcnt(AI) leaves only A1 in flight).
  static_for<0, AI>([&](auto U) { dma_a(0u, U); });
  advance_a();
  static_for<0, BI>([&](auto U) { dma_b((uint32_t)SLOT * 16u, U); });
  advance_b();
  if (nsl > 1) {
    static_for<0, AI>([&](auto U) { dma_a(2u * SLOT * 16u, U); });
    advance_a();
    if constexpr (AI == 8)
      asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
    else
      asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  } else {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
  __syncthreads();
  static_for<0, NR>([&](auto K) { read_item(0, SLOT, I<0>{}, I<0>{}, K); });

  // One slice: NCH chunks of NM MFMAs each.  The instruction order is fixed (a scheduling
  // fence after every MFMA slot) so that every non-MFMA instruction issues in the shadow
  // of a running MFMA:
  //   chunk c < NCH-1: the next chunk's NR fragment reads over the first NM/2 MFMAs;
  //   chunk 0 (MODE >= 1): the BI DMAs of B(s+1), evenly spread;
  //   chunks 1 and 2 (MODE 2): the AI DMAs of A(s+2), evenly spread;
  //   last chunk (MODE >= 1): after MFMA BAR the wave waits for its DMAs of A(s+1) and
  //     B(s+1) (not those of A(s+2)) and meets the others at the barrier (slice s+1 is
  //     then in LDS and nobody reads slice s any more), and the reads of slice s+1's
  //     first chunk go out over the remaining MFMAs.
  // MODE 2: slices with an A(s+2); 1: the second-to-last slice; 0: the last.
  int sa = 0;                                  // ring slot of the current A tile
  auto slice = [&](auto Mode) {
    constexpr int MODE = decltype(Mode)::value;
    const int a_cur = sa * SLOT, b_cur = wrap(sa + 1) * SLOT;
    const int a_nxt = wrap(sa + 2) * SLOT, b_nxt = wrap(sa + 3) * SLOT;
    const uint32_t b_load = (uint32_t)b_nxt * 16u;
    const uint32_t a_load = (uint32_t)(wrap(sa + 4) * SLOT) * 16u;
    static_for<0, NCH>([&](auto Cc) {
      constexpr int c = decltype(Cc)::value;
      constexpr int slot = c & 1;
      static_for<0, NM>([&](auto T) {
        constexpr int t = decltype(T)::value;
        constexpr int i = t / FN, j = t % FN;
        acc[i][j] = mfma_chunk<S>(af[slot][i], bfr[slot][j], acc[i][j]);
        if constexpr (c + 1 < NCH) {
          static_for<0, NR>([&](auto K) {
            if constexpr (spread_slot(decltype(K)::value, NR, 0, NM / 2) == t)
              read_item(a_cur, b_cur, I<c + 1>{}, I<slot ^ 1>{}, K);
          });
        }
        if constexpr (MODE >= 1 && c == 0) {
          static_for<0, BI>([&](auto U) {
            if constexpr (spread_slot(decltype(U)::value, BI, 0, NM) == t) dma_b(b_load, U);
          });
          if constexpr (t == NM - 1) advance_b();
        }
        if constexpr (MODE == 2 && (c == 1 || c == 2)) {
          static_for<0, AI>([&](auto U) {
            if constexpr (spread_slot(decltype(U)::value, AI, NM, 3 * NM) == c * NM + t)
              dma_a(a_load, U);
          });
          if constexpr (c == 2 && t == NM - 1) advance_a();
        }
        if constexpr (MODE >= 1 && c + 1 == NCH) {
          if constexpr (t == BAR) {
            if constexpr (MODE == 1)
              asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            else if constexpr (AI == 8)
              asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
            else
              asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
            __syncthreads();
          }
          static_for<0, NR>([&](auto K) {
            if constexpr (spread_slot(decltype(K)::value, NR, BAR, NM) == t)
              read_item(a_nxt, b_nxt, I<0>{}, I<slot ^ 1>{}, K);
          });
        }
        __builtin_amdgcn_sched_barrier(0);
      });
    });
    sa = wrap(sa + 2);
  };
  for (int s = 0; s + 2 < nsl; ++s) slice(I<2>{});
  if (nsl >= 2) slice(I<1>{});
  slice(I<0>{});
  __syncthreads();
  // bias table: the last NB floats of LDS, clear of the epilogue's staging rows
  float* const btab = reinterpret_cast<float*>(lds) + (NSLOT * SLOT * 4 - NB);
  if (tid < NB) btab[tid] = bias_v;
  __syncthreads();

  // ---- epilogue.  Each wave stages one 32-row block of its tile at a time through its
  // own quarter of the (now idle) LDS ring: the MFMA layout (lane = column, 16 rows per
  // lane) is written out as fp32 rows, then read back four consecutive columns per lane
  // so that global stores (and residual loads) are 16-byte-per-lane row segments.  The
  // residual segments go through a two-deep register ring of half blocks: the loads of
  // half block g + 2 are issued as soon as half block g is stored, so their latency
  // overlaps the following stores and staging.  The row bias of the transposed
  // projection is added after the read-back, once per 4-column segment.
  using OutT = typename std::conditional<EPI == EPI_BIAS_N_RES, float, S>::type;
  constexpr int RS = TN + 4;                           // staged row stride (floats)
  constexpr int QN = 32 * TN / 256;                    // 4-column segments per lane per block
  static_assert(32 * RS * 4 * 4 <= (int)sizeof(lds), "epilogue staging exceeds LDS");
  float* stage = reinterpret_cast<float*>(lds) + wave * 32 * RS;
  static_assert(4 * 32 * RS <= NSLOT * SLOT * 4 - NB, "staging rows overlap the bias table");
  const float* Rz = p.R ? p.R + z * p.sR : nullptr;
  OutT* Cz = static_cast<OutT*>(p.C) + z * p.sC;
  const bool vec_ok = (p.ldc & 3) == 0;
  float amax = 0.f;                                    // fp16 outputs: largest |value|
  // the whole tile inside C, with 16-byte-aligned row segments (uniform per workgroup)
  const bool interior = vec_ok && m0 + BM <= p.M && n0 + BN <= p.N;
  const int rows0 = m0 + wm * TM, cols0 = n0 + wn * TN;
  // segment q of block i: row ml, columns nl .. nl + 3 of the wave's sub-tile
  auto seg_ml = [&](int q) { return (q * 64 + lane) / (TN / 4); };
  auto seg_nl = [&](int q) { return ((q * 64 + lane) % (TN / 4)) * 4; };
  constexpr int QH = QN / 2;                           // segments per half block
  float4 rbuf[2][QH];
  auto load_res = [&](int g, float4* dst) {            // half block g = 2 i + h
#pragma unroll
    for (int qq = 0; qq < QH; ++qq) {
      const int q = (g & 1) * QH + qq;
      const int m = rows0 + (g >> 1) * 32 + seg_ml(q), n = cols0 + seg_nl(q);
      dst[qq] = (Rz && vec_ok && m < p.M && n + 3 < p.N)
                    ? *reinterpret_cast<const float4*>(Rz + (int64_t)m * p.ldc + n)
                    : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  if constexpr (EPI == EPI_BIAS_N_RES) {
    load_res(0, rbuf[0]);
    load_res(1, rbuf[1]);
  }
  float bnj[FN];                                       // column bias of the lane's columns
#pragma unroll
  for (int j = 0; j < FN; ++j) bnj[j] = (EPI != EPI_BIAS_M) ? btab[wn * TN + j * 32 + lrow] : 0.f;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int nl = j * 32 + lrow;
      const float bn = bnj[j];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ml = (r >> 2) * 8 + lhalf * 4 + (r & 3);
        float v = acc[i][j][r] + bn;
        if constexpr (EPI == EPI_BIAS_N_GELU) v = gelu_erf(v);
        stage[ml * RS + nl] = v;
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);      // lgkmcnt(0): this wave's LDS writes are done
    __builtin_amdgcn_wave_barrier();
    if (interior) {
      // No edge checks: each half block's QH staged segments are read back to back, so
      // the LDS latency is paid once per half block rather than once per segment.
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        if constexpr (EPI == EPI_BIAS_N_RES) {
          if (hb == 1 && 2 * i + 2 < 2 * FM) load_res(2 * i + 2, rbuf[0]);
        }
        float4 vq[QH];
        float bmq[QH];
#pragma unroll
        for (int qq = 0; qq < QH; ++qq) {
          const int q = hb * QH + qq;
          vq[qq] = *reinterpret_cast<const float4*>(stage + seg_ml(q) * RS + seg_nl(q));
          if constexpr (EPI == EPI_BIAS_M) bmq[qq] = btab[wm * TM + i * 32 + seg_ml(q)];
        }
#pragma unroll
        for (int qq = 0; qq < QH; ++qq) {
          const int q = hb * QH + qq;
          float4 v = vq[qq];
          if constexpr (EPI == EPI_BIAS_M) {
            v.x += bmq[qq]; v.y += bmq[qq]; v.z += bmq[qq]; v.w += bmq[qq];
          }
          if constexpr (EPI == EPI_BIAS_N_RES) {
            const float4 rr = rbuf[hb][qq];
            v.x += rr.x; v.y += rr.y; v.z += rr.z; v.w += rr.w;
          }
          const int m = rows0 + i * 32 + seg_ml(q), n = cols0 + seg_nl(q);
          track4<OutT>(amax, v);
          store4<OutT>(Cz + (int64_t)m * p.ldc + n, v);
        }
      }
    } else {
#pragma unroll
    for (int q = 0; q < QN; ++q) {
      if constexpr (EPI == EPI_BIAS_N_RES) {
        // half block 2i + h - 1 is fully stored: refill its ring slot two halves ahead
        if (q == QH && 2 * i + 2 < 2 * FM) load_res(2 * i + 2, rbuf[0]);
      }
      const int ml = seg_ml(q), nl = seg_nl(q);
      const int m = rows0 + i * 32 + ml, n = cols0 + nl;
      if (m >= p.M) continue;
      float4 v = *reinterpret_cast<const float4*>(stage + ml * RS + nl);
      if constexpr (EPI == EPI_BIAS_M) {
        const float bm = btab[wm * TM + i * 32 + ml];
        v.x += bm; v.y += bm; v.z += bm; v.w += bm;
      }
      OutT* dst = Cz + (int64_t)m * p.ldc + n;
      if (vec_ok && n + 3 < p.N) {
        if constexpr (EPI == EPI_BIAS_N_RES) {
          const float4 rr = rbuf[q / QH][q % QH];
          v.x += rr.x; v.y += rr.y; v.z += rr.z; v.w += rr.w;
        }
        track4<OutT>(amax, v);
        store4<OutT>(dst, v);
      } else {
        const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (n + k >= p.N) break;
          float o = vv[k];
          if constexpr (EPI == EPI_BIAS_N_RES) {
            if (Rz) o += Rz[(int64_t)m * p.ldc + n + k];
          }
          track4<OutT>(amax, make_float4(o, 0.f, 0.f, 0.f));
          store_val<OutT>(dst + k, o);
        }
      }
    }
    }
    if constexpr (EPI == EPI_BIAS_N_RES) {
      if (2 * i + 3 < 2 * FM) load_res(2 * i + 3, rbuf[1]);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
  }
  flag_overflow<OutT>(amax, p.ovf);
}

// XCD sharing of the tile raster (see the kernel): groups of four XCDs, when an XCD's 1/8
// of the tiles is a whole number of raster groups.  Measured on the FFN up projection of
// N = 8 sub-layers of width 2048 at 8192 tokens (8192 tiles): 4% faster than one XCD per
// sub-layer, the whole prefill 1.5-1.9% faster (groups of 2 and 8: 1.2-1.6%).
inline int gemm_xshare(int64_t total, int64_t group_sz) {
  return (total % 8 == 0 && (total / 8) % group_sz == 0) ? 4 : 1;
}

template <typename S, int BM, int BN>
hipError_t launch_cfg(const GemmDesc& g, hipStream_t s) {
  GemmParams p;
  p.A = g.A; p.B = g.B; p.C = g.C; p.bias = g.bias; p.R = g.R;
  p.M = g.M; p.N = g.N; p.K = g.K;
  p.lda = g.lda; p.ldb = g.ldb; p.ldc = g.ldc;
  p.sA = g.sA; p.sB = g.sB; p.sC = g.sC; p.sR = g.sR; p.sBias = g.sBias;
  p.kgroups = g.kgroups; p.gA = g.gA; p.gB = g.gB; p.gBmod = g.gBmod;
  p.tiles_m = (g.M + BM - 1) / BM;
  p.tiles_n = (g.N + BN - 1) / BN;
  p.batch = g.batch;
  p.ovf = g.ovf;
  const int64_t total = (int64_t)p.tiles_m * p.tiles_n * p.batch;
  p.xshare = gemm_xshare(total, (int64_t)GEMM_GROUP_M * p.tiles_n);
  dim3 grid((unsigned)total), block(256);
  switch (g.epi) {
    case EPI_BIAS_N:
      hipLaunchKernelGGL((gemm_kernel<S, BM, BN, EPI_BIAS_N>), grid, block, 0, s, p);
      break;
    case EPI_BIAS_N_GELU:
      hipLaunchKernelGGL((gemm_kernel<S, BM, BN, EPI_BIAS_N_GELU>), grid, block, 0, s, p);
      break;
    case EPI_BIAS_N_RES:
      hipLaunchKernelGGL((gemm_kernel<S, BM, BN, EPI_BIAS_N_RES>), grid, block, 0, s, p);
      break;
    case EPI_BIAS_M:
      hipLaunchKernelGGL((gemm_kernel<S, BM, BN, EPI_BIAS_M>), grid, block, 0, s, p);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ----------------------------------------------------------------------------- few rows
//
// GEMM for a few rows of A (M <= 64: the tokens of a decode step).  Then every weight
// element is used at most 64 times and the kernel is bound by streaming B (the weights)
// from HBM once, so the tiling is chosen for parallelism: a workgroup owns TW blocks of
// 16 output columns of one batch entry and all M rows, and its 4 waves split the
// (kgroups x K) reduction into 4 contiguous ranges, merged through LDS at the end.  Each
// step of 32 k is one v_mfma_f32_16x16x32 per (16-row block of A, column block): lane l
// supplies B column l % 16 and A row l % 16, k = 8 (l / 16) .. + 7 (one 16-byte load
// each), and gets D rows 4 (l / 16) .. + 3 of column l % 16.  A rows past M load row
// M - 1 and are masked to zero (whole 16-byte loads without branches: per-lane
// conditional loads compile to four 4-byte loads each and halved the throughput at 8
// rows); B columns past N load a clamped row and are not stored.
template <typename S>
__device__ __forceinline__ f32x4 mfma16(uint4 a, uint4 b, f32x4 c) {
  if constexpr (__is_same(S, bf16)) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  }
}

constexpr int SK_UNROLL = 8;   // steps of 32 k whose loads are issued together

// 16-byte weight load (plain: non-temporal loads measured the same, within 3%, on weight
// streams that do not fit the last-level cache).
__device__ __forceinline__ uint4 load_w16(const void* ptr) {
  return *reinterpret_cast<const uint4*>(ptr);
}

template <typename S, int MB, int TW, int EPI>
__global__ __launch_bounds__(256) void gemm_skinny_kernel(GemmParams p) {
  __shared__ float red[4][MB * TW][256];
  using OutT = std::conditional_t<EPI == EPI_BIAS_N_RES, float, S>;
  const int z = blockIdx.y;
  const int n0 = blockIdx.x * 16 * TW;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, kq = lane >> 4;
  const S* Bz[TW];
#pragma unroll
  for (int w = 0; w < TW; ++w)
    Bz[w] = static_cast<const S*>(p.B) + z * p.sB +
            (int64_t)min(n0 + w * 16 + col, p.N - 1) * p.ldb + kq * 8;
  // A rows past M load row M - 1 (whole 16-byte loads, no branches) and are masked to 0
  const S* Az[MB];
  uint32_t amask[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = mb * 16 + col;
    amask[mb] = m < p.M ? 0xffffffffu : 0u;
    Az[mb] = static_cast<const S*>(p.A) + z * p.sA + (int64_t)min(m, p.M - 1) * p.lda + kq * 8;
  }
  auto load_a = [&](int mb, int64_t off) {
    uint4 v = *reinterpret_cast<const uint4*>(Az[mb] + off);
    v.x &= amask[mb]; v.y &= amask[mb]; v.z &= amask[mb]; v.w &= amask[mb];
    return v;
  };
  const int steps_per_group = p.K / 32;
  const int steps = steps_per_group * p.kgroups;
  const int t0 = (int)((int64_t)steps * wave / 4), t1 = (int)((int64_t)steps * (wave + 1) / 4);
  f32x4 acc[MB * TW];
#pragma unroll
  for (int q = 0; q < MB * TW; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
  // step t covers k = 32 (t mod steps_per_group) .. + 31 of group g = t / steps_per_group;
  // (g, kk) is tracked incrementally from this wave's first step
  int g = t0 / steps_per_group, kk = (t0 - g * steps_per_group) * 32;
  int gb = g % p.gBmod;
  auto advance = [&]() {
    kk += 32;
    if (kk == p.K) {
      kk = 0;
      ++g;
      if (++gb == p.gBmod) gb = 0;
    }
  };
  int t = t0;
  for (; t + SK_UNROLL <= t1; t += SK_UNROLL) {
    uint4 bv[SK_UNROLL][TW], av[SK_UNROLL][MB];
    int64_t ao[SK_UNROLL], bo[SK_UNROLL];
#pragma unroll
    for (int u = 0; u < SK_UNROLL; ++u) {
      ao[u] = g * p.gA + kk;
      bo[u] = gb * p.gB + kk;
      advance();
    }
#pragma unroll
    for (int u = 0; u < SK_UNROLL; ++u)
#pragma unroll
      for (int w = 0; w < TW; ++w) bv[u][w] = load_w16(Bz[w] + bo[u]);
#pragma unroll
    for (int u = 0; u < SK_UNROLL; ++u)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        av[u][mb] = load_a(mb, ao[u]);
#pragma unroll
    for (int u = 0; u < SK_UNROLL; ++u)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int w = 0; w < TW; ++w)
          acc[mb * TW + w] = mfma16<S>(av[u][mb], bv[u][w], acc[mb * TW + w]);
  }
  for (; t < t1; ++t) {
    uint4 bv[TW];
#pragma unroll
    for (int w = 0; w < TW; ++w) bv[w] = load_w16(Bz[w] + gb * p.gB + kk);
    const int64_t ao = g * p.gA + kk;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const uint4 av = load_a(mb, ao);
#pragma unroll
      for (int w = 0; w < TW; ++w) acc[mb * TW + w] = mfma16<S>(av, bv[w], acc[mb * TW + w]);
    }
    advance();
  }
  // D row 4 kq + j, column col of each 16-row block -> red[wave][mb][row * 16 + col]
#pragma unroll
  for (int q = 0; q < MB * TW; ++q)
#pragma unroll
    for (int j = 0; j < 4; ++j) red[wave][q][(kq * 4 + j) * 16 + col] = acc[q][j];
  __syncthreads();
  const int tid = threadIdx.x;
  const float* biasz = p.bias ? p.bias + z * p.sBias : nullptr;
  float amax = 0.f;
#pragma unroll
  for (int w = 0; w < TW; ++w) {
    const int n = n0 + w * 16 + (tid & 15);
    if (n >= p.N) continue;
    const float bn = biasz ? biasz[n] : 0.f;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int m = mb * 16 + (tid >> 4);
      if (m >= p.M) break;
      const int q = mb * TW + w;
      float v = (red[0][q][tid] + red[1][q][tid]) + (red[2][q][tid] + red[3][q][tid]) + bn;
      if constexpr (EPI == EPI_BIAS_N_GELU) v = gelu_erf(v);
      if constexpr (EPI == EPI_BIAS_N_RES) {
        if (p.R) v += p.R[z * p.sR + (int64_t)m * p.ldc + n];
      }
      track4<OutT>(amax, make_float4(v, 0.f, 0.f, 0.f));
      store_val<OutT>(static_cast<OutT*>(p.C) + z * p.sC + (int64_t)m * p.ldc + n, v);
    }
  }
  flag_overflow<OutT>(amax, p.ovf);
}

template <typename S, int MB, int TW>
hipError_t launch_skinny(const GemmDesc& g, hipStream_t s) {
  GemmParams p;
  p.A = g.A; p.B = g.B; p.C = g.C; p.bias = g.bias; p.R = g.R;
  p.M = g.M; p.N = g.N; p.K = g.K;
  p.lda = g.lda; p.ldb = g.ldb; p.ldc = g.ldc;
  p.sA = g.sA; p.sB = g.sB; p.sC = g.sC; p.sR = g.sR; p.sBias = g.sBias;
  p.kgroups = g.kgroups; p.gA = g.gA; p.gB = g.gB; p.gBmod = g.gBmod;
  p.tiles_m = 1; p.tiles_n = (g.N + 16 * TW - 1) / (16 * TW); p.batch = g.batch; p.xshare = 1;
  p.ovf = g.ovf;
  dim3 grid((unsigned)p.tiles_n, (unsigned)g.batch), block(256);
  switch (g.epi) {
    case EPI_BIAS_N:
      hipLaunchKernelGGL((gemm_skinny_kernel<S, MB, TW, EPI_BIAS_N>), grid, block, 0, s, p);
      break;
    case EPI_BIAS_N_GELU:
      hipLaunchKernelGGL((gemm_skinny_kernel<S, MB, TW, EPI_BIAS_N_GELU>), grid, block, 0, s, p);
      break;
    case EPI_BIAS_N_RES:
      hipLaunchKernelGGL((gemm_skinny_kernel<S, MB, TW, EPI_BIAS_N_RES>), grid, block, 0, s, p);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Two 16-column blocks per wave (each A fragment feeds two MFMAs, halving the A loads per
// weight byte) for several rows and reductions up to 4096; one block (twice the
// workgroups) otherwise.  Measured on the N=8, d=2048 decode projections with weights
// streamed from HBM: one row, one block 5-18% faster for every projection (FFN down 54
// against 66 us); eight rows, two blocks 4-5% faster at K = 2048, one block 5% faster at
// K = 8192.
template <typename S, int MB>
hipError_t launch_skinny_tw(const GemmDesc& g, hipStream_t s) {
  if (g.M > 1 && (int64_t)g.K * g.kgroups <= 4096) return launch_skinny<S, MB, 2>(g, s);
  return launch_skinny<S, MB, 1>(g, s);
}

template <typename S>
hipError_t launch_skinny_rows(const GemmDesc& g, hipStream_t s) {
  if (g.M <= 16) return launch_skinny_tw<S, 1>(g, s);
  if (g.M <= 32) return launch_skinny_tw<S, 2>(g, s);
  return launch_skinny_tw<S, 4>(g, s);
}

}  // namespace

hipError_t launch_gemm(const GemmDesc& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0 || g.batch <= 0 || g.kgroups <= 0) return hipSuccess;
  const int bk = g.dt == DType::F32 ? 32 : 64;
  if (g.K <= 0 || g.K % bk != 0 || g.gBmod <= 0) return hipErrorInvalidValue;
  // the kernel addresses operand rows of one batch entry / K group with 32-bit byte offsets
  const int64_t es = (int64_t)dtype_size(g.dt);
  if ((int64_t)g.M * g.lda * es >= (1ll << 31) || (int64_t)g.N * g.ldb * es >= (1ll << 31))
    return hipErrorInvalidValue;
  // a few rows of 16-bit operands (a decode step): weight streaming
  if (g.M <= 64 && g.epi != EPI_BIAS_M && g.dt != DType::F32) {
    if (g.dt == DType::BF16) return launch_skinny_rows<bf16>(g, s);
    return launch_skinny_rows<f16>(g, s);
  }
  // 256 x 256 tiles when they give at least two waves of workgroups over the 256 CUs, else
  // 128 x 128, and 128 x 64 when those leave CUs idle (a prompt of ~100-200 tokens, where
  // the projections stream their weights and need workgroups in flight; measured on the
  // 65B and 175B 4-way engine shapes at 128 tokens: 156-232 workgroups of 128 x 128 ->
  // 128 x 64 7-10% faster, 464 -> 128 x 64 40% slower).
  const int64_t big = (int64_t)((g.M + 255) / 256) * ((g.N + 255) / 256) * g.batch;
  const int64_t mid = (int64_t)((g.M + 127) / 128) * ((g.N + 127) / 128) * g.batch;
  // 256 x 256 tiles need two waves of workgroups to hide their tail, except when one
  // tile per CU fills the chip exactly and the reduction is long (the W_concat shape)
  const bool one_round = big == 256 && (int64_t)g.K * g.kgroups >= 8192;
  const int cfg = (big >= 512 || one_round) ? 2 : mid >= 256 ? 1 : 0;
  switch (g.dt) {
    case DType::BF16:
      return cfg == 2 ? launch_cfg<bf16, 256, 256>(g, s)
           : cfg == 1 ? launch_cfg<bf16, 128, 128>(g, s) : launch_cfg<bf16, 128, 64>(g, s);
    case DType::F16:
      return cfg == 2 ? launch_cfg<f16, 256, 256>(g, s)
           : cfg == 1 ? launch_cfg<f16, 128, 128>(g, s) : launch_cfg<f16, 128, 64>(g, s);
    default:
      return cfg == 2 ? launch_cfg<float, 256, 256>(g, s)
           : cfg == 1 ? launch_cfg<float, 128, 128>(g, s) : launch_cfg<float, 128, 64>(g, s);
  }
}

}  // namespace kraken
