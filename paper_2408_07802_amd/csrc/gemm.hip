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
// (256 x 256 or 128 x 128); each wave owns a (BM/2) x (BN/2) sub-tile of 32x32
// MFMA blocks (v_mfma_f32_32x32x16_{bf16,f16} for 16-bit operands,
// v_mfma_f32_32x32x2_f32 for fp32).  K advances in 128-byte slices (64 16-bit or
// 32 fp32 elements).  Operand tiles go from HBM straight into LDS with
// global_load_lds_dwordx4 (no register staging) into the other half of a
// double-buffered LDS ring while the MFMAs consume the current half.  Tile rows
// are 128 bytes; 16-byte chunk c of row r is stored at chunk c ^ (r & 7), so the
// 8 lanes that read one chunk column of 8 consecutive rows hit distinct banks.
// The swizzle is applied on the load side: each lane of a DMA load writes the
// next 16 bytes of LDS, so it fetches the logical chunk that belongs there.
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
};

// GELU(v) = v/2 (1 + erf(v / sqrt 2)) with erf from Abramowitz & Stegun, Handbook of
// Mathematical Functions, formula 7.1.26: for x >= 0,
//   erf(x) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) exp(-x^2),  t = 1 / (1 + p x),
// |error| <= 1.5e-7; erf is odd.  GELU only needs erf to an absolute accuracy (it enters
// as 1 + erf), so the GELU error is below 1e-7 |v|.
__device__ __forceinline__ float gelu_erf(float v) {
  const float x = fabsf(v) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(1.0f + 0.3275911f * x);
  float poly = 1.061405429f;
  poly = poly * t - 1.453152027f;
  poly = poly * t + 1.421413741f;
  poly = poly * t - 0.284496736f;
  poly = poly * t + 0.254829592f;
  poly *= t;
  const float e = __builtin_amdgcn_exp2f(-x * x * 1.4426950408889634f);
  const float erf_abs = 1.0f - poly * e;
  return 0.5f * v * (1.0f + copysignf(erf_abs, v));
}

template <typename S>
__device__ __forceinline__ void store_val(S* p, float v) {
  *p = static_cast<S>(v);
}

template <typename S>
__device__ __forceinline__ void store4(S* p, float4 v);
template <>
__device__ __forceinline__ void store4<float>(float* p, float4 v) {
  *reinterpret_cast<float4*>(p) = v;
}
template <>
__device__ __forceinline__ void store4<bf16>(bf16* p, float4 v) {
  bf16x4 o;
  o[0] = (bf16)v.x; o[1] = (bf16)v.y; o[2] = (bf16)v.z; o[3] = (bf16)v.w;
  *reinterpret_cast<bf16x4*>(p) = o;
}
template <>
__device__ __forceinline__ void store4<f16>(f16* p, float4 v) {
  f16x4 o;
  o[0] = (f16)v.x; o[1] = (f16)v.y; o[2] = (f16)v.z; o[3] = (f16)v.w;
  *reinterpret_cast<f16x4*>(p) = o;
}

// Row-swizzled 16-byte chunk index inside a 128-byte tile row.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ (row & 7); }

typedef __attribute__((address_space(3))) void* lds_void_ptr;

// One 16-byte-per-lane DMA from global memory into LDS at `lds` + 16 * lane
// (global_load_lds_dwordx4 with the wave-uniform LDS address in M0).  It is issued from
// inline assembly so that the compiler does not order later LDS reads of the *other*
// stage behind it; the kernel orders it explicitly (s_waitcnt vmcnt(0) + barrier before
// the stage is read).
__device__ __forceinline__ void dma16(const void* g, void* lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_ptr)lds);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(l), "v"(g) : "memory", "m0");
}

template <typename S, int BM, int BN, int EPI>
__global__ __launch_bounds__(256, 1) void gemm_kernel(GemmParams p) {
  constexpr int NT = 256;
  constexpr int CH = 8;                        // 16-byte chunks per 128-byte row
  constexpr int EPC = 16 / sizeof(S);          // elements per chunk
  constexpr int BK = CH * EPC;                 // K elements per slice
  constexpr int TM = BM / 2, TN = BN / 2;      // wave tile
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int AI = BM / 32, BI = BN / 32;    // DMA instructions per wave per slice
  constexpr int STAGE = (BM + BN) * CH;        // uint4 per LDS stage

  __shared__ uint4 lds[2 * STAGE];

  // ---- tile scheduling: XCD-aware remap, then grouped raster inside a batch entry
  const int tiles_per_batch = p.tiles_m * p.tiles_n;
  const int total = tiles_per_batch * p.batch;
  int pid = blockIdx.x;
  if ((total & 7) == 0) pid = (pid & 7) * (total >> 3) + (pid >> 3);
  const int z = pid / tiles_per_batch;
  const int t = pid - z * tiles_per_batch;
  constexpr int GROUP_M = 8;
  const int group_sz = GROUP_M * p.tiles_n;
  const int gid = t / group_sz;
  const int first_m = gid * GROUP_M;
  const int gm = min(p.tiles_m - first_m, GROUP_M);
  const int tm = first_m + (t % group_sz) % gm;
  const int tn = (t % group_sz) / gm;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lrow = lane & 31, lhalf = lane >> 5;

  const S* Az = static_cast<const S*>(p.A) + z * p.sA;
  const S* Bz = static_cast<const S*>(p.B) + z * p.sB;

  // DMA source offsets: wave loads rows [wave*BM/4, +BM/4) of A in instructions of 8 rows;
  // lane writes row 8u + lane/8, physical chunk lane%8, so it fetches logical chunk
  // (lane % 8) ^ (lane / 8).
  const int dchunk = ((lane & 7) ^ (lane >> 3)) * EPC;
  // (32-bit offsets: the host guarantees rows * leading dimension < 2^31 per operand)
  uint32_t aoff[AI], boff[BI];
#pragma unroll
  for (int u = 0; u < AI; ++u) {
    const int m = min(m0 + wave * (BM / 4) + u * 8 + (lane >> 3), p.M - 1);
    aoff[u] = (uint32_t)m * (uint32_t)p.lda + dchunk;
  }
#pragma unroll
  for (int u = 0; u < BI; ++u) {
    const int n = min(n0 + wave * (BN / 4) + u * 8 + (lane >> 3), p.N - 1);
    boff[u] = (uint32_t)n * (uint32_t)p.ldb + dchunk;
  }

  const int ksl = p.K / BK;               // slices per group
  const int nsl = ksl * p.kgroups;        // total slices

  auto issue = [&](int s, uint4* base) {
    const int g = s / ksl;
    const int k0 = (s - g * ksl) * BK;
    const S* Ag = Az + g * p.gA + k0;
    const S* Bg = Bz + (g % p.gBmod) * p.gB + k0;
#pragma unroll
    for (int u = 0; u < AI; ++u) dma16(Ag + aoff[u], base + (wave * (BM / 4) + u * 8) * CH);
#pragma unroll
    for (int u = 0; u < BI; ++u)
      dma16(Bg + boff[u], base + (BM + wave * (BN / 4) + u * 8) * CH);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // LDS fragment addresses (uint4 index inside a stage): row-dependent part is fixed.
  int arow[FM], brow[FN];
#pragma unroll
  for (int i = 0; i < FM; ++i) arow[i] = (wm * TM + i * 32 + lrow) * CH;
#pragma unroll
  for (int j = 0; j < FN; ++j) brow[j] = (BM + wn * TN + j * 32 + lrow) * CH;
  const int sw = lrow & 7;   // (row & 7) is lrow & 7 for every fragment row

  uint4 af[2][FM], bfr[2][FN];
  auto read_frags = [&](const uint4* L, int c, int slot) {
    const int ch = (2 * c + lhalf) ^ sw;
#pragma unroll
    for (int i = 0; i < FM; ++i) af[slot][i] = L[arow[i] + ch];
#pragma unroll
    for (int j = 0; j < FN; ++j) bfr[slot][j] = L[brow[j] + ch];
  };

  issue(0, lds);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  read_frags(lds, 0, 0);

  // Software pipeline: the fragments of the next 16-deep K chunk are read while the
  // MFMAs of the current chunk run.  At the last chunk of a slice the wave first waits
  // for its own DMA, meets the others at the barrier (after which the next slice is in
  // LDS and nobody reads the current one any more) and reads the next slice's first
  // chunk, all before issuing this chunk's MFMAs, so the barrier and the reload
  // latency overlap matrix work already in flight.  The scheduling fences keep the
  // compiler from sinking the reads next to their uses.
  for (int s = 0; s < nsl; ++s) {
    const bool more = s + 1 < nsl;
    const uint4* cur_buf = lds + (s & 1) * STAGE;
    uint4* next_buf = lds + ((s + 1) & 1) * STAGE;
    if (more) issue(s + 1, next_buf);
#pragma unroll
    for (int c = 0; c < CH / 2; ++c) {
      const int cur = c & 1;
      if (c + 1 < CH / 2) {
        read_frags(cur_buf, c + 1, cur ^ 1);
      } else {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (more) read_frags(next_buf, 0, cur ^ 1);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma_chunk<S>(af[cur][i], bfr[cur][j], acc[i][j]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  __syncthreads();

  // ---- epilogue.  Each wave stages one 32-row block of its tile at a time through its
  // own quarter of the (now idle) LDS ring: the MFMA layout (lane = column, 16 rows per
  // lane) is written out as fp32 rows, then read back four consecutive columns per lane
  // so that global stores (and residual loads) are 16-byte-per-lane row segments.
  using OutT = typename std::conditional<EPI == EPI_BIAS_N_RES, float, S>::type;
  constexpr int RS = TN + 4;                           // staged row stride (floats)
  static_assert(32 * RS * 4 * 4 <= (int)sizeof(lds), "epilogue staging exceeds LDS");
  float* stage = reinterpret_cast<float*>(lds) + wave * 32 * RS;
  const float* biasz = p.bias ? p.bias + z * p.sBias : nullptr;
  const float* Rz = p.R ? p.R + z * p.sR : nullptr;
  OutT* Cz = static_cast<OutT*>(p.C) + z * p.sC;
  const bool vec_ok = (p.ldc & 3) == 0;
  const int rows0 = m0 + wm * TM, cols0 = n0 + wn * TN;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int nl = j * 32 + lrow;
      float bn = 0.f;
      if constexpr (EPI != EPI_BIAS_M)
        bn = (biasz && cols0 + nl < p.N) ? biasz[cols0 + nl] : 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ml = (r >> 2) * 8 + lhalf * 4 + (r & 3);
        float v = acc[i][j][r];
        if constexpr (EPI == EPI_BIAS_M) {
          const int m = rows0 + i * 32 + ml;
          v += (biasz && m < p.M) ? biasz[m] : 0.f;
        } else {
          v += bn;
        }
        if constexpr (EPI == EPI_BIAS_N_GELU) v = gelu_erf(v);
        stage[ml * RS + nl] = v;
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);      // lgkmcnt(0): this wave's LDS writes are done
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int q = 0; q < 32 * TN / 256; ++q) {
      const int e = q * 64 + lane;                     // float4 index inside the block
      const int ml = e / (TN / 4), nl = (e % (TN / 4)) * 4;
      const int m = rows0 + i * 32 + ml, n = cols0 + nl;
      if (m >= p.M) continue;
      float4 v = *reinterpret_cast<const float4*>(stage + ml * RS + nl);
      OutT* dst = Cz + (int64_t)m * p.ldc + n;
      if (vec_ok && n + 3 < p.N) {
        if constexpr (EPI == EPI_BIAS_N_RES) {
          if (Rz) {
            const float4 rr = *reinterpret_cast<const float4*>(Rz + (int64_t)m * p.ldc + n);
            v.x += rr.x; v.y += rr.y; v.z += rr.z; v.w += rr.w;
          }
        }
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
          store_val<OutT>(dst + k, o);
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
  }
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
  const int64_t total = (int64_t)p.tiles_m * p.tiles_n * p.batch;
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

}  // namespace

hipError_t launch_gemm(const GemmDesc& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0 || g.batch <= 0 || g.kgroups <= 0) return hipSuccess;
  const int bk = g.dt == DType::F32 ? 32 : 64;
  if (g.K <= 0 || g.K % bk != 0 || g.gBmod <= 0) return hipErrorInvalidValue;
  // the kernel addresses operand rows of one batch entry / K group with 32-bit byte offsets
  const int64_t es = (int64_t)dtype_size(g.dt);
  if ((int64_t)g.M * g.lda * es >= (1ll << 31) || (int64_t)g.N * g.ldb * es >= (1ll << 31))
    return hipErrorInvalidValue;
  // 256 x 256 tiles when they give at least two waves of workgroups over the 256 CUs,
  // else 128 x 128 (small token counts or narrow projections).
  const int64_t big = (int64_t)((g.M + 255) / 256) * ((g.N + 255) / 256) * g.batch;
  const bool use_big = big >= 512;
  switch (g.dt) {
    case DType::BF16:
      return use_big ? launch_cfg<bf16, 256, 256>(g, s) : launch_cfg<bf16, 128, 128>(g, s);
    case DType::F16:
      return use_big ? launch_cfg<f16, 256, 256>(g, s) : launch_cfg<f16, 128, 128>(g, s);
    default:
      return use_big ? launch_cfg<float, 256, 256>(g, s) : launch_cfg<float, 128, 128>(g, s);
  }
}

}  // namespace kraken
