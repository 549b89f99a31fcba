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
// Tiling (gfx950): a workgroup of WM x WN waves computes a BM x BN tile; each
// wave owns a (BM/WM) x (BN/WN) sub-tile built from 32x32 MFMA blocks
// (v_mfma_f32_32x32x16_{bf16,f16} for 16-bit operands, v_mfma_f32_32x32x2_f32 for
// fp32).  K advances in 128-byte slices (64 16-bit / 32 fp32 elements) staged through a
// double-buffered LDS ring; a 16-byte chunk c of tile row r lives at chunk
// c ^ (r & 7) so that the 8 lanes reading one chunk column hit distinct banks.
// Global loads for slice k+1 are issued before the MFMAs of slice k.
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

__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
}

template <typename S>
__device__ __forceinline__ void store_val(S* p, float v) {
  *p = static_cast<S>(v);
}

// Row-swizzled 16-byte chunk index inside a 128-byte tile row.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ (row & 7); }

template <typename S, int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(64 * WM * WN) void gemm_kernel(GemmParams p) {
  constexpr int NT = 64 * WM * WN;
  constexpr int CH = 8;                        // 16-byte chunks per 128-byte row
  constexpr int EPC = 16 / sizeof(S);          // elements per chunk
  constexpr int BK = CH * EPC;                 // K elements per slice
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int LA = BM * CH / NT, LB = BN * CH / NT;
  static_assert(LA * NT == BM * CH && LB * NT == BN * CH, "tile/threads mismatch");
  static_assert(FM >= 1 && FN >= 1, "wave tile too small");

  __shared__ uint4 lds[2][(BM + BN) * CH];

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
  const int wm = wave / WN, wn = wave % WN;

  const S* Az = static_cast<const S*>(p.A) + z * p.sA;
  const S* Bz = static_cast<const S*>(p.B) + z * p.sB;

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int ksl = p.K / BK;               // slices per group
  const int nsl = ksl * p.kgroups;        // total slices

  uint4 ra[LA], rb[LB];
  auto gload = [&](int s) {
    const int g = s / ksl;
    const int k0 = (s - g * ksl) * BK;
    const S* Ag = Az + g * p.gA;
    const S* Bg = Bz + (g % p.gBmod) * p.gB;
#pragma unroll
    for (int u = 0; u < LA; ++u) {
      const int q = tid + u * NT, row = q / CH, ch = q % CH;
      const int m = m0 + row;
      if (m < p.M)
        ra[u] = *reinterpret_cast<const uint4*>(Ag + (int64_t)m * p.lda + k0 + ch * EPC);
      else
        ra[u] = make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < LB; ++u) {
      const int q = tid + u * NT, row = q / CH, ch = q % CH;
      const int n = n0 + row;
      if (n < p.N)
        rb[u] = *reinterpret_cast<const uint4*>(Bg + (int64_t)n * p.ldb + k0 + ch * EPC);
      else
        rb[u] = make_uint4(0, 0, 0, 0);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int u = 0; u < LA; ++u) {
      const int q = tid + u * NT, row = q / CH, ch = q % CH;
      lds[buf][row * CH + swz(row, ch)] = ra[u];
    }
#pragma unroll
    for (int u = 0; u < LB; ++u) {
      const int q = tid + u * NT, row = q / CH, ch = q % CH;
      lds[buf][(BM + row) * CH + swz(row, ch)] = rb[u];
    }
  };

  gload(0);
  lstore(0);
  __syncthreads();

  const int lrow = lane & 31, lhalf = lane >> 5;
  for (int s = 0; s < nsl; ++s) {
    const int buf = s & 1;
    if (s + 1 < nsl) gload(s + 1);
    const uint4* As = lds[buf];
    const uint4* Bs = lds[buf] + BM * CH;
#pragma unroll
    for (int c = 0; c < CH / 2; ++c) {
      uint4 af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int row = wm * TM + i * 32 + lrow;
        af[i] = As[row * CH + swz(row, 2 * c + lhalf)];
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int row = wn * TN + j * 32 + lrow;
        bfr[j] = Bs[row * CH + swz(row, 2 * c + lhalf)];
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma_chunk<S>(af[i], bfr[j], acc[i][j]);
    }
    if (s + 1 < nsl) lstore(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: lane holds column lrow of each 32x32 block, rows (r/4)*8 + 4*lhalf + r%4
  const float* biasz = p.bias ? p.bias + z * p.sBias : nullptr;
  const float* Rz = p.R ? p.R + z * p.sR : nullptr;
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int n = n0 + wn * TN + j * 32 + lrow;
    if (n >= p.N) continue;
    float bn = 0.f;
    if constexpr (EPI != EPI_BIAS_M) bn = biasz ? biasz[n] : 0.f;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * TM + i * 32 + (r >> 2) * 8 + lhalf * 4 + (r & 3);
        if (m >= p.M) continue;
        const int64_t off = z * p.sC + (int64_t)m * p.ldc + n;
        float v = acc[i][j][r];
        if constexpr (EPI == EPI_BIAS_N) {
          store_val(static_cast<S*>(p.C) + off, v + bn);
        } else if constexpr (EPI == EPI_BIAS_N_GELU) {
          store_val(static_cast<S*>(p.C) + off, gelu_erf(v + bn));
        } else if constexpr (EPI == EPI_BIAS_N_RES) {
          v += bn;
          if (Rz) v += Rz[(int64_t)m * p.ldc + n];
          static_cast<float*>(p.C)[off] = v;
        } else {
          store_val(static_cast<S*>(p.C) + off, v + (biasz ? biasz[m] : 0.f));
        }
      }
    }
  }
}

template <typename S, int BM, int BN, int WM, int WN>
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
  dim3 grid((unsigned)total), block(64 * WM * WN);
  switch (g.epi) {
    case EPI_BIAS_N:
      hipLaunchKernelGGL((gemm_kernel<S, BM, BN, WM, WN, EPI_BIAS_N>), grid, block, 0, s, p);
      break;
    case EPI_BIAS_N_GELU:
      hipLaunchKernelGGL((gemm_kernel<S, BM, BN, WM, WN, EPI_BIAS_N_GELU>), grid, block, 0, s, p);
      break;
    case EPI_BIAS_N_RES:
      hipLaunchKernelGGL((gemm_kernel<S, BM, BN, WM, WN, EPI_BIAS_N_RES>), grid, block, 0, s, p);
      break;
    case EPI_BIAS_M:
      hipLaunchKernelGGL((gemm_kernel<S, BM, BN, WM, WN, EPI_BIAS_M>), grid, block, 0, s, p);
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
  switch (g.dt) {
    case DType::BF16: return launch_cfg<bf16, 128, 128, 2, 2>(g, s);
    case DType::F16: return launch_cfg<f16, 128, 128, 2, 2>(g, s);
    default: return launch_cfg<float, 128, 128, 2, 2>(g, s);
  }
}

}  // namespace kraken
