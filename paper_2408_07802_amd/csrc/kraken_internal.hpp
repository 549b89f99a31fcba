// Internal declarations shared by the Kraken HIP kernels and the runtime.
// Target: gfx950 (CDNA4), 64-lane wavefronts, MFMA matrix cores.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kraken {

typedef __bf16 bf16;
typedef _Float16 f16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Element types.  For a model, the storage type is what the caller's weight blob and
// input use; the compute type is the MFMA operand type of every GEMM and of attention.
enum class DType : int { F32 = 0, BF16 = 1, F16 = 2 };

inline size_t dtype_size(DType t) { return t == DType::F32 ? 4 : 2; }

template <typename S>
struct IsHalfWidth {
  static constexpr bool value = sizeof(S) == 2;
};

// One 16-byte operand chunk per lane into a 32x32 MFMA block.
// 16-bit types: the chunk is 8 consecutive k of the lane's row (k = 8*half + j), one
//   v_mfma_f32_32x32x16_{bf16,f16}.
// fp32: the chunk is 4 consecutive k; MFMA q (0..3) takes element q of both halves, so
//   lane half h supplies k = 4*h + q, the same permutation of k for A and B.
template <typename S>
__device__ __forceinline__ f32x16 mfma_chunk(uint4 a, uint4 b, f32x16 c) {
  if constexpr (__is_same(S, bf16)) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  } else if constexpr (__is_same(S, f16)) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  } else {
    const f32x4 a4 = __builtin_bit_cast(f32x4, a), b4 = __builtin_bit_cast(f32x4, b);
#pragma unroll
    for (int q = 0; q < 4; ++q) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[q], b4[q], c, 0, 0, 0);
    return c;
  }
}

// Epilogues of the batched GEMM C = epi(A B^T).
enum GemmEpi : int {
  EPI_BIAS_N = 0,       // C (storage type) = acc + bias[n]
  EPI_BIAS_N_GELU = 1,  // C (storage type) = GELU(acc + bias[n]), exact erf form
  EPI_BIAS_N_RES = 2,   // C (float32)      = acc + bias[n] + R[m][n]   (bias, R optional)
  EPI_BIAS_M = 3        // C (storage type) = acc + bias[m]
};

// C[z][m][n] = epi( sum_g sum_k A[z][g][m][k] * B[z][g mod gBmod][n][k] )
// A element (z,g,m,k) at A + z*sA + g*gA + m*lda + k; B likewise with ldb/sB/gB;
// C element at C + z*sC + m*ldc + n; R at R + z*sR + m*ldc + n; bias at bias + z*sBias.
struct GemmDesc {
  DType dt;
  int epi;
  const void* A;
  const void* B;
  void* C;
  const float* bias;
  const float* R;
  int M, N, K;  // K per group, multiple of 64 (bf16) / 32 (fp32)
  int lda, ldb, ldc;
  int64_t sA, sB, sC, sR, sBias;
  int batch;
  int kgroups;
  int64_t gA, gB;
  int gBmod;
  // fp16 outputs only: set to 1 (vector store) when a finite fp32 result rounds to an
  // fp16 infinity (|v| >= 65520); NULL: no check
  int* ovf;
};

hipError_t launch_gemm(const GemmDesc& g, hipStream_t s);

// Causal flash attention over packed sequences; n_kv_heads key/value heads (query head
// h reads head h / (n_heads / n_kv_heads)), dkv = n_kv_heads * hd.
struct AttnDesc {
  DType dt;
  const void* qk;   // [n][T][d + dkv]   (Q | K per row)
  const void* vt;   // [n][dkv][ldv]     (V transposed)
  void* out;        // [n][T][d]
  int n, T, d, n_heads, n_kv_heads;
  const int32_t* cu_host;  // host cu_seqlens [num_seqs + 1]
  int num_seqs;
  int q_prescaled;          // the Q columns already carry log2(e) / sqrt(hd)
};

hipError_t launch_attention(const AttnDesc& a, hipStream_t s);

// Row stride (elements) of the transposed V buffer for T tokens: a multiple of 64,
// so that every 8-token group of a row starts on a 16-byte boundary.
inline int vt_ld(int T) { return (T + 63) & ~63; }

// Sets columns [c0, c1) of `rows` rows (row stride ld elements) to zero.
hipError_t launch_zero_cols(DType dt, void* base, int64_t rows, int64_t ld, int c0, int c1,
                            hipStream_t s);

// LayerNorm of n rows-sets: out[i][t] = LN(x[i*xs + t*d]) with per-i gamma/beta.  Rows are
// d wide (the stored width); the statistics cover the first dl (logical width, a multiple
// of 4; padding columns past it hold zeros and have gamma = beta = 0).
// ovf (fp16 outputs; may be NULL): set to 1 when an output overflows the fp16 range.
hipError_t launch_layernorm(DType dt, const float* x, int64_t x_batch_stride, const float* gamma,
                            const float* beta, void* out, int n, int T, int d, int dl, float eps,
                            int* ovf, hipStream_t s);

// out[i][t] = LN(h[i][t] + y[t]); y = shared[t] or sum_k x[k][t].  d, dl, ovf as for LN1.
hipError_t launch_combine_ln2(DType dt, const float* x, const float* shared, const float* h,
                              const float* gamma, const float* beta, void* out, int n, int T,
                              int d, int dl, float eps, int* ovf, hipStream_t s);

// dst[r * dst_ld + pad(c)] = float(src[r * src_ld + c]) for r < R, c < C, with
// pad(c) = (c / g) * gp + c % g (logical element c of group c / g, placed in a group of gp
// slots; g = gp: no padding).  Untouched destination elements keep their values.
hipError_t launch_to_f32_2d(DType st, const void* src, int64_t src_ld, float* dst,
                            int64_t dst_ld, int R, int C, int g, int gp, hipStream_t s);

// dst[r * dst_ld + c] = Dst(src[r * src_ld + c]) for r < R, c < C; *overflow as for
// launch_transpose.
hipError_t launch_convert_2d(DType src_t, const void* src, int64_t src_ld, DType dst_t, void* dst,
                             int64_t dst_ld, int R, int C, int* overflow, hipStream_t s);

// X[t][c] = tok[ids[t]][c] + pos[pos_ids[t]][c] for c < dp (device ids and positions).
hipError_t launch_embed(DType dt, const int* ids, const int* pos_ids, const void* tok,
                        const float* pos, float* X, int T, int dp, hipStream_t s);

// dst[b][:] = src[rows[b]][:], fp32 rows of dp elements (device rows).
hipError_t launch_gather_rows(const float* src, const int* rows, float* dst, int B, int dp,
                              hipStream_t s);

// dst[k] = float(src[k]) for k < count.
hipError_t launch_to_f32(DType dt, const void* src, float* dst, int64_t count, hipStream_t s);

// Two-term split of fp32 values in a 16-bit type: hi = S(v), lo = S(v - hi);
// hi at dst, lo at dst + count (elements).  ovf as for LN1 (a hi part that overflows fp16).
hipError_t launch_split16(DType dt, const float* src, void* dst, int64_t count, int* ovf,
                          hipStream_t s);

// dst[pad_c(c)][pad_r(r)] = Dst(src[r*src_ld + c]) for r < R, c < C, dst row stride dst_ld,
// with pad_r(r) = (r / gr) * grp + r % gr and pad_c likewise with (gc, gcp) (see
// launch_to_f32_2d; gr = grp and gc = gcp: a plain transpose).  When the destination is
// fp16 and a finite source value does not fit, *overflow is set to 1.
hipError_t launch_transpose(DType src_t, const void* src, int64_t src_ld, DType dst_t, void* dst,
                            int64_t dst_ld, int R, int C, int* overflow, hipStream_t s,
                            int gr = 1, int grp = 1, int gc = 1, int gcp = 1);

// KV cache of one layer: [n][2 (K, V)][max_seqs][n_kv_heads][capacity][hd], compute
// type; dkv = n_kv_heads * hd.  Prefill: K from columns d .. d+dkv-1 of qk [n][T][d + dkv],
// V from vt [n][dkv][vt_ld(T)]; token t of sequence b (cu_host[b] <= t < cu_host[b+1])
// goes to position t - cu_host[b] of slot b.
hipError_t launch_kv_store(DType dt, const void* qk, const void* vt, void* cache_layer, int n,
                           int T, int d, int n_heads, int n_kv_heads, const int32_t* cu_host,
                           int num_seqs, int max_seqs, int capacity, hipStream_t s);

// Decode: the K columns of qk [n][B][d + dkv] and v [n][B][dkv] at position lens_host[b]
// of slot b.
hipError_t launch_kv_append(DType dt, const void* qk, const void* v, void* cache_layer, int n,
                            int B, int d, int n_heads, int n_kv_heads, const int32_t* lens_host,
                            int max_seqs, int capacity, hipStream_t s);

// fp32 elements of the decode-attention partials for `splits` key chunks.
int64_t decode_partial_floats(int n, int B, int n_heads, int hd, int splits);

// out [n][B][d] = attention of the Q columns of qk [n][B][d + dkv] over keys
// 0..lens_host[b] of slot b (the new token's own included, already appended).  part: fp32
// scratch of part_floats elements; the key range is split into as many chunks as it holds.
// q_prescaled: the Q columns already carry log2(e) / sqrt(hd).
hipError_t launch_decode_attention(DType dt, const void* qk, const void* cache_layer,
                                   float* part, int64_t part_floats, void* out, int n, int B,
                                   int d, int n_heads, int n_kv_heads, const int32_t* lens_host,
                                   int max_seqs, int capacity, int q_prescaled, hipStream_t s);

// p[k] *= c for k < count (operand type dt).
hipError_t launch_scale(DType dt, void* p, int64_t count, float c, hipStream_t s);

}  // namespace kraken
