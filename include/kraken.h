/*
 * kraken.h -- C ABI of the MI355X (gfx950) Kraken prefill library.
 *
 * Method: Prabhakar, Zhang and Wentzlaff, "Kraken: Inherently Parallel
 * Transformers For Efficient Multi-Device Inference" (arXiv 2408.07802).
 *
 * A Kraken model is a stack of L layers; every layer holds N independent
 * pre-LN Transformer sub-layers of width d (Section 3.1).  Sub-layer i of
 * layer j runs Algorithm 1 ("Kraken Sub-Layer: Forward Pass"):
 *
 *     h_i      = x_i + MHA_i(LN1_i(x_i))
 *     x_i(j+1) = h_i + FFN_i(LN2_i(h_i + y(j)))
 *
 * with y(1) = X (the first layer replaces the AllReduce by the identity) and
 * y(j) = sum_k x_k(j) for j >= 2 (the element-wise sum of the previous
 * layer's N outputs, Section 3.1).  All first-layer sub-layers read the same
 * input X.  After layer L the outputs are combined by one linear map,
 * out = [Y_1 | ... | Y_N] W_concat with W_concat of shape (N d) x d
 * (Section 3.1).  MHA is causal scaled dot-product attention per head,
 * softmax(Q K^T / sqrt(hd)) V with hd = d / heads, heads combined by the
 * output projection; FFN is Linear -> exact GELU -> Linear (Section 2.1).
 * LayerNorm uses the biased variance.  On one GPU the N sub-layers of a layer
 * run as batched work and the paper's cross-device AllReduce becomes an
 * on-device N-way sum fused into the FFN LayerNorm.
 *
 * Conventions shared by every call
 *   - All calls return a kraken_status; no C++ exception crosses this ABI.
 *     On failure kraken_last_error() returns a thread-local detail string.
 *   - Validation happens before anything is enqueued: a call that fails
 *     validation has enqueued no work.  Launch failures return
 *     KRAKEN_ERR_HIP; faults inside kernels surface at the caller's next
 *     synchronisation of the stream.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Device work is asynchronous and ordered on that stream.
 *   - Device pointers must be device memory of the device that was current
 *     when the model was created; that device must be current at every call.
 *   - Debug switch: with the environment variable KRAKEN_DEBUG_SYNC set to a
 *     value other than "0" when a model is created, every kernel launch of that
 *     model's prefill / decode calls is followed by a synchronisation of the
 *     stream; a launch or execution error is then returned (KRAKEN_ERR_HIP,
 *     naming the kernel) by the call that enqueued it instead of surfacing at a
 *     later synchronisation.  Results are bit-identical to a normal run.
 */
#ifndef KRAKEN_H_
#define KRAKEN_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  KRAKEN_OK = 0,
  KRAKEN_ERR_INVALID_ARG = 1,  /* a null pointer, a bad size, a bad cu_seqlens */
  KRAKEN_ERR_UNSUPPORTED = 2,  /* a valid configuration the library does not implement */
  KRAKEN_ERR_OOM = 3,          /* device allocation failed; nothing is leaked */
  KRAKEN_ERR_STATE = 4,        /* e.g. kraken_prefill before kraken_load_weights */
  KRAKEN_ERR_HIP = 5,          /* a HIP runtime call or kernel launch failed */
  KRAKEN_ERR_OVERFLOW = 6      /* kraken_sync: an activation exceeded the fp16 operand range */
} kraken_status;

typedef enum {
  KRAKEN_DTYPE_F32 = 0,
  KRAKEN_DTYPE_BF16 = 1,
  KRAKEN_DTYPE_F16 = 2
} kraken_dtype;

/* MFMA operand type of every projection and of attention (accumulation is
 * always fp32, and so are the residual stream, LayerNorm statistics and the
 * softmax).  KRAKEN_COMPUTE_STORAGE uses the storage dtype.  Weights are
 * converted once at load; a weight that does not fit the operand type (an
 * fp16 overflow) makes kraken_load_weights fail with UNSUPPORTED. */
typedef enum {
  KRAKEN_COMPUTE_STORAGE = 0,
  KRAKEN_COMPUTE_F32 = 1,
  KRAKEN_COMPUTE_BF16 = 2,
  KRAKEN_COMPUTE_F16 = 3
} kraken_compute;

/* Layer architecture (Section 4.3 compares Kraken with the two others at equal sizes). */
typedef enum {
  KRAKEN_ARCH_KRAKEN = 0,    /* N sub-layers per layer, combine y, W_concat (Algorithm 1) */
  KRAKEN_ARCH_GPT = 1,       /* standard pre-LN layer: h = x + MHA(LN1(x)), h + FFN(LN2(h)) */
  KRAKEN_ARCH_PARALLEL = 2   /* parallel attention + FFN (GPT-J, PaLM): u = LN1(x),
                                x + MHA(u) + FFN(u); its weight record has no ln2 */
} kraken_arch;

/*
 * Model shape (Section 3.1; heads are per sub-layer as in the paper's engine
 * table, Section 4.3).
 *   n_sub      N >= 1, parallel sub-layers per layer (1 for the GPT-like and
 *              parallel architectures)
 *   n_layers   L >= 1
 *   d_model    d, width of one sub-layer; multiple of 4.  Widths that are not
 *              multiples of 64 (the engine table's 1248, 3120, 5472, ...) are stored
 *              padded to the next multiple of 64; results are those of width d.
 *   n_heads    heads per sub-layer
 *   d_ff       MLP width; 0 means 4 d (Section 2.1; the engine table's Kraken
 *              models use 2 d, Section 3.2); multiple of 4
 *   max_tokens largest packed token count T a prefill may use (>= 1; at most
 *              4194304, and max_tokens * (the widest stored activation row) * 4 < 2^31)
 *   dtype      a kraken_dtype: element type of the weight blob and of hidden_in
 *   compute    a kraken_compute: MFMA operand type (0 = same as dtype)
 *   ln_eps     LayerNorm epsilon; 0 means 1e-5
 *   n_kv_heads key/value heads per sub-layer; 0 means n_heads (multi-head
 *              attention).  Fewer is grouped-query attention, 1 multi-query
 *              attention (the paper's suggested way to shrink the KV cache,
 *              appendix on the KV cache size): the n_heads query heads form
 *              n_kv_heads groups of consecutive heads, and query head h reads
 *              key/value head h / (n_heads / n_kv_heads).  Must divide n_heads,
 *              and n_kv_heads * (stored head size) must be a multiple of 64.
 *   arch       a kraken_arch (0 = Kraken)
 *   head_dim   hd, the head size; 0 means d / n_heads (d must then be a multiple of
 *              n_heads; Section 4.3: the width divided by the heads).  A multiple of 8
 *              in 8..128; head sizes other than 32, 64 and 128 (the engine table's
 *              72, 96, 104) are stored padded to the next of those, with the softmax
 *              scale 1 / sqrt(hd) of the logical size.  The query width is
 *              n_heads * hd (it may differ from d, as in GPT-3 13B: d = 5140, 40
 *              heads of 128).
 *   vocab      0: no embeddings (kraken_prefill takes the first-layer rows).  > 0:
 *              token embedding rows, used again (tied) by the unembedding of
 *              kraken_forward_tokens (Section 3.1: one set of embeddings, kept for
 *              weight tying)
 *   max_positions  position embedding rows (>= 1 when vocab > 0): the longest
 *              sequence kraken_forward_tokens accepts
 *   Weights: d_ff * d * es, (query + key/value widths) * d * es, n_sub * d^2 * es
 *   (Kraken) and vocab * d * es (stored widths; es = 4 bytes for fp32 MFMA operands,
 *   2 for 16-bit ones) must stay below 2^31 (32-bit byte offsets of the repacked
 *   weights); d (stored) at most 16384.
 */
typedef struct {
  int32_t n_sub;
  int32_t n_layers;
  int32_t d_model;
  int32_t n_heads;
  int32_t d_ff;
  int32_t max_tokens;
  int32_t dtype;
  int32_t compute;
  float ln_eps;
  int32_t n_kv_heads;
  int32_t arch;
  int32_t head_dim;
  int32_t vocab;
  int32_t max_positions;
} kraken_config;

typedef struct kraken_model kraken_model;

/* Largest number of packed sequences one kraken_prefill call accepts. */
#define KRAKEN_MAX_SEQS 256

/* Row stride of the transposed-V operand of kraken_op_attention for T tokens. */
#define KRAKEN_VT_LD(T) ((((T) + 63) / 64) * 64)

/*
 * Creates a model on the current device and allocates all device memory it
 * will use (weights and the activation workspace for max_tokens tokens).
 * The model owns that memory until kraken_destroy.  *out is set to NULL on
 * failure.  Errors: INVALID_ARG (null pointers, non-positive sizes, an unknown
 * arch, n_sub != 1 for the GPT-like or parallel architecture), UNSUPPORTED (d or
 * d_ff not a multiple of 4, a head size outside 8..128 or not a multiple of 8,
 * unknown dtype, sizes past the 32-bit offset limits above), OOM.
 */
kraken_status kraken_create(const kraken_config* cfg, kraken_model** out);

/*
 * Number of elements of the weight blob for cfg (0 for an invalid cfg), with the
 * logical query width dq = n_heads * hd and key/value width dkv = n_kv_heads * hd:
 *   L * N * (2 d dq + 2 d dkv + 2 d F + 5 d + dq + 2 dkv + F + 2 d [no ln2 in
 *   the parallel architecture]) + N d^2 [Kraken] + (vocab + max_positions) d + 2 d
 *   [vocab > 0].  (The Kraken model with dq = dkv = d and no embeddings:
 *   L * N * (4 d^2 + 2 d F + 9 d + F) + N d^2.)
 */
size_t kraken_weight_blob_elems(const kraken_config* cfg);

/*
 * Loads the weights.  The blob holds elements of the model's dtype in this
 * logical order: for j in 0..L-1, for i in 0..N-1 (sub-layer i of layer j):
 *   ln1_g[d] ln1_b[d] Wqkv[d][d + 2 dkv] bqkv[d + 2 dkv] Wo[d][d] bo[d]
 *   ln2_g[d] ln2_b[d] W1[d][F] b1[F] W2[F][d] b2[d]
 * and then W_concat[N d][d] (Kraken only), then, when vocab > 0,
 *   tok_emb[vocab][d] pos_emb[max_positions][d] lnf_g[d] lnf_b[d].
 * The GPT-like and parallel architectures have one record per layer (N = 1);
 * the parallel record omits ln2_g and ln2_b.  Matrices are row-major and
 * multiply as x W ([in][out]); Wqkv is [d][dq + 2 dkv] with columns [Q | K | V],
 * query head h owns columns h*hd .. h*hd+hd-1 of Q and key/value head g columns
 * g*hd .. g*hd+hd-1 of K and of V; Wo is [dq][d]; W_concat's row block i
 * multiplies Y_i.
 * blob_is_device selects whether `blob` is device or host memory.  The call
 * copies and repacks the blob into the model's own layout; the caller keeps
 * ownership and may free or reuse the blob once the stream has synchronised.
 * Errors: INVALID_ARG (null, nbytes != elems * dtype size), UNSUPPORTED (a
 * weight outside the range of the compute type; the call then synchronises
 * the stream to read the check), HIP.  A host blob is uploaded through a
 * staging buffer and the call returns after the upload.
 */
kraken_status kraken_load_weights(kraken_model* m, const void* blob, size_t nbytes,
                                  int blob_is_device, void* stream);

/*
 * Prefill forward pass of the whole stack (Algorithm 1 over L layers, then
 * W_concat) for a packed batch of num_seqs causal sequences.
 *   hidden_in   device [T][d], model dtype: the shared first-layer input X
 *               (token + position embeddings, Section 3.1), sequences packed
 *               back to back with no padding.
 *   cu_seqlens  HOST int32[num_seqs + 1]: cu[0] = 0, strictly increasing
 *               (no empty sequence), T = cu[num_seqs] <= max_tokens.
 *               Tokens cu[b] .. cu[b+1]-1 form sequence b; attention is
 *               causal within a sequence and never crosses sequences.
 *   num_seqs    1 .. KRAKEN_MAX_SEQS.
 *   hidden_out  device float32 [T][d]: out = [Y_1|...|Y_N] W_concat.
 *   sub_out     NULL or device float32 [N][T][d]: the final sub-layer
 *               outputs Y_i before W_concat.
 * Outputs are fp32 whatever the storage dtype (the residual stream and all
 * accumulation are fp32).  Outputs must not overlap the input or each other.
 * The call enqueues the whole pass on `stream` and returns; it keeps no
 * pointer to caller memory.  One prefill at a time per model: concurrent
 * calls on one model must be serialised by the caller (e.g. one stream).
 * Errors: INVALID_ARG, STATE (weights not loaded), HIP.
 */
kraken_status kraken_prefill(kraken_model* m, const void* hidden_in, const int32_t* cu_seqlens,
                             int32_t num_seqs, float* hidden_out, float* sub_out, void* stream);

/*
 * The whole model on packed token sequences (Section 2.1: embeddings, the layer
 * stack, the unembedding; Section 3.1: one token and position embedding shared by
 * the first layer's sub-layers, W_concat's output feeds the unembedding).  Needs a
 * model with vocab > 0.
 *   token_ids   HOST int32[T], each in 0 .. vocab-1; T = cu_seqlens[num_seqs].
 *   cu_seqlens  HOST, as for kraken_prefill; every sequence at most max_positions
 *               long.  Token t of sequence b has position t - cu[b].
 *   logits      device float32 [num_seqs][vocab]: the next-token logits of each
 *               sequence's last token, LN_f(h) tok_emb^T (the unembedding tied to
 *               the token embedding, after a final LayerNorm), where h is the
 *               stack's output row (W_concat's, for Kraken).
 *   hidden_out  NULL or device float32 [T][d]: h for every token.
 * The ids are copied through a pinned host buffer the model owns; the call returns
 * once the copy is enqueued (a following call waits for it before reusing the
 * buffer).  Errors: INVALID_ARG (an id out of range, a sequence longer than
 * max_positions, overlapping outputs, bad cu_seqlens), STATE (no embeddings, weights
 * not loaded), HIP.  Activation overflow of fp16 operands: see kraken_sync.
 */
kraken_status kraken_forward_tokens(kraken_model* m, const int32_t* token_ids,
                                    const int32_t* cu_seqlens, int32_t num_seqs, float* logits,
                                    float* hidden_out, void* stream);

/* ------------------------------------------------------------------------
 * KV cache and one-token decode (Section 2.1, KV cache: the keys and values
 * of every processed token are kept so that later tokens attend to them
 * without recomputing them).  Every sub-layer of every layer has its own
 * keys and values.
 *
 * Cache: caller-owned device memory of kraken_kv_cache_bytes(cfg, max_seqs,
 * capacity) bytes, 16-byte aligned, elements of the MFMA operand type (the
 * compute type; the storage type when compute is KRAKEN_COMPUTE_STORAGE):
 *   [L][N][2 (K, V)][max_seqs][n_kv_heads][capacity][hd]
 * Slot b holds sequence b; position p of slot b holds the key (value) row of
 * that sequence's p-th token, projection bias included, as the attention of
 * kraken_prefill consumes it.  Positions at or above a sequence's length
 * are never read.
 *
 * Returns 0 for an invalid cfg, max_seqs outside 1..KRAKEN_MAX_SEQS or a
 * capacity below 1.
 */
size_t kraken_kv_cache_bytes(const kraken_config* cfg, int32_t max_seqs, int32_t capacity);

/*
 * kraken_prefill that also fills the cache: sequence b of the packed batch
 * (cu_seqlens as for kraken_prefill) writes positions 0 .. S_b - 1 of slot b
 * (S_b = cu[b+1] - cu[b] <= capacity, num_seqs <= max_seqs).  Other slots
 * and positions are left as they are.  hidden_out and sub_out are those of
 * kraken_prefill, bit for bit.  The cache must not overlap the other
 * buffers.  Errors: those of kraken_prefill; INVALID_ARG for a null or
 * misaligned cache, a sequence longer than capacity, num_seqs > max_seqs.
 */
kraken_status kraken_prefill_kv(kraken_model* m, const void* hidden_in, const int32_t* cu_seqlens,
                                int32_t num_seqs, float* hidden_out, float* sub_out,
                                void* kv_cache, int32_t max_seqs, int32_t capacity, void* stream);

/*
 * One decode step for num_seqs sequences, one new token each: the new token
 * of sequence b sits at position lens[b] (the number of tokens slot b
 * already holds), attends causally to positions 0 .. lens[b] of slot b, and
 * its keys and values are written to position lens[b] (the cache then holds
 * lens[b] + 1 tokens of slot b; the caller advances lens).  The result
 * equals row lens[b] of a kraken_prefill over the sequence extended by the
 * new token (causality, Section 2.1), up to rounding.
 *   hidden_in   device [num_seqs][d], model dtype: the new tokens' X rows.
 *   lens        HOST int32[num_seqs], 0 <= lens[b] < capacity.
 *   num_seqs    1 .. min(max_seqs, max_tokens); sequence b uses slot b.
 *   hidden_out  device float32 [num_seqs][d].
 *   sub_out     NULL or device float32 [N][num_seqs][d].
 * The model's workspace holds the step's activations and the attention's
 * per-chunk partial results; one model runs one call at a time.
 * Errors: INVALID_ARG (null or misaligned pointers, lens out of range,
 * overlapping buffers), STATE (weights not loaded), HIP.
 */
kraken_status kraken_decode(kraken_model* m, const void* hidden_in, const int32_t* lens,
                            int32_t num_seqs, float* hidden_out, float* sub_out, void* kv_cache,
                            int32_t max_seqs, int32_t capacity, void* stream);

/*
 * Waits for `stream` and reports the model's fp16 activation overflow flag.
 * With fp16 MFMA operands (compute type KRAKEN_COMPUTE_F16, or fp16 storage),
 * every activation converted to fp16 for a matrix product (the LayerNorm
 * outputs, the Q|K and V projections, the GELU output and the high half of
 * the W_concat operand) is checked on the device: a finite fp32 value of
 * magnitude >= 65520 rounds to an fp16 infinity and sets a sticky flag.  (The
 * attention output is a convex combination of V rows and cannot exceed the
 * V projection's range.)  Returns KRAKEN_ERR_OVERFLOW, and clears the flag, if
 * any kraken_prefill / kraken_prefill_kv / kraken_decode of this model since
 * the last kraken_sync overflowed: their outputs are then not valid.  Returns
 * KRAKEN_OK otherwise.  Errors: INVALID_ARG, HIP.
 */
kraken_status kraken_sync(kraken_model* m, void* stream);

/* Waits for the model's device work, frees everything it owns.  NULL is a no-op. */
kraken_status kraken_destroy(kraken_model* m);

const char* kraken_status_string(kraken_status s);
const char* kraken_last_error(void);

/* ------------------------------------------------------------------------
 * Per-kernel timing of kraken_prefill (measurement support).
 * When enabled, every launch of a prefill is bracketed by a pair of HIP
 * events on the prefill's stream; kraken_profile_read returns, per kernel
 * class, the summed device time in ms and the number of launches since the
 * last reset.  Reading waits for the recorded events.  Kernel classes:
 */
enum {
  KRAKEN_K_LN1 = 0,        /* LayerNorm before MHA */
  KRAKEN_K_GEMM_QK = 1,    /* Q,K projection */
  KRAKEN_K_GEMM_VT = 2,    /* V projection (written transposed) */
  KRAKEN_K_ATTN = 3,       /* causal flash attention */
  KRAKEN_K_GEMM_O = 4,     /* output projection + residual */
  KRAKEN_K_COMBINE = 5,    /* N-way sum + residual + LayerNorm before FFN (GPT-like: LN2) */
  KRAKEN_K_GEMM_UP = 6,    /* FFN up projection + GELU */
  KRAKEN_K_GEMM_DOWN = 7,  /* FFN down projection + residual */
  KRAKEN_K_CONCAT = 8,     /* W_concat (and its operand split) */
  KRAKEN_K_OTHER = 9,      /* input conversion, output copies, embedding, final LayerNorm */
  KRAKEN_K_KV = 10,        /* KV cache writes (kraken_prefill_kv, kraken_decode) */
  KRAKEN_K_UNEMBED = 11,   /* unembedding GEMM (kraken_forward_tokens) */
  KRAKEN_K_COUNT = 12
};
kraken_status kraken_profile_enable(kraken_model* m, int enable);
kraken_status kraken_profile_read(kraken_model* m, int kernel_class, double* total_ms,
                                  int64_t* launches);
kraken_status kraken_profile_reset(kraken_model* m);
/* Algorithmic FLOPs (matrix products and attention, causal pairs only) of one
 * prefill over `cu_seqlens`, per kernel class: returns 0 for classes that do
 * no matrix work. */
double kraken_class_flops(const kraken_config* cfg, int kernel_class, const int32_t* cu_seqlens,
                          int32_t num_seqs);

/* ------------------------------------------------------------------------
 * Single-kernel entry points: the same kernels kraken_prefill launches, on
 * caller buffers, for per-kernel parity tests.  All pointers are device
 * pointers; `dtype` is a kraken_dtype naming the operand type "S" below.
 *
 * kraken_op_layernorm (Algorithm 1, LN1): out[i][t][:] = LN(x_i[t][:]; g_i, b_i)
 *   x float32 at x + i*x_batch_stride + t*d (x_batch_stride may be 0: shared
 *   input), g/b float32 [n][d], out S [n][T][d].
 */
kraken_status kraken_op_layernorm(int32_t dtype, const float* x, int64_t x_batch_stride,
                                  const float* gamma, const float* beta, void* out,
                                  int32_t n, int32_t T, int32_t d, float eps, void* stream);

/*
 * kraken_op_combine_ln2 (Algorithm 1, second LayerNorm; Section 3.1 combine):
 *   y[t] = shared[t] if shared != NULL, else sum_k x[k][t]  (k < n)
 *   out[i][t] = LN(h[i][t] + y[t]; g_i, b_i)
 *   x, h float32 [n][T][d]; shared float32 [T][d] or NULL; out S [n][T][d].
 */
kraken_status kraken_op_combine_ln2(int32_t dtype, const float* x, const float* shared,
                                    const float* h, const float* gamma, const float* beta,
                                    void* out, int32_t n, int32_t T, int32_t d, float eps,
                                    void* stream);

/*
 * kraken_op_gemm: batched C[z] = epilogue(A[z] B[z]^T), z < batch, with
 *   A S [M][K] (row stride K, batch stride sA), B S [N][K] (row stride K,
 *   batch stride sB), fp32 accumulation.  epilogue:
 *     0  C = acc + bias[n]              C is S     (bias float32 [batch][N])
 *     1  C = GELU(acc + bias[n])        C is S     (exact erf GELU)
 *     2  C = acc + bias[n] + R[m][n]    C is float32, R float32 with batch
 *                                       stride sR (may be 0)
 *     3  C = acc + bias[m]              C is S     (bias float32 [batch][M])
 *   Row stride of C and R is N; batch strides are in elements; bias may be
 *   NULL (no bias).  K must be a multiple of 64 elements.
 */
kraken_status kraken_op_gemm(int32_t dtype, int32_t epilogue, const void* A, const void* B,
                             void* C, const float* bias, const float* R, int32_t M, int32_t N,
                             int32_t K, int32_t batch, int64_t sA, int64_t sB, int64_t sC,
                             int64_t sR, void* stream);

/*
 * Test support: fills the model's whole activation workspace with 0xFF bytes
 * (a NaN in every element type) on `stream`.  A following prefill or decode
 * must give the same result as without it: every workspace element a kernel
 * reads has been written earlier in the same call.  Errors: INVALID_ARG, HIP.
 */
kraken_status kraken_debug_poison_workspace(kraken_model* m, void* stream);

/*
 * kraken_op_attention (Section 2.1, causal MHA core; packed sequences), with
 * n_kv_heads key/value heads (0 = n_heads; query head h reads key/value head
 * h / (n_heads / n_kv_heads)) and dkv = n_kv_heads * hd:
 *   qk S [n][T][d + dkv] (row t: Q then K, query head h at columns h*hd,
 *      key head g at columns d + g*hd),
 *   vt S [n][dkv][ldv] (V transposed: row c is feature c over tokens), with
 *      ldv = T rounded up to a multiple of 64 (KRAKEN_VT_LD(T)); the padding
 *      columns [T, ldv) must hold finite values (they meet zero probabilities),
 *   out S [n][T][d]: out = softmax(Q K^T / sqrt(hd) + causal mask) V per head.
 *   q_prescaled 0: Q as above.  1: the Q columns already carry the factor
 *      log2(e) / sqrt(hd), as kraken_prefill's Q projection does (its weights are
 *      scaled at load), and the kernel computes softmax with base-2 exponentials
 *      of Q K^T directly: out = softmax(ln(2) Q K^T + mask) V.  This is the
 *      variant the prefill launches.
 *   cu_seqlens is a HOST int32[num_seqs+1] array as in kraken_prefill.
 *   16-bit operands with hd = 128 run the ping-pong kernel the prefill uses as long
 *   as one layer's qk rows fit 32-bit byte offsets (T * (d + dkv) * 2 < 2^32);
 *   larger inputs, and every other case, run the one-phase kernel.  Same results
 *   either way, within each kernel's rounding.
 */
kraken_status kraken_op_attention(int32_t dtype, const void* qk, const void* vt, void* out,
                                  int32_t n, int32_t d, int32_t n_heads, int32_t n_kv_heads,
                                  int32_t q_prescaled, const int32_t* cu_seqlens,
                                  int32_t num_seqs, void* stream);

/*
 * kraken_op_decode_attention (Section 2.1, attention of one new token per
 * sequence over its KV cache; the kernels kraken_decode launches), with
 * n_kv_heads key/value heads as for kraken_op_attention:
 *   qk       S [n][B][d + dkv]: row b's first d columns are the new token's
 *            query of sequence b (B = num_seqs); the K columns are not read.
 *   kv_layer S, one layer of a KV cache as kraken.h lays it out,
 *            [n][2][max_seqs][n_kv_heads][capacity][hd], holding keys and values
 *            at positions 0 .. lens[b] of slot b (the new token's own at lens[b]).
 *   out      S [n][B][d]: softmax(q K^T / sqrt(hd)) V per head over those
 *            lens[b] + 1 positions.
 *   lens     HOST int32[num_seqs], 0 <= lens[b] < capacity.
 *   work     device float32 scratch of work_floats elements, at least
 *            n * B * n_heads * (hd + 2): per-chunk (max, sum, output) partials.
 *            The key range is split into as many chunks (multiples of 256 keys)
 *            as the scratch holds; the result does not depend on the split
 *            beyond rounding.
 */
kraken_status kraken_op_decode_attention(int32_t dtype, const void* qk, const void* kv_layer,
                                         void* out, int32_t n, int32_t d, int32_t n_heads,
                                         int32_t n_kv_heads, const int32_t* lens,
                                         int32_t num_seqs, int32_t max_seqs, int32_t capacity,
                                         float* work, int64_t work_floats, void* stream);

/*
 * kraken_op_decode_attention_noalloc: kraken_op_decode_attention without the `work`
 * argument, for callers that cannot allocate device memory (code being captured into a
 * HIP graph, tight serving loops, harnesses that forbid hipMalloc).  The per-chunk
 * partials live in a static device array of KRAKEN_NOALLOC_SCRATCH_FLOATS floats (32 MiB)
 * that the library holds on every GPU it runs on until the process ends; the call itself
 * allocates and frees nothing.  Arguments and result are those of
 * kraken_op_decode_attention with work_floats = KRAKEN_NOALLOC_SCRATCH_FLOATS (the same
 * key split, so the same bits).
 * Limit: n * num_seqs * n_heads * (hd + 2) must not exceed KRAKEN_NOALLOC_SCRATCH_FLOATS
 * (one key chunk's partials), else KRAKEN_ERR_UNSUPPORTED with a message.
 * Every call on one GPU shares that GPU's array (nothing in it needs to start at zero:
 * each call writes every partial it reads): calls that overlap in time on one GPU, e.g.
 * on two streams, race and must be serialised by the caller.
 * Errors: INVALID_ARG, UNSUPPORTED, HIP (including a failed lookup of the array's
 * device address on the first call on a device).
 */
#define KRAKEN_NOALLOC_SCRATCH_FLOATS (8 * 1024 * 1024)
kraken_status kraken_op_decode_attention_noalloc(int32_t dtype, const void* qk,
                                                 const void* kv_layer, void* out, int32_t n,
                                                 int32_t d, int32_t n_heads, int32_t n_kv_heads,
                                                 const int32_t* lens, int32_t num_seqs,
                                                 int32_t max_seqs, int32_t capacity,
                                                 void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KRAKEN_H_ */
