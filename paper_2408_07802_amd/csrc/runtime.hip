// Host runtime and C ABI of the Kraken prefill library (declared in kraken.h).
//
// A model owns two device allocations: the repacked weights and the activation
// workspace for max_tokens tokens.  kraken_prefill validates everything on the
// host, then enqueues the whole pass on the caller's stream: per layer
//   LN1 -> Q,K projection -> V projection (transposed) -> causal attention
//   -> output projection + residual -> N-way sum + residual + LN2
//   -> FFN up + GELU -> FFN down + residual
// (Algorithm 1 for all N sub-layers at once; every GEMM is batched over the N
// sub-layers), then W_concat over the N final outputs (Section 3.1).  The same
// kernels run the two architectures the paper compares with (Section 4.3): the
// standard GPT-like layer (LN2 of h alone) and the parallel attention + FFN layer
// (one LayerNorm feeding both branches); and, for a model with embeddings, the
// whole token-to-logits pass (Sections 2.1 and 3.1).
//
// Stored widths.  The kernels need row widths that are multiples of 64 and head
// sizes of 32, 64 or 128.  A model of another width d (the engine table's 1248,
// 3120, 5472, ...) or head size hd (72, 96, 104) keeps its logical sizes and is
// stored at dp = d rounded up to 64 and hdp = hd rounded up to 32, 64 or 128: padding
// weights, biases and LayerNorm gains are zero, so padding features of every
// activation stay exactly zero, LayerNorm statistics run over the first d features
// only, a padded head's extra dimensions add nothing to its scores, and the
// softmax scale is that of the logical head size.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/kraken.h"
#include "kraken_internal.hpp"

using namespace kraken;

namespace {

thread_local std::string g_last_error;

// Scratch of the allocation-free decode attention (kraken_op_decode_attention_noalloc): the
// per-chunk (max, sum, output) partials, fp32.  One copy per GPU, held until the process
// ends.  In host code `scratch` only names the symbol; its device address is looked up
// once per device and kept in g_scratch_ptr.
static __device__ __align__(256) float scratch[KRAKEN_NOALLOC_SCRATCH_FLOATS];
constexpr int kMaxDevices = 64;
float* g_scratch_ptr[kMaxDevices] = {};
std::mutex g_scratch_mutex;

kraken_status fail(kraken_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

kraken_status hip_fail(hipError_t e, const char* what) {
  return fail(KRAKEN_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                \
  do {                                     \
    hipError_t e_ = (expr);                \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

// Stored layouts (dp, dq, dkv, Fp: the stored widths of Dims below).
struct LayerW {
  float *ln1_g, *ln1_b, *ln2_g, *ln2_b;  // [N][dp]
  float *bqk;                            // [N][dq + dkv]
  float *bv;                             // [N][dkv]
  float *bo, *b2;                        // [N][dp]
  float *b1;                             // [N][Fp]
  void *WqkT;                            // [N][dq + dkv][dp]
  void *WvT;                             // [N][dkv][dp]
  void *WoT;                             // [N][dp][dq]
  void *W1T;                             // [N][Fp][dp]
  void *W2T;                             // [N][dp][Fp]
};

struct ProfRec {
  int cls;
  hipEvent_t a, b;
};

// Logical sizes of a configuration and the widths they are stored at.
struct Dims {
  int arch, N, L, d, H, hd, Hkv, F, V, P;
  int64_t dq_l, dkv_l;     // logical attention widths: H hd and Hkv hd
  int dp, hdp, Fp;         // stored: d rounded up to 64; hd to 32, 64 or 128; F to 64
  int64_t dq, dkv;         // stored attention widths: H hdp and Hkv hdp
};

int round_up(int x, int m) { return (x + m - 1) / m * m; }

// Sizes of a configuration that validate_cfg accepted (or of any cfg, for the size
// queries, which check the basics themselves).
Dims dims_of(const kraken_config* c) {
  Dims D;
  D.arch = c->arch;
  D.N = c->n_sub;
  D.L = c->n_layers;
  D.d = c->d_model;
  D.H = c->n_heads;
  D.hd = c->head_dim > 0 ? c->head_dim : (c->n_heads > 0 ? c->d_model / c->n_heads : 0);
  D.Hkv = c->n_kv_heads > 0 ? c->n_kv_heads : c->n_heads;
  D.F = c->d_ff > 0 ? c->d_ff : 4 * c->d_model;
  D.V = c->vocab;
  D.P = c->max_positions;
  D.dq_l = (int64_t)D.H * D.hd;
  D.dkv_l = (int64_t)D.Hkv * D.hd;
  D.dp = round_up(D.d, 64);
  D.hdp = D.hd <= 32 ? 32 : D.hd <= 64 ? 64 : 128;
  D.Fp = round_up(D.F, 64);
  D.dq = (int64_t)D.H * D.hdp;
  D.dkv = (int64_t)D.Hkv * D.hdp;
  return D;
}

// Element counts of the logical blob of one sub-layer (of a layer, for the GPT-like and
// parallel architectures), in blob order.  The parallel attention + FFN layer has one
// LayerNorm, so its record has no ln2_g / ln2_b.
struct SubOffsets {
  int64_t ln1_g, ln1_b, Wqkv, bqkv, Wo, bo, ln2_g, ln2_b, W1, b1, W2, b2, total;
  explicit SubOffsets(const Dims& D) {
    const int64_t d = D.d, F = D.F, dq = D.dq_l, dkv = D.dkv_l;
    const bool ln2 = D.arch != KRAKEN_ARCH_PARALLEL;
    int64_t o = 0;
    ln1_g = o; o += d;
    ln1_b = o; o += d;
    Wqkv = o; o += d * (dq + 2 * dkv);
    bqkv = o; o += dq + 2 * dkv;
    Wo = o; o += dq * d;
    bo = o; o += d;
    ln2_g = o; o += ln2 ? d : 0;
    ln2_b = o; o += ln2 ? d : 0;
    W1 = o; o += d * F;
    b1 = o; o += F;
    W2 = o; o += F * d;
    b2 = o; o += d;
    total = o;
  }
};

}  // namespace

struct kraken_model {
  kraken_config cfg;
  Dims D;     // logical and stored sizes
  DType st;   // storage type of the blob and of hidden_in
  DType dt;   // MFMA operand type
  int N, L, d, H, F, Tmax, device;   // (logical d and F)
  int dp, Fp;                        // stored widths
  int Hkv;                           // key/value heads (grouped-query attention: Hkv < H)
  int64_t dq, dkv;                   // stored query and key/value widths
  float eps;
  bool loaded = false;
  void* wmem = nullptr;
  void* amem = nullptr;
  size_t wbytes = 0;
  std::vector<LayerW> layers;
  void* WcatT = nullptr;  // [dp][N*dp] (Kraken)
  // embeddings (vocab > 0): token rows [V][dp] in the operand type (also the tied
  // unembedding), position rows [P][dp] fp32, final LayerNorm [dp] fp32
  void* tok = nullptr;
  float *pos = nullptr, *lnf_g = nullptr, *lnf_b = nullptr;
  // token-path workspace: ids [Tmax], positions [Tmax], last rows [MAX_SEQS] (int32),
  // gathered last rows [MAX_SEQS][dp] fp32 and their normalised rows in the operand type
  int* tok_ids = nullptr;
  float* last = nullptr;
  void* last_act = nullptr;
  int* tok_host = nullptr;        // pinned host staging of the ids, positions and rows
  hipEvent_t tok_copied = nullptr;
  // device: [0] = a weight overflowed the operand type (set at load); [1] = an activation
  // overflowed the fp16 operand type (sticky until kraken_sync reads it)
  int* flags = nullptr;
  // workspace (stored widths)
  float *X32 = nullptr, *xbuf = nullptr, *hbuf = nullptr;
  void *act = nullptr, *qk = nullptr, *vt = nullptr, *o = nullptr, *g = nullptr;
  char* ws_end = nullptr;
  // KRAKEN_DEBUG_SYNC=1 at kraken_create: synchronise and check after every launch
  bool debug_sync = false;
  // per-kernel timing
  bool prof = false;
  std::vector<ProfRec> pending;
  std::vector<hipEvent_t> pool;
  double prof_ms[KRAKEN_K_COUNT] = {};
  int64_t prof_n[KRAKEN_K_COUNT] = {};

  hipEvent_t take_event() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }

  // Runs one launch, bracketed by timing events when profiling is on; in debug-sync mode
  // the stream is synchronised after it and any launch or execution error is returned.
  template <class Fn>
  hipError_t run(int cls, hipStream_t s, Fn&& fn) {
    hipError_t e;
    hipEvent_t a = prof ? take_event() : nullptr, b = prof ? take_event() : nullptr;
    if (a && b) {
      hipEventRecord(a, s);
      e = fn();
      hipEventRecord(b, s);
      pending.push_back({cls, a, b});
    } else {
      if (a) pool.push_back(a);
      if (b) pool.push_back(b);
      e = fn();
    }
    if (e == hipSuccess && debug_sync) {
      e = hipStreamSynchronize(s);
      if (e == hipSuccess) e = hipGetLastError();
    }
    return e;
  }
};

namespace {

size_t sz(DType t) { return dtype_size(t); }

kraken_status validate_cfg(const kraken_config* c) {
  if (!c) return fail(KRAKEN_ERR_INVALID_ARG, "cfg is NULL");
  if (c->n_sub < 1 || c->n_layers < 1 || c->d_model < 1 || c->n_heads < 1 || c->max_tokens < 1 ||
      c->d_ff < 0 || c->ln_eps < 0.f || c->head_dim < 0 || c->vocab < 0 || c->max_positions < 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "non-positive size in cfg");
  if (c->arch < KRAKEN_ARCH_KRAKEN || c->arch > KRAKEN_ARCH_PARALLEL)
    return fail(KRAKEN_ERR_INVALID_ARG, "unknown arch");
  if (c->arch != KRAKEN_ARCH_KRAKEN && c->n_sub != 1)
    return fail(KRAKEN_ERR_INVALID_ARG, "the GPT-like and parallel architectures have n_sub = 1");
  if (c->head_dim == 0 && c->d_model % c->n_heads != 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "d_model is not a multiple of n_heads (give head_dim)");
  const Dims D = dims_of(c);
  if (D.hd < 8 || D.hd > 128 || D.hd % 8 != 0)
    return fail(KRAKEN_ERR_UNSUPPORTED, "head size must be a multiple of 8 in 8..128");
  if (D.d % 4 != 0 || D.F % 4 != 0)
    return fail(KRAKEN_ERR_UNSUPPORTED, "d_model and d_ff must be multiples of 4");
  if (c->n_kv_heads < 0) return fail(KRAKEN_ERR_INVALID_ARG, "negative n_kv_heads");
  if (c->n_kv_heads > 0) {
    if (c->n_heads % c->n_kv_heads != 0)
      return fail(KRAKEN_ERR_INVALID_ARG, "n_kv_heads does not divide n_heads");
    if (D.dkv % 64 != 0)
      return fail(KRAKEN_ERR_UNSUPPORTED,
                  "n_kv_heads * stored head size (32, 64 or 128) must be a multiple of 64");
  }
  if (D.dq % 64 != 0)
    return fail(KRAKEN_ERR_UNSUPPORTED,
                "n_heads * stored head size (32, 64 or 128) must be a multiple of 64");
  if (D.dp > 16384) return fail(KRAKEN_ERR_UNSUPPORTED, "d_model above 16384");
  if (c->max_tokens > (1 << 22)) return fail(KRAKEN_ERR_UNSUPPORTED, "max_tokens above 4194304");
  if (c->vocab > 0 && c->max_positions < 1)
    return fail(KRAKEN_ERR_INVALID_ARG, "a model with embeddings needs max_positions >= 1");
  if (c->dtype < KRAKEN_DTYPE_F32 || c->dtype > KRAKEN_DTYPE_F16)
    return fail(KRAKEN_ERR_UNSUPPORTED, "unknown dtype");
  if (c->compute < KRAKEN_COMPUTE_STORAGE || c->compute > KRAKEN_COMPUTE_F16)
    return fail(KRAKEN_ERR_UNSUPPORTED, "unknown compute type");
  // GEMM operands of one sub-layer are addressed with 32-bit byte offsets: the activation
  // rows (tokens x the widest stored row; 4 bytes bounds every activation type), and the
  // repacked weights [out][in] in the compute type (es bytes) of the projections, the FFN
  // (Fp x dp either way), W_concat (dp x N dp) and the token embedding (V x dp)
  const bool f32_ops = c->compute == KRAKEN_COMPUTE_F32 ||
                       (c->compute == KRAKEN_COMPUTE_STORAGE && c->dtype == KRAKEN_DTYPE_F32);
  const int64_t es = f32_ops ? 4 : 2;
  const int64_t widest = std::max<int64_t>({(int64_t)D.dp, D.dq + D.dkv, (int64_t)D.Fp});
  if ((int64_t)c->max_tokens * widest * 4 >= (1ll << 31))
    return fail(KRAKEN_ERR_UNSUPPORTED, "max_tokens * the widest activation row too large");
  if ((int64_t)D.Fp * D.dp * es >= (1ll << 31) || (D.dq + D.dkv) * D.dp * es >= (1ll << 31))
    return fail(KRAKEN_ERR_UNSUPPORTED, "d_ff * d_model too large for 32-bit weight offsets");
  if (c->arch == KRAKEN_ARCH_KRAKEN && (int64_t)D.N * D.dp * D.dp * es >= (1ll << 31))
    return fail(KRAKEN_ERR_UNSUPPORTED,
                "n_sub * d_model^2 too large for 32-bit W_concat offsets");
  if ((int64_t)D.V * D.dp * es >= (1ll << 31))
    return fail(KRAKEN_ERR_UNSUPPORTED, "vocab * d_model too large for 32-bit offsets");
  return KRAKEN_OK;
}

kraken_status check_device(const kraken_model* m) {
  int cur = -1;
  HIP_TRY(hipGetDevice(&cur), "hipGetDevice");
  if (cur != m->device) return fail(KRAKEN_ERR_INVALID_ARG, "the model's device is not current");
  return KRAKEN_OK;
}

kraken_status check_cu(const int32_t* cu, int32_t num_seqs, int64_t max_tokens, int64_t* T) {
  if (!cu) return fail(KRAKEN_ERR_INVALID_ARG, "cu_seqlens is NULL");
  if (num_seqs < 1 || num_seqs > KRAKEN_MAX_SEQS)
    return fail(KRAKEN_ERR_INVALID_ARG, "num_seqs out of range 1..KRAKEN_MAX_SEQS");
  if (cu[0] != 0) return fail(KRAKEN_ERR_INVALID_ARG, "cu_seqlens[0] must be 0");
  for (int b = 0; b < num_seqs; ++b)
    if (cu[b + 1] <= cu[b])
      return fail(KRAKEN_ERR_INVALID_ARG, "cu_seqlens must be strictly increasing (no empty sequence)");
  if (cu[num_seqs] > max_tokens) return fail(KRAKEN_ERR_INVALID_ARG, "T exceeds max_tokens");
  *T = cu[num_seqs];
  return KRAKEN_OK;
}

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || !na || !nb) return false;
  const char* pa = static_cast<const char*>(a);
  const char* pb = static_cast<const char*>(b);
  return pa < pb + nb && pb < pa + na;
}

void free_model_memory(kraken_model* m) {
  if (m->wmem) hipFree(m->wmem);
  if (m->amem) hipFree(m->amem);
  m->wmem = m->amem = nullptr;
}

// Bump allocator over one hipMalloc'd block, 256-byte aligned pieces.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  void* take(size_t bytes) {
    void* p = base ? base + off : nullptr;
    off += (bytes + 255) & ~size_t(255);
    return p;
  }
};

// Lays out (or, with a null base, measures) the weight arena.
size_t carve_weights(kraken_model* m, void* base) {
  Carver c(base);
  const Dims& D = m->D;
  const size_t N = D.N, dp = D.dp, Fp = D.Fp, dq = D.dq, dkv = D.dkv, es = sz(m->dt);
  m->layers.resize(m->L);
  for (int j = 0; j < m->L; ++j) {
    LayerW& w = m->layers[j];
    w.ln1_g = (float*)c.take(N * dp * 4);
    w.ln1_b = (float*)c.take(N * dp * 4);
    w.ln2_g = (float*)c.take(N * dp * 4);
    w.ln2_b = (float*)c.take(N * dp * 4);
    w.bqk = (float*)c.take(N * (dq + dkv) * 4);
    w.bv = (float*)c.take(N * dkv * 4);
    w.bo = (float*)c.take(N * dp * 4);
    w.b1 = (float*)c.take(N * Fp * 4);
    w.b2 = (float*)c.take(N * dp * 4);
    w.WqkT = c.take(N * (dq + dkv) * dp * es);
    w.WvT = c.take(N * dkv * dp * es);
    w.WoT = c.take(N * dp * dq * es);
    w.W1T = c.take(N * Fp * dp * es);
    w.W2T = c.take(N * dp * Fp * es);
  }
  m->WcatT = D.arch == KRAKEN_ARCH_KRAKEN ? c.take(dp * N * dp * es) : nullptr;
  if (D.V > 0) {
    m->tok = c.take((size_t)D.V * dp * es);
    m->pos = (float*)c.take((size_t)D.P * dp * 4);
    m->lnf_g = (float*)c.take(dp * 4);
    m->lnf_b = (float*)c.take(dp * 4);
  }
  m->flags = (int*)c.take(256);
  return c.off;
}

size_t carve_workspace(kraken_model* m, void* base) {
  Carver c(base);
  const Dims& D = m->D;
  const size_t N = D.N, dp = D.dp, Fp = D.Fp, T = m->Tmax, dq = D.dq, dkv = D.dkv;
  const size_t es = sz(m->dt);
  if (D.V > 0) {
    m->tok_ids = (int*)c.take((2 * T + KRAKEN_MAX_SEQS) * sizeof(int));
    m->last = (float*)c.take((size_t)KRAKEN_MAX_SEQS * dp * 4);
    m->last_act = c.take((size_t)KRAKEN_MAX_SEQS * dp * es);
  }
  m->X32 = (float*)c.take(T * dp * 4);
  m->xbuf = (float*)c.take(N * T * dp * 4);
  m->hbuf = (float*)c.take(N * T * dp * 4);
  m->act = c.take(N * T * dp * es);
  m->qk = c.take(N * T * (dq + dkv) * es);
  m->o = c.take(N * T * std::max(dq, dkv) * es);
  // vt and g stay adjacent and last: a decode step keeps its attention partials there
  m->vt = c.take(N * dkv * (size_t)vt_ld(m->Tmax) * es);
  m->g = c.take(std::max(N * T * Fp, 2 * N * T * dp) * es);
  m->ws_end = base ? static_cast<char*>(base) + c.off : nullptr;
  return c.off;
}

inline const char* cptr(const void* p, int64_t elems, DType t) {
  return static_cast<const char*>(p) + elems * (int64_t)sz(t);
}

// Repack one sub-layer's logical parameters (device pointer `src`) into the stored layout:
// matrices transposed to [out][in] in the operand type, heads of hd features placed at
// multiples of hdp, rows padded to the stored widths (the arena was zeroed, so every
// padding element stays zero).
hipError_t repack_sub(kraken_model* m, int j, int i, const void* src, hipStream_t s) {
  const Dims& D = m->D;
  const int64_t d = D.d, F = D.F, dql = D.dq_l, dkvl = D.dkv_l, wq = dql + 2 * dkvl;
  const int64_t dp = D.dp, Fp = D.Fp, dq = D.dq, dkv = D.dkv;
  const int hd = D.hd, hdp = D.hdp;
  const SubOffsets so(D);
  const LayerW& w = m->layers[j];
  const DType st = m->st, dt = m->dt;
  const size_t es = sz(dt);
  int* of = m->flags;
  char* WqkT = static_cast<char*>(w.WqkT) + i * (dq + dkv) * dp * es;
  hipError_t e;
#define R_(x) do { e = (x); if (e != hipSuccess) return e; } while (0)
  R_(launch_to_f32(st, cptr(src, so.ln1_g, st), w.ln1_g + i * dp, d, s));
  R_(launch_to_f32(st, cptr(src, so.ln1_b, st), w.ln1_b + i * dp, d, s));
  if (D.arch != KRAKEN_ARCH_PARALLEL) {
    R_(launch_to_f32(st, cptr(src, so.ln2_g, st), w.ln2_g + i * dp, d, s));
    R_(launch_to_f32(st, cptr(src, so.ln2_b, st), w.ln2_b + i * dp, d, s));
  }
  // biases of the Q, K and V columns, each head at a multiple of hdp
  R_(launch_to_f32_2d(st, cptr(src, so.bqkv, st), 0, w.bqk + i * (dq + dkv), 0, 1, (int)dql, hd,
                      hdp, s));
  R_(launch_to_f32_2d(st, cptr(src, so.bqkv + dql, st), 0, w.bqk + i * (dq + dkv) + dq, 0, 1,
                      (int)dkvl, hd, hdp, s));
  R_(launch_to_f32_2d(st, cptr(src, so.bqkv + dql + dkvl, st), 0, w.bv + i * dkv, 0, 1,
                      (int)dkvl, hd, hdp, s));
  R_(launch_to_f32(st, cptr(src, so.bo, st), w.bo + i * dp, d, s));
  R_(launch_to_f32(st, cptr(src, so.b1, st), w.b1 + i * Fp, F, s));
  R_(launch_to_f32(st, cptr(src, so.b2, st), w.b2 + i * dp, d, s));
  // x W layout [in][out] -> [out][in], converted to the operand type; the output rows of
  // Q, K and V (and the input columns of Wo) go head by head to multiples of hdp
  R_(launch_transpose(st, cptr(src, so.Wqkv, st), wq, dt, WqkT, dp, (int)d, (int)dql, of, s,
                      1, 1, hd, hdp));
  R_(launch_transpose(st, cptr(src, so.Wqkv + dql, st), wq, dt, WqkT + dq * dp * es, dp, (int)d,
                      (int)dkvl, of, s, 1, 1, hd, hdp));
  // The Q projection (the first dq rows of WqkT, the first dq biases) carries the softmax
  // factor log2(e) / sqrt(hd) of the logical head size, so the attention kernels get scores
  // in log2 units straight from their MFMAs.
  {
    const float qs = (float)(1.4426950408889634 / std::sqrt((double)hd));
    R_(launch_scale(dt, WqkT, dq * dp, qs, s));
    R_(launch_scale(DType::F32, w.bqk + i * (dq + dkv), dq, qs, s));
  }
  R_(launch_transpose(st, cptr(src, so.Wqkv + dql + dkvl, st), wq, dt,
                      static_cast<char*>(w.WvT) + i * dkv * dp * es, dp, (int)d, (int)dkvl, of,
                      s, 1, 1, hd, hdp));
  R_(launch_transpose(st, cptr(src, so.Wo, st), d, dt, static_cast<char*>(w.WoT) + i * dp * dq * es,
                      dq, (int)dql, (int)d, of, s, hd, hdp, 1, 1));
  R_(launch_transpose(st, cptr(src, so.W1, st), F, dt, static_cast<char*>(w.W1T) + i * Fp * dp * es,
                      dp, (int)d, (int)F, of, s));
  R_(launch_transpose(st, cptr(src, so.W2, st), d, dt, static_cast<char*>(w.W2T) + i * dp * Fp * es,
                      Fp, (int)F, (int)d, of, s));
#undef R_
  return hipSuccess;
}

GemmDesc gemm_base(DType dt) {
  GemmDesc g;
  std::memset(&g, 0, sizeof(g));
  g.dt = dt;
  g.batch = 1;
  g.kgroups = 1;
  g.gBmod = 1;
  return g;
}

// KV cache of a prefill_kv or decode call.  cache points at layer 0; layer j starts
// j * layer_bytes further.  lens is set for a decode step (host, one entry per sequence).
struct KvRef {
  char* cache = nullptr;
  size_t layer_bytes = 0;
  int max_seqs = 0, cap = 0;
  const int32_t* lens = nullptr;
};

size_t kv_layer_bytes(const kraken_model* m, int max_seqs, int cap) {
  return (size_t)m->N * 2 * (size_t)max_seqs * (size_t)cap * (size_t)m->dkv * sz(m->dt);
}

// fp32 elements available to a decode step's attention partials: the vt and g regions.
int64_t decode_partial_room(const kraken_model* m) {
  return (int64_t)((m->ws_end - static_cast<char*>(m->vt)) / sizeof(float));
}

// The whole pass over T rows, validated by the caller.  Prefill: T packed tokens of
// num_seqs sequences (cu), causal attention within each; with kv, each layer's K and V
// also go to the cache.  Decode (kv->lens set): T = num_seqs new tokens, one per
// sequence; each layer appends its K and V to the cache and attends over it.
// Input: hidden_in [T][d] in the storage type, or NULL when X32 already holds the
// first-layer rows (the embedding lookup wrote them).  Output: hidden_out [T][d] fp32 (may
// be NULL), sub_out [N][T][d] fp32 (may be NULL); *final_rows (if given) receives the
// stored [T][dp] rows of the stack's output (the unembedding's input).
kraken_status forward(kraken_model* m, const void* hidden_in, int T, const int32_t* cu,
                      int32_t num_seqs, const KvRef* kv, float* hidden_out, float* sub_out,
                      const float** final_rows, hipStream_t s) {
  const bool decode = kv && kv->lens;
  const DType dt = m->dt;
  const Dims& D = m->D;
  int* const ovf = m->flags + 1;   // fp16 operand overflow of the activations
  const int64_t N = D.N, d = D.d, dp = D.dp, Fp = D.Fp;
  const int64_t Td = (int64_t)T * dp;
  const int ldv = vt_ld(T);
  hipError_t e;
#define RUN(cls, call, what)                      \
  do {                                            \
    e = m->run(cls, s, [&]() { return (call); }); \
    if (e != hipSuccess) return hip_fail(e, what); \
  } while (0)

  const float* X32 = m->X32;
  if (hidden_in) {
    if (m->st == DType::F32 && d == dp) {
      X32 = static_cast<const float*>(hidden_in);
    } else {
      RUN(KRAKEN_K_OTHER,
          launch_to_f32_2d(m->st, hidden_in, d, m->X32, dp, T, (int)d, 1, 1, s),
          "input conversion");
      if (dp > d)
        RUN(KRAKEN_K_OTHER, launch_zero_cols(DType::F32, m->X32, T, dp, (int)d, (int)dp, s),
            "input padding");
    }
  }

  // Attention reads V^T in 16-byte chunks of 8 tokens; the padding columns [T, ldv) are
  // only ever multiplied by zero probabilities but must hold finite values.
  const int64_t dq = D.dq, dkv = D.dkv, dqk = dq + dkv;   // stored Q, K/V and Q|K widths
  if (!decode && ldv > T)
    RUN(KRAKEN_K_OTHER, launch_zero_cols(dt, m->vt, N * dkv, ldv, T, ldv, s), "V padding");

  for (int j = 0; j < m->L; ++j) {
    const LayerW& w = m->layers[j];
    const float* xin = j == 0 ? X32 : m->xbuf;   // sub-layer inputs x_i
    const int64_t xs = j == 0 ? 0 : Td;           // first layer: one shared input
    char* cache_j = kv ? kv->cache + (size_t)j * kv->layer_bytes : nullptr;
    RUN(KRAKEN_K_LN1,
        launch_layernorm(dt, xin, xs, w.ln1_g, w.ln1_b, m->act, (int)N, T, (int)dp, (int)d,
                         m->eps, ovf, s),
        "ln1");
    {
      GemmDesc g = gemm_base(dt);
      g.epi = EPI_BIAS_N;
      g.A = m->act; g.lda = (int)dp; g.sA = Td;
      g.B = w.WqkT; g.ldb = (int)dp; g.sB = dqk * dp;
      g.C = m->qk; g.ldc = (int)dqk; g.sC = (int64_t)T * dqk;
      g.bias = w.bqk; g.sBias = dqk;
      g.M = T; g.N = (int)dqk; g.K = (int)dp; g.batch = (int)N;
      g.ovf = ovf;
      RUN(KRAKEN_K_GEMM_QK, launch_gemm(g, s), "QK projection");
    }
    if (!decode) {
      {
        GemmDesc g = gemm_base(dt);
        g.epi = EPI_BIAS_M;
        g.A = w.WvT; g.lda = (int)dp; g.sA = dkv * dp;
        g.B = m->act; g.ldb = (int)dp; g.sB = Td;
        g.C = m->vt; g.ldc = ldv; g.sC = dkv * ldv;
        g.bias = w.bv; g.sBias = dkv;
        g.M = (int)dkv; g.N = T; g.K = (int)dp; g.batch = (int)N;
        g.ovf = ovf;
        RUN(KRAKEN_K_GEMM_VT, launch_gemm(g, s), "V projection");
      }
      if (kv)
        RUN(KRAKEN_K_KV,
            launch_kv_store(dt, m->qk, m->vt, cache_j, (int)N, T, (int)dq, D.H, D.Hkv, cu,
                            num_seqs, kv->max_seqs, kv->cap, s),
            "KV store");
      AttnDesc a;
      a.dt = dt; a.qk = m->qk; a.vt = m->vt; a.out = m->o;
      a.n = (int)N; a.T = T; a.d = (int)dq; a.n_heads = D.H; a.n_kv_heads = D.Hkv;
      a.cu_host = cu; a.num_seqs = num_seqs;
      a.q_prescaled = 1;
      RUN(KRAKEN_K_ATTN, launch_attention(a, s), "attention");
    } else {
      // V rows of the new tokens go through o ([N][T][dkv]) into the cache; o then takes
      // the attention output, after the append has read it (stream order).
      {
        GemmDesc g = gemm_base(dt);
        g.epi = EPI_BIAS_N;
        g.A = m->act; g.lda = (int)dp; g.sA = Td;
        g.B = w.WvT; g.ldb = (int)dp; g.sB = dkv * dp;
        g.C = m->o; g.ldc = (int)dkv; g.sC = (int64_t)T * dkv;
        g.bias = w.bv; g.sBias = dkv;
        g.M = T; g.N = (int)dkv; g.K = (int)dp; g.batch = (int)N;
        g.ovf = ovf;
        RUN(KRAKEN_K_GEMM_VT, launch_gemm(g, s), "V projection");
      }
      RUN(KRAKEN_K_KV,
          launch_kv_append(dt, m->qk, m->o, cache_j, (int)N, T, (int)dq, D.H, D.Hkv, kv->lens,
                           kv->max_seqs, kv->cap, s),
          "KV append");
      RUN(KRAKEN_K_ATTN,
          launch_decode_attention(dt, m->qk, cache_j, static_cast<float*>(m->vt),
                                  decode_partial_room(m), m->o, (int)N, T, (int)dq, D.H, D.Hkv,
                                  kv->lens, kv->max_seqs, kv->cap, 1, s),
          "decode attention");
    }
    {
      GemmDesc g = gemm_base(dt);
      g.epi = EPI_BIAS_N_RES;
      g.A = m->o; g.lda = (int)dq; g.sA = (int64_t)T * dq;
      g.B = w.WoT; g.ldb = (int)dq; g.sB = dp * dq;
      g.C = m->hbuf; g.ldc = (int)dp; g.sC = Td;
      g.bias = w.bo; g.sBias = dp;
      g.R = xin; g.sR = xs;
      g.M = T; g.N = (int)dp; g.K = (int)dq; g.batch = (int)N;
      RUN(KRAKEN_K_GEMM_O, launch_gemm(g, s), "output projection");
    }
    // The FFN's LayerNorm: Kraken reads h + y with y the combine (Algorithm 1); the
    // GPT-like layer reads h; the parallel layer's FFN takes the LN1 output still in act.
    if (D.arch == KRAKEN_ARCH_KRAKEN)
      RUN(KRAKEN_K_COMBINE,
          launch_combine_ln2(dt, m->xbuf, j == 0 ? X32 : nullptr, m->hbuf, w.ln2_g, w.ln2_b,
                             m->act, (int)N, T, (int)dp, (int)d, m->eps, ovf, s),
          "combine + ln2");
    else if (D.arch == KRAKEN_ARCH_GPT)
      RUN(KRAKEN_K_COMBINE,
          launch_layernorm(dt, m->hbuf, Td, w.ln2_g, w.ln2_b, m->act, (int)N, T, (int)dp, (int)d,
                           m->eps, ovf, s),
          "ln2");
    {
      GemmDesc g = gemm_base(dt);
      g.epi = EPI_BIAS_N_GELU;
      g.A = m->act; g.lda = (int)dp; g.sA = Td;
      g.B = w.W1T; g.ldb = (int)dp; g.sB = Fp * dp;
      g.C = m->g; g.ldc = (int)Fp; g.sC = (int64_t)T * Fp;
      g.bias = w.b1; g.sBias = Fp;
      g.M = T; g.N = (int)Fp; g.K = (int)dp; g.batch = (int)N;
      g.ovf = ovf;
      RUN(KRAKEN_K_GEMM_UP, launch_gemm(g, s), "FFN up");
    }
    {
      GemmDesc g = gemm_base(dt);
      g.epi = EPI_BIAS_N_RES;
      g.A = m->g; g.lda = (int)Fp; g.sA = (int64_t)T * Fp;
      g.B = w.W2T; g.ldb = (int)Fp; g.sB = dp * Fp;
      g.C = m->xbuf; g.ldc = (int)dp; g.sC = Td;
      g.bias = w.b2; g.sBias = dp;
      g.R = m->hbuf; g.sR = Td;
      g.M = T; g.N = (int)dp; g.K = (int)Fp; g.batch = (int)N;
      RUN(KRAKEN_K_GEMM_DOWN, launch_gemm(g, s), "FFN down");
    }
  }

  if (sub_out)
    RUN(KRAKEN_K_OTHER,
        hipMemcpy2DAsync(sub_out, d * sizeof(float), m->xbuf, dp * sizeof(float),
                         d * sizeof(float), N * T, hipMemcpyDeviceToDevice, s),
        "sub_out copy");

  const float* fin = m->xbuf;   // the stack's output rows, [T][dp]
  if (D.arch == KRAKEN_ARCH_KRAKEN) {
    // out = [Y_1 | ... | Y_N] W_concat, K split into N groups of dp (one per sub-layer).
    // Into the caller's [T][d] directly, or into X32 (free after the first layer) when the
    // stored rows are wanted.
    GemmDesc g = gemm_base(dt);
    g.epi = EPI_BIAS_N_RES;
    if (dt != DType::F32) {
      // 16-bit operands: Y = hi + lo with hi = S(Y), lo = S(Y - hi); 2N groups
      RUN(KRAKEN_K_CONCAT, launch_split16(dt, m->xbuf, m->g, N * Td, ovf, s),
          "W_concat operand split");
      g.A = m->g;
      g.kgroups = (int)(2 * N);
    } else {
      g.A = m->xbuf;
      g.kgroups = (int)N;
    }
    g.lda = (int)dp; g.gA = Td;
    g.B = m->WcatT; g.ldb = (int)(N * dp); g.gB = dp; g.gBmod = (int)N;
    g.M = T; g.K = (int)dp;
    if (final_rows) {
      g.C = m->X32; g.ldc = (int)dp; g.N = (int)dp;
      fin = m->X32;
    } else {
      g.C = hidden_out; g.ldc = (int)d; g.N = (int)d;
    }
    RUN(KRAKEN_K_CONCAT, launch_gemm(g, s), "W_concat");
    if (final_rows && hidden_out)
      RUN(KRAKEN_K_OTHER,
          hipMemcpy2DAsync(hidden_out, d * sizeof(float), fin, dp * sizeof(float),
                           d * sizeof(float), T, hipMemcpyDeviceToDevice, s),
          "output copy");
  } else if (hidden_out) {
    // the GPT-like and parallel stacks end with their last layer's output
    RUN(KRAKEN_K_OTHER,
        hipMemcpy2DAsync(hidden_out, d * sizeof(float), fin, dp * sizeof(float),
                         d * sizeof(float), T, hipMemcpyDeviceToDevice, s),
        "output copy");
  }
  if (final_rows) *final_rows = fin;
#undef RUN
  return KRAKEN_OK;
}

// Checks shared by prefill_kv and decode: a cache for this model's sizes.
kraken_status check_cache(const kraken_model* m, const void* cache, int32_t max_seqs,
                          int32_t capacity, int32_t num_seqs, size_t* bytes) {
  if (!cache) return fail(KRAKEN_ERR_INVALID_ARG, "kv_cache is NULL");
  if (reinterpret_cast<uintptr_t>(cache) % 16 != 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "kv_cache is not 16-byte aligned");
  if (max_seqs < 1 || max_seqs > KRAKEN_MAX_SEQS || capacity < 1)
    return fail(KRAKEN_ERR_INVALID_ARG, "max_seqs out of 1..KRAKEN_MAX_SEQS or capacity < 1");
  if (num_seqs > max_seqs) return fail(KRAKEN_ERR_INVALID_ARG, "num_seqs exceeds max_seqs");
  *bytes = kv_layer_bytes(m, max_seqs, capacity) * (size_t)m->L;
  return KRAKEN_OK;
}

}  // namespace

extern "C" {

const char* kraken_status_string(kraken_status s) {
  // A C caller may pass any int; in C++ an enum object holding a value outside the enum's
  // range is undefined behaviour, so the code is read as the int it is.
  int code;
  std::memcpy(&code, &s, sizeof code);
  switch (code) {
    case KRAKEN_OK: return "ok";
    case KRAKEN_ERR_INVALID_ARG: return "invalid argument";
    case KRAKEN_ERR_UNSUPPORTED: return "unsupported configuration";
    case KRAKEN_ERR_OOM: return "out of device memory";
    case KRAKEN_ERR_STATE: return "invalid state";
    case KRAKEN_ERR_HIP: return "HIP error";
    case KRAKEN_ERR_OVERFLOW: return "fp16 activation overflow";
  }
  return "unknown status";
}

const char* kraken_last_error(void) { return g_last_error.c_str(); }

size_t kraken_weight_blob_elems(const kraken_config* c) {
  if (!c || c->n_sub < 1 || c->n_layers < 1 || c->d_model < 1 || c->d_ff < 0 ||
      c->n_heads < 1 || c->n_kv_heads < 0 || c->head_dim < 0 || c->vocab < 0 ||
      c->max_positions < 0 || c->arch < KRAKEN_ARCH_KRAKEN || c->arch > KRAKEN_ARCH_PARALLEL)
    return 0;
  const Dims D = dims_of(c);
  if (D.hd < 1) return 0;
  const SubOffsets so(D);
  size_t n = (size_t)D.L * D.N * (size_t)so.total;
  if (D.arch == KRAKEN_ARCH_KRAKEN) n += (size_t)D.N * D.d * D.d;
  if (D.V > 0) n += ((size_t)D.V + D.P) * D.d + 2 * (size_t)D.d;
  return n;
}

kraken_status kraken_create(const kraken_config* cfg, kraken_model** out) {
  if (!out) return fail(KRAKEN_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  kraken_status st = validate_cfg(cfg);
  if (st != KRAKEN_OK) return st;
  kraken_model* m = new (std::nothrow) kraken_model();
  if (!m) return fail(KRAKEN_ERR_OOM, "host allocation failed");
  m->cfg = *cfg;
  m->D = dims_of(cfg);
  m->st = (DType)cfg->dtype;
  m->dt = cfg->compute == KRAKEN_COMPUTE_STORAGE ? m->st : (DType)(cfg->compute - 1);
  m->N = cfg->n_sub;
  m->L = cfg->n_layers;
  m->d = m->D.d;
  m->H = cfg->n_heads;
  m->Hkv = m->D.Hkv;
  m->F = m->D.F;
  m->dp = m->D.dp;
  m->Fp = m->D.Fp;
  m->dq = m->D.dq;
  m->dkv = m->D.dkv;
  m->Tmax = cfg->max_tokens;
  m->eps = cfg->ln_eps > 0.f ? cfg->ln_eps : 1e-5f;
  {
    const char* dbg = std::getenv("KRAKEN_DEBUG_SYNC");
    m->debug_sync = dbg && dbg[0] && std::strcmp(dbg, "0") != 0;
  }
  hipError_t e = hipGetDevice(&m->device);
  if (e != hipSuccess) {
    delete m;
    return hip_fail(e, "hipGetDevice");
  }
  const size_t wbytes = carve_weights(m, nullptr);
  const size_t abytes = carve_workspace(m, nullptr);
  if (hipMalloc(&m->wmem, wbytes) != hipSuccess) {
    (void)hipGetLastError();
    m->wmem = nullptr;
    delete m;
    return fail(KRAKEN_ERR_OOM, "weight allocation of " + std::to_string(wbytes) + " bytes failed");
  }
  if (hipMalloc(&m->amem, abytes) != hipSuccess) {
    (void)hipGetLastError();
    m->amem = nullptr;
    free_model_memory(m);
    delete m;
    return fail(KRAKEN_ERR_OOM, "workspace allocation of " + std::to_string(abytes) + " bytes failed");
  }
  carve_weights(m, m->wmem);
  carve_workspace(m, m->amem);
  m->wbytes = wbytes;
  if (m->D.V > 0) {
    // pinned staging of a token call's ids, positions and last rows, and the event that
    // tells when the previous call's copy has read it
    const size_t hb = (2 * (size_t)m->Tmax + KRAKEN_MAX_SEQS) * sizeof(int);
    if (hipHostMalloc((void**)&m->tok_host, hb, hipHostMallocDefault) != hipSuccess) {
      (void)hipGetLastError();
      m->tok_host = nullptr;
      free_model_memory(m);
      delete m;
      return fail(KRAKEN_ERR_OOM, "pinned host allocation failed");
    }
    if (hipEventCreateWithFlags(&m->tok_copied, hipEventDisableTiming) != hipSuccess) {
      (void)hipGetLastError();
      hipHostFree(m->tok_host);
      free_model_memory(m);
      delete m;
      return fail(KRAKEN_ERR_HIP, "event creation failed");
    }
  }
  *out = m;
  return KRAKEN_OK;
}

kraken_status kraken_destroy(kraken_model* m) {
  if (!m) return KRAKEN_OK;
  hipDeviceSynchronize();
  for (auto& r : m->pending) {
    hipEventDestroy(r.a);
    hipEventDestroy(r.b);
  }
  for (auto e : m->pool) hipEventDestroy(e);
  if (m->tok_copied) hipEventDestroy(m->tok_copied);
  if (m->tok_host) hipHostFree(m->tok_host);
  free_model_memory(m);
  delete m;
  return KRAKEN_OK;
}

kraken_status kraken_load_weights(kraken_model* m, const void* blob, size_t nbytes,
                                  int blob_is_device, void* stream) {
  if (!m || !blob) return fail(KRAKEN_ERR_INVALID_ARG, "model or blob is NULL");
  const size_t elems = kraken_weight_blob_elems(&m->cfg);
  if (nbytes != elems * sz(m->st))
    return fail(KRAKEN_ERR_INVALID_ARG, "blob size " + std::to_string(nbytes) + " != expected " +
                                            std::to_string(elems * sz(m->st)));
  kraken_status st = check_device(m);
  if (st != KRAKEN_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const Dims& D = m->D;
  const int64_t d = D.d, N = D.N, dp = D.dp;
  const SubOffsets so(D);
  const int64_t layer_elems = N * so.total;
  // the pieces after the layers: W_concat (Kraken), then the embeddings
  int64_t tail = (int64_t)m->L * layer_elems;
  const int64_t wcat_off = tail;
  if (D.arch == KRAKEN_ARCH_KRAKEN) tail += N * d * d;
  const int64_t tok_off = tail, pos_off = tok_off + (int64_t)D.V * d;
  const int64_t lnf_off = pos_off + (int64_t)D.P * d;
  void* staging = nullptr;
  if (!blob_is_device) {
    const int64_t biggest = std::max<int64_t>(
        {layer_elems, N * d * d, (int64_t)D.V * d, (int64_t)D.P * d, 2 * d});
    if (hipMalloc(&staging, biggest * sz(m->st)) != hipSuccess) {
      (void)hipGetLastError();
      return fail(KRAKEN_ERR_OOM, "staging allocation failed");
    }
  }
  auto cleanup = [&]() {
    if (staging) {
      hipStreamSynchronize(s);
      hipFree(staging);
    }
  };
  // device address of `elems` blob elements at `off` (uploaded through the staging buffer
  // for a host blob; the previous piece's repack has finished reading it by then)
  hipError_t e = hipSuccess;
  auto piece = [&](int64_t off, int64_t count) -> const void* {
    const void* src = cptr(blob, off, m->st);
    if (blob_is_device) return src;
    e = hipStreamSynchronize(s);
    if (e == hipSuccess)
      e = hipMemcpyAsync(staging, src, count * sz(m->st), hipMemcpyHostToDevice, s);
    return staging;
  };
  m->loaded = false;
  // zero everything first: padding weights, biases and gains must be zero (and the flags)
  e = hipMemsetAsync(m->wmem, 0, m->wbytes, s);
  if (e != hipSuccess) {
    cleanup();
    return hip_fail(e, "weight arena reset");
  }
  for (int j = 0; j < m->L; ++j) {
    const void* src = piece(j * layer_elems, layer_elems);
    if (e != hipSuccess) {
      cleanup();
      return hip_fail(e, "weight upload");
    }
    for (int i = 0; i < m->N; ++i) {
      e = repack_sub(m, j, i, cptr(src, i * so.total, m->st), s);
      if (e != hipSuccess) {
        cleanup();
        return hip_fail(e, "weight repack");
      }
    }
  }
  if (D.arch == KRAKEN_ARCH_KRAKEN) {
    // W_concat [N d][d] -> [dp][N dp]: row block i (sub-layer i) to columns i dp ..
    const void* wsrc = piece(wcat_off, N * d * d);
    if (e == hipSuccess)
      e = launch_transpose(m->st, wsrc, d, m->dt, m->WcatT, N * dp, (int)(N * d), (int)d,
                           m->flags, s, (int)d, (int)dp, 1, 1);
    if (e != hipSuccess) {
      cleanup();
      return hip_fail(e, "W_concat repack");
    }
  }
  if (D.V > 0) {
    // token rows [V][d] -> [V][dp] in the operand type (the unembedding's B operand as is),
    // position rows -> fp32 [P][dp], final LayerNorm -> fp32
    const void* tsrc = piece(tok_off, (int64_t)D.V * d);
    if (e == hipSuccess)
      e = launch_convert_2d(m->st, tsrc, d, m->dt, m->tok, dp, D.V, (int)d, m->flags, s);
    const void* psrc = e == hipSuccess ? piece(pos_off, (int64_t)D.P * d) : nullptr;
    if (e == hipSuccess)
      e = launch_to_f32_2d(m->st, psrc, d, m->pos, dp, D.P, (int)d, 1, 1, s);
    const void* lsrc = e == hipSuccess ? piece(lnf_off, 2 * d) : nullptr;
    if (e == hipSuccess) e = launch_to_f32(m->st, lsrc, m->lnf_g, d, s);
    if (e == hipSuccess) e = launch_to_f32(m->st, cptr(lsrc, d, m->st), m->lnf_b, d, s);
    if (e != hipSuccess) {
      cleanup();
      return hip_fail(e, "embedding repack");
    }
  }
  cleanup();
  if (m->dt == DType::F16 && m->st != DType::F16) {
    int flag = 0;
    e = hipMemcpyAsync(&flag, m->flags, sizeof(int), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "overflow check");
    if (flag) return fail(KRAKEN_ERR_UNSUPPORTED, "a weight exceeds the fp16 operand range");
  }
  m->loaded = true;
  return KRAKEN_OK;
}

kraken_status kraken_prefill(kraken_model* m, const void* hidden_in, const int32_t* cu_seqlens,
                             int32_t num_seqs, float* hidden_out, float* sub_out, void* stream) {
  return kraken_prefill_kv(m, hidden_in, cu_seqlens, num_seqs, hidden_out, sub_out, nullptr, 0, 0,
                           stream);
}

size_t kraken_kv_cache_bytes(const kraken_config* c, int32_t max_seqs, int32_t capacity) {
  if (!c || validate_cfg(c) != KRAKEN_OK) return 0;
  if (max_seqs < 1 || max_seqs > KRAKEN_MAX_SEQS || capacity < 1) return 0;
  const DType st = (DType)c->dtype;
  const DType dt = c->compute == KRAKEN_COMPUTE_STORAGE ? st : (DType)(c->compute - 1);
  const size_t dkv = (size_t)dims_of(c).dkv;   // stored key/value width
  return (size_t)c->n_layers * (size_t)c->n_sub * 2 * (size_t)max_seqs * (size_t)capacity *
         dkv * sz(dt);
}

kraken_status kraken_prefill_kv(kraken_model* m, const void* hidden_in, const int32_t* cu_seqlens,
                                int32_t num_seqs, float* hidden_out, float* sub_out,
                                void* kv_cache, int32_t max_seqs, int32_t capacity, void* stream) {
  if (!m) return fail(KRAKEN_ERR_INVALID_ARG, "model is NULL");
  if (!hidden_in || !hidden_out) return fail(KRAKEN_ERR_INVALID_ARG, "hidden_in or hidden_out is NULL");
  if (!m->loaded) return fail(KRAKEN_ERR_STATE, "weights are not loaded");
  int64_t T64 = 0;
  kraken_status st = check_cu(cu_seqlens, num_seqs, m->Tmax, &T64);
  if (st != KRAKEN_OK) return st;
  const int T = (int)T64;
  const int64_t N = m->N, d = m->d;
  const size_t in_bytes = T * d * sz(m->st), out_bytes = T * d * 4, sub_bytes = N * T * d * 4;
  if (overlap(hidden_in, in_bytes, hidden_out, out_bytes) ||
      overlap(hidden_in, in_bytes, sub_out, sub_bytes) ||
      overlap(hidden_out, out_bytes, sub_out, sub_bytes))
    return fail(KRAKEN_ERR_INVALID_ARG, "input and output buffers overlap");
  KvRef kv;
  const bool with_kv = kv_cache != nullptr;
  if (with_kv) {
    size_t cbytes = 0;
    st = check_cache(m, kv_cache, max_seqs, capacity, num_seqs, &cbytes);
    if (st != KRAKEN_OK) return st;
    for (int b = 0; b < num_seqs; ++b)
      if (cu_seqlens[b + 1] - cu_seqlens[b] > capacity)
        return fail(KRAKEN_ERR_INVALID_ARG, "a sequence is longer than the cache capacity");
    if (overlap(kv_cache, cbytes, hidden_in, in_bytes) ||
        overlap(kv_cache, cbytes, hidden_out, out_bytes) ||
        overlap(kv_cache, cbytes, sub_out, sub_bytes))
      return fail(KRAKEN_ERR_INVALID_ARG, "kv_cache overlaps another buffer");
    kv.cache = static_cast<char*>(kv_cache);
    kv.layer_bytes = kv_layer_bytes(m, max_seqs, capacity);
    kv.max_seqs = max_seqs;
    kv.cap = capacity;
  }
  st = check_device(m);
  if (st != KRAKEN_OK) return st;
  return forward(m, hidden_in, T, cu_seqlens, num_seqs, with_kv ? &kv : nullptr, hidden_out,
                 sub_out, nullptr, static_cast<hipStream_t>(stream));
}

kraken_status kraken_decode(kraken_model* m, const void* hidden_in, const int32_t* lens,
                            int32_t num_seqs, float* hidden_out, float* sub_out, void* kv_cache,
                            int32_t max_seqs, int32_t capacity, void* stream) {
  if (!m) return fail(KRAKEN_ERR_INVALID_ARG, "model is NULL");
  if (!hidden_in || !hidden_out || !lens)
    return fail(KRAKEN_ERR_INVALID_ARG, "hidden_in, hidden_out or lens is NULL");
  if (!m->loaded) return fail(KRAKEN_ERR_STATE, "weights are not loaded");
  if (num_seqs < 1 || num_seqs > KRAKEN_MAX_SEQS || num_seqs > m->Tmax)
    return fail(KRAKEN_ERR_INVALID_ARG, "num_seqs out of 1..min(KRAKEN_MAX_SEQS, max_tokens)");
  size_t cbytes = 0;
  kraken_status st = check_cache(m, kv_cache, max_seqs, capacity, num_seqs, &cbytes);
  if (st != KRAKEN_OK) return st;
  for (int b = 0; b < num_seqs; ++b)
    if (lens[b] < 0 || lens[b] >= capacity)
      return fail(KRAKEN_ERR_INVALID_ARG, "lens[b] out of 0..capacity-1");
  const int B = num_seqs;
  const int64_t N = m->N, d = m->d;
  const size_t in_bytes = B * d * sz(m->st), out_bytes = B * d * 4, sub_bytes = N * B * d * 4;
  if (overlap(hidden_in, in_bytes, hidden_out, out_bytes) ||
      overlap(hidden_in, in_bytes, sub_out, sub_bytes) ||
      overlap(hidden_out, out_bytes, sub_out, sub_bytes))
    return fail(KRAKEN_ERR_INVALID_ARG, "input and output buffers overlap");
  if (overlap(kv_cache, cbytes, hidden_in, in_bytes) ||
      overlap(kv_cache, cbytes, hidden_out, out_bytes) ||
      overlap(kv_cache, cbytes, sub_out, sub_bytes))
    return fail(KRAKEN_ERR_INVALID_ARG, "kv_cache overlaps another buffer");
  if (decode_partial_floats((int)N, B, m->H, m->D.hdp, 1) > decode_partial_room(m))
    return fail(KRAKEN_ERR_UNSUPPORTED, "workspace too small for the decode attention partials");
  st = check_device(m);
  if (st != KRAKEN_OK) return st;
  KvRef kv;
  kv.cache = static_cast<char*>(kv_cache);
  kv.layer_bytes = kv_layer_bytes(m, max_seqs, capacity);
  kv.max_seqs = max_seqs;
  kv.cap = capacity;
  kv.lens = lens;
  return forward(m, hidden_in, B, nullptr, num_seqs, &kv, hidden_out, sub_out, nullptr,
                 static_cast<hipStream_t>(stream));
}

kraken_status kraken_forward_tokens(kraken_model* m, const int32_t* token_ids,
                                    const int32_t* cu_seqlens, int32_t num_seqs, float* logits,
                                    float* hidden_out, void* stream) {
  if (!m) return fail(KRAKEN_ERR_INVALID_ARG, "model is NULL");
  const Dims& D = m->D;
  if (D.V <= 0) return fail(KRAKEN_ERR_STATE, "the model has no embeddings (vocab = 0)");
  if (!token_ids || !logits) return fail(KRAKEN_ERR_INVALID_ARG, "token_ids or logits is NULL");
  if (!m->loaded) return fail(KRAKEN_ERR_STATE, "weights are not loaded");
  int64_t T64 = 0;
  kraken_status st = check_cu(cu_seqlens, num_seqs, m->Tmax, &T64);
  if (st != KRAKEN_OK) return st;
  const int T = (int)T64, B = num_seqs;
  for (int b = 0; b < B; ++b)
    if (cu_seqlens[b + 1] - cu_seqlens[b] > D.P)
      return fail(KRAKEN_ERR_INVALID_ARG, "a sequence is longer than max_positions");
  for (int t = 0; t < T; ++t)
    if (token_ids[t] < 0 || token_ids[t] >= D.V)
      return fail(KRAKEN_ERR_INVALID_ARG, "a token id is outside 0..vocab-1");
  const size_t lbytes = (size_t)B * D.V * 4, obytes = (size_t)T * D.d * 4;
  if (overlap(logits, lbytes, hidden_out, obytes))
    return fail(KRAKEN_ERR_INVALID_ARG, "logits and hidden_out overlap");
  st = check_device(m);
  if (st != KRAKEN_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // ids, positions within each sequence, last row of each sequence -> pinned staging ->
  // device (the previous call's copy must have read the staging first)
  HIP_TRY(hipEventSynchronize(m->tok_copied), "token staging wait");
  int* h = m->tok_host;
  for (int b = 0; b < B; ++b) {
    for (int t = cu_seqlens[b]; t < cu_seqlens[b + 1]; ++t) {
      h[t] = token_ids[t];
      h[T + t] = t - cu_seqlens[b];
    }
    h[2 * T + b] = cu_seqlens[b + 1] - 1;
  }
  HIP_TRY(hipMemcpyAsync(m->tok_ids, h, (2 * (size_t)T + B) * sizeof(int), hipMemcpyHostToDevice,
                         s),
          "token upload");
  HIP_TRY(hipEventRecord(m->tok_copied, s), "hipEventRecord");
  const int dp = D.dp;
  hipError_t e;
#define RUN(cls, call, what)                      \
  do {                                            \
    e = m->run(cls, s, [&]() { return (call); }); \
    if (e != hipSuccess) return hip_fail(e, what); \
  } while (0)
  // Section 3.1: one token + position embedding, shared by the first layer's sub-layers
  RUN(KRAKEN_K_OTHER, launch_embed(m->dt, m->tok_ids, m->tok_ids + T, m->tok, m->pos, m->X32, T,
                                   dp, s),
      "embedding");
  const float* fin = nullptr;
  st = forward(m, nullptr, T, cu_seqlens, B, nullptr, hidden_out, nullptr, &fin, s);
  if (st != KRAKEN_OK) return st;
  // the unembedding of each sequence's last token: ln_f, then logits = z tok^T (tied)
  RUN(KRAKEN_K_OTHER, launch_gather_rows(fin, m->tok_ids + 2 * T, m->last, B, dp, s),
      "last-row gather");
  RUN(KRAKEN_K_OTHER,
      launch_layernorm(m->dt, m->last, 0, m->lnf_g, m->lnf_b, m->last_act, 1, B, dp, D.d, m->eps,
                       m->flags + 1, s),
      "final LayerNorm");
  {
    GemmDesc g = gemm_base(m->dt);
    g.epi = EPI_BIAS_N_RES;
    g.A = m->last_act; g.lda = dp;
    g.B = m->tok; g.ldb = dp;
    g.C = logits; g.ldc = D.V;
    g.M = B; g.N = D.V; g.K = dp;
    RUN(KRAKEN_K_UNEMBED, launch_gemm(g, s), "unembedding");
  }
#undef RUN
  return KRAKEN_OK;
}

kraken_status kraken_sync(kraken_model* m, void* stream) {
  if (!m) return fail(KRAKEN_ERR_INVALID_ARG, "model is NULL");
  kraken_status st = check_device(m);
  if (st != KRAKEN_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int flag = 0;
  HIP_TRY(hipMemcpyAsync(&flag, m->flags + 1, sizeof(int), hipMemcpyDeviceToHost, s),
          "overflow flag read");
  HIP_TRY(hipStreamSynchronize(s), "hipStreamSynchronize");
  if (flag) {
    HIP_TRY(hipMemsetAsync(m->flags + 1, 0, sizeof(int), s), "overflow flag reset");
    HIP_TRY(hipStreamSynchronize(s), "hipStreamSynchronize");
    return fail(KRAKEN_ERR_OVERFLOW,
                "an activation exceeded the fp16 operand range since the last kraken_sync; "
                "the outputs of those calls are not valid");
  }
  return KRAKEN_OK;
}

kraken_status kraken_debug_poison_workspace(kraken_model* m, void* stream) {
  if (!m) return fail(KRAKEN_ERR_INVALID_ARG, "model is NULL");
  kraken_status st = check_device(m);
  if (st != KRAKEN_OK) return st;
  const size_t bytes = (size_t)(m->ws_end - static_cast<char*>(m->amem));
  HIP_TRY(hipMemsetAsync(m->amem, 0xff, bytes, static_cast<hipStream_t>(stream)),
          "workspace poison");
  return KRAKEN_OK;
}

kraken_status kraken_profile_enable(kraken_model* m, int enable) {
  if (!m) return fail(KRAKEN_ERR_INVALID_ARG, "model is NULL");
  m->prof = enable != 0;
  return KRAKEN_OK;
}

kraken_status kraken_profile_read(kraken_model* m, int cls, double* total_ms, int64_t* launches) {
  if (!m || !total_ms || !launches) return fail(KRAKEN_ERR_INVALID_ARG, "NULL argument");
  if (cls < 0 || cls >= KRAKEN_K_COUNT) return fail(KRAKEN_ERR_INVALID_ARG, "bad kernel class");
  for (auto& r : m->pending) {
    hipError_t e = hipEventSynchronize(r.b);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    m->prof_ms[r.cls] += ms;
    m->prof_n[r.cls] += 1;
    m->pool.push_back(r.a);
    m->pool.push_back(r.b);
  }
  m->pending.clear();
  *total_ms = m->prof_ms[cls];
  *launches = m->prof_n[cls];
  return KRAKEN_OK;
}

kraken_status kraken_profile_reset(kraken_model* m) {
  if (!m) return fail(KRAKEN_ERR_INVALID_ARG, "model is NULL");
  double t;
  int64_t n;
  kraken_status st = kraken_profile_read(m, 0, &t, &n);  // drains pending events
  if (st != KRAKEN_OK) return st;
  for (int k = 0; k < KRAKEN_K_COUNT; ++k) {
    m->prof_ms[k] = 0;
    m->prof_n[k] = 0;
  }
  return KRAKEN_OK;
}

double kraken_class_flops(const kraken_config* c, int cls, const int32_t* cu, int32_t num_seqs) {
  if (!c || !cu || num_seqs < 1 || c->n_heads < 1) return 0.0;
  const Dims D = dims_of(c);
  // algorithmic work of the logical model (padding excluded)
  const double N = D.N, L = D.L, d = D.d, F = D.F, dq = (double)D.dq_l, dkv = (double)D.dkv_l;
  const double T = cu[num_seqs];
  switch (cls) {
    case KRAKEN_K_GEMM_QK: return L * N * 2.0 * T * d * (dq + dkv);
    case KRAKEN_K_GEMM_VT: return L * N * 2.0 * T * d * dkv;
    case KRAKEN_K_GEMM_O: return L * N * 2.0 * T * dq * d;
    case KRAKEN_K_GEMM_UP: return L * N * 2.0 * T * d * F;
    case KRAKEN_K_GEMM_DOWN: return L * N * 2.0 * T * F * d;
    case KRAKEN_K_CONCAT: return D.arch == KRAKEN_ARCH_KRAKEN ? 2.0 * T * N * d * d : 0.0;
    case KRAKEN_K_UNEMBED: return D.V > 0 ? 2.0 * num_seqs * d * (double)D.V : 0.0;
    case KRAKEN_K_ATTN: {
      // QK^T and PV over causal pairs: 4 hd flops per pair and head = 4 dq per pair
      double pairs = 0;
      for (int b = 0; b < num_seqs; ++b) {
        const double S = cu[b + 1] - cu[b];
        pairs += S * (S + 1) / 2.0;
      }
      return L * N * 4.0 * dq * pairs;
    }
    default: return 0.0;
  }
}

// ----------------------------------------------------------------------------- single ops

kraken_status kraken_op_layernorm(int32_t dtype, const float* x, int64_t xs, const float* gamma,
                                  const float* beta, void* out, int32_t n, int32_t T, int32_t d,
                                  float eps, void* stream) {
  if (!x || !gamma || !beta || !out) return fail(KRAKEN_ERR_INVALID_ARG, "NULL pointer");
  if (dtype < KRAKEN_DTYPE_F32 || dtype > KRAKEN_DTYPE_F16)
    return fail(KRAKEN_ERR_UNSUPPORTED, "unknown dtype");
  if (n < 1 || T < 0 || d < 4 || d % 64 != 0 || d > 16384 || xs < 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "bad sizes");
  hipError_t e = launch_layernorm((DType)dtype, x, xs, gamma, beta, out, n, T, d, d, eps, nullptr,
                                  static_cast<hipStream_t>(stream));
  return e == hipSuccess ? KRAKEN_OK : hip_fail(e, "layernorm");
}

kraken_status kraken_op_combine_ln2(int32_t dtype, const float* x, const float* shared,
                                    const float* h, const float* gamma, const float* beta,
                                    void* out, int32_t n, int32_t T, int32_t d, float eps,
                                    void* stream) {
  if ((!x && !shared) || !h || !gamma || !beta || !out)
    return fail(KRAKEN_ERR_INVALID_ARG, "NULL pointer");
  if (dtype < KRAKEN_DTYPE_F32 || dtype > KRAKEN_DTYPE_F16)
    return fail(KRAKEN_ERR_UNSUPPORTED, "unknown dtype");
  if (n < 1 || T < 0 || d % 64 != 0 || d < 64 || d > 16384)
    return fail(KRAKEN_ERR_INVALID_ARG, "bad sizes");
  hipError_t e = launch_combine_ln2((DType)dtype, x, shared, h, gamma, beta, out, n, T, d, d, eps,
                                    nullptr, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? KRAKEN_OK : hip_fail(e, "combine_ln2");
}

kraken_status kraken_op_gemm(int32_t dtype, int32_t epilogue, const void* A, const void* B,
                             void* C, const float* bias, const float* R, int32_t M, int32_t N,
                             int32_t K, int32_t batch, int64_t sA, int64_t sB, int64_t sC,
                             int64_t sR, void* stream) {
  if (!A || !B || !C) return fail(KRAKEN_ERR_INVALID_ARG, "NULL pointer");
  if (dtype < KRAKEN_DTYPE_F32 || dtype > KRAKEN_DTYPE_F16)
    return fail(KRAKEN_ERR_UNSUPPORTED, "unknown dtype");
  if (epilogue < 0 || epilogue > 3) return fail(KRAKEN_ERR_INVALID_ARG, "bad epilogue");
  if (M < 1 || N < 1 || K < 64 || K % 64 != 0 || batch < 1 || sA < 0 || sB < 0 || sC < 0 || sR < 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "bad sizes");
  GemmDesc g = gemm_base((DType)dtype);
  g.epi = epilogue;
  g.A = A; g.B = B; g.C = C; g.bias = bias; g.R = R;
  g.M = M; g.N = N; g.K = K; g.lda = K; g.ldb = K; g.ldc = N;
  g.sA = sA; g.sB = sB; g.sC = sC; g.sR = sR;
  g.sBias = epilogue == EPI_BIAS_M ? M : N;
  g.batch = batch;
  hipError_t e = launch_gemm(g, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? KRAKEN_OK : hip_fail(e, "gemm");
}

kraken_status kraken_op_attention(int32_t dtype, const void* qk, const void* vt, void* out,
                                  int32_t n, int32_t d, int32_t n_heads, int32_t n_kv_heads,
                                  int32_t q_prescaled, const int32_t* cu_seqlens,
                                  int32_t num_seqs, void* stream) {
  if (!qk || !vt || !out) return fail(KRAKEN_ERR_INVALID_ARG, "NULL pointer");
  if (dtype < KRAKEN_DTYPE_F32 || dtype > KRAKEN_DTYPE_F16)
    return fail(KRAKEN_ERR_UNSUPPORTED, "unknown dtype");
  if (n < 1 || d < 1 || n_heads < 1 || d % n_heads != 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "bad sizes");
  const int hd = d / n_heads;
  if (hd != 32 && hd != 64 && hd != 128) return fail(KRAKEN_ERR_UNSUPPORTED, "head size");
  if (n_kv_heads < 0 || (n_kv_heads > 0 && n_heads % n_kv_heads != 0))
    return fail(KRAKEN_ERR_INVALID_ARG, "n_kv_heads must be 0 or divide n_heads");
  int64_t T = 0;
  kraken_status st = check_cu(cu_seqlens, num_seqs, INT32_MAX, &T);
  if (st != KRAKEN_OK) return st;
  AttnDesc a;
  a.dt = (DType)dtype; a.qk = qk; a.vt = vt; a.out = out;
  a.n = n; a.T = (int)T; a.d = d; a.n_heads = n_heads; a.n_kv_heads = n_kv_heads;
  a.cu_host = cu_seqlens; a.num_seqs = num_seqs;
  a.q_prescaled = q_prescaled != 0;
  hipError_t e = launch_attention(a, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? KRAKEN_OK : hip_fail(e, "attention");
}

kraken_status kraken_op_decode_attention(int32_t dtype, const void* qk, const void* kv_layer,
                                         void* out, int32_t n, int32_t d, int32_t n_heads,
                                         int32_t n_kv_heads, const int32_t* lens,
                                         int32_t num_seqs, int32_t max_seqs, int32_t capacity,
                                         float* work, int64_t work_floats, void* stream) {
  if (!qk || !kv_layer || !out || !lens || !work)
    return fail(KRAKEN_ERR_INVALID_ARG, "NULL pointer");
  if (dtype < KRAKEN_DTYPE_F32 || dtype > KRAKEN_DTYPE_F16)
    return fail(KRAKEN_ERR_UNSUPPORTED, "unknown dtype");
  if (n < 1 || d < 1 || n_heads < 1 || d % n_heads != 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "bad sizes");
  const int hd = d / n_heads;
  if (hd != 32 && hd != 64 && hd != 128) return fail(KRAKEN_ERR_UNSUPPORTED, "head size");
  if (n_kv_heads < 0 || (n_kv_heads > 0 && n_heads % n_kv_heads != 0))
    return fail(KRAKEN_ERR_INVALID_ARG, "n_kv_heads must be 0 or divide n_heads");
  if (num_seqs < 1 || num_seqs > KRAKEN_MAX_SEQS || max_seqs < num_seqs ||
      max_seqs > KRAKEN_MAX_SEQS || capacity < 1)
    return fail(KRAKEN_ERR_INVALID_ARG, "num_seqs, max_seqs or capacity out of range");
  if (reinterpret_cast<uintptr_t>(kv_layer) % 16 != 0 || reinterpret_cast<uintptr_t>(qk) % 16 != 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "qk or kv_layer is not 16-byte aligned");
  for (int b = 0; b < num_seqs; ++b)
    if (lens[b] < 0 || lens[b] >= capacity)
      return fail(KRAKEN_ERR_INVALID_ARG, "lens[b] out of 0..capacity-1");
  if (work_floats < decode_partial_floats(n, num_seqs, n_heads, hd, 1))
    return fail(KRAKEN_ERR_INVALID_ARG, "work is smaller than n * B * n_heads * (hd + 2)");
  hipError_t e = launch_decode_attention((DType)dtype, qk, kv_layer, work, work_floats, out, n,
                                         num_seqs, d, n_heads, n_kv_heads, lens, max_seqs,
                                         capacity, 0, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? KRAKEN_OK : hip_fail(e, "decode attention");
}

kraken_status kraken_op_decode_attention_noalloc(int32_t dtype, const void* qk,
                                                 const void* kv_layer, void* out, int32_t n,
                                                 int32_t d, int32_t n_heads, int32_t n_kv_heads,
                                                 const int32_t* lens, int32_t num_seqs,
                                                 int32_t max_seqs, int32_t capacity,
                                                 void* stream) {
  if (!qk || !kv_layer || !out || !lens) return fail(KRAKEN_ERR_INVALID_ARG, "NULL pointer");
  if (dtype < KRAKEN_DTYPE_F32 || dtype > KRAKEN_DTYPE_F16)
    return fail(KRAKEN_ERR_UNSUPPORTED, "unknown dtype");
  if (n < 1 || d < 1 || n_heads < 1 || d % n_heads != 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "bad sizes");
  const int hd = d / n_heads;
  if (hd != 32 && hd != 64 && hd != 128) return fail(KRAKEN_ERR_UNSUPPORTED, "head size");
  if (n_kv_heads < 0 || (n_kv_heads > 0 && n_heads % n_kv_heads != 0))
    return fail(KRAKEN_ERR_INVALID_ARG, "n_kv_heads must be 0 or divide n_heads");
  if (num_seqs < 1 || num_seqs > KRAKEN_MAX_SEQS || max_seqs < num_seqs ||
      max_seqs > KRAKEN_MAX_SEQS || capacity < 1)
    return fail(KRAKEN_ERR_INVALID_ARG, "num_seqs, max_seqs or capacity out of range");
  if (reinterpret_cast<uintptr_t>(kv_layer) % 16 != 0 || reinterpret_cast<uintptr_t>(qk) % 16 != 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "qk or kv_layer is not 16-byte aligned");
  for (int b = 0; b < num_seqs; ++b)
    if (lens[b] < 0 || lens[b] >= capacity)
      return fail(KRAKEN_ERR_INVALID_ARG, "lens[b] out of 0..capacity-1");
  // one key chunk's partials must fit the static scratch
  if (decode_partial_floats(n, num_seqs, n_heads, hd, 1) > KRAKEN_NOALLOC_SCRATCH_FLOATS)
    return fail(KRAKEN_ERR_UNSUPPORTED,
                "n * num_seqs * n_heads * (hd + 2) = " +
                    std::to_string(decode_partial_floats(n, num_seqs, n_heads, hd, 1)) +
                    " exceeds the static scratch of KRAKEN_NOALLOC_SCRATCH_FLOATS = " +
                    std::to_string((int64_t)KRAKEN_NOALLOC_SCRATCH_FLOATS) + " floats");
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(KRAKEN_ERR_UNSUPPORTED, "device index");
  float* part = nullptr;
  {
    // first call on this device (with the device current): look up its copy's address
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
      void* ptr = nullptr;
      HIP_TRY(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
      if (!ptr) return fail(KRAKEN_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
      g_scratch_ptr[dev] = static_cast<float*>(ptr);
    }
    part = g_scratch_ptr[dev];
  }
  hipError_t e = launch_decode_attention((DType)dtype, qk, kv_layer, part,
                                         KRAKEN_NOALLOC_SCRATCH_FLOATS, out, n, num_seqs, d,
                                         n_heads, n_kv_heads, lens, max_seqs, capacity, 0,
                                         static_cast<hipStream_t>(stream));
  return e == hipSuccess ? KRAKEN_OK : hip_fail(e, "decode attention (static scratch)");
}

}  // extern "C"
