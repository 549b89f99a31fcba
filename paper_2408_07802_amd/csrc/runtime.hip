// Host runtime and C ABI of the Kraken prefill library (declared in kraken.h).
//
// A model owns two device allocations: the repacked weights and the activation
// workspace for max_tokens tokens.  kraken_prefill validates everything on the
// host, then enqueues the whole pass on the caller's stream: per layer
//   LN1 -> Q,K projection -> V projection (transposed) -> causal attention
//   -> output projection + residual -> N-way sum + residual + LN2
//   -> FFN up + GELU -> FFN down + residual
// (Algorithm 1 for all N sub-layers at once; every GEMM is batched over the N
// sub-layers), then W_concat over the N final outputs (Section 3.1).
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

struct LayerW {
  float *ln1_g, *ln1_b, *ln2_g, *ln2_b;  // [N][d]
  float *bqk;                            // [N][d + dkv]
  float *bv;                             // [N][dkv]
  float *bo, *b2;                        // [N][d]
  float *b1;                             // [N][F]
  void *WqkT;                            // [N][d + dkv][d]
  void *WvT;                             // [N][dkv][d]
  void *WoT;                             // [N][d][d]
  void *W1T;                             // [N][F][d]
  void *W2T;                             // [N][d][F]
};

struct ProfRec {
  int cls;
  hipEvent_t a, b;
};

// Element counts of the logical blob of one sub-layer, in blob order.
struct SubOffsets {
  int64_t ln1_g, ln1_b, Wqkv, bqkv, Wo, bo, ln2_g, ln2_b, W1, b1, W2, b2, total;
  SubOffsets(int64_t d, int64_t F, int64_t dkv) {
    int64_t o = 0;
    ln1_g = o; o += d;
    ln1_b = o; o += d;
    Wqkv = o; o += d * (d + 2 * dkv);
    bqkv = o; o += d + 2 * dkv;
    Wo = o; o += d * d;
    bo = o; o += d;
    ln2_g = o; o += d;
    ln2_b = o; o += d;
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
  DType st;   // storage type of the blob and of hidden_in
  DType dt;   // MFMA operand type
  int N, L, d, H, F, Tmax, device;
  int Hkv, dkv;   // key/value heads and width (grouped-query attention: Hkv < H)
  float eps;
  bool loaded = false;
  void* wmem = nullptr;
  void* amem = nullptr;
  std::vector<LayerW> layers;
  void* WcatT = nullptr;  // [d][N*d]
  // device: [0] = a weight overflowed the operand type (set at load); [1] = an activation
  // overflowed the fp16 operand type (sticky until kraken_sync reads it)
  int* flags = nullptr;
  // workspace
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
      c->d_ff < 0 || c->ln_eps < 0.f)
    return fail(KRAKEN_ERR_INVALID_ARG, "non-positive size in cfg");
  if (c->d_model % c->n_heads != 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "d_model is not a multiple of n_heads");
  const int hd = c->d_model / c->n_heads;
  if (hd != 32 && hd != 64 && hd != 128)
    return fail(KRAKEN_ERR_UNSUPPORTED, "head size must be 32, 64 or 128");
  const int F = c->d_ff ? c->d_ff : 4 * c->d_model;
  if (c->d_model % 64 != 0 || F % 64 != 0)
    return fail(KRAKEN_ERR_UNSUPPORTED, "d_model and d_ff must be multiples of 64");
  if (c->n_kv_heads < 0) return fail(KRAKEN_ERR_INVALID_ARG, "negative n_kv_heads");
  if (c->n_kv_heads > 0) {
    if (c->n_heads % c->n_kv_heads != 0)
      return fail(KRAKEN_ERR_INVALID_ARG, "n_kv_heads does not divide n_heads");
    if ((c->n_kv_heads * hd) % 64 != 0)
      return fail(KRAKEN_ERR_UNSUPPORTED, "n_kv_heads * head size must be a multiple of 64");
  }
  if (c->d_model > 8192) return fail(KRAKEN_ERR_UNSUPPORTED, "d_model above 8192");
  if (c->max_tokens > (1 << 22)) return fail(KRAKEN_ERR_UNSUPPORTED, "max_tokens above 4194304");
  // GEMM operands of one sub-layer are addressed with 32-bit byte offsets: the activation
  // rows (tokens x the widest row), and the repacked weights [out][in] of the FFN (F x d
  // either way) and of W_concat (d x N d); 4 bytes bounds every element type
  if ((int64_t)c->max_tokens * std::max(2 * c->d_model, F) * 4 >= (1ll << 31))
    return fail(KRAKEN_ERR_UNSUPPORTED, "max_tokens * max(2 d_model, d_ff) too large");
  if ((int64_t)F * c->d_model * 4 >= (1ll << 31))
    return fail(KRAKEN_ERR_UNSUPPORTED, "d_ff * d_model too large for 32-bit weight offsets");
  if ((int64_t)c->n_sub * c->d_model * c->d_model * 4 >= (1ll << 31))
    return fail(KRAKEN_ERR_UNSUPPORTED,
                "n_sub * d_model^2 too large for 32-bit W_concat offsets");
  if (c->dtype < KRAKEN_DTYPE_F32 || c->dtype > KRAKEN_DTYPE_F16)
    return fail(KRAKEN_ERR_UNSUPPORTED, "unknown dtype");
  if (c->compute < KRAKEN_COMPUTE_STORAGE || c->compute > KRAKEN_COMPUTE_F16)
    return fail(KRAKEN_ERR_UNSUPPORTED, "unknown compute type");
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
  const size_t N = m->N, d = m->d, F = m->F, dkv = m->dkv, es = sz(m->dt);
  m->layers.resize(m->L);
  for (int j = 0; j < m->L; ++j) {
    LayerW& w = m->layers[j];
    w.ln1_g = (float*)c.take(N * d * 4);
    w.ln1_b = (float*)c.take(N * d * 4);
    w.ln2_g = (float*)c.take(N * d * 4);
    w.ln2_b = (float*)c.take(N * d * 4);
    w.bqk = (float*)c.take(N * (d + dkv) * 4);
    w.bv = (float*)c.take(N * dkv * 4);
    w.bo = (float*)c.take(N * d * 4);
    w.b1 = (float*)c.take(N * F * 4);
    w.b2 = (float*)c.take(N * d * 4);
    w.WqkT = c.take(N * (d + dkv) * d * es);
    w.WvT = c.take(N * dkv * d * es);
    w.WoT = c.take(N * d * d * es);
    w.W1T = c.take(N * F * d * es);
    w.W2T = c.take(N * d * F * es);
  }
  m->WcatT = c.take(d * N * d * es);
  m->flags = (int*)c.take(256);
  return c.off;
}

size_t carve_workspace(kraken_model* m, void* base) {
  Carver c(base);
  const size_t N = m->N, d = m->d, F = m->F, T = m->Tmax, dkv = m->dkv, es = sz(m->dt);
  m->X32 = (float*)c.take(T * d * 4);
  m->xbuf = (float*)c.take(N * T * d * 4);
  m->hbuf = (float*)c.take(N * T * d * 4);
  m->act = c.take(N * T * d * es);
  m->qk = c.take(N * T * (d + dkv) * es);
  m->o = c.take(N * T * d * es);
  // vt and g stay adjacent and last: a decode step keeps its attention partials there
  m->vt = c.take(N * dkv * (size_t)vt_ld(m->Tmax) * es);
  m->g = c.take(std::max(N * T * F, 2 * N * T * d) * es);
  m->ws_end = base ? static_cast<char*>(base) + c.off : nullptr;
  return c.off;
}

inline const char* cptr(const void* p, int64_t elems, DType t) {
  return static_cast<const char*>(p) + elems * (int64_t)sz(t);
}

// Repack one sub-layer's logical parameters (device pointer `src`) into the model layout.
hipError_t repack_sub(kraken_model* m, int j, int i, const void* src, hipStream_t s) {
  const int64_t d = m->d, F = m->F, dkv = m->dkv, wq = d + 2 * dkv;   // Wqkv row width
  const SubOffsets so(d, F, dkv);
  const LayerW& w = m->layers[j];
  const DType st = m->st, dt = m->dt;
  const size_t es = sz(dt);
  int* of = m->flags;
  hipError_t e;
#define R_(x) do { e = (x); if (e != hipSuccess) return e; } while (0)
  R_(launch_to_f32(st, cptr(src, so.ln1_g, st), w.ln1_g + i * d, d, s));
  R_(launch_to_f32(st, cptr(src, so.ln1_b, st), w.ln1_b + i * d, d, s));
  R_(launch_to_f32(st, cptr(src, so.ln2_g, st), w.ln2_g + i * d, d, s));
  R_(launch_to_f32(st, cptr(src, so.ln2_b, st), w.ln2_b + i * d, d, s));
  R_(launch_to_f32(st, cptr(src, so.bqkv, st), w.bqk + i * (d + dkv), d + dkv, s));
  R_(launch_to_f32(st, cptr(src, so.bqkv + d + dkv, st), w.bv + i * dkv, dkv, s));
  R_(launch_to_f32(st, cptr(src, so.bo, st), w.bo + i * d, d, s));
  R_(launch_to_f32(st, cptr(src, so.b1, st), w.b1 + i * F, F, s));
  R_(launch_to_f32(st, cptr(src, so.b2, st), w.b2 + i * d, d, s));
  // x W layout [in][out] -> [out][in], converted to the operand type
  R_(launch_transpose(st, cptr(src, so.Wqkv, st), wq, dt,
                      static_cast<char*>(w.WqkT) + i * (d + dkv) * d * es, d, (int)d,
                      (int)(d + dkv), of, s));
  // The Q projection (the first d rows of WqkT, the first d biases) carries the softmax
  // factor log2(e) / sqrt(hd), so the attention kernels get scores in log2 units straight
  // from their MFMAs.
  {
    const float qs = (float)(1.4426950408889634 / std::sqrt((double)(d / m->H)));
    R_(launch_scale(dt, static_cast<char*>(w.WqkT) + i * (d + dkv) * d * es, d * d, qs, s));
    R_(launch_scale(DType::F32, w.bqk + i * (d + dkv), d, qs, s));
  }
  R_(launch_transpose(st, cptr(src, so.Wqkv + d + dkv, st), wq, dt,
                      static_cast<char*>(w.WvT) + i * dkv * d * es, d, (int)d, (int)dkv, of, s));
  R_(launch_transpose(st, cptr(src, so.Wo, st), d, dt, static_cast<char*>(w.WoT) + i * d * d * es,
                      d, (int)d, (int)d, of, s));
  R_(launch_transpose(st, cptr(src, so.W1, st), F, dt, static_cast<char*>(w.W1T) + i * F * d * es,
                      d, (int)d, (int)F, of, s));
  R_(launch_transpose(st, cptr(src, so.W2, st), d, dt, static_cast<char*>(w.W2T) + i * d * F * es,
                      F, (int)F, (int)d, of, s));
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
kraken_status forward(kraken_model* m, const void* hidden_in, int T, const int32_t* cu,
                      int32_t num_seqs, const KvRef* kv, float* hidden_out, float* sub_out,
                      hipStream_t s) {
  const bool decode = kv && kv->lens;
  const DType dt = m->dt;
  int* const ovf = m->flags + 1;   // fp16 operand overflow of the activations
  const int64_t N = m->N, d = m->d, F = m->F;
  const int64_t Td = (int64_t)T * d;
  const int ldv = vt_ld(T);
  hipError_t e;
#define RUN(cls, call, what)                      \
  do {                                            \
    e = m->run(cls, s, [&]() { return (call); }); \
    if (e != hipSuccess) return hip_fail(e, what); \
  } while (0)

  const float* X32 = static_cast<const float*>(hidden_in);
  if (m->st != DType::F32) {
    RUN(KRAKEN_K_OTHER, launch_to_f32(m->st, hidden_in, m->X32, Td, s), "input conversion");
    X32 = m->X32;
  }

  // Attention reads V^T in 16-byte chunks of 8 tokens; the padding columns [T, ldv) are
  // only ever multiplied by zero probabilities but must hold finite values.
  const int64_t dkv = m->dkv, dqk = d + dkv;   // key/value width, Q|K row width
  if (!decode && ldv > T)
    RUN(KRAKEN_K_OTHER, launch_zero_cols(dt, m->vt, N * dkv, ldv, T, ldv, s), "V padding");

  for (int j = 0; j < m->L; ++j) {
    const LayerW& w = m->layers[j];
    const float* xin = j == 0 ? X32 : m->xbuf;   // sub-layer inputs x_i
    const int64_t xs = j == 0 ? 0 : Td;           // first layer: one shared input
    char* cache_j = kv ? kv->cache + (size_t)j * kv->layer_bytes : nullptr;
    RUN(KRAKEN_K_LN1,
        launch_layernorm(dt, xin, xs, w.ln1_g, w.ln1_b, m->act, (int)N, T, (int)d, m->eps, ovf,
                         s),
        "ln1");
    {
      GemmDesc g = gemm_base(dt);
      g.epi = EPI_BIAS_N;
      g.A = m->act; g.lda = (int)d; g.sA = Td;
      g.B = w.WqkT; g.ldb = (int)d; g.sB = dqk * d;
      g.C = m->qk; g.ldc = (int)dqk; g.sC = (int64_t)T * dqk;
      g.bias = w.bqk; g.sBias = dqk;
      g.M = T; g.N = (int)dqk; g.K = (int)d; g.batch = (int)N;
      g.ovf = ovf;
      RUN(KRAKEN_K_GEMM_QK, launch_gemm(g, s), "QK projection");
    }
    if (!decode) {
      {
        GemmDesc g = gemm_base(dt);
        g.epi = EPI_BIAS_M;
        g.A = w.WvT; g.lda = (int)d; g.sA = dkv * d;
        g.B = m->act; g.ldb = (int)d; g.sB = Td;
        g.C = m->vt; g.ldc = ldv; g.sC = dkv * ldv;
        g.bias = w.bv; g.sBias = dkv;
        g.M = (int)dkv; g.N = T; g.K = (int)d; g.batch = (int)N;
        g.ovf = ovf;
        RUN(KRAKEN_K_GEMM_VT, launch_gemm(g, s), "V projection");
      }
      if (kv)
        RUN(KRAKEN_K_KV,
            launch_kv_store(dt, m->qk, m->vt, cache_j, (int)N, T, (int)d, m->H, m->Hkv, cu,
                            num_seqs, kv->max_seqs, kv->cap, s),
            "KV store");
      AttnDesc a;
      a.dt = dt; a.qk = m->qk; a.vt = m->vt; a.out = m->o;
      a.n = (int)N; a.T = T; a.d = (int)d; a.n_heads = m->H; a.n_kv_heads = m->Hkv;
      a.cu_host = cu; a.num_seqs = num_seqs;
      a.q_prescaled = 1;
      RUN(KRAKEN_K_ATTN, launch_attention(a, s), "attention");
    } else {
      // V rows of the new tokens go through o ([N][T][dkv]) into the cache; o then takes
      // the attention output, after the append has read it (stream order).
      {
        GemmDesc g = gemm_base(dt);
        g.epi = EPI_BIAS_N;
        g.A = m->act; g.lda = (int)d; g.sA = Td;
        g.B = w.WvT; g.ldb = (int)d; g.sB = dkv * d;
        g.C = m->o; g.ldc = (int)dkv; g.sC = (int64_t)T * dkv;
        g.bias = w.bv; g.sBias = dkv;
        g.M = T; g.N = (int)dkv; g.K = (int)d; g.batch = (int)N;
        g.ovf = ovf;
        RUN(KRAKEN_K_GEMM_VT, launch_gemm(g, s), "V projection");
      }
      RUN(KRAKEN_K_KV,
          launch_kv_append(dt, m->qk, m->o, cache_j, (int)N, T, (int)d, m->H, m->Hkv, kv->lens,
                           kv->max_seqs, kv->cap, s),
          "KV append");
      RUN(KRAKEN_K_ATTN,
          launch_decode_attention(dt, m->qk, cache_j, static_cast<float*>(m->vt),
                                  decode_partial_room(m), m->o, (int)N, T, (int)d, m->H,
                                  m->Hkv, kv->lens, kv->max_seqs, kv->cap, 1, s),
          "decode attention");
    }
    {
      GemmDesc g = gemm_base(dt);
      g.epi = EPI_BIAS_N_RES;
      g.A = m->o; g.lda = (int)d; g.sA = Td;
      g.B = w.WoT; g.ldb = (int)d; g.sB = d * d;
      g.C = m->hbuf; g.ldc = (int)d; g.sC = Td;
      g.bias = w.bo; g.sBias = d;
      g.R = xin; g.sR = xs;
      g.M = T; g.N = (int)d; g.K = (int)d; g.batch = (int)N;
      RUN(KRAKEN_K_GEMM_O, launch_gemm(g, s), "output projection");
    }
    RUN(KRAKEN_K_COMBINE,
        launch_combine_ln2(dt, m->xbuf, j == 0 ? X32 : nullptr, m->hbuf, w.ln2_g, w.ln2_b, m->act,
                           (int)N, T, (int)d, m->eps, ovf, s),
        "combine + ln2");
    {
      GemmDesc g = gemm_base(dt);
      g.epi = EPI_BIAS_N_GELU;
      g.A = m->act; g.lda = (int)d; g.sA = Td;
      g.B = w.W1T; g.ldb = (int)d; g.sB = F * d;
      g.C = m->g; g.ldc = (int)F; g.sC = (int64_t)T * F;
      g.bias = w.b1; g.sBias = F;
      g.M = T; g.N = (int)F; g.K = (int)d; g.batch = (int)N;
      g.ovf = ovf;
      RUN(KRAKEN_K_GEMM_UP, launch_gemm(g, s), "FFN up");
    }
    {
      GemmDesc g = gemm_base(dt);
      g.epi = EPI_BIAS_N_RES;
      g.A = m->g; g.lda = (int)F; g.sA = (int64_t)T * F;
      g.B = w.W2T; g.ldb = (int)F; g.sB = d * F;
      g.C = m->xbuf; g.ldc = (int)d; g.sC = Td;
      g.bias = w.b2; g.sBias = d;
      g.R = m->hbuf; g.sR = Td;
      g.M = T; g.N = (int)d; g.K = (int)F; g.batch = (int)N;
      RUN(KRAKEN_K_GEMM_DOWN, launch_gemm(g, s), "FFN down");
    }
  }

  if (sub_out)
    RUN(KRAKEN_K_OTHER,
        hipMemcpyAsync(sub_out, m->xbuf, N * Td * sizeof(float), hipMemcpyDeviceToDevice, s),
        "sub_out copy");

  // out = [Y_1 | ... | Y_N] W_concat, K split into N groups of d (one per sub-layer).
  {
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
    g.lda = (int)d; g.gA = Td;
    g.B = m->WcatT; g.ldb = (int)(N * d); g.gB = d; g.gBmod = (int)N;
    g.C = hidden_out; g.ldc = (int)d;
    g.M = T; g.N = (int)d; g.K = (int)d;
    RUN(KRAKEN_K_CONCAT, launch_gemm(g, s), "W_concat");
  }
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
  switch (s) {
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
      c->n_heads < 1 || c->n_kv_heads < 0)
    return 0;
  const uint64_t N = c->n_sub, L = c->n_layers, d = c->d_model;
  const uint64_t F = c->d_ff ? c->d_ff : 4 * d;
  const uint64_t dkv = c->n_kv_heads ? (uint64_t)c->n_kv_heads * (d / c->n_heads) : d;
  return (size_t)(L * N * (2 * d * d + 2 * d * dkv + 2 * d * F + 7 * d + 2 * dkv + F) +
                  N * d * d);
}

kraken_status kraken_create(const kraken_config* cfg, kraken_model** out) {
  if (!out) return fail(KRAKEN_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  kraken_status st = validate_cfg(cfg);
  if (st != KRAKEN_OK) return st;
  kraken_model* m = new (std::nothrow) kraken_model();
  if (!m) return fail(KRAKEN_ERR_OOM, "host allocation failed");
  m->cfg = *cfg;
  m->st = (DType)cfg->dtype;
  m->dt = cfg->compute == KRAKEN_COMPUTE_STORAGE ? m->st : (DType)(cfg->compute - 1);
  m->N = cfg->n_sub;
  m->L = cfg->n_layers;
  m->d = cfg->d_model;
  m->H = cfg->n_heads;
  m->Hkv = cfg->n_kv_heads > 0 ? cfg->n_kv_heads : cfg->n_heads;
  m->dkv = m->Hkv * (cfg->d_model / cfg->n_heads);
  m->F = cfg->d_ff ? cfg->d_ff : 4 * cfg->d_model;
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
  const int64_t d = m->d, N = m->N;
  const SubOffsets so(d, m->F, m->dkv);
  const int64_t layer_elems = N * so.total;
  const int64_t wcat_off = (int64_t)m->L * layer_elems;
  void* staging = nullptr;
  if (!blob_is_device) {
    const size_t sbytes = std::max<int64_t>(layer_elems, N * d * d) * sz(m->st);
    if (hipMalloc(&staging, sbytes) != hipSuccess) {
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
  m->loaded = false;
  hipError_t e = hipMemsetAsync(m->flags, 0, 256, s);
  if (e != hipSuccess) {
    cleanup();
    return hip_fail(e, "flag reset");
  }
  for (int j = 0; j < m->L; ++j) {
    const void* src = cptr(blob, j * layer_elems, m->st);
    if (!blob_is_device) {
      e = hipStreamSynchronize(s);  // staging is free again
      if (e == hipSuccess)
        e = hipMemcpyAsync(staging, src, layer_elems * sz(m->st), hipMemcpyHostToDevice, s);
      if (e != hipSuccess) {
        cleanup();
        return hip_fail(e, "weight upload");
      }
      src = staging;
    }
    for (int i = 0; i < m->N; ++i) {
      e = repack_sub(m, j, i, cptr(src, i * so.total, m->st), s);
      if (e != hipSuccess) {
        cleanup();
        return hip_fail(e, "weight repack");
      }
    }
  }
  const void* wsrc = cptr(blob, wcat_off, m->st);
  if (!blob_is_device) {
    e = hipStreamSynchronize(s);
    if (e == hipSuccess)
      e = hipMemcpyAsync(staging, wsrc, N * d * d * sz(m->st), hipMemcpyHostToDevice, s);
    if (e != hipSuccess) {
      cleanup();
      return hip_fail(e, "W_concat upload");
    }
    wsrc = staging;
  }
  e = launch_transpose(m->st, wsrc, d, m->dt, m->WcatT, N * d, (int)(N * d), (int)d, m->flags, s);
  if (e != hipSuccess) {
    cleanup();
    return hip_fail(e, "W_concat repack");
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
  const size_t dkv = c->n_kv_heads > 0 ? (size_t)c->n_kv_heads * (c->d_model / c->n_heads)
                                        : (size_t)c->d_model;
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
                 sub_out, static_cast<hipStream_t>(stream));
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
  if (decode_partial_floats((int)N, B, m->H, (int)d / m->H, 1) > decode_partial_room(m))
    return fail(KRAKEN_ERR_UNSUPPORTED, "workspace too small for the decode attention partials");
  st = check_device(m);
  if (st != KRAKEN_OK) return st;
  KvRef kv;
  kv.cache = static_cast<char*>(kv_cache);
  kv.layer_bytes = kv_layer_bytes(m, max_seqs, capacity);
  kv.max_seqs = max_seqs;
  kv.cap = capacity;
  kv.lens = lens;
  return forward(m, hidden_in, B, nullptr, num_seqs, &kv, hidden_out, sub_out,
                 static_cast<hipStream_t>(stream));
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
  if (!c || !cu || num_seqs < 1) return 0.0;
  const double N = c->n_sub, L = c->n_layers, d = c->d_model;
  const double F = c->d_ff ? c->d_ff : 4.0 * d;
  const double T = cu[num_seqs];
  const double dkv =
      (c->n_kv_heads > 0 && c->n_heads > 0) ? (double)c->n_kv_heads * (c->d_model / c->n_heads) : d;
  switch (cls) {
    case KRAKEN_K_GEMM_QK: return L * N * 2.0 * T * d * (d + dkv);
    case KRAKEN_K_GEMM_VT: return L * N * 2.0 * T * d * dkv;
    case KRAKEN_K_GEMM_O: return L * N * 2.0 * T * d * d;
    case KRAKEN_K_GEMM_UP: return L * N * 2.0 * T * d * F;
    case KRAKEN_K_GEMM_DOWN: return L * N * 2.0 * T * F * d;
    case KRAKEN_K_CONCAT: return 2.0 * T * N * d * d;
    case KRAKEN_K_ATTN: {
      // QK^T and PV over causal pairs: 4 hd flops per pair and head = 4 d per pair
      double pairs = 0;
      for (int b = 0; b < num_seqs; ++b) {
        const double S = cu[b + 1] - cu[b];
        pairs += S * (S + 1) / 2.0;
      }
      return L * N * 4.0 * d * pairs;
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
  if (n < 1 || T < 0 || d < 4 || d % 64 != 0 || d > 8192 || xs < 0)
    return fail(KRAKEN_ERR_INVALID_ARG, "bad sizes");
  hipError_t e = launch_layernorm((DType)dtype, x, xs, gamma, beta, out, n, T, d, eps, nullptr,
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
  if (n < 1 || T < 0 || d % 64 != 0 || d < 64 || d > 8192)
    return fail(KRAKEN_ERR_INVALID_ARG, "bad sizes");
  hipError_t e = launch_combine_ln2((DType)dtype, x, shared, h, gamma, beta, out, n, T, d, eps,
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
