// Host-side paths of the C ABI under AddressSanitizer and UndefinedBehaviorSanitizer.
//
// Built from the library's sources compiled for the host only (no device code), so every
// call here must finish on the host: argument and configuration checks, the size and
// FLOP queries, status strings and error messages.  A configuration that passes its
// checks goes on to the device (hipGetDevice); with no GPU that call fails and takes the
// error path, with a GPU the model is created and destroyed.  Exits 0 when every result
// is the documented one; the sanitizers abort on any memory error or undefined behaviour.
#include <cstdio>
#include <cstring>

#include "kraken.h"

namespace {

int failures = 0;

void expect(bool ok, const char* what) {
  if (!ok) {
    std::fprintf(stderr, "FAIL: %s (last error: %s)\n", what, kraken_last_error());
    ++failures;
  }
}

kraken_config base() {
  kraken_config c;
  std::memset(&c, 0, sizeof c);
  c.n_sub = 2;
  c.n_layers = 2;
  c.d_model = 128;
  c.n_heads = 4;
  c.max_tokens = 64;
  c.dtype = KRAKEN_DTYPE_BF16;
  return c;
}

kraken_status create(const kraken_config& c) {
  kraken_model* m = reinterpret_cast<kraken_model*>(&failures);   // must be reset to NULL
  const kraken_status s = kraken_create(&c, &m);
  if (s == KRAKEN_OK) {
    expect(m != nullptr, "create OK returns a model");
    kraken_destroy(m);
  } else {
    expect(m == nullptr, "create failure sets *out to NULL");
    expect(std::strlen(kraken_last_error()) > 0, "create failure sets a message");
  }
  return s;
}

}  // namespace

int main() {
  // status strings, including codes past the enum
  for (int s = -3; s < 12; ++s)
    expect(kraken_status_string(static_cast<kraken_status>(s)) != nullptr, "status string");

  // configuration checks that end on the host
  struct Bad {
    void (*edit)(kraken_config&);
    kraken_status want;
    const char* what;
  };
  const Bad bad[] = {
      {[](kraken_config& c) { c.n_sub = 0; }, KRAKEN_ERR_INVALID_ARG, "n_sub 0"},
      {[](kraken_config& c) { c.d_model = -8; }, KRAKEN_ERR_INVALID_ARG, "negative d"},
      {[](kraken_config& c) { c.arch = 9; }, KRAKEN_ERR_INVALID_ARG, "unknown arch"},
      {[](kraken_config& c) { c.arch = KRAKEN_ARCH_GPT; }, KRAKEN_ERR_INVALID_ARG,
       "gpt with n_sub 2"},
      {[](kraken_config& c) { c.d_model = 130; }, KRAKEN_ERR_INVALID_ARG, "d % heads"},
      {[](kraken_config& c) { c.head_dim = 136; }, KRAKEN_ERR_UNSUPPORTED, "head 136"},
      {[](kraken_config& c) { c.d_model = 16448; c.n_heads = 128; c.head_dim = 128; },
       KRAKEN_ERR_UNSUPPORTED, "d above 16384"},
      {[](kraken_config& c) { c.max_tokens = 1 << 23; }, KRAKEN_ERR_UNSUPPORTED,
       "max_tokens"},
      {[](kraken_config& c) { c.d_model = 8192; c.n_heads = 64; c.d_ff = 131072;
                              c.max_tokens = 1; }, KRAKEN_ERR_UNSUPPORTED, "FFN offsets"},
      {[](kraken_config& c) { c.vocab = 100; }, KRAKEN_ERR_INVALID_ARG, "vocab without positions"},
      {[](kraken_config& c) { c.n_kv_heads = 3; }, KRAKEN_ERR_INVALID_ARG, "kv heads"},
      {[](kraken_config& c) { c.dtype = 7; }, KRAKEN_ERR_UNSUPPORTED, "dtype"},
      {[](kraken_config& c) { c.compute = 9; }, KRAKEN_ERR_UNSUPPORTED, "compute"},
  };
  for (const Bad& b : bad) {
    kraken_config c = base();
    b.edit(c);
    expect(create(c) == b.want, b.what);
  }
  expect(kraken_create(nullptr, nullptr) == KRAKEN_ERR_INVALID_ARG, "create NULL");

  // a valid configuration reaches the device: an error without a GPU, a model with one
  {
    kraken_config c = base();
    const kraken_status s = create(c);
    expect(s == KRAKEN_OK || s == KRAKEN_ERR_HIP, "valid config");
  }

  // size and FLOP queries (host arithmetic), every architecture, padded widths
  const int32_t cu[3] = {0, 3, 10};
  for (int arch = KRAKEN_ARCH_KRAKEN; arch <= KRAKEN_ARCH_PARALLEL; ++arch) {
    kraken_config c = base();
    c.arch = arch;
    if (arch != KRAKEN_ARCH_KRAKEN) c.n_sub = 1;
    c.d_model = 200;
    c.n_heads = 5;
    c.vocab = 777;
    c.max_positions = 64;
    expect(kraken_weight_blob_elems(&c) > 0, "blob elems");
    expect(kraken_kv_cache_bytes(&c, 3, 100) > 0, "cache bytes");
    double total = 0.0;
    for (int k = 0; k < KRAKEN_K_COUNT; ++k) total += kraken_class_flops(&c, k, cu, 2);
    expect(total > 0.0, "class flops");
    expect(kraken_class_flops(&c, KRAKEN_K_COUNT, cu, 2) == 0.0, "class past the end");
  }
  expect(kraken_weight_blob_elems(nullptr) == 0, "blob elems NULL");
  expect(kraken_kv_cache_bytes(nullptr, 1, 1) == 0, "cache bytes NULL");
  {
    kraken_config c = base();
    expect(kraken_kv_cache_bytes(&c, 0, 4) == 0, "cache bytes 0 slots");
    expect(kraken_kv_cache_bytes(&c, KRAKEN_MAX_SEQS + 1, 4) == 0, "cache bytes slots");
  }

  // model calls on NULL and op entry points with bad arguments: rejected before launch
  const int32_t cu1[2] = {0, 4};
  expect(kraken_prefill(nullptr, nullptr, cu1, 1, nullptr, nullptr, nullptr) ==
             KRAKEN_ERR_INVALID_ARG, "prefill NULL");
  expect(kraken_sync(nullptr, nullptr) == KRAKEN_ERR_INVALID_ARG, "sync NULL");
  expect(kraken_debug_poison_workspace(nullptr, nullptr) == KRAKEN_ERR_INVALID_ARG,
         "poison NULL");
  expect(kraken_destroy(nullptr) == KRAKEN_OK, "destroy NULL");
  expect(kraken_op_gemm(1, 0, nullptr, nullptr, nullptr, nullptr, nullptr, 1, 1, 64, 1, 0, 0,
                        0, 0, nullptr) == KRAKEN_ERR_INVALID_ARG, "gemm NULL");
  expect(kraken_op_layernorm(1, nullptr, 0, nullptr, nullptr, nullptr, 1, 4, 128, 1e-5f,
                             nullptr) == KRAKEN_ERR_INVALID_ARG, "layernorm NULL");
  expect(kraken_op_attention(1, nullptr, nullptr, nullptr, 1, 128, 2, 0, 0, cu1, 1,
                             nullptr) == KRAKEN_ERR_INVALID_ARG, "attention NULL");
  expect(kraken_op_decode_attention_noalloc(1, nullptr, nullptr, nullptr, 1, 128, 2, 0,
                                            nullptr, 1, 1, 4, nullptr) ==
             KRAKEN_ERR_INVALID_ARG, "decode noalloc NULL");

  if (failures) {
    std::fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  std::printf("host paths clean under the sanitizers\n");
  return 0;
}
