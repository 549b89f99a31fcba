"""Host-side checks of the C ABI that need no GPU: the library loads, exports every
symbol the header declares, sizes the weight blob as the oracle counts parameters,
and rejects bad arguments before touching the device."""

import ctypes
import os
import re

import pytest

from oracle import kraken_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kraken.h")


def K():
    from paper_2408_07802_amd import kraken
    return kraken


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kraken_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = header_functions()
    assert len(names) >= 15
    L = K().lib()
    for name in names:
        assert hasattr(L, name), name


def test_blob_elems_matches_oracle_parameter_count():
    for (N, L, d, F) in [(2, 2, 128, 512), (4, 12, 768, 3072), (8, 24, 2048, 8192),
                         (4, 36, 1280, 5120), (3, 1, 64, 0)]:
        cfg = K().Config(n_sub=N, n_layers=L, d_model=d, n_heads=2, d_ff=F, max_tokens=16)
        want = O.kraken_param_count(N, L, d, F or 4 * d, biases=True, layer_norms=True,
                                    w_concat=True)
        assert K().weight_blob_elems(cfg) == want


def _create_status(**kw):
    base = dict(n_sub=2, n_layers=2, d_model=128, n_heads=4, d_ff=0, max_tokens=64, dtype="bf16")
    arch = kw.pop("arch", None)
    base.update(kw)
    cfg = K().Config(**base)
    c = cfg.c_struct()
    if arch is not None:
        c.arch = arch
    h = ctypes.c_void_p()
    st = K().lib().kraken_create(ctypes.byref(c), ctypes.byref(h))
    assert not h.value
    return st


@pytest.mark.parametrize("kw,status", [
    (dict(n_sub=0), 1), (dict(n_layers=0), 1), (dict(d_model=0), 1), (dict(n_heads=0), 1),
    (dict(max_tokens=0), 1), (dict(d_ff=-1), 1), (dict(d_model=130, n_heads=4), 1),
    (dict(d_model=120, n_heads=10), 2),       # head size 12: not a multiple of 8
    (dict(d_model=130, n_heads=2, head_dim=64), 2),   # d not a multiple of 4
    (dict(d_model=1280, n_heads=4), 2),       # head size 320
    (dict(head_dim=136), 2),                  # head size above 128
    (dict(d_ff=102), 2), (dict(max_tokens=1 << 23), 2),
    (dict(arch=5), 1), (dict(n_sub=2, arch=1), 1), (dict(n_sub=2, arch=2), 1),
    (dict(vocab=100, max_positions=0), 1), (dict(vocab=-1), 1),
    (dict(d_model=2048, n_heads=16, d_ff=8192, max_tokens=65536), 2),   # 32-bit GEMM offsets
    (dict(d_model=16448, n_heads=128, head_dim=128, d_ff=64, max_tokens=1), 2),  # width
])
def test_create_rejects_bad_configs_before_allocating(kw, status):
    assert _create_status(**kw) == status
    assert K().lib().kraken_last_error()


def test_create_rejects_unknown_dtype():
    c = K().Config(n_sub=1, n_layers=1, d_model=64, n_heads=2, max_tokens=4).c_struct()
    c.dtype = 7
    h = ctypes.c_void_p()
    assert K().lib().kraken_create(ctypes.byref(c), ctypes.byref(h)) == K().ERR_UNSUPPORTED


def test_null_arguments_are_rejected():
    L = K().lib()
    cu = (ctypes.c_int32 * 2)(0, 4)
    assert L.kraken_prefill(None, None, cu, 1, None, None, None) == K().ERR_INVALID_ARG
    assert L.kraken_load_weights(None, None, 0, 0, None) == K().ERR_INVALID_ARG
    assert L.kraken_create(None, None) == K().ERR_INVALID_ARG
    assert L.kraken_destroy(None) == K().OK
    assert L.kraken_op_gemm(1, 0, None, None, None, None, None, 1, 1, 64, 1, 0, 0, 0, 0,
                            None) == K().ERR_INVALID_ARG
    assert L.kraken_status_string(K().ERR_STATE) == b"invalid state"


def test_class_flops_formula():
    cfg = K().Config(n_sub=8, n_layers=24, d_model=2048, n_heads=16, d_ff=8192, max_tokens=8192)
    cu = [0, 8192]
    N, L, d, F, T = 8, 24, 2048, 8192, 8192
    total = sum(K().class_flops(cfg, k, cu) for k in range(K().K_COUNT))
    want = N * L * (T * (8 * d * d + 4 * d * F) + 2 * d * T * (T + 1)) + 2 * T * N * d * d
    assert abs(total - want) / want < 1e-12
    assert abs(total - 2.117e14) / 2.117e14 < 1e-3      # the algorithmic FLOPs of this workload
    # ragged: attention counts causal pairs within each sequence only
    cu2 = [0, 3, 10]
    att = K().class_flops(cfg, K().K_ATTN, cu2)
    assert att == L * N * 4.0 * d * (3 * 4 / 2 + 7 * 8 / 2)


def test_kv_cache_bytes():
    # [L][N][2][max_seqs][heads][capacity][hd] elements of the compute type
    for dtype, compute, es in [("bf16", "storage", 2), ("f32", "storage", 4), ("bf16", "f16", 2),
                               ("bf16", "f32", 4), ("f16", "bf16", 2)]:
        cfg = K().Config(n_sub=8, n_layers=24, d_model=2048, n_heads=16, d_ff=8192,
                         max_tokens=8192, dtype=dtype, compute=compute)
        c = cfg.c_struct()
        got = K().lib().kraken_kv_cache_bytes(ctypes.byref(c), 3, 8193)
        assert got == 24 * 8 * 2 * 3 * 8193 * 2048 * es
    # one token of one sequence costs 2 L N d elements: N times a single-stack model of width d
    cfg = K().Config(n_sub=4, n_layers=2, d_model=128, n_heads=4, max_tokens=4, dtype="bf16")
    c = cfg.c_struct()
    assert K().lib().kraken_kv_cache_bytes(ctypes.byref(c), 1, 1) == 2 * 2 * 4 * 128 * 2
    for ms, cap in [(0, 4), (K().MAX_SEQS + 1, 4), (1, 0), (1, -3)]:
        assert K().lib().kraken_kv_cache_bytes(ctypes.byref(c), ms, cap) == 0
    bad = K().Config(n_sub=0, n_layers=2, d_model=128, n_heads=4, max_tokens=4).c_struct()
    assert K().lib().kraken_kv_cache_bytes(ctypes.byref(bad), 1, 4) == 0


def test_grouped_query_sizes():
    # weight blob, KV cache and projection FLOPs with n_kv_heads key/value heads
    N, L, d, F, H = 4, 3, 512, 1024, 16
    hd = d // H
    for Hkv in (16, 8, 4, 2):
        dkv = Hkv * hd
        cfg = K().Config(n_sub=N, n_layers=L, d_model=d, n_heads=H, d_ff=F, max_tokens=16,
                         n_kv_heads=Hkv)
        want = O.kraken_param_count(N, L, d, F, biases=True, layer_norms=True, w_concat=True,
                                    kv_width=dkv)
        assert K().weight_blob_elems(cfg) == want
        c = cfg.c_struct()
        assert K().lib().kraken_kv_cache_bytes(ctypes.byref(c), 2, 100) == \
            L * N * 2 * 2 * 100 * dkv * 2
        cu = [0, 100]
        assert K().class_flops(cfg, K().K_GEMM_QK, cu) == L * N * 2.0 * 100 * d * (d + dkv)
        assert K().class_flops(cfg, K().K_GEMM_VT, cu) == L * N * 2.0 * 100 * d * dkv
    # n_kv_heads = n_heads is the multi-head model
    a = K().Config(n_sub=N, n_layers=L, d_model=d, n_heads=H, d_ff=F, max_tokens=16)
    b = K().Config(n_sub=N, n_layers=L, d_model=d, n_heads=H, d_ff=F, max_tokens=16,
                   n_kv_heads=H)
    assert K().weight_blob_elems(a) == K().weight_blob_elems(b)


@pytest.mark.parametrize("kw,status", [
    (dict(n_kv_heads=3), 1),                   # does not divide 4 heads
    (dict(n_kv_heads=-1), 1),
    (dict(d_model=256, n_heads=8, n_kv_heads=1), 2),   # 1 x 32 features: not a multiple of 64
])
def test_create_rejects_bad_kv_heads(kw, status):
    assert _create_status(**kw) == status


@pytest.mark.parametrize("kw", [
    # repacked FFN weights F x d past 2^31 bytes: fp32 operands (4 bytes an element), and
    # 16-bit operands (2 bytes)
    dict(d_model=8192, n_heads=64, d_ff=65536, max_tokens=1, dtype="f32"),
    dict(d_model=8192, n_heads=64, d_ff=131072, max_tokens=1),
    # W_concat^T d x N d past 2^31 bytes at 2 bytes an element
    dict(n_sub=32, d_model=8192, n_heads=64, d_ff=8192, max_tokens=1),
])
def test_create_rejects_weight_offsets_past_32_bits(kw):
    assert _create_status(**kw) == K().ERR_UNSUPPORTED
    assert b"32-bit" in K().lib().kraken_last_error()


def test_sync_and_poison_reject_null_model():
    L = K().lib()
    assert L.kraken_sync(None, None) == K().ERR_INVALID_ARG
    assert L.kraken_debug_poison_workspace(None, None) == K().ERR_INVALID_ARG
    assert L.kraken_status_string(K().ERR_OVERFLOW) == b"fp16 activation overflow"


def test_op_attention_validates_before_launch():
    # a head size the kernels do not have, and a bad cu_seqlens: rejected on the host
    L = K().lib()
    cu = (ctypes.c_int32 * 2)(0, 4)
    dummy = ctypes.c_void_p(16)
    assert L.kraken_op_attention(2, dummy, dummy, dummy, 1, 96, 1, 0, 1, cu, 1,
                                 None) == K().ERR_UNSUPPORTED
    bad = (ctypes.c_int32 * 3)(0, 4, 4)
    assert L.kraken_op_attention(2, dummy, dummy, dummy, 1, 256, 2, 0, 1, bad, 2,
                                 None) == K().ERR_INVALID_ARG


# ------------------------------------------- the binding's buffer checks (no GPU needed)

def _cfg():
    return K().Config(n_sub=2, n_layers=1, d_model=128, n_heads=4, max_tokens=16, dtype="bf16")


def test_binding_rejects_host_tensors():
    import torch
    x = torch.zeros((8, 128), dtype=torch.bfloat16)          # CPU: would be a host pointer
    with pytest.raises(ValueError, match="GPU tensor"):
        K().check_call_buffers(_cfg(), x, 8, None, None)


class _FakeCuda:
    """Stands in for a CUDA tensor on a host without a GPU: the attributes the binding's
    buffer checks read, taken from a CPU tensor."""

    def __init__(self, t, index=0):
        self._t = t
        self.is_cuda = True
        self.device = __import__("torch").device("cuda", index)
        self.dtype = t.dtype

    def is_contiguous(self):
        return self._t.is_contiguous()

    def numel(self):
        return self._t.numel()


def test_binding_rejects_wrong_dtype_size_layout_and_device():
    import torch
    cfg = _cfg()
    ok = _FakeCuda(torch.zeros((8, 128), dtype=torch.bfloat16))
    out_ok = _FakeCuda(torch.zeros((8, 128), dtype=torch.float32))
    sub_ok = _FakeCuda(torch.zeros((2, 8, 128), dtype=torch.float32))
    K().check_call_buffers(cfg, ok, 8, out_ok, sub_ok)            # accepted
    cases = [
        (dict(hidden=_FakeCuda(torch.zeros((8, 128), dtype=torch.float32))), "dtype"),
        (dict(hidden=_FakeCuda(torch.zeros((7, 128), dtype=torch.bfloat16))), "elements"),
        (dict(hidden=_FakeCuda(torch.zeros((128, 8), dtype=torch.bfloat16).t())), "contiguous"),
        (dict(out=_FakeCuda(torch.zeros((8, 128), dtype=torch.bfloat16))), "dtype"),
        (dict(out=_FakeCuda(torch.zeros((8, 128), dtype=torch.float32), index=1)), "is on"),
        (dict(out=torch.zeros((8, 128), dtype=torch.float32)), "GPU tensor"),
        (dict(sub_out=_FakeCuda(torch.zeros((1, 8, 128), dtype=torch.float32))), "elements"),
    ]
    for kw, pat in cases:
        args = dict(hidden=ok, out=out_ok, sub_out=sub_ok)
        args.update(kw)
        with pytest.raises(ValueError, match=pat):
            K().check_call_buffers(cfg, args["hidden"], 8, args["out"], args["sub_out"])


def test_noalloc_scratch_size_matches_the_header():
    text = open(HEADER).read()
    m = re.search(r"#define KRAKEN_NOALLOC_SCRATCH_FLOATS \((\d+) \* (\d+) \* (\d+)\)", text)
    assert m and int(m[1]) * int(m[2]) * int(m[3]) == K().NOALLOC_SCRATCH_FLOATS


def test_blob_elems_of_the_three_architectures_and_the_embeddings():
    # GPT-like and parallel: one record per layer, no W_concat; parallel without ln2;
    # head size other than d / heads; embeddings after the layers
    d, F, H, hd, L, V, P = 320, 1280, 2, 128, 3, 1000, 64
    for arch in ("gpt", "parallel", "kraken"):
        N = 3 if arch == "kraken" else 1
        cfg = K().Config(n_sub=N, n_layers=L, d_model=d, n_heads=H, d_ff=F, max_tokens=16,
                         arch=arch, head_dim=hd, vocab=V, max_positions=P)
        dq = H * hd
        per = d * 3 * dq + 3 * dq + dq * d + d + 2 * d * F + F + d + 2 * d
        per += 2 * d if arch != "parallel" else 0
        want = L * N * per + (N * d * d if arch == "kraken" else 0) + (V + P) * d + 2 * d
        assert K().weight_blob_elems(cfg) == want, arch
    # the engine table's parameter counts (Section 4.3) with F = 2d and no biases: the
    # blob minus biases and LayerNorms is N * 8 d^2 per layer
    for N, d, H in [(4, 1248, 12), (8, 960, 10), (4, 3120, 30), (8, 2304, 32)]:
        cfg = K().Config(n_sub=N, n_layers=1, d_model=d, n_heads=H, d_ff=2 * d, max_tokens=16)
        extra = N * (4 * d + 3 * d + d + 2 * d + d) + N * d * d   # biases, LNs, W_concat
        assert K().weight_blob_elems(cfg) - extra == N * 8 * d * d


def test_forward_tokens_rejects_bad_arguments_before_the_device():
    L = K().lib()
    ids = (ctypes.c_int32 * 4)(0, 1, 2, 3)
    cu = (ctypes.c_int32 * 2)(0, 4)
    assert L.kraken_forward_tokens(None, ids, cu, 1, None, None, None) == K().ERR_INVALID_ARG


def test_class_flops_of_the_comparison_architectures():
    cu = [0, 128]
    for arch, N in (("gpt", 1), ("parallel", 1), ("kraken", 4)):
        cfg = K().Config(n_sub=N, n_layers=2, d_model=320, n_heads=2, d_ff=1280, head_dim=128,
                         max_tokens=128, arch=arch, vocab=1000, max_positions=128)
        dq = 256
        assert K().class_flops(cfg, K().K_GEMM_QK, cu) == 2 * N * 2.0 * 128 * 320 * 2 * dq
        assert K().class_flops(cfg, K().K_GEMM_O, cu) == 2 * N * 2.0 * 128 * dq * 320
        assert K().class_flops(cfg, K().K_ATTN, cu) == 2 * N * 4.0 * dq * 128 * 129 / 2
        assert K().class_flops(cfg, K().K_UNEMBED, cu) == 2.0 * 1 * 320 * 1000
        assert (K().class_flops(cfg, K().K_CONCAT, cu) > 0) == (arch == "kraken")
