"""Per-kernel parity: each HIP kernel of the prefill, through its C-ABI entry point,
against the fp64 oracle's pieces (or the plain definition of the op) on the same inputs."""

import math

import numpy as np
import pytest
import torch

from oracle import kraken_oracle as O

pytestmark = pytest.mark.gpu

DEV = "cuda"


def K():
    from paper_2408_07802_amd import kraken
    return kraken


def tdt(name):
    return {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[name]


def f64(t):
    return t.detach().double().cpu().numpy()


def check_close(got, ref, dtype_name, what, rel_elem=None, rel_rms=None):
    got, ref = np.asarray(got, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), what
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    if rel_elem is None:
        rel_elem = {"bf16": 2.0 ** -8, "f16": 2.0 ** -11, "f32": 1e-6}[dtype_name]
    if rel_rms is None:
        rel_rms = {"bf16": 2e-3, "f16": 2.5e-4, "f32": 2e-6}[dtype_name]
    bound = rel_elem * np.abs(ref) + rel_rms * rms + 1e-30
    bad = np.abs(got - ref) > bound
    if bad.any():
        idx = np.unravel_index(np.argmax(np.abs(got - ref) - bound), ref.shape)
        raise AssertionError(f"{what}: {bad.sum()} elements out of bound; worst at {idx}: "
                             f"got {got[idx]!r} ref {ref[idx]!r} bound {bound[idx]!r}")


# ----------------------------------------------------------------------------- LayerNorm

@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("n,T,d,shared", [(3, 37, 128, False), (2, 5, 2048, True),
                                          (4, 130, 768, False), (1, 1, 64, False),
                                          (2, 9, 8192, False), (8, 3, 2048, True),
                                          (2, 3, 12288, False), (1, 2, 16384, True)])
def test_layernorm(dtype, n, T, d, shared):
    g = torch.Generator(device="cpu").manual_seed(n * 1000 + T * 7 + d)
    x = (torch.randn((1 if shared else n, T, d), generator=g) * 3 + 1.5).to(DEV)
    gamma = (1 + 0.3 * torch.randn((n, d), generator=g)).to(DEV)
    beta = (0.3 * torch.randn((n, d), generator=g)).to(DEV)
    out = torch.full((n, T, d), float("nan"), dtype=tdt(dtype), device=DEV)
    K().op_layernorm(x, 0 if shared else T * d, gamma, beta, out, n, T, d, 1e-5)
    torch.cuda.synchronize()
    xs, gs, bs = f64(x), f64(gamma), f64(beta)
    for i in range(n):
        ref = O.layer_norm(xs[0 if shared else i], gs[i], bs[i])
        check_close(f64(out[i]), ref, dtype, f"layernorm sub-layer {i}")


# ------------------------------------------------------------------- combine + LN2

@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("n,T,d,shared", [(2, 64, 128, True), (2, 64, 128, False),
                                          (4, 33, 768, False), (8, 17, 2048, False),
                                          (1, 5, 1280, False), (3, 2, 4096, True),
                                          (2, 3, 12288, False), (1, 2, 16384, True)])
def test_combine_ln2(dtype, n, T, d, shared):
    g = torch.Generator(device="cpu").manual_seed(n * 31 + T + d)
    x = torch.randn((n, T, d), generator=g).to(DEV)
    h = torch.randn((n, T, d), generator=g).to(DEV) * 2
    X = torch.randn((T, d), generator=g).to(DEV) if shared else None
    gamma = (1 + 0.3 * torch.randn((n, d), generator=g)).to(DEV)
    beta = (0.3 * torch.randn((n, d), generator=g)).to(DEV)
    out = torch.full((n, T, d), float("nan"), dtype=tdt(dtype), device=DEV)
    K().op_combine_ln2(None if shared else x, X, h, gamma, beta, out, n, T, d, 1e-5)
    torch.cuda.synchronize()
    y = f64(X) if shared else f64(x).sum(axis=0)
    hs, gs, bs = f64(h), f64(gamma), f64(beta)
    for i in range(n):
        ref = O.layer_norm(hs[i] + y, gs[i], bs[i])
        check_close(f64(out[i]), ref, dtype, f"combine_ln2 sub-layer {i}")


# ----------------------------------------------------------------------------- GEMM

GEMM_SHAPES = [  # (M, N, K, batch)
    (128, 128, 64, 1), (200, 96, 128, 2), (1, 300, 64, 1), (333, 129, 192, 3),
    (64, 1536, 768, 2), (257, 2048, 256, 1), (1000, 64, 3072, 1),
]


# Shapes of at least 512 256 x 256 tiles, which select the large-tile configuration of
# 16-bit operands: ragged M and N edges, and the shortest K values (one, two and three
# 64-element slices: the operand ring's prologue alone, then with its second-to-last
# slice, then with one slice that loads two ahead).
GEMM_BIG_SHAPES = [(2000, 1100, 320, 15), (1024, 1024, 64, 32), (1024, 1024, 128, 32),
                   (1024, 1024, 192, 32)]
# a few rows (decode steps): 16-column tiles, the reduction split over 4 waves in blocks of
# 8 steps of 32 k plus a remainder, 1, 2 or 4 blocks of 16 rows
GEMM_SKINNY_SHAPES = [(1, 2048, 8192, 2), (5, 1000, 2048, 3), (16, 4096, 2048, 1),
                      (17, 33, 320, 2), (33, 130, 64, 1), (64, 2048, 1024, 2),
                      (9, 520, 2112, 2), (3, 7, 64, 1), (1, 4096, 2048, 8), (20, 300, 8192, 2)]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("epi", [0, 1, 2, 3])
@pytest.mark.parametrize("shape", GEMM_SHAPES)
def test_gemm(dtype, epi, shape):
    _check_gemm(dtype, epi, shape)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("epi", [0, 1, 2, 3])
@pytest.mark.parametrize("shape", GEMM_BIG_SHAPES)
def test_gemm_big_tiles(dtype, epi, shape):
    _check_gemm(dtype, epi, shape)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("epi", [0, 1, 2, 3])
@pytest.mark.parametrize("shape", GEMM_SKINNY_SHAPES)
def test_gemm_few_rows(dtype, epi, shape):
    _check_gemm(dtype, epi, shape)


def _check_gemm(dtype, epi, shape):
    M, N, Kd, batch = shape
    g = torch.Generator(device="cpu").manual_seed(M * 7 + N * 3 + Kd + batch + epi * 101)
    dt = tdt(dtype)
    A = (torch.randn((batch, M, Kd), generator=g)).to(dt).to(DEV)
    B = (torch.randn((batch, N, Kd), generator=g) * (1.0 / math.sqrt(Kd))).to(dt).to(DEV)
    nb = M if epi == 3 else N
    bias = (0.5 * torch.randn((batch, nb), generator=g)).to(DEV)
    R = torch.randn((batch, M, N), generator=g).to(DEV) if epi == 2 else None
    out_dt = torch.float32 if epi == 2 else dt
    C = torch.full((batch, M, N), float("nan"), dtype=out_dt, device=DEV)
    K().op_gemm(epi, A, B, C, bias, R, M, N, Kd, batch, M * Kd, N * Kd, M * N, M * N)
    torch.cuda.synchronize()
    a, b, bi = f64(A), f64(B), f64(bias)
    for z in range(batch):
        acc = a[z] @ b[z].T
        if epi == 0:
            ref = acc + bi[z][None, :]
        elif epi == 1:
            ref = O.gelu(acc + bi[z][None, :])
        elif epi == 2:
            ref = acc + bi[z][None, :] + f64(R[z])
        else:
            ref = acc + bi[z][:, None]
        odt = "f32" if epi == 2 else dtype
        # fp32 outputs of bf16 products: only accumulation-order error remains
        kw = {"rel_elem": 1e-5, "rel_rms": 1e-5} if odt == "f32" else {}
        check_close(f64(C[z]), ref, odt, f"gemm epi={epi} batch {z}", **kw)


def test_gemm_without_bias_or_residual():
    M, N, Kd = 70, 130, 128
    g = torch.Generator(device="cpu").manual_seed(3)
    A = torch.randn((M, Kd), generator=g).to(torch.bfloat16).to(DEV)
    B = torch.randn((N, Kd), generator=g).to(torch.bfloat16).to(DEV)
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
    K().op_gemm(2, A, B, C, None, None, M, N, Kd, 1, 0, 0, 0, 0)
    torch.cuda.synchronize()
    check_close(f64(C), f64(A) @ f64(B).T, "f32", "gemm plain", rel_elem=1e-5, rel_rms=1e-5)


def test_gemm_gelu_epilogue_accuracy():
    """The GELU epilogue alone: an fp32 GEMM whose products are exactly v (one nonzero k)
    feeds a grid of arguments to it, and the result must stay within twice the
    approximation's absolute error of 1e-7 |v| (plus fp32 rounding of the few operations and
    of the hardware reciprocal and exp2) of the exact erf form, for both signs and far into
    either tail."""
    M, N, Kd = 4096, 64, 64
    v = np.concatenate([np.linspace(-12.0, 12.0, M - 6), [0.0, -0.0, 1e-30, -1e-30, 40.0, -40.0]])
    A = torch.zeros((M, Kd), dtype=torch.float32)
    A[:, 0] = torch.from_numpy(v).float()
    B = torch.zeros((N, Kd), dtype=torch.float32)
    B[:, 0] = 1.0
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
    K().op_gemm(1, A.to(DEV), B.to(DEV), C, None, None, M, N, Kd, 1, 0, 0, 0, 0)
    torch.cuda.synchronize()
    x = f64(A[:, 0])                                   # the fp32 arguments
    ref = np.array([0.5 * t * (1.0 + math.erf(t / math.sqrt(2.0))) for t in x])
    got = f64(C)
    bound = 2e-7 * np.abs(x) + 8 * 2.0 ** -24 * np.abs(ref) + 1e-37
    err = np.abs(got - ref[:, None])
    assert np.all(np.isfinite(got))
    assert np.all(err <= bound[:, None]), (float(np.max(err / bound[:, None])),
                                           x[np.argmax(np.max(err, axis=1) / bound)])
    assert np.all(got[x == 0.0] == 0.0)


@pytest.mark.parametrize("epi", [0, 2])
def test_gemm_one_tile_per_cu_long_k(epi):
    """256 tiles of 256 x 256 with K = 8192: the one-round large-tile configuration (the
    W_concat shape).  Sampled rows of every batch entry against fp64."""
    M, N, Kd, batch = 2048, 2048, 8192, 4
    g = torch.Generator(device="cpu").manual_seed(77 + epi)
    A = torch.randn((batch, M, Kd), generator=g).to(torch.float16).to(DEV)
    B = (torch.randn((batch, N, Kd), generator=g) / math.sqrt(Kd)).to(torch.float16).to(DEV)
    bias = (0.5 * torch.randn((batch, N), generator=g)).to(DEV)
    R = torch.randn((batch, M, N), generator=g).to(DEV) if epi == 2 else None
    C = torch.full((batch, M, N), float("nan"),
                   dtype=torch.float32 if epi == 2 else torch.float16, device=DEV)
    K().op_gemm(epi, A, B, C, bias, R, M, N, Kd, batch, M * Kd, N * Kd, M * N, M * N)
    torch.cuda.synchronize()
    rows = torch.arange(0, M, 61)
    for z in range(batch):
        ref = f64(A[z, rows]) @ f64(B[z]).T + f64(bias[z])[None, :]
        if epi == 2:
            ref = ref + f64(R[z, rows])
            check_close(f64(C[z, rows]), ref, "f32", f"one-round gemm {z}", rel_elem=1e-5,
                        rel_rms=1e-5)
        else:
            check_close(f64(C[z, rows]), ref, "f16", f"one-round gemm {z}")


def test_gemm_shared_residual_batch_stride_zero():
    M, N, Kd, batch = 50, 64, 64, 3
    g = torch.Generator(device="cpu").manual_seed(4)
    A = torch.randn((batch, M, Kd), generator=g).to(torch.bfloat16).to(DEV)
    B = torch.randn((batch, N, Kd), generator=g).to(torch.bfloat16).to(DEV)
    R = torch.randn((M, N), generator=g).to(DEV)
    C = torch.empty((batch, M, N), dtype=torch.float32, device=DEV)
    K().op_gemm(2, A, B, C, None, R, M, N, Kd, batch, M * Kd, N * Kd, M * N, 0)
    torch.cuda.synchronize()
    for z in range(batch):
        check_close(f64(C[z]), f64(A[z]) @ f64(B[z]).T + f64(R), "f32", f"gemm shared R {z}",
                    rel_elem=1e-5, rel_rms=1e-5)


# ----------------------------------------------------------------------------- attention

ATTN_CASES = [  # (n, d, heads, seq_lens)
    (1, 128, 4, [64]), (2, 128, 4, [1, 7, 64, 5]), (2, 256, 4, [300]),
    (1, 256, 2, [129, 1, 250]), (3, 768, 12, [200, 57]), (1, 512, 4, [513]),
    (2, 2048, 16, [130]), (1, 1280, 20, [31, 97, 160]),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("case", ATTN_CASES)
def test_attention(dtype, case):
    n, d, H, lens = case
    cu = [0]
    for s in lens:
        cu.append(cu[-1] + s)
    T = cu[-1]
    ldv = K().vt_ld(T)
    dt = tdt(dtype)
    g = torch.Generator(device="cpu").manual_seed(T * 13 + d + n)
    qk = (torch.randn((n, T, 2 * d), generator=g) * 1.5).to(dt).to(DEV)
    v = torch.randn((n, T, d), generator=g).to(dt)
    vt = torch.zeros((n, d, ldv), dtype=dt)
    vt[:, :, :T] = v.transpose(1, 2)
    vt = vt.to(DEV)
    out = torch.full((n, T, d), float("nan"), dtype=dt, device=DEV)
    K().op_attention(qk, vt, out, n, d, H, cu)
    torch.cuda.synchronize()
    q64, v64 = f64(qk), f64(v)
    for i in range(n):
        ref = O.causal_attention(q64[i][:, :d], q64[i][:, d:], v64[i], cu, H)
        check_attention(f64(out[i]), ref, q64[i], np.abs(v64[i]), cu, H, dtype,
                        f"attention sub-layer {i}")


GQA_ATTN_CASES = [  # (n, d, heads, kv heads, seq_lens): groups of 2, 4, 8 and 3 heads
    (2, 256, 4, 2, [300, 17]), (1, 256, 4, 1, [129, 200]), (2, 512, 16, 4, [130]),
    (1, 2048, 16, 2, [257, 64]), (1, 384, 6, 2, [100]), (1, 512, 16, 2, [70]),
]


@pytest.mark.parametrize("dtype", ["f32", "f16"])
@pytest.mark.parametrize("case", GQA_ATTN_CASES)
def test_attention_grouped_query(dtype, case):
    n, d, H, Hkv, lens = case
    dkv = Hkv * (d // H)
    cu = [0]
    for s in lens:
        cu.append(cu[-1] + s)
    T = cu[-1]
    ldv = K().vt_ld(T)
    dt = tdt(dtype)
    g = torch.Generator(device="cpu").manual_seed(T * 7 + d + H + Hkv)
    qk = (torch.randn((n, T, d + dkv), generator=g) * 1.5).to(dt).to(DEV)
    v = torch.randn((n, T, dkv), generator=g).to(dt)
    vt = torch.zeros((n, dkv, ldv), dtype=dt)
    vt[:, :, :T] = v.transpose(1, 2)
    vt = vt.to(DEV)
    out = torch.full((n, T, d), float("nan"), dtype=dt, device=DEV)
    K().op_attention(qk, vt, out, n, d, H, cu, n_kv_heads=Hkv)
    torch.cuda.synchronize()
    q64, v64 = f64(qk), f64(v)
    for i in range(n):
        ref = O.causal_attention(q64[i][:, :d], q64[i][:, d:], v64[i], cu, H, Hkv)
        check_attention(f64(out[i]), ref, q64[i], np.abs(v64[i]), cu, H, dtype,
                        f"grouped-query attention sub-layer {i}", d=d, Hkv=Hkv)


def check_attention(got, ref, qk64, vabs, cu, H, dtype, what, d=None, Hkv=None):
    """Elementwise bound from the rounding model of the kernel.

    bf16: the probabilities p are rounded to bf16 (relative error <= 2^-8) before the
    P V product and the output is rounded to bf16, so
    |err| <= 2^-8 (sum_k p_k |v_k| + |out|) plus fp32 accumulation error; the sum is
    the oracle's attention applied to |V|.  fp32: the score error (fp32 dot products of
    up to 128 terms, |s| up to ~30) moves each p by a relative ~1e-6 |s| through the
    exponential; 2^-16 covers it.
    """
    d = d or qk64.shape[1] // 2
    weighted_abs = O.causal_attention(qk64[:, :d], qk64[:, d:], vabs, cu, H, Hkv)
    u = {"bf16": 2.0 ** -8, "f16": 2.0 ** -11, "f32": 2.0 ** -16}[dtype]
    bound = u * (weighted_abs + np.abs(ref)) + 1e-6 * np.sqrt(np.mean(ref ** 2))
    assert np.all(np.isfinite(got)), what
    bad = np.abs(got - ref) > bound
    if bad.any():
        idx = np.unravel_index(np.argmax(np.abs(got - ref) / bound), ref.shape)
        raise AssertionError(f"{what}: {bad.sum()} elements out of bound; worst at {idx}: "
                             f"got {got[idx]!r} ref {ref[idx]!r} bound {bound[idx]!r}")


def test_attention_large_logits_stay_finite():
    n, d, H, lens = 1, 256, 2, [200]
    T = 200
    ldv = K().vt_ld(T)
    g = torch.Generator(device="cpu").manual_seed(9)
    qk = (torch.randn((n, T, 2 * d), generator=g) * 6).to(torch.bfloat16).to(DEV)
    v = torch.randn((n, T, d), generator=g).to(torch.bfloat16)
    vt = torch.zeros((n, d, ldv), dtype=torch.bfloat16)
    vt[:, :, :T] = v.transpose(1, 2)
    out = torch.empty((n, T, d), dtype=torch.bfloat16, device=DEV)
    K().op_attention(qk, vt.to(DEV), out, n, d, H, [0, T])
    torch.cuda.synchronize()
    ref = O.causal_attention(f64(qk[0])[:, :d], f64(qk[0])[:, d:], f64(v[0]), [0, T], H)
    check_attention(f64(out[0]), ref, f64(qk[0]), np.abs(f64(v[0])), [0, T], H, "bf16",
                    "attention large logits")


# ------------------------------------------- attention with pre-scaled Q (the product form)

LOG2E = 1.4426950408889634

PRESCALED_CASES = [  # (n, d, heads, seq_lens, heads checked per sub-layer or None = all)
    (2, 256, 2, [300, 1, 129], None),            # head size 128: ping-pong kernel
    (1, 512, 8, [513, 64], None),                # head size 64: one-phase kernel, scale 1
    (2, 128, 4, [200, 7], None),                 # head size 32
    (2, 1024, 8, [4500, 700], None),             # 71 + 11 key tiles, ragged tail
    # the benchmark's attention launch for 4 of its 8 sub-layers: one 8192-token sequence,
    # 16 heads of 128, 2048 workgroups in the head-grouped XCD order, all 128 key tiles
    (4, 2048, 16, [8192], [0, 5, 10, 15]),
    # ragged lengths of the packed 8-sequence workload at head size 128: the grouped order
    # over an uneven tile prefix
    (4, 2048, 16, [3585, 2177, 3101, 3452, 1119, 2039, 1665, 1442], [0, 9, 15]),
]


def prescaled_inputs(n, d, H, T, dt, seed):
    """Q|K rows and V^T as the prefill hands them to attention: the Q columns carry
    log2(e) / sqrt(hd) (rounded once to the operand type).  Returns the device operands and
    the fp64 Q, K, V the oracle takes (Q divided back by the factor, exactly in fp64)."""
    hd = d // H
    c = LOG2E / math.sqrt(hd)
    g = torch.Generator(device="cpu").manual_seed(seed)
    q = torch.randn((n, T, d), generator=g) * 1.5
    k = torch.randn((n, T, d), generator=g) * 1.5
    v = torch.randn((n, T, d), generator=g)
    qk = torch.cat([(q * c).to(dt), k.to(dt)], dim=2)
    v = v.to(dt)
    ldv = K().vt_ld(T)
    vt = torch.zeros((n, d, ldv), dtype=dt)
    vt[:, :, :T] = v.transpose(1, 2)
    q64 = qk[:, :, :d].double().numpy() / c
    return qk, vt, q64, qk[:, :, d:].double().numpy(), v.double().numpy()


def check_heads(got, q64, k64, v64, cu, H, heads, dtype, what):
    """The kernel's output against the oracle's causal attention, for the given heads
    (each head is independent: the oracle runs on those heads' columns alone)."""
    hd = q64.shape[1] // H
    heads = list(range(H)) if heads is None else heads
    cols = np.concatenate([np.arange(h * hd, (h + 1) * hd) for h in heads])
    qs, ks, vs = q64[:, cols], k64[:, cols], v64[:, cols]
    ref = O.causal_attention(qs, ks, vs, cu, len(heads))
    check_attention(got[:, cols], ref, np.concatenate([qs, ks], axis=1), np.abs(vs), cu,
                    len(heads), dtype, what)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("case", PRESCALED_CASES)
def test_attention_prescaled_q(dtype, case):
    n, d, H, lens, heads = case
    if heads is not None and dtype == "bf16":
        heads = heads[:2]
    cu = [0]
    for s_ in lens:
        cu.append(cu[-1] + s_)
    T = cu[-1]
    print(f"[attention q_prescaled] n={n} d={d} H={H} lens={lens} {dtype}", flush=True)
    qk, vt, q64, k64, v64 = prescaled_inputs(n, d, H, T, tdt(dtype), T * 31 + d + n)
    out = torch.full((n, T, d), float("nan"), dtype=tdt(dtype), device=DEV)
    K().op_attention(qk.to(DEV), vt.to(DEV), out, n, d, H, cu, q_prescaled=True)
    torch.cuda.synchronize()
    got = f64(out)
    for i in range(n):
        check_heads(got[i], q64[i], k64[i], v64[i], cu, H, heads, dtype,
                    f"pre-scaled attention sub-layer {i}")


@pytest.mark.parametrize("pre", [True, False])
@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_attention_rising_scores_take_every_softmax_path(dtype, pre):
    """Ping-pong attention (head size 128, Q pre-scaled or not) on scores that climb by ~2.5
    (log2 units) per 64-key tile over the first 1100 keys and then drop by 10.  The
    running maximum outgrows the exponent base every few tiles (rescales of O); most
    tiles in between have packed row sums of 2^8 or more while staying within 8 of the
    base (the exact path, which then keeps the base); the low tail takes the shortcut
    without a maximum.  Every query sees the same profile up to its own position."""
    n, d, H, T = 1, 256, 2, 1700
    hd = d // H
    cu = [0, T]
    dt = tdt(dtype)
    g = torch.Generator(device="cpu").manual_seed(77)
    q = torch.randn((n, T, d), generator=g) * 0.1           # Q in log2-unit scale
    k = torch.randn((n, T, d), generator=g) * 0.1
    v = torch.randn((n, T, d), generator=g).to(dt)
    t = torch.arange(T, dtype=torch.float32)
    score = torch.where(t < 1100, 2.5 * t / 64, torch.full_like(t, 2.5 * 1100 / 64 - 10))
    score = score + 0.5 * torch.sin(t)
    for h in range(H):
        q[:, :, h * hd] = 1.0
        k[:, :, h * hd] = score
    c = LOG2E / math.sqrt(hd)
    qk = torch.cat([(q if pre else q / c).to(dt), k.to(dt)], dim=2)
    vt = torch.zeros((n, d, K().vt_ld(T)), dtype=dt)
    vt[:, :, :T] = v.transpose(1, 2)
    print(f"[attention rising scores] T={T} {dtype} q_prescaled={pre}", flush=True)
    out = torch.full((n, T, d), float("nan"), dtype=dt, device=DEV)
    K().op_attention(qk.to(DEV), vt.to(DEV), out, n, d, H, cu, q_prescaled=pre)
    torch.cuda.synchronize()
    q64 = qk[0, :, :d].double().numpy() / (c if pre else 1.0)
    check_heads(f64(out[0]), q64, qk[0, :, d:].double().numpy(), v[0].double().numpy(), cu,
                H, None, dtype, "attention with rising scores")


def test_attention_dma_base_with_bit31_of_the_low_address_word_set_and_clear():
    """Regression test of a fixed fault.  The ping-pong attention kernel rebuilds each
    wave-uniform 64-bit DMA base from two 32-bit halves; the low half must be widened as
    unsigned, or an address whose low word has bit 31 set sign-extends over the high word.
    Whether a tile base has that bit set depends on where the allocator puts the operands,
    so here they are placed inside one allocation of more than 2 GiB at addresses whose low
    word has bit 31 set, then clear, and the result is checked against the oracle."""
    n, d, H, lens = 2, 256, 2, [1000, 300]
    cu = [0, 1000, 1300]
    T = cu[-1]
    dt = torch.float16
    qk, vt, q64, k64, v64 = prescaled_inputs(n, d, H, T, dt, 4242)
    sizes = [qk.numel() * 2, vt.numel() * 2, n * T * d * 2]
    offs = [0]
    for sz in sizes[:-1]:
        offs.append(offs[-1] + (sz + 4095) // 4096 * 4096)
    need = offs[-1] + sizes[-1]
    big = torch.empty(2 ** 31 + 2 * need + 8192, dtype=torch.uint8, device=DEV)
    base = big.data_ptr()
    for bit in (1, 0):
        # first 4 KiB-aligned window of `need` bytes whose addresses all have bit 31 == bit
        a = (base + 4095) // 4096 * 4096
        if ((a >> 31) & 1) != bit or (((a + need - 1) >> 31) & 1) != bit:
            a = ((a >> 31) + 1) << 31
            if ((a >> 31) & 1) != bit:
                a = ((a >> 31) + 1) << 31
        assert a + need <= base + big.numel()
        assert ((a >> 31) & 1) == bit and (((a + need - 1) >> 31) & 1) == bit
        o = a - base
        views = []
        for off, sz, shape in zip(offs, sizes, [qk.shape, vt.shape, (n, T, d)]):
            views.append(big[o + off:o + off + sz].view(dt).view(shape))
        views[0].copy_(qk.to(DEV))
        views[1].copy_(vt.to(DEV))
        views[2].fill_(float("nan"))
        for pre in (True, False):
            if pre:          # the Q columns carry log2(e) / sqrt(hd)
                q_ref = q64
            else:            # plain Q: the operand holds unscaled values
                plain = torch.from_numpy(q64).to(dt)
                views[0][:, :, :d].copy_(plain.to(DEV))
                q_ref = plain.double().numpy()
            print(f"[attention dma base] low-word bit 31 = {bit}, q_prescaled={pre}",
                  flush=True)
            K().op_attention(views[0], views[1], views[2], n, d, H, cu, q_prescaled=pre)
            torch.cuda.synchronize()
            got = f64(views[2])
            for i in range(n):
                check_heads(got[i], q_ref[i], k64[i], v64[i], cu, H, None, "f16",
                            f"bit31={bit} pre={pre} sub-layer {i}")
    del big
    torch.cuda.empty_cache()


@pytest.mark.timeout(600)
def test_attention_past_32_bit_qk_offsets_takes_the_one_phase_kernel():
    """One layer's Q|K rows of more than 4 GiB (T (d + dkv) 2 bytes > 2^32, here 65,537
    tokens of d = dkv = 16,384, 128 heads of 128): the ping-pong kernel addresses them with
    32-bit byte offsets, so the launch takes the one-phase kernel.  Sampled query rows of
    two heads against the oracle's single-row attention (a row attends to itself and the
    keys before it), under the elementwise bound of the kernel's rounding model."""
    n, d, H, hd = 1, 16384, 128, 128
    T = (1 << 32) // (2 * d * 2) + 1
    assert T * 2 * d * 2 > (1 << 32) - 1
    dt = torch.float16
    c = LOG2E / math.sqrt(hd)
    g = torch.Generator(device=DEV).manual_seed(1729)
    qk = torch.empty((n, T, 2 * d), dtype=dt, device=DEV)
    qk[:, :, :d] = (torch.randn((n, T, d), generator=g, device=DEV) * (1.5 * c)).to(dt)
    qk[:, :, d:] = (torch.randn((n, T, d), generator=g, device=DEV) * 1.5).to(dt)
    v = torch.randn((n, T, d), generator=g, device=DEV).to(dt)
    vt = torch.zeros((n, d, K().vt_ld(T)), dtype=dt, device=DEV)
    vt[:, :, :T] = v.transpose(1, 2)
    out = torch.full((n, T, d), float("nan"), dtype=dt, device=DEV)
    print(f"[attention 32-bit fallback] T={T} d={d} H={H}", flush=True)
    K().op_attention(qk, vt, out, n, d, H, [0, T], q_prescaled=True)
    torch.cuda.synchronize()
    rows = [0, 1, 63, 64, 4095, 30001, T - 2, T - 1]
    for h in (0, 77):
        cols = slice(h * hd, (h + 1) * hd)
        q64 = f64(qk[0, :, cols]) / c
        k64 = f64(qk[0, :, d + h * hd:d + (h + 1) * hd])
        v64 = f64(v[0, :, cols])
        got = f64(out[0, rows, cols])
        for j, r in enumerate(rows):
            args = (q64[r:r + 1], k64[r:r + 1])
            ref = O.cached_attention(*args, v64[r:r + 1], [k64[:r]], [v64[:r]], 1)[0]
            wabs = O.cached_attention(*args, np.abs(v64[r:r + 1]), [k64[:r]],
                                      [np.abs(v64[:r])], 1)[0]
            bound = 2.0 ** -11 * (wabs + np.abs(ref)) + 1e-6 * np.sqrt(np.mean(ref ** 2))
            err = np.abs(got[j] - ref)
            assert np.all(np.isfinite(got[j])), (h, r)
            assert np.all(err <= bound), (h, r, float(np.max(err / bound)))
    del qk, vt, v, out
    torch.cuda.empty_cache()


# ----------------------------------------------------------------------- decode attention

DECODE_ATTN_CASES = [
    # n, d, H, lens (cached tokens before the new one), max_seqs, capacity, work splits
    (2, 128, 4, [0, 1, 255, 256, 257], 6, 300, None),        # hd 32, chunk edges
    (1, 256, 4, [5000, 17, 0], 3, 5001, None),               # hd 64, 20 chunks
    (3, 256, 2, [1023, 4096], 2, 4100, None),                 # hd 128
    (2, 256, 2, [9000, 300, 0], 4, 9001, 2),                  # 2 chunks of 4608 keys
    (1, 128, 1, [777], 1, 800, 1),                            # hd 128, one chunk, 4 pieces
]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("case", DECODE_ATTN_CASES)
def test_decode_attention(dtype, case):
    n, d, H, lens, max_seqs, cap, splits = case
    _check_decode_attention(dtype, n, d, H, H, lens, max_seqs, cap, splits)


DECODE_GQA_CASES = [
    # n, d, H, Hkv, lens, max_seqs, capacity, work splits: groups of 2, 4, 8 and 3 heads
    # (workgroups of 2, 4, 4 and 1 query heads), chunk edges, an empty cache
    (2, 256, 4, 2, [0, 255, 256, 1500], 4, 1600, None),
    (1, 512, 16, 4, [3000, 1], 2, 3001, 3),
    (1, 512, 16, 2, [777, 0], 2, 800, None),
    (2, 384, 6, 2, [513, 40], 3, 600, None),
    (1, 2048, 16, 1, [8192], 1, 8193, None),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("case", DECODE_GQA_CASES)
def test_decode_attention_grouped_query(dtype, case):
    n, d, H, Hkv, lens, max_seqs, cap, splits = case
    _check_decode_attention(dtype, n, d, H, Hkv, lens, max_seqs, cap, splits)


def _check_decode_attention(dtype, n, d, H, Hkv, lens, max_seqs, cap, splits):
    hd, B = d // H, len(lens)
    dkv = Hkv * hd
    dt = tdt(dtype)
    g = torch.Generator(device="cpu").manual_seed(sum(lens) + 7 * d + n + 31 * Hkv)
    qk = (torch.randn((n, B, d + dkv), generator=g) * 2.0).to(dt)
    cache = torch.full((n, 2, max_seqs, Hkv, cap, hd), float("nan"), dtype=dt)
    rows_k, rows_v = [], []
    for i in range(n):
        rk, rv = [], []
        for b in range(B):
            # keys and values at positions 0..lens[b]; the new token's own at lens[b]
            k = (torch.randn((lens[b] + 1, dkv), generator=g) * 2.0).to(dt)
            v = torch.randn((lens[b] + 1, dkv), generator=g).to(dt)
            cache[i, 0, b, :, :lens[b] + 1] = k.view(-1, Hkv, hd).transpose(0, 1)
            cache[i, 1, b, :, :lens[b] + 1] = v.view(-1, Hkv, hd).transpose(0, 1)
            rk.append(f64(k))
            rv.append(f64(v))
        rows_k.append(rk)
        rows_v.append(rv)
    per_split = n * B * H * (hd + 2)
    work = torch.empty(per_split * (splits or 64), dtype=torch.float32, device=DEV)
    out = torch.full((n, B, d), float("nan"), dtype=dt, device=DEV)
    K().op_decode_attention(qk.to(DEV), cache.to(DEV), out, n, d, H, lens, max_seqs, cap, work,
                            n_kv_heads=Hkv)
    torch.cuda.synchronize()
    q64 = f64(qk)
    for i in range(n):
        q = q64[i][:, :d]
        k_new = np.stack([rows_k[i][b][-1] for b in range(B)])
        v_new = np.stack([rows_v[i][b][-1] for b in range(B)])
        K_c = [rows_k[i][b][:-1] for b in range(B)]
        V_c = [rows_v[i][b][:-1] for b in range(B)]
        ref = O.cached_attention(q, k_new, v_new, K_c, V_c, H, Hkv)
        wabs = O.cached_attention(q, k_new, np.abs(v_new), K_c, [np.abs(x) for x in V_c], H,
                                  Hkv)
        # fp32 scores, probabilities and accumulation; one rounding of the output to S
        u = {"bf16": 2.0 ** -8, "f16": 2.0 ** -11, "f32": 0.0}[dtype]
        bound = u * np.abs(ref) + 2.0 ** -16 * wabs + 1e-6 * np.sqrt(np.mean(ref ** 2))
        got = f64(out[i])
        assert np.all(np.isfinite(got))
        bad = np.abs(got - ref) > bound
        assert not bad.any(), (i, int(bad.sum()), float(np.max(np.abs(got - ref) - bound)))


def test_decode_attention_rejects_small_work_and_bad_lens():
    n, d, H, B, cap = 1, 128, 2, 2, 8
    qk = torch.zeros((n, B, 2 * d), dtype=torch.bfloat16, device=DEV)
    cache = torch.zeros((n, 2, B, H, cap, d // H), dtype=torch.bfloat16, device=DEV)
    out = torch.empty((n, B, d), dtype=torch.bfloat16, device=DEV)
    small_work = torch.empty(n * B * H * (d // H + 2) - 1, dtype=torch.float32, device=DEV)
    work = torch.empty(n * B * H * (d // H + 2), dtype=torch.float32, device=DEV)
    with pytest.raises(K().KrakenError):
        K().op_decode_attention(qk, cache, out, n, d, H, [0, 0], B, cap, small_work)
    with pytest.raises(K().KrakenError):
        K().op_decode_attention(qk, cache, out, n, d, H, [0, cap], B, cap, work)
    with pytest.raises(K().KrakenError):
        K().op_decode_attention(qk, cache, out, n, d, H, [0, 0, 0], B, cap, work)
