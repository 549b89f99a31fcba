"""Seeded synthetic workloads for the Kraken prefill.

This module only draws numbers: it holds none of the method's arithmetic, and it
is the one thing the HIP path and the fp64 oracle share (the same input arrays,
not code).  Every tensor is keyed by ``(seed, tensor id, layer, sub-layer)`` so any
single tensor can be regenerated on its own, on the host or on a device.  Values
are drawn in fp32 and rounded once (round-to-nearest-even) to the workload's
storage dtype; both sides then use exactly those values.

Workload shapes and distributions follow the paper's TTFT setting (random
weights, batch 1, causal prefill; Section 4.3) at the sizes listed in
``WORKLOADS``: hidden input ~ N(0, 1), weights ~ N(0, 0.02), LayerNorm
gamma = 1 / beta = 0 and zero biases, with the 1/sqrt(2L)-scaled residual
projections where a workload asks for them (Section 3.1 describes that kind of
scaled initialisation).  ``affine="random"`` draws biases ~ N(0, 0.02),
gamma ~ 1 + N(0, 0.1) and beta ~ N(0, 0.02) instead, so that those code paths
are exercised by the parity tests.

``compute`` names the MFMA operand type a workload runs with.  The bf16-storage
workloads run with fp16 operands (bf16 weights convert to fp16 exactly in the
normal range): with bf16 operands the rounding of every GEMM operand alone puts
the deepest stacks at the edge of the 2e-2 parity bound.
"""

from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

__all__ = ["Workload", "WORKLOADS", "workload", "seq_lens", "cu_seqlens",
           "gen_hidden", "gen_sub_layer", "gen_layer", "gen_w_concat", "torch_dtype",
           "compute_dtype", "gen_cached_kv", "ENGINES", "engine_workload", "gen_tokens",
           "gen_embeddings"]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n_sub: int                 # N parallel sub-layers per layer
    n_layers: int              # L
    d_model: int               # d, width of one sub-layer
    n_heads: int               # heads per sub-layer
    d_ff: int                  # MLP width
    dtype: str                 # "f32", "bf16" or "f16" storage dtype
    seq_lens: Optional[Sequence[int]] = None   # fixed lengths (None: drawn, see ragged)
    ragged: Optional[tuple] = None             # (count, lo, hi): lengths ~ U{lo..hi}
    w_std: float = 0.02
    out_proj_std: Optional[float] = None       # std of Wo and W2 (None: w_std)
    compute: str = "storage"                   # MFMA operand type the prefill runs with
    n_kv_heads: int = 0                        # key/value heads (0: n_heads)
    arch: str = "kraken"                       # "kraken", "gpt" or "parallel"
    head_size: int = 0                         # 0: d_model / n_heads
    vocab: int = 0                             # token embedding rows (0: no embeddings)
    max_positions: int = 0                     # position embedding rows

    @property
    def head_dim(self) -> int:
        return self.head_size or self.d_model // self.n_heads

    @property
    def kv_heads(self) -> int:
        return self.n_kv_heads or self.n_heads

    @property
    def kv_width(self) -> int:
        return self.kv_heads * self.head_dim


WORKLOADS: Dict[str, Workload] = {w.name: w for w in [
    Workload("kraken-n2-l2-d128-h4-s64-f32", 2, 2, 128, 4, 512, "f32", seq_lens=(64,)),
    Workload("kraken-n4-l12-d768-h12-s2048-bf16", 4, 12, 768, 12, 3072, "bf16",
             seq_lens=(2048,), compute="f16"),
    Workload("kraken-n4-l24-d1024-h16-s4096-bf16", 4, 24, 1024, 16, 4096, "bf16",
             seq_lens=(4096,), out_proj_std=0.02 / math.sqrt(2 * 24), compute="f16"),
    Workload("kraken-n8-l24-d2048-h16-s8192-bf16", 8, 24, 2048, 16, 8192, "bf16",
             seq_lens=(8192,), compute="f16"),
    Workload("kraken-n4-l36-d1280-h20-ragged8x512-4096-bf16", 4, 36, 1280, 20, 5120, "bf16",
             ragged=(8, 512, 4096), compute="f16"),
    # the benchmark shape with grouped-query attention: 4 key/value heads per sub-layer
    Workload("kraken-n8-l24-d2048-h16-kv4-s8192-bf16", 8, 24, 2048, 16, 8192, "bf16",
             seq_lens=(8192,), compute="f16", n_kv_heads=4),
    # the paper's 4-way Kraken engines of the 65B and 175B models (engine table: d_ff = 2d,
    # heads per sub-layer), built like the paper's with a quarter of the layers, fp16, one
    # sequence of 128 or 2048 tokens
    Workload("kraken-n4-l20-d4992-h39-f9984-s2048-f16", 4, 20, 4992, 39, 9984, "f16",
             seq_lens=(2048,)),
    Workload("kraken-n4-l20-d4992-h39-f9984-s128-f16", 4, 20, 4992, 39, 9984, "f16",
             seq_lens=(128,)),
    Workload("kraken-n4-l24-d7424-h58-f14848-s2048-f16", 4, 24, 7424, 58, 14848, "f16",
             seq_lens=(2048,)),
    Workload("kraken-n4-l24-d7424-h58-f14848-s128-f16", 4, 24, 7424, 58, 14848, "f16",
             seq_lens=(128,)),
]}

# The workload the throughput benchmark runs: N=8 sub-layers of width 2048, 24 layers,
# one causal sequence of 8192 tokens.
BENCH_WORKLOAD = "kraken-n8-l24-d2048-h16-s8192-bf16"

# The paper's TTFT engines (Section 4.3, table of engine configurations): layers, the
# GPT-like width and heads (shared by the parallel attention + FFN engine), and the 4-way
# and 8-way Kraken widths and heads per sub-layer.  The GPT-like engines have an FFN of 4d,
# the Kraken engines of 2d (Section 3.2).  The 65B and 175B engines were built with a
# quarter of the layers; the 13B GPT-like width 5140 with 40 heads has heads of 128 (the
# GPT-3 13B configuration; 5140 / 40 is not an integer).  Vocabulary 51,200 and prompts of
# up to 2048 tokens (Section 4.3).
ENGINES = {
    "1.3b": dict(layers=24, gpt=(2048, 16), kraken4=(1248, 12), kraken8=(960, 10)),
    "6.7b": dict(layers=32, gpt=(4096, 32), kraken4=(2496, 24), kraken8=(1920, 20)),
    "13b": dict(layers=40, gpt=(5140, 40), kraken4=(3120, 30), kraken8=(2304, 32),
                gpt_head=128),
    "65b": dict(layers=20, gpt=(8192, 64), kraken4=(4992, 39), kraken8=(3648, 38)),
    "175b": dict(layers=24, gpt=(12288, 96), kraken4=(7424, 58), kraken8=(5472, 57)),
}
ENGINE_VOCAB = 51200
ENGINE_POSITIONS = 2048


def engine_workload(model: str, arch: str, ctx: int, layers: Optional[int] = None,
                    dtype: str = "f16") -> "Workload":
    """The engine of ``model`` for architecture ``arch`` ("gpt", "parallel", "kraken4" or
    "kraken8"), one prompt of ``ctx`` tokens, random weights, fp16 (Section 4.3)."""
    e = ENGINES[model]
    L = layers or e["layers"]
    if arch in ("gpt", "parallel"):
        d, H = e["gpt"]
        return Workload(f"{arch}-{model}-l{L}-s{ctx}", 1, L, d, H, 4 * d, dtype,
                        seq_lens=(ctx,), arch=arch, head_size=e.get("gpt_head", 0),
                        vocab=ENGINE_VOCAB, max_positions=ENGINE_POSITIONS)
    n = {"kraken4": 4, "kraken8": 8}[arch]
    d, H = e[arch]
    return Workload(f"kraken{n}-{model}-l{L}-s{ctx}", n, L, d, H, 2 * d, dtype,
                    seq_lens=(ctx,), vocab=ENGINE_VOCAB, max_positions=ENGINE_POSITIONS)


_TENSOR_IDS = {"hidden": 1, "ln1_g": 2, "ln1_b": 3, "Wqkv": 4, "bqkv": 5, "Wo": 6, "bo": 7,
               "ln2_g": 8, "ln2_b": 9, "W1": 10, "b1": 11, "W2": 12, "b2": 13,
               "W_concat": 14, "lens": 15, "cache_k": 16, "cache_v": 17, "tokens": 18,
               "tok_emb": 19, "pos_emb": 20, "lnf_g": 21, "lnf_b": 22}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def torch_dtype(w: Workload) -> torch.dtype:
    return {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[w.dtype]


def _key(*parts: int) -> int:
    h = hashlib.sha256(",".join(str(int(p)) for p in parts).encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def _normal(shape, key: int, std: float, mean: float, device, dtype) -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(key)
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    if mean != 0.0:
        t.add_(mean)
    return t.to(dtype)


def seq_lens(w: Workload, seed: int = 0) -> List[int]:
    if w.seq_lens is not None:
        return list(w.seq_lens)
    count, lo, hi = w.ragged
    rng = np.random.default_rng([seed, _TENSOR_IDS["lens"]])
    return [int(v) for v in rng.integers(lo, hi + 1, size=count)]


def cu_seqlens(lens: Sequence[int]) -> List[int]:
    cu = [0]
    for s in lens:
        cu.append(cu[-1] + int(s))
    return cu


def gen_hidden(w: Workload, n_tokens: int, seed: int = 0, device="cpu") -> torch.Tensor:
    """Shared first-layer input ``[T, d]`` ~ N(0, 1)."""
    return _normal((n_tokens, w.d_model), _key(seed, _TENSOR_IDS["hidden"]), 1.0, 0.0,
                   device, torch_dtype(w))


def gen_sub_layer(w: Workload, layer: int, sub: int, seed: int = 0, device="cpu",
                  affine: str = "plain") -> Dict[str, torch.Tensor]:
    """Parameters of sub-layer ``sub`` of layer ``layer`` (x @ W layout, [in, out]); the
    attention width is n_heads * head_dim (d unless a head size is given).  A parallel
    attention + FFN layer has no second LayerNorm."""
    d, f, dkv = w.d_model, w.d_ff, w.kv_width
    dq = w.n_heads * w.head_dim
    dt = torch_dtype(w)
    ostd = w.out_proj_std if w.out_proj_std is not None else w.w_std

    def mat(name, shape, std):
        return _normal(shape, _key(seed, _TENSOR_IDS[name], layer, sub), std, 0.0, device, dt)

    def vec(name, n, kind):
        if affine == "plain":
            fill = 1.0 if kind == "gamma" else 0.0
            return torch.full((n,), fill, dtype=dt, device=device)
        std, mean = {"gamma": (0.1, 1.0), "beta": (0.02, 0.0), "bias": (0.02, 0.0)}[kind]
        return _normal((n,), _key(seed, _TENSOR_IDS[name], layer, sub, 1), std, mean,
                       device, dt)

    if affine not in ("plain", "random"):
        raise ValueError(f"unknown affine variant {affine!r}")
    p = {
        "ln1_g": vec("ln1_g", d, "gamma"), "ln1_b": vec("ln1_b", d, "beta"),
        "Wqkv": mat("Wqkv", (d, dq + 2 * dkv), w.w_std),
        "bqkv": vec("bqkv", dq + 2 * dkv, "bias"),
        "Wo": mat("Wo", (dq, d), ostd), "bo": vec("bo", d, "bias"),
        "ln2_g": vec("ln2_g", d, "gamma"), "ln2_b": vec("ln2_b", d, "beta"),
        "W1": mat("W1", (d, f), w.w_std), "b1": vec("b1", f, "bias"),
        "W2": mat("W2", (f, d), ostd), "b2": vec("b2", d, "bias"),
    }
    if w.arch == "parallel":
        del p["ln2_g"], p["ln2_b"]
    return p


def gen_layer(w: Workload, layer: int, seed: int = 0, device="cpu",
              affine: str = "plain") -> List[Dict[str, torch.Tensor]]:
    return [gen_sub_layer(w, layer, i, seed, device, affine) for i in range(w.n_sub)]


def gen_w_concat(w: Workload, seed: int = 0, device="cpu") -> torch.Tensor:
    """``W_concat`` ``[N*d, d]`` ~ N(0, 0.02)."""
    return _normal((w.n_sub * w.d_model, w.d_model), _key(seed, _TENSOR_IDS["W_concat"]),
                   w.w_std, 0.0, device, torch_dtype(w))


def gen_tokens(w: Workload, n_tokens: int, seed: int = 0) -> np.ndarray:
    """Token ids ~ U{0 .. vocab - 1} (int32, host): a prompt of random tokens."""
    rng = np.random.default_rng([seed, _TENSOR_IDS["tokens"]])
    return rng.integers(0, w.vocab, size=n_tokens).astype(np.int32)


def gen_embeddings(w: Workload, seed: int = 0, device="cpu",
                   affine: str = "plain") -> Dict[str, torch.Tensor]:
    """Token embedding ``[vocab, d]`` and position embedding ``[max_positions, d]`` ~
    N(0, 0.02), the final LayerNorm (gamma = 1, beta = 0, or the random affine variant)."""
    d, dt = w.d_model, torch_dtype(w)
    out = {"tok_emb": _normal((w.vocab, d), _key(seed, _TENSOR_IDS["tok_emb"]), w.w_std, 0.0,
                              device, dt),
           "pos_emb": _normal((w.max_positions, d), _key(seed, _TENSOR_IDS["pos_emb"]), w.w_std,
                              0.0, device, dt)}
    if affine == "plain":
        out["lnf_g"] = torch.ones(d, dtype=dt, device=device)
        out["lnf_b"] = torch.zeros(d, dtype=dt, device=device)
    else:
        out["lnf_g"] = _normal((d,), _key(seed, _TENSOR_IDS["lnf_g"]), 0.1, 1.0, device, dt)
        out["lnf_b"] = _normal((d,), _key(seed, _TENSOR_IDS["lnf_b"]), 0.02, 0.0, device, dt)
    return out


def compute_dtype(w: Workload) -> torch.dtype:
    """MFMA operand type of the workload (the element type of its KV cache)."""
    name = w.dtype if w.compute == "storage" else w.compute
    return {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[name]


def gen_cached_kv(w: Workload, n_tokens: int, layer: int, sub: int, seq: int, seed: int = 0,
                  k_std: float = 1.0, v_std: float = 1.0, device="cpu"):
    """Stand-in cached keys and values ``(K, V)``, each ``[n_tokens, dkv]`` ~ N(0, std^2) in
    the compute type, for sequence ``seq`` of sub-layer ``sub`` of layer ``layer``: the
    earlier tokens of a decode step whose prefill is not run."""
    dt = compute_dtype(w)
    K = _normal((n_tokens, w.kv_width), _key(seed, _TENSOR_IDS["cache_k"], layer, sub, seq),
                k_std, 0.0, device, dt)
    V = _normal((n_tokens, w.kv_width), _key(seed, _TENSOR_IDS["cache_v"], layer, sub, seq),
                v_std, 0.0, device, dt)
    return K, V
