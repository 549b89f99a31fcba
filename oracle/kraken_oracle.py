"""Plain fp64 CPU oracle for the Kraken prefill forward pass.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import this module:
it is used by ``tests/``, by ``__graft_entry__.smoke()`` and by the
``cpu_baseline`` leg of ``bench.py``, and by nothing else.  It shares no code
with the HIP path (no kernels, headers, layouts or helpers); the two meet only
in the seeded input arrays that the tests hand to both.

What it computes (Prabhakar, Zhang and Wentzlaff, "Kraken: Inherently Parallel
Transformers For Efficient Multi-Device Inference", arXiv 2408.07802):

* Algorithm 1 ("Kraken Sub-Layer: Forward Pass"): for one sub-layer with
  input ``x`` and the combined activations ``y`` of the previous layer,
      h   = x + MHA(LN1(x))
      out = h + FFN(LN2(h + y)).
  The first layer uses ``y = x`` (the AllReduce is replaced by the identity).
* Section 3.1 (layer construction): ``y`` is the element-wise sum of the N
  sub-layer outputs of the previous layer, added before the FFN LayerNorm;
  all first-layer sub-layers share one input; after the last layer the N
  outputs are concatenated and multiplied by ``W_concat`` (Nd x d).
* Section 2.1 (background): MHA is ``softmax(Q K^T / sqrt(h)) V`` per head with
  ``h`` the head dimension, heads combined by the output projection; the FFN is
  two linears with a GELU in between; LayerNorms sit before MHA and FFN
  (pre-LN).

Readings where the paper is silent or ambiguous:
LayerNorm uses the biased variance and eps = 1e-5; GELU is the exact erf form;
all four linears carry a bias, ``W_concat`` does not; the causal mask applies
within each packed sequence only; ``y`` includes the sub-layer's own input
(an AllReduce sums every participant).

Every function works in float64 on whatever values it is given; callers pass
the exact dtype-rounded inputs and weights of the run being checked.

Decode (the autoregressive phase after the prefill; Section 2.1 on the KV
cache: the keys and values of every token are cached, and each decode step
appends its own): a new token of a sequence runs the same layer stack on its own
row; its attention sees the keys and values of every earlier token of its
sequence, cached by the prefill (and earlier decode steps) per layer and
sub-layer, plus its own.  By causality a decode step equals the last row of the
prefill of the extended sequence; the pins in ``tests/test_oracle_pins.py``
check exactly that.

Grouped-query attention (the Kraken paper's suggested way to shrink its larger KV
cache, citing multi-query and grouped-query attention; appendix on the KV cache
size): with ``n_kv_heads`` = Hkv < H key/value heads, the H query heads form Hkv
groups of G = H / Hkv consecutive heads and every head of group g uses key/value
head g (head h reads K/V head ``h // G``); Hkv = 1 is multi-query attention and
Hkv = H the standard multi-head attention.  Only the key and value projections
narrow, to dkv = Hkv * hd columns each.

The whole model (``model_forward``): token and position embeddings shared by the
first layer (Section 3.1), the layer stack, W_concat for Kraken, a final
LayerNorm and the unembedding tied to the token embedding, giving the
next-token logits of each sequence's last token (Section 2.1).  Besides the
Kraken stack it runs the two architectures the paper compares with at the same
sizes (Section 4.3, engine configurations): the standard GPT-like layer and the
parallel attention + FFN layer of GPT-J / PaLM.  The head size may differ from
the width divided by the heads (``head_dim``), as in the GPT-3 13B configuration.

Weight layout taken by this module (a convention, not mathematics): every
matrix multiplies as ``u @ W`` (row-major ``[in, out]``); ``Wqkv`` has
columns ``[Q | K | V]`` (widths dq = heads * hd, dkv, dkv) and head ``h`` owns
columns ``h*hd:(h+1)*hd`` of Q, key/value head ``g`` columns ``g*hd:(g+1)*hd`` of
K and V; ``Wo`` is ``[dq, d]``.
"""

from __future__ import annotations

import math
from typing import Iterable, Mapping, Sequence

import numpy as np
from scipy.special import erf as _erf

LN_EPS = 1e-5

# Names of the per-(layer, sub-layer) parameters, as the oracle reads them.
PARAM_NAMES = ("ln1_g", "ln1_b", "Wqkv", "bqkv", "Wo", "bo",
               "ln2_g", "ln2_b", "W1", "b1", "W2", "b2")


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def layer_norm(v: np.ndarray, gamma, beta, eps: float = LN_EPS) -> np.ndarray:
    """Pre-LN LayerNorm over the last axis (Section 2.1; Algorithm 1).

    ``gamma * (v - mean) / sqrt(var + eps) + beta`` with the biased variance.
    """
    v = _f64(v)
    mu = v.mean(axis=-1, keepdims=True)
    var = ((v - mu) ** 2).mean(axis=-1, keepdims=True)
    return _f64(gamma) * (v - mu) / np.sqrt(var + eps) + _f64(beta)


def gelu(z: np.ndarray) -> np.ndarray:
    """Exact GELU, ``z * Phi(z) = z/2 * (1 + erf(z / sqrt 2))`` (Section 2.1)."""
    z = _f64(z)
    return 0.5 * z * (1.0 + _erf(z / math.sqrt(2.0)))


def causal_attention(Q, K, V, cu_seqlens: Sequence[int], n_heads: int,
                     n_kv_heads: int | None = None) -> np.ndarray:
    """Scaled dot-product attention with a causal mask, per head and per sequence.

    Section 2.1: each head computes ``softmax(Q K^T / sqrt(hd)) V``.  ``Q`` is
    ``[T, d]`` with head ``h`` in columns ``h*hd:(h+1)*hd``; ``K, V`` are
    ``[T, n_kv_heads*hd]`` and head ``h`` uses their head ``h // (n_heads /
    n_kv_heads)`` (grouped-query attention; by default every head has its own).
    Tokens of packed sequence ``b`` are rows ``cu[b]:cu[b+1]`` and attend to
    themselves and to earlier tokens of the same sequence only.  Returns the heads
    concatenated, ``[T, d]``.
    """
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    T, d = Q.shape
    hd = d // n_heads
    group = n_heads // (n_kv_heads or n_heads)
    out = np.zeros((T, d), dtype=np.float64)
    for b in range(len(cu_seqlens) - 1):
        s0, s1 = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        S = s1 - s0
        future = np.triu(np.ones((S, S), dtype=bool), k=1)   # key index > query index
        for h in range(n_heads):
            cols = slice(h * hd, (h + 1) * hd)
            kv = slice((h // group) * hd, (h // group + 1) * hd)
            scores = Q[s0:s1, cols] @ K[s0:s1, kv].T / math.sqrt(hd)
            scores[future] = -np.inf
            scores -= scores.max(axis=1, keepdims=True)
            p = np.exp(scores)
            p /= p.sum(axis=1, keepdims=True)
            out[s0:s1, cols] = p @ V[s0:s1, kv]
    return out


def multi_head_attention(u, p: Mapping, cu_seqlens, n_heads: int,
                         kv_out: list | None = None,
                         n_kv_heads: int | None = None,
                         head_dim: int | None = None) -> np.ndarray:
    """MHA block: QKV projection, per-head causal attention, output projection.

    ``Wqkv`` has ``dq + 2 dkv`` columns ``[Q | K | V]`` with dq = n_heads * hd and
    dkv = n_kv_heads * hd; hd = ``head_dim``, by default d / n_heads (Section 4.3:
    the model width divided by the number of heads), and ``Wo`` is ``[dq, d]``.
    With ``kv_out`` (a list), appends this block's keys and values ``(K, V)``
    (``[T, dkv]`` each, the projections the attention used).
    """
    u = _f64(u)
    d = u.shape[1]
    hd = head_dim or d // n_heads
    dq, dkv = n_heads * hd, hd * (n_kv_heads or n_heads)
    qkv = u @ _f64(p["Wqkv"]) + _f64(p["bqkv"])
    Q, K, V = qkv[:, :dq], qkv[:, dq:dq + dkv], qkv[:, dq + dkv:]
    if kv_out is not None:
        kv_out.append((K, V))
    return (causal_attention(Q, K, V, cu_seqlens, n_heads, n_kv_heads) @ _f64(p["Wo"])
            + _f64(p["bo"]))


def feed_forward(u, p: Mapping) -> np.ndarray:
    """FFN block: two linears with the exact GELU between them (Section 2.1)."""
    u = _f64(u)
    return gelu(u @ _f64(p["W1"]) + _f64(p["b1"])) @ _f64(p["W2"]) + _f64(p["b2"])


def sub_layer_forward(x, y, p: Mapping, cu_seqlens, n_heads: int,
                      eps: float = LN_EPS, kv_out: list | None = None,
                      n_kv_heads: int | None = None,
                      head_dim: int | None = None) -> np.ndarray:
    """One Kraken sub-layer (Algorithm 1) given its input ``x`` and combined ``y``.

    ``h = x + MHA(LN1(x))``; returns ``h + FFN(LN2(h + y))``.  ``kv_out``,
    ``n_kv_heads``, ``head_dim``: see ``multi_head_attention``.
    """
    x = _f64(x)
    h = x + multi_head_attention(layer_norm(x, p["ln1_g"], p["ln1_b"], eps),
                                 p, cu_seqlens, n_heads, kv_out, n_kv_heads, head_dim)
    return h + feed_forward(layer_norm(h + _f64(y), p["ln2_g"], p["ln2_b"], eps), p)


def kraken_prefill(X, cu_seqlens: Sequence[int], layers: Iterable[Sequence[Mapping]],
                   W_concat, n_heads: int, eps: float = LN_EPS, return_kv: bool = False,
                   n_kv_heads: int | None = None, head_dim: int | None = None):
    """Forward pass of a stack of Kraken layers followed by ``W_concat``.

    ``X`` is the shared first-layer input ``[T, d]`` (Section 3.1: one set of
    embeddings feeds every first-layer sub-layer).  ``layers`` yields, per layer,
    a sequence of N parameter mappings (one per sub-layer); it may be a lazy
    iterable so that large stacks are materialised one layer at a time.

    Per layer j: ``y = X`` if j is the first layer (Algorithm 1's comment), else
    ``y = sum_k x_k`` over the N outputs of the previous layer (Section 3.1,
    element-wise addition); then every sub-layer runs Algorithm 1.

    Returns ``(out, sub_out)``: ``sub_out[i]`` is sub-layer i's output after the
    last layer (``[N, T, d]``) and ``out = [Y_1 | ... | Y_N] @ W_concat``
    (``[T, d]``; Section 3.1, final combine).  With ``return_kv``, also the key
    and value projections of every layer and sub-layer, ``kv[j][i] = (K, V)``
    (``[T, dkv]`` each): what a decode step attends to.  ``n_kv_heads``: key/value
    heads per sub-layer (grouped-query attention; default ``n_heads``).
    """
    X = _f64(X)
    xs = None
    kv = []
    for j, layer in enumerate(layers):
        n_sub = len(layer)
        if j == 0:
            xs = [X] * n_sub
            y = X
        else:
            if len(xs) != n_sub:
                raise ValueError("every layer must have the same number of sub-layers")
            y = np.sum(xs, axis=0)
        kv_j = []
        xs = [sub_layer_forward(xs[i], y, layer[i], cu_seqlens, n_heads, eps,
                                kv_j if return_kv else None, n_kv_heads, head_dim)
              for i in range(n_sub)]
        kv.append(kv_j)
    if xs is None:
        raise ValueError("at least one layer is required")
    Y = np.concatenate(xs, axis=1)          # [T, N*d]
    out = Y @ _f64(W_concat)
    if return_kv:
        return out, np.stack(xs), kv
    return out, np.stack(xs)


def cached_attention(q, k_new, v_new, K_cache, V_cache, n_heads: int,
                     n_kv_heads: int | None = None) -> np.ndarray:
    """Attention of one new token per sequence over its cached keys and its own.

    ``q`` is ``[B, d]`` and ``k_new, v_new`` are ``[B, dkv]`` (row b: the new token
    of sequence b); ``K_cache[b], V_cache[b]`` are ``[S_b, dkv]`` (the earlier
    tokens, ``S_b >= 0``).  Row b attends to the ``S_b + 1`` keys
    ``[K_cache[b]; k_new[b]]`` with the scaled dot-product softmax of Section 2.1
    (no mask is needed: every cached token precedes the new one); head ``h`` uses
    key/value head ``h // (n_heads / n_kv_heads)``.  Returns ``[B, d]``, heads
    concatenated.
    """
    q, k_new, v_new = _f64(q), _f64(k_new), _f64(v_new)
    B, d = q.shape
    hd = d // n_heads
    group = n_heads // (n_kv_heads or n_heads)
    dkv = k_new.shape[1]
    out = np.zeros((B, d), dtype=np.float64)
    for b in range(B):
        Kb = np.concatenate([_f64(K_cache[b]).reshape(-1, dkv), k_new[b:b + 1]], axis=0)
        Vb = np.concatenate([_f64(V_cache[b]).reshape(-1, dkv), v_new[b:b + 1]], axis=0)
        for h in range(n_heads):
            cols = slice(h * hd, (h + 1) * hd)
            kv = slice((h // group) * hd, (h // group + 1) * hd)
            scores = Kb[:, kv] @ q[b, cols] / math.sqrt(hd)
            scores -= scores.max()
            p = np.exp(scores)
            out[b, cols] = (p / p.sum()) @ Vb[:, kv]
    return out


def kraken_decode(X_new, kv_cache, layers: Iterable[Sequence[Mapping]], W_concat,
                  n_heads: int, eps: float = LN_EPS, n_kv_heads: int | None = None):
    """One decode step: the next token of each of B sequences through the stack.

    ``X_new`` is ``[B, d]`` (row b: the new token of sequence b; its first-layer
    input, shared by the N sub-layers as in the prefill).  ``kv_cache[j][i] =
    (K, V)`` where ``K[b], V[b]`` are the ``[S_b, d]`` keys and values of sequence
    b's earlier tokens at layer j, sub-layer i (``[S_b, dkv]`` with grouped-query
    attention).  Each layer runs Algorithm 1 on the new rows (combine ``y`` as in the
    prefill: ``X_new`` at the first layer, else the sum of the N previous outputs),
    the attention being ``cached_attention``.

    Returns ``(out [B, d], sub_out [N, B, d], kv_new)`` with ``kv_new[j][i] = (k, v)``,
    the new tokens' keys and values (``[B, dkv]`` each), which a following step appends.
    """
    X = _f64(X_new)
    xs = None
    kv_new = []
    for j, layer in enumerate(layers):
        n_sub = len(layer)
        y = X if j == 0 else np.sum(xs, axis=0)
        if j == 0:
            xs = [X] * n_sub
        nxt, kv_j = [], []
        for i in range(n_sub):
            p = layer[i]
            x = xs[i]
            d = x.shape[1]
            dkv = d // n_heads * (n_kv_heads or n_heads)
            u = layer_norm(x, p["ln1_g"], p["ln1_b"], eps)
            qkv = u @ _f64(p["Wqkv"]) + _f64(p["bqkv"])
            q, k, v = qkv[:, :d], qkv[:, d:d + dkv], qkv[:, d + dkv:]
            kv_j.append((k, v))
            K_c, V_c = kv_cache[j][i]
            a = cached_attention(q, k, v, K_c, V_c, n_heads, n_kv_heads)
            h = x + a @ _f64(p["Wo"]) + _f64(p["bo"])
            nxt.append(h + feed_forward(layer_norm(h + y, p["ln2_g"], p["ln2_b"], eps), p))
        xs = nxt
        kv_new.append(kv_j)
    if xs is None:
        raise ValueError("at least one layer is required")
    out = np.concatenate(xs, axis=1) @ _f64(W_concat)
    return out, np.stack(xs), kv_new


def split_kv(kv, cu_seqlens: Sequence[int]):
    """Per-sequence view of a prefill's keys and values: ``kv[j][i] = (K, V)`` with
    ``K, V [T, d]`` -> ``(K_list, V_list)`` with one ``[S_b, d]`` block per sequence."""
    out = []
    for kv_j in kv:
        row = []
        for K, V in kv_j:
            row.append(([K[cu_seqlens[b]:cu_seqlens[b + 1]] for b in range(len(cu_seqlens) - 1)],
                        [V[cu_seqlens[b]:cu_seqlens[b + 1]] for b in range(len(cu_seqlens) - 1)]))
        out.append(row)
    return out


# ------------------------------------------------------------------ the whole model
#
# Section 2.1 (background): a decoder-only model turns the tokens into embeddings that
# carry each token and its position, runs the layer stack, and feeds the last layer's
# activations to the unembedding, which gives the next-token logits.  Section 3.1: a
# Kraken model keeps one set of token and position embeddings, shared by all first-layer
# sub-layers (for compatibility with weight tying), and its W_concat output is the
# unembedding's input.  Section 4.3 compares Kraken with two other architectures built
# at the same sizes: the standard GPT-like model (Section 2.1: sequential pre-LN
# attention and FFN blocks) and the parallel attention + FFN layer of GPT-J and PaLM
# (the FFN runs beside the attention instead of after it).
#
# Readings: positions count from 0 inside each packed sequence; a final LayerNorm
# (weights lnf_g, lnf_b) precedes the unembedding, as in the GPT-2 models the paper's
# training code builds on; the unembedding is tied to the token embedding (logits =
# LN_f(h) @ tok_emb^T); the parallel layer has one LayerNorm whose output feeds both
# branches, x + MHA(LN(x)) + FFN(LN(x)) (the PaLM formulation); the standard layer is
# h = x + MHA(LN1(x)), x' = h + FFN(LN2(h)).

ARCHS = ("kraken", "gpt", "parallel")


def embed(token_ids, cu_seqlens: Sequence[int], tok_emb, pos_emb) -> np.ndarray:
    """First-layer input: ``tok_emb[id] + pos_emb[position]``, the position of token t of
    packed sequence b being ``t - cu[b]`` (Section 2.1; Section 3.1 shares this one input
    across the first layer's sub-layers)."""
    ids = np.asarray(token_ids, dtype=np.int64)
    tok, pos = _f64(tok_emb), _f64(pos_emb)
    X = np.empty((len(ids), tok.shape[1]), dtype=np.float64)
    for b in range(len(cu_seqlens) - 1):
        s0, s1 = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        X[s0:s1] = tok[ids[s0:s1]] + pos[:s1 - s0]
    return X


def gpt_block_forward(x, p: Mapping, cu_seqlens, n_heads: int, eps: float = LN_EPS,
                      head_dim: int | None = None) -> np.ndarray:
    """Standard pre-LN layer (Section 2.1): ``h = x + MHA(LN1(x))``, returns
    ``h + FFN(LN2(h))``."""
    x = _f64(x)
    h = x + multi_head_attention(layer_norm(x, p["ln1_g"], p["ln1_b"], eps), p, cu_seqlens,
                                 n_heads, head_dim=head_dim)
    return h + feed_forward(layer_norm(h, p["ln2_g"], p["ln2_b"], eps), p)


def parallel_block_forward(x, p: Mapping, cu_seqlens, n_heads: int, eps: float = LN_EPS,
                           head_dim: int | None = None) -> np.ndarray:
    """Parallel attention + FFN layer (Section 4.3, the GPT-J / PaLM comparison): one
    LayerNorm ``u = LN(x)`` (weights ln1_g, ln1_b) feeds both branches; returns
    ``x + MHA(u) + FFN(u)``."""
    x = _f64(x)
    u = layer_norm(x, p["ln1_g"], p["ln1_b"], eps)
    return x + multi_head_attention(u, p, cu_seqlens, n_heads, head_dim=head_dim) + \
        feed_forward(u, p)


def stack_forward(X, cu_seqlens: Sequence[int], arch: str,
                  layers: Iterable[Sequence[Mapping]], n_heads: int, W_concat=None,
                  eps: float = LN_EPS, head_dim: int | None = None,
                  n_kv_heads: int | None = None) -> np.ndarray:
    """The layer stack on first-layer rows ``X``: for "kraken" the Kraken layers and
    W_concat (``kraken_prefill``'s ``out``); for "gpt" / "parallel" the standard or the
    parallel layers (one parameter mapping per layer) in sequence, returning the last
    layer's output."""
    if arch not in ARCHS:
        raise ValueError(f"unknown architecture {arch!r}")
    if arch == "kraken":
        out, _ = kraken_prefill(X, cu_seqlens, layers, W_concat, n_heads, eps,
                                n_kv_heads=n_kv_heads, head_dim=head_dim)
        return out
    block = gpt_block_forward if arch == "gpt" else parallel_block_forward
    hidden = _f64(X)
    for layer in layers:
        (p,) = layer
        hidden = block(hidden, p, cu_seqlens, n_heads, eps, head_dim)
    return hidden


def unembed(h, lnf_g, lnf_b, tok_emb, eps: float = LN_EPS) -> np.ndarray:
    """Next-token logits of the rows of ``h``: ``LN_f(h) @ tok_emb^T`` (tied weights)."""
    return layer_norm(h, lnf_g, lnf_b, eps) @ _f64(tok_emb).T


def model_forward(token_ids, cu_seqlens: Sequence[int], arch: str,
                  layers: Iterable[Sequence[Mapping]], emb: Mapping, n_heads: int,
                  W_concat=None, eps: float = LN_EPS, head_dim: int | None = None,
                  n_kv_heads: int | None = None):
    """The whole model on packed token sequences.

    ``emb`` holds ``tok_emb [V, d]``, ``pos_emb [P, d]``, ``lnf_g``, ``lnf_b``.
    ``arch`` "kraken": the Kraken stack (``layers`` yields N sub-layer mappings per layer)
    and W_concat; "gpt" / "parallel": one mapping per layer, the standard or parallel
    layer, no W_concat.  Returns ``(logits, hidden)``: the logits ``[num_seqs, V]`` of the
    last token of every sequence (the first generated token's distribution, what the
    time to first token measures) and the unembedding's input ``hidden [T, d]``.
    """
    X = embed(token_ids, cu_seqlens, emb["tok_emb"], emb["pos_emb"])
    hidden = stack_forward(X, cu_seqlens, arch, layers, n_heads, W_concat, eps, head_dim,
                           n_kv_heads)
    last = [int(c) - 1 for c in cu_seqlens[1:]]
    return unembed(hidden[last], emb["lnf_g"], emb["lnf_b"], emb["tok_emb"], eps), hidden


def kraken_param_count(n_sub: int, n_layers: int, d: int, d_ff: int,
                       vocab: int = 0, biases: bool = True, layer_norms: bool = True,
                       w_concat: bool = True, positions: int = 0,
                       kv_width: int | None = None) -> int:
    """Number of parameters of a Kraken model.

    Per sub-layer: QKV (3d^2) + output projection (d^2) + FFN (2 d d_ff), plus
    optional biases (3d + d + d_ff + d) and two LayerNorms (4d) -- Section 3.2's
    closed form counts only the matrices.  ``W_concat`` adds N d^2 (Section 3.1),
    token and position embeddings add ``(vocab + positions) * d``.  With grouped-query
    attention the key and value projections are ``kv_width`` (= n_kv_heads * hd)
    wide instead of d: QKV is ``d (d + 2 kv_width)`` and its bias ``d + 2 kv_width``.
    """
    dkv = d if kv_width is None else kv_width
    per_sub = d * (d + 2 * dkv) + d * d + 2 * d * d_ff
    if biases:
        per_sub += (d + 2 * dkv) + d + d_ff + d
    if layer_norms:
        per_sub += 4 * d
    total = n_layers * n_sub * per_sub
    if w_concat:
        total += n_sub * d * d
    total += (vocab + positions) * d
    return total
