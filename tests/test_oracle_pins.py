"""Pins of the fp64 oracle against facts the paper and the mathematics fix.

None of these tests compares the oracle with itself: each check is a brute-force
restatement on tiny inputs, a library routine (torch on the CPU, in float64), a
closed form, an invariant of the Kraken layer, or a number printed in the paper.
"""

import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import kraken_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------- helpers

def rand_params(rng, d, f, scale=0.3, affine=True, dkv=None):
    """Random fp64 sub-layer parameters (x @ W layout); K and V are dkv wide."""
    w = d + 2 * (d if dkv is None else dkv)
    p = {
        "Wqkv": rng.normal(0, scale, (d, w)), "Wo": rng.normal(0, scale, (d, d)),
        "W1": rng.normal(0, scale, (d, f)), "W2": rng.normal(0, scale, (f, d)),
    }
    if affine:
        p.update(ln1_g=1 + rng.normal(0, 0.2, d), ln1_b=rng.normal(0, 0.2, d),
                 ln2_g=1 + rng.normal(0, 0.2, d), ln2_b=rng.normal(0, 0.2, d),
                 bqkv=rng.normal(0, 0.2, w), bo=rng.normal(0, 0.2, d),
                 b1=rng.normal(0, 0.2, f), b2=rng.normal(0, 0.2, d))
    else:
        p.update(ln1_g=np.ones(d), ln1_b=np.zeros(d), ln2_g=np.ones(d), ln2_b=np.zeros(d),
                 bqkv=np.zeros(w), bo=np.zeros(d), b1=np.zeros(f), b2=np.zeros(d))
    return p


def zero_params(d, f):
    return {"Wqkv": np.zeros((d, 3 * d)), "Wo": np.zeros((d, d)), "W1": np.zeros((d, f)),
            "W2": np.zeros((f, d)), "ln1_g": np.ones(d), "ln1_b": np.zeros(d),
            "ln2_g": np.ones(d), "ln2_b": np.zeros(d), "bqkv": np.zeros(3 * d),
            "bo": np.zeros(d), "b1": np.zeros(f), "b2": np.zeros(d)}


def rel_err(a, b):
    a, b = np.asarray(a), np.asarray(b)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ------------------------------------------------------ P1: brute-force attention, S <= 8

def brute_attention(Q, K, V, cu, n_heads):
    """Explicit loops with math.exp: softmax(q.k / sqrt(hd)) v over keys t' <= t."""
    T, d = len(Q), len(Q[0])
    hd = d // n_heads
    out = [[0.0] * d for _ in range(T)]
    for b in range(len(cu) - 1):
        for h in range(n_heads):
            c0 = h * hd
            for t in range(cu[b], cu[b + 1]):
                logits = []
                for u in range(cu[b], t + 1):
                    s = 0.0
                    for c in range(hd):
                        s += Q[t][c0 + c] * K[u][c0 + c]
                    logits.append(s / math.sqrt(hd))
                mx = max(logits)
                w = [math.exp(v - mx) for v in logits]
                z = sum(w)
                for c in range(hd):
                    acc = 0.0
                    for k, u in enumerate(range(cu[b], t + 1)):
                        acc += w[k] / z * V[u][c0 + c]
                    out[t][c0 + c] = acc
    return out


@pytest.mark.parametrize("lens,n_heads,d", [([1], 1, 4), ([8], 2, 8), ([3, 5], 2, 6),
                                            ([2, 1, 4], 3, 9), ([7], 4, 8)])
def test_p1_attention_brute_force(lens, n_heads, d):
    rng = np.random.default_rng(sum(lens) * 31 + d)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(int)
    T = int(cu[-1])
    Q, K, V = (rng.normal(0, 1.5, (T, d)) for _ in range(3))
    got = O.causal_attention(Q, K, V, cu, n_heads)
    want = np.array(brute_attention(Q.tolist(), K.tolist(), V.tolist(), cu.tolist(), n_heads))
    assert rel_err(got, want) <= 1e-12


def test_p1_causality_future_perturbation():
    rng = np.random.default_rng(5)
    T, d, H = 8, 8, 2
    Q, K, V = (rng.normal(size=(T, d)) for _ in range(3))
    base = O.causal_attention(Q, K, V, [0, T], H)
    for t in range(T - 1):
        K2, V2 = K.copy(), V.copy()
        K2[t + 1:] += rng.normal(size=(T - t - 1, d)) * 10
        V2[t + 1:] -= 7.0
        pert = O.causal_attention(Q, K2, V2, [0, T], H)
        np.testing.assert_array_equal(pert[:t + 1], base[:t + 1])
        assert not np.allclose(pert[t + 1:], base[t + 1:])


# --------------------------------------------- P2: library routines (torch CPU, float64)

def test_p2_attention_matches_torch_sdpa():
    rng = np.random.default_rng(11)
    lens, H, d = [17, 5, 30], 4, 32
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    Q, K, V = (rng.normal(0, 2.0, (T, d)) for _ in range(3))
    got = O.causal_attention(Q, K, V, cu, H)
    hd = d // H
    for b in range(len(lens)):
        s0, s1 = cu[b], cu[b + 1]

        def heads(a):
            return torch.from_numpy(a[s0:s1]).reshape(s1 - s0, H, hd).transpose(0, 1)

        ref = F.scaled_dot_product_attention(heads(Q), heads(K), heads(V), is_causal=True)
        ref = ref.transpose(0, 1).reshape(s1 - s0, d).numpy()
        assert rel_err(got[s0:s1], ref) <= 1e-12


def test_p2_layer_norm_matches_torch():
    rng = np.random.default_rng(12)
    v = rng.normal(3.0, 5.0, (9, 48))
    g, b = rng.normal(1, 0.3, 48), rng.normal(0, 0.3, 48)
    ref = F.layer_norm(torch.from_numpy(v), (48,), torch.from_numpy(g), torch.from_numpy(b),
                       eps=1e-5).numpy()
    assert rel_err(O.layer_norm(v, g, b), ref) <= 1e-12
    # near-constant rows: eps matters, and it is 1e-5 on the biased variance
    v2 = 1.0 + rng.normal(0, 1e-3, (4, 48))
    ref2 = F.layer_norm(torch.from_numpy(v2), (48,), eps=1e-5).numpy()
    assert rel_err(O.layer_norm(v2, np.ones(48), np.zeros(48)), ref2) <= 1e-11


def test_p2_gelu_matches_torch_exact():
    z = np.linspace(-9, 9, 2001)
    ref = F.gelu(torch.from_numpy(z), approximate="none").numpy()
    assert np.max(np.abs(O.gelu(z) - ref)) <= 1e-15 * 10
    tanh = F.gelu(torch.from_numpy(z), approximate="tanh").numpy()
    assert np.max(np.abs(O.gelu(z) - tanh)) > 1e-4   # the tanh form is a different function


# ------------------------------------------------ P11: GELU identities and scalar erf

def test_p11_gelu_identities():
    z = np.random.default_rng(3).normal(0, 3, 1000)
    np.testing.assert_allclose(O.gelu(z) - O.gelu(-z), z, rtol=0, atol=1e-14)
    assert O.gelu(np.array([0.0]))[0] == 0.0
    for v in (-4.0, -2.7, -1.0, -0.1, 0.3, 1.0, 2.5, 6.0):
        want = 0.5 * v * (1 + math.erf(v / math.sqrt(2)))
        assert abs(O.gelu(np.array([v]))[0] - want) <= 1e-15 * max(1, abs(v))


# ------------------------------------- P3: N = 1 restated as a GPT-2 block (torch, fp64)

def torch_block(x, p, cu, n_heads, ln2_extra):
    """GPT-2 pre-LN block from torch primitives, FFN LayerNorm reading h + ln2_extra."""
    t = {k: torch.from_numpy(np.asarray(v, dtype=np.float64)) for k, v in p.items()}
    x = torch.from_numpy(np.asarray(x, dtype=np.float64))
    T, d = x.shape
    hd = d // n_heads
    a = F.layer_norm(x, (d,), t["ln1_g"], t["ln1_b"], eps=1e-5)
    qkv = F.linear(a, t["Wqkv"].T, t["bqkv"])
    q, k, v = qkv.split(d, dim=1)
    o = torch.empty_like(q)
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])

        def heads(m):
            return m[s0:s1].reshape(s1 - s0, n_heads, hd).transpose(0, 1)

        att = F.scaled_dot_product_attention(heads(q), heads(k), heads(v), is_causal=True)
        o[s0:s1] = att.transpose(0, 1).reshape(s1 - s0, d)
    h = x + F.linear(o, t["Wo"].T, t["bo"])
    extra = torch.from_numpy(np.asarray(ln2_extra, dtype=np.float64))
    z = F.layer_norm(h + extra, (d,), t["ln2_g"], t["ln2_b"], eps=1e-5)
    m = F.linear(F.gelu(F.linear(z, t["W1"].T, t["b1"])), t["W2"].T, t["b2"])
    return (h + m).numpy()


@pytest.mark.parametrize("n_layers", [1, 3])
def test_p3_single_sub_layer_is_gpt2_block_with_h_plus_x(n_layers):
    rng = np.random.default_rng(100 + n_layers)
    d, f, H, cu = 16, 40, 4, [0, 9, 20]
    X = rng.normal(size=(cu[-1], d))
    layers = [[rand_params(rng, d, f)] for _ in range(n_layers)]
    Wc = rng.normal(0, 0.3, (d, d))
    out, sub = O.kraken_prefill(X, cu, layers, Wc, H)
    x = X
    for j in range(n_layers):
        x = torch_block(x, layers[j][0], cu, H, ln2_extra=x)
    assert rel_err(sub[0], x) <= 1e-12
    assert rel_err(out, x @ Wc) <= 1e-12
    # the companion: a vanilla GPT-2 block (no combine term) is a different function
    xv = X
    for j in range(n_layers):
        xv = torch_block(xv, layers[j][0], cu, H, ln2_extra=np.zeros_like(xv))
    assert rel_err(sub[0], xv) > 1e-3


# ------------------------------------------ P4: layer-1 independence of sub-layers

def test_p4_first_layer_sub_layers_are_independent():
    rng = np.random.default_rng(7)
    d, f, H, N, cu = 12, 24, 3, 3, [0, 11]
    X = rng.normal(size=(11, d))
    layer = [rand_params(rng, d, f) for _ in range(N)]
    Wc = rng.normal(0, 0.3, (N * d, d))
    out, sub = O.kraken_prefill(X, cu, [layer], Wc, H)
    want_out = np.zeros_like(out)
    for i in range(N):
        yi = torch_block(X, layer[i], cu, H, ln2_extra=X)
        assert rel_err(sub[i], yi) <= 1e-12
        want_out += yi @ Wc[i * d:(i + 1) * d]     # row block i of W_concat multiplies Y_i
    assert rel_err(out, want_out) <= 1e-12


# ---------------------------------------------------- P5: sub-layer permutation

def test_p5_permuting_sub_layers_with_w_concat_blocks():
    rng = np.random.default_rng(8)
    d, f, H, N, L, cu = 8, 16, 2, 4, 3, [0, 6, 13]
    X = rng.normal(size=(13, d))
    layers = [[rand_params(rng, d, f) for _ in range(N)] for _ in range(L)]
    Wc = rng.normal(0, 0.3, (N * d, d))
    out, sub = O.kraken_prefill(X, cu, layers, Wc, H)
    perm = [2, 0, 3, 1]
    layers_p = [[layer[k] for k in perm] for layer in layers]
    Wc_p = np.concatenate([Wc[k * d:(k + 1) * d] for k in perm])
    out_p, sub_p = O.kraken_prefill(X, cu, layers_p, Wc_p, H)
    assert rel_err(out_p, out) <= 1e-13
    for new, old in enumerate(perm):
        assert rel_err(sub_p[new], sub[old]) <= 1e-13


# -------------------------------------------- P6: causal prefix, P7: packing

def test_p6_causal_prefix():
    rng = np.random.default_rng(9)
    d, f, H, N, L, S = 8, 16, 2, 2, 3, 15
    X = rng.normal(size=(S, d))
    layers = [[rand_params(rng, d, f) for _ in range(N)] for _ in range(L)]
    Wc = rng.normal(0, 0.3, (N * d, d))
    out, sub = O.kraken_prefill(X, [0, S], layers, Wc, H)
    for Sp in (1, 2, 7, 14):
        out_p, sub_p = O.kraken_prefill(X[:Sp], [0, Sp], layers, Wc, H)
        assert rel_err(out_p, out[:Sp]) <= 1e-12
        assert rel_err(sub_p, sub[:, :Sp]) <= 1e-12


def test_p7_packing_equals_separate_runs():
    rng = np.random.default_rng(10)
    d, f, H, N, L = 8, 16, 2, 3, 2
    lens = [5, 1, 9]
    cu = np.concatenate([[0], np.cumsum(lens)])
    X = rng.normal(size=(cu[-1], d))
    layers = [[rand_params(rng, d, f) for _ in range(N)] for _ in range(L)]
    Wc = rng.normal(0, 0.3, (N * d, d))
    out, sub = O.kraken_prefill(X, cu, layers, Wc, H)
    for b in range(len(lens)):
        s0, s1 = cu[b], cu[b + 1]
        out_b, sub_b = O.kraken_prefill(X[s0:s1], [0, s1 - s0], layers, Wc, H)
        assert rel_err(out_b, out[s0:s1]) <= 1e-12
        assert rel_err(sub_b, sub[:, s0:s1]) <= 1e-12


# ------------------------------------------ P8: zero model, P9: constant V, P10: S=1

def test_p8_zero_model_closed_form():
    rng = np.random.default_rng(13)
    d, f, H, N, L = 8, 32, 2, 3, 4
    X = rng.normal(size=(10, d))
    layers = [[zero_params(d, f) for _ in range(N)] for _ in range(L)]
    Wc = rng.normal(0, 0.3, (N * d, d))
    out, sub = O.kraken_prefill(X, [0, 4, 10], layers, Wc, H)
    for i in range(N):
        np.testing.assert_array_equal(sub[i], X)
    Wsum = sum(Wc[i * d:(i + 1) * d] for i in range(N))
    assert rel_err(out, X @ Wsum) <= 1e-13


def test_p9_constant_values_give_constant_attention():
    rng = np.random.default_rng(14)
    d, H, T = 12, 3, 9
    p = rand_params(rng, d, 4)
    p["Wqkv"][:, 2 * d:] = 0.0                      # V columns of the projection are zero
    c = rng.normal(size=d)
    p["bqkv"][2 * d:] = c                           # so every V row is the bias c
    p["Wo"] = np.eye(d)
    p["bo"] = np.zeros(d)
    u = rng.normal(size=(T, d))
    got = O.multi_head_attention(u, p, [0, 2, 9], H)
    np.testing.assert_allclose(got, np.broadcast_to(c, (T, d)), rtol=0, atol=1e-14)


def test_p10_single_token_attention_returns_v():
    rng = np.random.default_rng(15)
    Q, K, V = (rng.normal(size=(3, 8)) for _ in range(3))
    got = O.causal_attention(Q, K, V, [0, 1, 2, 3], 2)       # three sequences of length 1
    np.testing.assert_allclose(got, V, rtol=0, atol=1e-15)


# ------------------------------------------- P12: zero sub-layer pins the N-way sum

def test_p12_zero_sub_layer_pins_the_sum():
    rng = np.random.default_rng(16)
    d, f, H, L, cu = 8, 24, 2, 4, [0, 7, 12]
    X = rng.normal(size=(12, d))
    live = [rand_params(rng, d, f) for _ in range(L)]
    layers = [[live[j], zero_params(d, f)] for j in range(L)]
    Wc = rng.normal(0, 0.3, (2 * d, d))
    out, sub = O.kraken_prefill(X, cu, layers, Wc, H)
    np.testing.assert_array_equal(sub[1], X)
    x1 = X
    for j in range(L):
        y = X if j == 0 else x1 + X            # first layer: identity; then x_1 + x_2 = x_1 + X
        x1 = torch_block(x1, live[j], cu, H, ln2_extra=y)
    assert rel_err(sub[0], x1) <= 1e-12
    assert rel_err(out, x1 @ Wc[:d] + X @ Wc[d:]) <= 1e-12


# ----------------------------------- brute force of the whole stack on tiny inputs

def _ln_py(v, g, b):
    mu = sum(v) / len(v)
    var = sum((a - mu) ** 2 for a in v) / len(v)
    return [g[c] * (v[c] - mu) / math.sqrt(var + 1e-5) + b[c] for c in range(len(v))]


def _vecmat(v, W, bias):
    return [sum(v[k] * W[k][c] for k in range(len(v))) + bias[c] for c in range(len(W[0]))]


def _sub_layer_py(x, y, p, cu, H):
    d = len(x[0])
    pl = {k: np.asarray(v).tolist() for k, v in p.items()}
    qkv = [_vecmat(_ln_py(row, pl["ln1_g"], pl["ln1_b"]), pl["Wqkv"], pl["bqkv"]) for row in x]
    att = brute_attention([r[:d] for r in qkv], [r[d:2 * d] for r in qkv],
                          [r[2 * d:] for r in qkv], cu, H)
    h = [[x[t][c] + v for c, v in enumerate(_vecmat(att[t], pl["Wo"], pl["bo"]))]
         for t in range(len(x))]
    out = []
    for t in range(len(x)):
        z = _ln_py([h[t][c] + y[t][c] for c in range(d)], pl["ln2_g"], pl["ln2_b"])
        g = [0.5 * a * (1 + math.erf(a / math.sqrt(2))) for a in _vecmat(z, pl["W1"], pl["b1"])]
        m = _vecmat(g, pl["W2"], pl["b2"])
        out.append([h[t][c] + m[c] for c in range(d)])
    return out


def test_whole_stack_brute_force_tiny():
    rng = np.random.default_rng(17)
    d, f, H, N, L, cu = 4, 6, 2, 3, 3, [0, 3, 5]
    X = rng.normal(size=(5, d))
    layers = [[rand_params(rng, d, f, scale=0.6) for _ in range(N)] for _ in range(L)]
    Wc = rng.normal(0, 0.5, (N * d, d))
    out, sub = O.kraken_prefill(X, cu, layers, Wc, H)
    xs = [X.tolist()] * N
    for j in range(L):
        if j == 0:
            y = X.tolist()
        else:
            y = [[sum(xs[k][t][c] for k in range(N)) for c in range(d)] for t in range(5)]
        xs = [_sub_layer_py(xs[i], y, layers[j][i], cu, H) for i in range(N)]
    Y = [[v for i in range(N) for v in xs[i][t]] for t in range(5)]
    want = [[sum(Y[t][k] * Wc[k][c] for k in range(N * d)) for c in range(d)] for t in range(5)]
    assert rel_err(sub, np.array(xs)) <= 1e-12
    assert rel_err(out, np.array(want)) <= 1e-12


# ------------------------------------- P13: parameter counts printed by the paper

def _rows(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return [ln.split() for ln in fh if ln.strip() and not ln.startswith("#")]


def test_p13_engine_per_layer_counts():
    for r in _rows("engine_model_dims.txt"):
        unit = float(r[11])
        d_std, p_std = int(r[2]), float(r[3])
        got = O.kraken_param_count(1, 1, d_std, 4 * d_std, biases=False, layer_norms=False,
                                   w_concat=False) / 1e6
        assert abs(got - p_std) <= unit, (r[0], "standard", got, p_std)
        for n_sub, dcol, pcol in ((4, 5, 6), (8, 8, 9)):
            d, printed = int(r[dcol]), float(r[pcol])
            got = O.kraken_param_count(n_sub, 1, d, 2 * d, biases=False, layer_norms=False,
                                       w_concat=False) / 1e6
            # one unit of the printed precision: 4 x 8 x 1248^2 = 49.84M is printed 49.9M
            assert abs(got - printed) <= unit, (r[0], n_sub, got, printed)


def test_p13_model_totals():
    for r in _rows("model_configurations.txt"):
        n_sub, L, d, printed = int(r[0]), int(r[1]), int(r[2]), float(r[3])
        got = O.kraken_param_count(n_sub, L, d, 2 * d, vocab=50257, positions=1024,
                                   biases=False, layer_norms=False) / 1e6
        assert abs(got - printed) <= 0.35, (r, got)
        # without W_concat the totals fall short by N d^2 (> 0.35M for every row)
        no_cat = O.kraken_param_count(n_sub, L, d, 2 * d, vocab=50257, positions=1024,
                                      biases=False, layer_norms=False, w_concat=False) / 1e6
        assert printed - no_cat > 0.35


# ---------------------------------- decode: one token past a cached prefix (Section 2.1)
#
# The decode oracle is pinned to the (already pinned) prefill oracle by causality: the
# new token's row of a prefill over the extended sequence is exactly what a decode step
# over the prefix's cached keys and values must produce, and the extended prefill's keys
# and values are the prefix's plus the decode step's.  The cached attention itself is
# checked against the explicit-loop brute force above.

def _stack(rng, n_sub, n_layers, d, f, affine=True, scale=0.3):
    return [[rand_params(rng, d, f, scale=scale, affine=affine) for _ in range(n_sub)]
            for _ in range(n_layers)]


def _decode_case(seed=5, n_sub=2, n_layers=3, d=8, f=16, H=2, lens=(5, 1, 3)):
    rng = np.random.default_rng(seed)
    layers = _stack(rng, n_sub, n_layers, d, f)
    wcat = rng.normal(0, 0.3, (n_sub * d, d))
    X_full = [rng.normal(0, 1, (S + 2, d)) for S in lens]   # prefix + two decode tokens
    return layers, wcat, X_full, H


def _prefill(seqs, layers, wcat, H):
    cu = [0]
    for s in seqs:
        cu.append(cu[-1] + len(s))
    out, sub, kv = O.kraken_prefill(np.concatenate(seqs), cu, layers, wcat, H, return_kv=True)
    return cu, out, sub, kv


def test_decode_step_equals_last_row_of_extended_prefill():
    layers, wcat, X_full, H = _decode_case()
    lens = [len(x) - 2 for x in X_full]
    cu_p, _, _, kv_p = _prefill([x[:-2] for x in X_full], layers, wcat, H)
    cu_e, out_e, sub_e, _ = _prefill([x[:-1] for x in X_full], layers, wcat, H)
    X_new = np.stack([x[-2] for x in X_full])
    out_d, sub_d, _ = O.kraken_decode(X_new, O.split_kv(kv_p, cu_p), layers, wcat, H)
    last = [cu_e[b + 1] - 1 for b in range(len(lens))]
    assert rel_err(out_d, out_e[last]) < 1e-12
    assert rel_err(sub_d, sub_e[:, last]) < 1e-12


def test_two_decode_steps_equal_extended_prefill_and_its_cache():
    layers, wcat, X_full, H = _decode_case(seed=11, lens=(4, 2))
    cu_p, _, _, kv_p = _prefill([x[:-2] for x in X_full], layers, wcat, H)
    cu_e, out_e, sub_e, kv_e = _prefill(X_full, layers, wcat, H)
    cache = O.split_kv(kv_p, cu_p)
    outs = []
    for step in (2, 1):
        X_new = np.stack([x[-step] for x in X_full])
        out_d, _, kv_new = O.kraken_decode(X_new, cache, layers, wcat, H)
        outs.append(out_d)
        # append the step's keys and values to each sequence's cache
        cache = [[([np.vstack([Kc[b], kv_new[j][i][0][b:b + 1]]) for b in range(len(Kc))],
                   [np.vstack([Vc[b], kv_new[j][i][1][b:b + 1]]) for b in range(len(Vc))])
                  for i, (Kc, Vc) in enumerate(row)] for j, row in enumerate(cache)]
    for k, step in enumerate((2, 1)):
        rows = [cu_e[b + 1] - step for b in range(len(X_full))]
        assert rel_err(outs[k], out_e[rows]) < 1e-12
    # the cache after two steps is the extended prefill's keys and values
    full = O.split_kv(kv_e, cu_e)
    for j in range(len(layers)):
        for i in range(len(layers[0])):
            for b in range(len(X_full)):
                assert rel_err(cache[j][i][0][b], full[j][i][0][b]) < 1e-12
                assert rel_err(cache[j][i][1][b], full[j][i][1][b]) < 1e-12


def test_decode_with_empty_cache_is_a_one_token_prefill():
    layers, wcat, X_full, H = _decode_case(seed=2, lens=(0, 0))
    d = X_full[0].shape[1]
    empty = [[([np.zeros((0, d))] * 2, [np.zeros((0, d))] * 2) for _ in row] for row in layers]
    X_new = np.stack([x[0] for x in X_full])
    out_d, sub_d, _ = O.kraken_decode(X_new, empty, layers, wcat, H)
    cu = [0, 1, 2]
    out_p, sub_p = O.kraken_prefill(X_new, cu, layers, wcat, H)
    assert rel_err(out_d, out_p) < 1e-12 and rel_err(sub_d, sub_p) < 1e-12


def test_cached_attention_matches_brute_force():
    rng = np.random.default_rng(7)
    d, H = 6, 3
    lens = [4, 0, 2]
    Kc = [rng.normal(0, 1, (S, d)) for S in lens]
    Vc = [rng.normal(0, 1, (S, d)) for S in lens]
    q, k, v = (rng.normal(0, 1, (len(lens), d)) for _ in range(3))
    got = O.cached_attention(q, k, v, Kc, Vc, H)
    for b, S in enumerate(lens):
        # the new token is the last of a sequence [cache; new]: brute force over it
        Q = [list(r) for r in np.vstack([np.zeros((S, d)), q[b:b + 1]])]
        K = [list(r) for r in np.vstack([Kc[b], k[b:b + 1]])]
        V = [list(r) for r in np.vstack([Vc[b], v[b:b + 1]])]
        ref = brute_attention(Q, K, V, [0, S + 1], H)[S]
        assert rel_err(got[b], ref) < 1e-12


# ------------------------------------------------ grouped-query and multi-query attention
# With Hkv key/value heads, query head h of a group of G = H / Hkv consecutive heads uses
# key/value head h // G.  That is multi-head attention whose key and value weights repeat
# each shared head's columns for every query head of its group: the pins build that
# multi-head model explicitly and compare whole stacks, prefill and decode.

def _repeat_kv_heads(p, d, H, Hkv):
    """Multi-head parameters equal to grouped-query ``p``: K/V head columns repeated."""
    hd, G = d // H, H // Hkv
    dkv = Hkv * hd
    W, bias = p["Wqkv"], p["bqkv"]
    q_w, k_w, v_w = W[:, :d], W[:, d:d + dkv], W[:, d + dkv:]
    q_b, k_b, v_b = bias[:d], bias[d:d + dkv], bias[d + dkv:]
    k_cols, v_cols, kb, vb = [], [], [], []
    for h in range(H):
        g = h // G                     # the shared head this query head reads
        k_cols.append(k_w[:, g * hd:(g + 1) * hd])
        v_cols.append(v_w[:, g * hd:(g + 1) * hd])
        kb.append(k_b[g * hd:(g + 1) * hd])
        vb.append(v_b[g * hd:(g + 1) * hd])
    out = dict(p)
    out["Wqkv"] = np.concatenate([q_w] + k_cols + v_cols, axis=1)
    out["bqkv"] = np.concatenate([q_b] + kb + vb)
    return out


@pytest.mark.parametrize("H,Hkv", [(4, 2), (4, 1), (6, 3), (6, 2)])
def test_gqa_prefill_equals_mha_with_repeated_kv_heads(H, Hkv):
    rng = np.random.default_rng(40 + H * 10 + Hkv)
    d, f, n_sub, n_layers = 12, 20, 2, 2
    hd = d // H
    layers = [[rand_params(rng, d, f, dkv=Hkv * hd) for _ in range(n_sub)]
              for _ in range(n_layers)]
    mha = [[_repeat_kv_heads(p, d, H, Hkv) for p in row] for row in layers]
    wcat = rng.normal(0, 0.3, (n_sub * d, d))
    cu = [0, 5, 6, 9]
    X = rng.normal(0, 1, (9, d))
    out_g, sub_g, kv_g = O.kraken_prefill(X, cu, layers, wcat, H, return_kv=True,
                                          n_kv_heads=Hkv)
    out_m, sub_m = O.kraken_prefill(X, cu, mha, wcat, H)
    assert rel_err(out_g, out_m) < 1e-12 and rel_err(sub_g, sub_m) < 1e-12
    assert kv_g[0][0][0].shape == (9, Hkv * hd)
    # a wrong grouping (head h reading shared head h mod Hkv) would differ
    if 1 < Hkv < H:
        wrong = O.causal_attention(X, X[:, :Hkv * hd], X[:, :Hkv * hd], cu, H, Hkv)
        alt = np.zeros_like(wrong)
        for h in range(H):
            g = h % Hkv
            alt[:, h * hd:(h + 1) * hd] = O.causal_attention(
                X[:, h * hd:(h + 1) * hd], X[:, g * hd:(g + 1) * hd],
                X[:, g * hd:(g + 1) * hd], cu, 1)
        assert rel_err(wrong, alt) > 1e-3


def brute_mqa(Q, K, V, cu, n_heads):
    """Multi-query attention with explicit loops: every head uses the single K/V head."""
    T, d = len(Q), len(Q[0])
    hd = d // n_heads
    out = [[0.0] * d for _ in range(T)]
    for b in range(len(cu) - 1):
        for h in range(n_heads):
            for t in range(cu[b], cu[b + 1]):
                logits = []
                for u in range(cu[b], t + 1):
                    s = 0.0
                    for c in range(hd):
                        s += Q[t][h * hd + c] * K[u][c]
                    logits.append(s / math.sqrt(hd))
                mx = max(logits)
                w = [math.exp(v - mx) for v in logits]
                z = sum(w)
                for c in range(hd):
                    out[t][h * hd + c] = sum(w[k] / z * V[u][c]
                                             for k, u in enumerate(range(cu[b], t + 1)))
    return out


def test_mqa_attention_brute_force():
    rng = np.random.default_rng(3)
    H, hd = 3, 2
    cu = [0, 4, 7]
    Q = rng.normal(0, 1, (7, H * hd))
    K = rng.normal(0, 1, (7, hd))
    V = rng.normal(0, 1, (7, hd))
    got = O.causal_attention(Q, K, V, cu, H, 1)
    ref = brute_mqa(Q.tolist(), K.tolist(), V.tolist(), cu, H)
    assert rel_err(got, ref) < 1e-12


@pytest.mark.parametrize("Hkv", [1, 2])
def test_gqa_decode_equals_last_row_of_extended_prefill(Hkv):
    rng = np.random.default_rng(17 + Hkv)
    d, f, H, n_sub, n_layers = 8, 16, 4, 2, 2
    layers = [[rand_params(rng, d, f, dkv=Hkv * d // H) for _ in range(n_sub)]
              for _ in range(n_layers)]
    wcat = rng.normal(0, 0.3, (n_sub * d, d))
    X_full = [rng.normal(0, 1, (S + 1, d)) for S in (3, 1, 5)]
    cu_p = [0]
    for x in X_full:
        cu_p.append(cu_p[-1] + len(x) - 1)
    _, _, kv_p = O.kraken_prefill(np.concatenate([x[:-1] for x in X_full]), cu_p, layers,
                                  wcat, H, return_kv=True, n_kv_heads=Hkv)
    cu_e = [0]
    for x in X_full:
        cu_e.append(cu_e[-1] + len(x))
    out_e, sub_e = O.kraken_prefill(np.concatenate(X_full), cu_e, layers, wcat, H,
                                    n_kv_heads=Hkv)
    X_new = np.stack([x[-1] for x in X_full])
    out_d, sub_d, kv_new = O.kraken_decode(X_new, O.split_kv(kv_p, cu_p), layers, wcat, H,
                                           n_kv_heads=Hkv)
    last = [cu_e[b + 1] - 1 for b in range(len(X_full))]
    assert rel_err(out_d, out_e[last]) < 1e-12
    assert rel_err(sub_d, sub_e[:, last]) < 1e-12
    assert kv_new[0][0][0].shape == (3, Hkv * d // H)
    # the same step through the repeated-head multi-head model
    mha = [[_repeat_kv_heads(p, d, H, Hkv) for p in row] for row in layers]
    _, _, kv_m = O.kraken_prefill(np.concatenate([x[:-1] for x in X_full]), cu_p, mha, wcat,
                                  H, return_kv=True)
    out_m, _, _ = O.kraken_decode(X_new, O.split_kv(kv_m, cu_p), mha, wcat, H)
    assert rel_err(out_d, out_m) < 1e-12


def test_gqa_parameter_count():
    # the key and value projections narrow from d to Hkv * hd columns each
    d, f, N, L, H = 2048, 8192, 8, 24, 16
    full = O.kraken_param_count(N, L, d, f)
    for Hkv in (16, 4, 1):
        dkv = Hkv * d // H
        got = O.kraken_param_count(N, L, d, f, kv_width=dkv)
        assert full - got == N * L * 2 * (d - dkv) * (d + 1)


# ------------------------------------------------------------ the whole model (NEXT-4)

def torch_mha(a, t, cu, n_heads, hd):
    """Causal multi-head attention block from torch primitives (QKV, SDPA, Wo)."""
    dq = n_heads * hd
    qkv = F.linear(a, t["Wqkv"].T, t["bqkv"])
    q, k, v = qkv[:, :dq], qkv[:, dq:2 * dq], qkv[:, 2 * dq:]
    o = torch.empty_like(q)
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])

        def heads(m):
            return m[s0:s1].reshape(s1 - s0, n_heads, hd).transpose(0, 1)

        att = F.scaled_dot_product_attention(heads(q), heads(k), heads(v), is_causal=True)
        o[s0:s1] = att.transpose(0, 1).reshape(s1 - s0, dq)
    return F.linear(o, t["Wo"].T, t["bo"])


def torch_ffn(z, t):
    return F.linear(F.gelu(F.linear(z, t["W1"].T, t["b1"])), t["W2"].T, t["b2"])


def tt(p):
    return {k: torch.from_numpy(np.asarray(v, dtype=np.float64)) for k, v in p.items()}


def torch_gpt_block(x, p, cu, n_heads, hd):
    t, d = tt(p), x.shape[1]
    h = x + torch_mha(F.layer_norm(x, (d,), t["ln1_g"], t["ln1_b"], eps=1e-5), t, cu, n_heads, hd)
    return h + torch_ffn(F.layer_norm(h, (d,), t["ln2_g"], t["ln2_b"], eps=1e-5), t)


def torch_parallel_block(x, p, cu, n_heads, hd):
    t, d = tt(p), x.shape[1]
    u = F.layer_norm(x, (d,), t["ln1_g"], t["ln1_b"], eps=1e-5)
    return x + torch_mha(u, t, cu, n_heads, hd) + torch_ffn(u, t)


def rand_params_hd(rng, d, f, n_heads, hd, scale=0.3):
    """Sub-layer parameters with an attention width n_heads * hd that may differ from d."""
    dq = n_heads * hd
    return {"Wqkv": rng.normal(0, scale, (d, 3 * dq)), "bqkv": rng.normal(0, 0.2, 3 * dq),
            "Wo": rng.normal(0, scale, (dq, d)), "bo": rng.normal(0, 0.2, d),
            "W1": rng.normal(0, scale, (d, f)), "b1": rng.normal(0, 0.2, f),
            "W2": rng.normal(0, scale, (f, d)), "b2": rng.normal(0, 0.2, d),
            "ln1_g": 1 + rng.normal(0, 0.2, d), "ln1_b": rng.normal(0, 0.2, d),
            "ln2_g": 1 + rng.normal(0, 0.2, d), "ln2_b": rng.normal(0, 0.2, d)}


def rand_emb(rng, V, P, d):
    return {"tok_emb": rng.normal(0, 1.0, (V, d)), "pos_emb": rng.normal(0, 0.5, (P, d)),
            "lnf_g": 1 + rng.normal(0, 0.2, d), "lnf_b": rng.normal(0, 0.2, d)}


def test_embed_is_token_plus_position_within_each_sequence():
    rng = np.random.default_rng(50)
    V, P, d = 11, 9, 6
    emb = rand_emb(rng, V, P, d)
    cu = [0, 4, 5, 9]
    ids = rng.integers(0, V, 9)
    X = O.embed(ids, cu, emb["tok_emb"], emb["pos_emb"])
    pos = torch.tensor([0, 1, 2, 3, 0, 0, 1, 2, 3])        # positions restart per sequence
    want = F.embedding(torch.from_numpy(ids), torch.from_numpy(emb["tok_emb"])) + \
        F.embedding(pos, torch.from_numpy(emb["pos_emb"]))
    assert rel_err(X, want.numpy()) <= 1e-15
    # one-hot form: X = onehot(ids) tok_emb + onehot(pos) pos_emb
    oh = np.eye(V)[ids] @ emb["tok_emb"] + np.eye(P)[pos.numpy()] @ emb["pos_emb"]
    assert rel_err(X, oh) <= 1e-14


@pytest.mark.parametrize("hd", [None, 5])
def test_gpt_block_is_the_vanilla_pre_ln_block(hd):
    # hd = 5 with 3 heads and d = 16: an attention width (15) that differs from d, as in a
    # GPT-3 13B layer (d = 5140, 40 heads of 128)
    rng = np.random.default_rng(51)
    d, f, H, cu = 16, 40, 3 if hd else 4, [0, 9, 20]
    hd_ = hd or d // H
    x = rng.normal(size=(cu[-1], d))
    p = rand_params_hd(rng, d, f, H, hd_)
    got = O.gpt_block_forward(x, p, cu, H, head_dim=hd)
    want = torch_gpt_block(torch.from_numpy(x), p, cu, H, hd_).numpy()
    assert rel_err(got, want) <= 1e-12
    # it is not the Kraken sub-layer with N = 1 (whose FFN LayerNorm reads h + x)
    if hd is None:
        assert rel_err(O.sub_layer_forward(x, x, p, cu, H), got) > 1e-3


def test_parallel_block_against_torch_and_its_two_reductions():
    rng = np.random.default_rng(52)
    d, f, H, cu = 16, 40, 4, [0, 7, 19]
    x = rng.normal(size=(cu[-1], d))
    p = rand_params_hd(rng, d, f, H, d // H)
    got = O.parallel_block_forward(x, p, cu, H)
    want = torch_parallel_block(torch.from_numpy(x), p, cu, H, d // H).numpy()
    assert rel_err(got, want) <= 1e-12
    # FFN off (W1, b1, W2, b2 = 0): both layer forms are x + MHA(LN1(x))
    q = dict(p, W1=np.zeros_like(p["W1"]), b1=np.zeros(f), W2=np.zeros_like(p["W2"]),
             b2=np.zeros(d))
    assert rel_err(O.parallel_block_forward(x, q, cu, H), O.gpt_block_forward(x, q, cu, H)) <= 1e-13
    # attention off (Wqkv, bqkv, bo = 0, so MHA = 0) and LN2 = LN1: both are x + FFN(LN(x))
    r = dict(p, Wqkv=np.zeros_like(p["Wqkv"]), bqkv=np.zeros_like(p["bqkv"]), bo=np.zeros(d),
             ln2_g=p["ln1_g"], ln2_b=p["ln1_b"])
    assert rel_err(O.parallel_block_forward(x, r, cu, H), O.gpt_block_forward(x, r, cu, H)) <= 1e-13
    # with both branches on, the two forms differ
    assert rel_err(got, O.gpt_block_forward(x, p, cu, H)) > 1e-3


def test_unembed_against_torch_and_loops():
    rng = np.random.default_rng(53)
    V, d = 7, 5
    emb = rand_emb(rng, V, 3, d)
    h = rng.normal(size=(3, d)) * 4 + 2
    got = O.unembed(h, emb["lnf_g"], emb["lnf_b"], emb["tok_emb"])
    t = tt(emb)
    want = F.linear(F.layer_norm(torch.from_numpy(h), (d,), t["lnf_g"], t["lnf_b"], eps=1e-5),
                    t["tok_emb"]).numpy()
    assert rel_err(got, want) <= 1e-13
    for r in range(3):          # logit v is the dot product with token v's embedding
        mu = sum(h[r]) / d
        var = sum((a - mu) ** 2 for a in h[r]) / d
        z = [emb["lnf_g"][c] * (h[r][c] - mu) / math.sqrt(var + 1e-5) + emb["lnf_b"][c]
             for c in range(d)]
        for v in range(V):
            assert abs(got[r][v] - sum(z[c] * emb["tok_emb"][v][c] for c in range(d))) <= 1e-12


def torch_model(ids, cu, arch, layers, emb, H, hd, Wc=None):
    """The whole model from torch primitives: embeddings, blocks, (W_concat), ln_f, tied
    unembedding of each sequence's last token."""
    t = tt(emb)
    pos = torch.cat([torch.arange(cu[b + 1] - cu[b]) for b in range(len(cu) - 1)])
    x = F.embedding(torch.from_numpy(np.asarray(ids)), t["tok_emb"]) + F.embedding(pos, t["pos_emb"])
    d = x.shape[1]
    if arch == "kraken":
        xs, y = [x] * len(layers[0]), x
        for j, layer in enumerate(layers):
            if j > 0:
                y = sum(xs)
            nxt = []
            for i, p in enumerate(layer):
                q = tt(p)
                h = xs[i] + torch_mha(F.layer_norm(xs[i], (d,), q["ln1_g"], q["ln1_b"], eps=1e-5),
                                      q, cu, H, hd)
                nxt.append(h + torch_ffn(F.layer_norm(h + y, (d,), q["ln2_g"], q["ln2_b"],
                                                      eps=1e-5), q))
            xs = nxt
        x = torch.cat(xs, dim=1) @ torch.from_numpy(Wc)
    else:
        blk = torch_gpt_block if arch == "gpt" else torch_parallel_block
        for (p,) in layers:
            x = blk(x, p, cu, H, hd)
    last = [c - 1 for c in cu[1:]]
    return F.linear(F.layer_norm(x[last], (d,), t["lnf_g"], t["lnf_b"], eps=1e-5),
                    t["tok_emb"]).numpy()


@pytest.mark.parametrize("arch", ["kraken", "gpt", "parallel"])
def test_model_forward_against_torch_model(arch):
    rng = np.random.default_rng(54)
    V, P, d, f, H, L = 13, 12, 12, 24, 3, 2
    N = 3 if arch == "kraken" else 1
    cu = [0, 5, 12]
    ids = rng.integers(0, V, 12)
    emb = rand_emb(rng, V, P, d)
    layers = [[rand_params_hd(rng, d, f, H, d // H) for _ in range(N)] for _ in range(L)]
    Wc = rng.normal(0, 0.3, (N * d, d)) if arch == "kraken" else None
    logits, hidden = O.model_forward(ids, cu, arch, layers, emb, H, W_concat=Wc)
    assert logits.shape == (2, V) and hidden.shape == (12, d)
    want = torch_model(ids, cu, arch, layers, emb, H, d // H, Wc)
    assert rel_err(logits, want) <= 1e-12


@pytest.mark.parametrize("arch", ["kraken", "gpt", "parallel"])
def test_model_forward_packing_equals_separate_sequences(arch):
    # positions restart in every packed sequence and attention never crosses sequences, so
    # each sequence's last-token logits equal a run of that sequence alone
    rng = np.random.default_rng(55)
    V, P, d, f, H = 9, 10, 8, 16, 2
    N = 2 if arch == "kraken" else 1
    emb = rand_emb(rng, V, P, d)
    layers = [[rand_params_hd(rng, d, f, H, d // H) for _ in range(N)] for _ in range(2)]
    Wc = rng.normal(0, 0.3, (N * d, d)) if arch == "kraken" else None
    lens = [4, 1, 7]
    ids = rng.integers(0, V, sum(lens))
    cu = [0, 4, 5, 12]
    packed, _ = O.model_forward(ids, cu, arch, layers, emb, H, W_concat=Wc)
    for b, s in enumerate(lens):
        alone, _ = O.model_forward(ids[cu[b]:cu[b + 1]], [0, s], arch, layers, emb, H, W_concat=Wc)
        assert rel_err(packed[b], alone[0]) <= 1e-12
