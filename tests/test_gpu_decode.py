"""KV-cache prefill and one-token decode (kraken_prefill_kv, kraken_decode) against the
fp64 oracle, through the C ABI.

Section 2.1 (KV cache): a decode step of a token at position p of a sequence equals row
p of a prefill of the sequence extended by that token; the oracle's ``kraken_decode``
is pinned to exactly that on the CPU.  Here:
  * prefill_kv returns kraken_prefill's outputs bit for bit, and its cache holds the
    oracle's keys and values of every (layer, sub-layer, sequence, position), while
    slots and positions past the sequences keep what they held;
  * decode steps after prefill_kv match the oracle's decode over the oracle's cache,
    and append the oracle's new keys and values at position lens[b];
  * decode over stand-in caches (seeded values written into the cache) of several
    thousand keys, where the key range is split into chunks, matches the oracle;
  * decode over an empty cache is a one-token prefill.
Metric and bound as for the prefill: max |gpu - oracle| / RMS(oracle), 2e-2 for 16-bit
operands and 1e-4 for fp32.
"""

import numpy as np
import pytest
import torch

from oracle import kraken_oracle as O
from paper_2408_07802_amd import synth
from test_gpu_prefill import DEV, TOL, build_model, f64, oracle_layers, rel_err, say, small

pytestmark = pytest.mark.gpu

SENTINEL = 7.0


def K():
    from paper_2408_07802_amd import kraken
    return kraken


def tol(w):
    return TOL["f32"] if synth.compute_dtype(w) == torch.float32 else TOL["bf16"]


def cache_rows(cv, j, i, kv, b, n):
    """Rows 0..n-1 of slot b ([n, d]) from a cache view [L, N, 2, S, H, cap, hd]."""
    t = cv[j, i, kv, b, :, :n, :]           # [H, n, hd]
    return t.permute(1, 0, 2).reshape(n, -1)


def write_cache_rows(cv, j, i, kv, b, rows):
    n = rows.shape[0]
    H, hd = cv.shape[4], cv.shape[6]
    cv[j, i, kv, b, :, :n, :] = rows.view(n, H, hd).permute(1, 0, 2)


def wconcat(w, seed=0):
    return f64(synth.gen_w_concat(w, seed, DEV))


def check(name, got, ref, bound):
    e = rel_err(f64(got), ref)
    say(f"    {name}: max|err|/rms {e:.3e} (bound {bound})")
    assert e <= bound, (name, e)


def prefill_then_decode(w, lens, steps=2, seed=0, affine="random", capacity=None):
    cu = synth.cu_seqlens(lens)
    T, B = cu[-1], len(lens)
    cap = capacity or max(lens) + steps + 3
    say(f"[decode parity] {w.name} compute={w.compute} lens={lens} steps={steps} cap={cap}")
    model = build_model(w, T, seed, affine)
    max_seqs = min(B + 1, K().MAX_SEQS)        # one unused slot when there is room
    cache = model.new_kv_cache(max_seqs, cap)
    cache.buf.view(synth.compute_dtype(w)).fill_(SENTINEL)
    cv = cache.view(model.cfg)
    X = synth.gen_hidden(w, T, seed, DEV)
    out_p, sub_p = model.prefill(X, cu, sub_out=True)
    model.poison_workspace()           # no stale value of the plain prefill may be read
    out, sub = model.prefill_kv(X, cu, cache, sub_out=True)
    model.sync()
    assert torch.equal(out, out_p) and torch.equal(sub, sub_p), "prefill_kv != prefill"

    layers = [list(l) for l in oracle_layers(w, seed, affine)]
    out_o, _, kv = O.kraken_prefill(f64(X), cu, layers, wconcat(w, seed), w.n_heads,
                                    return_kv=True, n_kv_heads=w.kv_heads)
    check("prefill out", out, out_o, tol(w))
    bound = tol(w)
    for j in range(w.n_layers):
        for i in range(w.n_sub):
            for b in range(B):
                for kvi in range(2):
                    ref = kv[j][i][kvi][cu[b]:cu[b + 1]]
                    e = rel_err(f64(cache_rows(cv, j, i, kvi, b, lens[b])), ref)
                    assert e <= bound, ("cache", j, i, b, kvi, e)
                # positions past the sequence are untouched
                assert bool((cv[j, i, :, b, :, lens[b]:, :] == SENTINEL).all())
    if max_seqs > B:
        assert bool((cv[:, :, :, B] == SENTINEL).all()), "an unused slot was written"

    cache_o = O.split_kv(kv, cu)
    cur = list(lens)
    for step in range(steps):
        Xn = synth.gen_hidden(w, B, seed + 1 + step, DEV)
        model.poison_workspace()
        out_d, sub_d = model.decode(Xn, cur, cache, sub_out=True)
        model.sync()
        out_do, sub_do, kv_new = O.kraken_decode(f64(Xn), cache_o, layers, wconcat(w, seed),
                                                 w.n_heads, n_kv_heads=w.kv_heads)
        check(f"step {step} out", out_d, out_do, bound)
        check(f"step {step} sub_out", sub_d, sub_do, bound)
        for j in range(w.n_layers):
            for i in range(w.n_sub):
                k_new, v_new = kv_new[j][i]
                for b in range(B):
                    for kvi, ref in ((0, k_new[b]), (1, v_new[b])):
                        got = f64(cv[j, i, kvi, b, :, cur[b], :].reshape(-1))
                        e = rel_err(got, ref)
                        assert e <= bound, ("appended", step, j, i, b, kvi, e)
                    cache_o[j][i][0][b] = np.vstack([cache_o[j][i][0][b], k_new[b:b + 1]])
                    cache_o[j][i][1][b] = np.vstack([cache_o[j][i][1][b], v_new[b:b + 1]])
        cur = [c + 1 for c in cur]
    model.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_prefill_kv_then_two_decode_steps_head32(dtype):
    w = small("kv-n2-l2-d128-h4", dtype=dtype)
    prefill_then_decode(w, [5, 70, 33])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_prefill_kv_then_decode_head64_head128(dtype):
    w = small("kv-n3-l2-d256-h4", n_sub=3, d_model=256, n_heads=4, d_ff=512, dtype=dtype)
    prefill_then_decode(w, [1, 130, 300], steps=1)
    w = small("kv-n2-l2-d256-h2", n_sub=2, d_model=256, n_heads=2, d_ff=512, dtype=dtype)
    prefill_then_decode(w, [257, 2], steps=2)


def test_prefill_kv_then_decode_fp16_operands():
    w = small("kv-n4-l2-d128-h2-f16", n_sub=4, d_model=128, n_heads=2, d_ff=256, dtype="bf16",
              compute="f16")
    prefill_then_decode(w, [40, 9, 100, 1], steps=2)


@pytest.mark.parametrize("B,dtype", [(70, "bf16"), (256, "f32")])
def test_decode_large_batches(B, dtype):
    # 70 rows: the projections leave the few-row GEMM for the tiled one; 256: the most
    # sequences one call takes
    rng = np.random.default_rng(B)
    lens = [int(v) for v in rng.integers(1, 13 if B < 100 else 6, size=B)]
    w = small(f"dec-batch{B}-n2-l2-d128-h4", dtype=dtype)
    prefill_then_decode(w, lens, steps=1)


def decode_over_standin_cache(w, lens, decode_tokens, seed=3, k_std=4.0):
    """Decode with a model sized for `decode_tokens` rows (so the attention partials must
    share a small workspace) over seeded stand-in caches of lens[b] tokens."""
    B = len(lens)
    cap = max(lens) + 1
    say(f"[decode stand-in cache] {w.name} compute={w.compute} lens={lens} cap={cap}")
    model = build_model(w, decode_tokens, seed, "random")
    cache = model.new_kv_cache(B, cap)
    cv = cache.view(model.cfg)
    cache_o = []
    for j in range(w.n_layers):
        row = []
        for i in range(w.n_sub):
            Ks, Vs = [], []
            for b in range(B):
                Kb, Vb = synth.gen_cached_kv(w, lens[b], j, i, b, seed, k_std=k_std, device=DEV)
                if lens[b]:
                    write_cache_rows(cv, j, i, 0, b, Kb)
                    write_cache_rows(cv, j, i, 1, b, Vb)
                Ks.append(f64(Kb))
                Vs.append(f64(Vb))
            row.append((Ks, Vs))
        cache_o.append(row)
    Xn = synth.gen_hidden(w, B, seed + 1, DEV)
    out, sub = model.decode(Xn, lens, cache, sub_out=True)
    torch.cuda.synchronize()
    model.close()
    layers = [list(l) for l in oracle_layers(w, seed, "random")]
    out_o, sub_o, _ = O.kraken_decode(f64(Xn), cache_o, layers, wconcat(w, seed), w.n_heads,
                                      n_kv_heads=w.kv_heads)
    check("out", out, out_o, tol(w))
    check("sub_out", sub, sub_o, tol(w))


@pytest.mark.parametrize("compute", ["storage", "f16"])
def test_decode_long_standin_cache_chunk_split(compute):
    # head size 128; the one-row workspace holds 32 chunk partials, so 9000 keys take
    # 512-key chunks
    w = small("dec-n2-l1-d256-h2", n_sub=2, n_layers=1, d_model=256, n_heads=2, d_ff=512,
              dtype="bf16", compute=compute, out_proj_std=0.1)
    decode_over_standin_cache(w, [9000], decode_tokens=1)


def test_decode_standin_cache_ragged_batch():
    # chunks past the end of the shorter sequences, an empty cache among them
    w = small("dec-n2-l2-d256-h4", n_sub=2, n_layers=2, d_model=256, n_heads=4, d_ff=512,
              dtype="bf16", out_proj_std=0.1)
    decode_over_standin_cache(w, [9000, 0, 300], decode_tokens=3)
    w = small("dec-n2-l1-d128-h4-f32", n_sub=2, n_layers=1, d_model=128, n_heads=4, d_ff=256,
              dtype="f32", out_proj_std=0.1)
    decode_over_standin_cache(w, [1, 511, 512, 513, 2048], decode_tokens=5)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decode_over_empty_cache_is_one_token_prefill(dtype):
    w = small("dec0-n2-l2-d128-h4", dtype=dtype)
    B = 3
    model = build_model(w, B, 0, "random")
    cache = model.new_kv_cache(B, 4)
    Xn = synth.gen_hidden(w, B, 5, DEV)
    out, sub = model.decode(Xn, [0] * B, cache, sub_out=True)
    out_p, sub_p = model.prefill(Xn, list(range(B + 1)), sub_out=True)
    torch.cuda.synchronize()
    model.close()
    layers = [list(l) for l in oracle_layers(w, 0, "random")]
    out_o, sub_o = O.kraken_prefill(f64(Xn), list(range(B + 1)), layers, wconcat(w), w.n_heads)
    check("decode out", out, out_o, tol(w))
    check("decode sub_out", sub, sub_o, tol(w))
    check("prefill out", out_p, out_o, tol(w))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("H,Hkv,d", [(4, 2, 256), (4, 1, 256), (16, 2, 512), (16, 4, 512),
                                     (6, 2, 384)])
def test_grouped_query_prefill_kv_then_decode(dtype, H, Hkv, d):
    # decode workgroups serve 4, 2 or 1 query heads of a key/value group (groups of 2, 4,
    # 8 and 3 heads here); the cache holds Hkv heads
    w = small(f"gqa-kv-n2-l2-d{d}-h{H}-kv{Hkv}", n_sub=2, d_model=d, n_heads=H, d_ff=2 * d,
              dtype=dtype, n_kv_heads=Hkv)
    prefill_then_decode(w, [3, 70, 33], steps=2)


@pytest.mark.parametrize("H,Hkv", [(16, 4), (16, 1)])
def test_grouped_query_decode_long_standin_cache(H, Hkv):
    w = small(f"gqa-dec-n2-l1-d2048-h{H}-kv{Hkv}", n_sub=2, n_layers=1, d_model=2048,
              n_heads=H, d_ff=2048, dtype="bf16", compute="f16", out_proj_std=0.05,
              n_kv_heads=Hkv)
    decode_over_standin_cache(w, [5000, 1], decode_tokens=2)


def test_decode_and_prefill_kv_argument_errors():
    w = small("err-n2-l1-d128-h4", n_layers=1, dtype="bf16")
    model = build_model(w, 8, 0, "plain")
    cache = model.new_kv_cache(2, 4)
    X = synth.gen_hidden(w, 8, 0, DEV)
    kr = K()

    def status(fn):
        with pytest.raises(kr.KrakenError) as ei:
            fn()
        return ei.value.status

    # lens at capacity, negative, more sequences than slots
    assert status(lambda: model.decode(X[:2], [4, 0], cache)) == kr.ERR_INVALID_ARG
    assert status(lambda: model.decode(X[:2], [-1, 0], cache)) == kr.ERR_INVALID_ARG
    assert status(lambda: model.decode(X[:3], [0, 0, 0], cache)) == kr.ERR_INVALID_ARG
    # a sequence longer than the capacity; more sequences than slots
    assert status(lambda: model.prefill_kv(X, [0, 5, 8], cache)) == kr.ERR_INVALID_ARG
    assert status(lambda: model.prefill_kv(X[:6], [0, 2, 4, 6], cache)) == kr.ERR_INVALID_ARG
    # a misaligned cache (large enough, 8 bytes off the 16-byte alignment)
    roomy = model.new_kv_cache(2, 5)
    bad = kr.KVCache(roomy.buf[8:], cache.max_seqs, cache.capacity)
    assert status(lambda: model.decode(X[:2], [0, 0], bad)) == kr.ERR_INVALID_ARG
    # a cache buffer shorter than its max_seqs and capacity need: refused by the binding
    short = kr.KVCache(cache.buf[:-16], cache.max_seqs, cache.capacity)
    with pytest.raises(ValueError, match="cache holds"):
        model.decode(X[:2], [0, 0], short)
    # input and output buffers of the wrong type, size or device: refused by the binding
    with pytest.raises(ValueError, match="dtype"):
        model.decode(X[:2].float(), [0, 0], cache)
    with pytest.raises(ValueError, match="GPU tensor"):
        model.prefill(X.cpu(), [0, 8])
    with pytest.raises(ValueError, match="elements"):
        model.prefill(X, [0, 4])
    with pytest.raises(ValueError, match="elements"):
        model.prefill(X, [0, 8], out=torch.empty((4, w.d_model), device=DEV))
    # the cache overlapping an output
    out = cache.buf.view(torch.float32)[: 2 * w.d_model].view(2, w.d_model)
    assert status(lambda: model.decode(X[:2], [0, 0], cache, out=out)) == kr.ERR_INVALID_ARG
    model.close()


# -------------------------------------- the benchmark model (N=8, L=24, d=2048), 8192 tokens

class _StandinCache:
    """Oracle view of a stand-in cache: ``[j][i] -> (K list, V list)``, generated on
    demand one (layer, sub-layer) at a time, so that the fp64 copy of a full-depth
    8192-token cache never has to be held at once."""

    def __init__(self, w, lens, seed, k_std):
        self.w, self.lens, self.seed, self.k_std = w, lens, seed, k_std

    def __getitem__(self, j):
        outer = self

        class _Row:
            def __getitem__(self, i):
                Ks, Vs = [], []
                for b, n in enumerate(outer.lens):
                    Kb, Vb = synth.gen_cached_kv(outer.w, n, j, i, b, outer.seed,
                                                 k_std=outer.k_std, device=DEV)
                    Ks.append(f64(Kb))
                    Vs.append(f64(Vb))
                return Ks, Vs
        return _Row()


def test_bench_model_decode_over_8192_token_standin_cache():
    # the step a decode benchmark times: one new token after 8192 cached ones, the model
    # sized for the 8192-token prefill (so the attention splits into 256-key chunks)
    w = synth.workload(synth.BENCH_WORKLOAD)
    lens, seed = [8192], 11
    say(f"[decode full size] {w.name} lens={lens}")
    model = build_model(w, 8192, seed, "plain")
    cache = model.new_kv_cache(1, 8193)
    cv = cache.view(model.cfg)
    for j in range(w.n_layers):
        for i in range(w.n_sub):
            Kb, Vb = synth.gen_cached_kv(w, lens[0], j, i, 0, seed, k_std=2.0, device=DEV)
            write_cache_rows(cv, j, i, 0, 0, Kb)
            write_cache_rows(cv, j, i, 1, 0, Vb)
    Xn = synth.gen_hidden(w, 1, seed + 1, DEV)
    out, sub = model.decode(Xn, lens, cache, sub_out=True)
    torch.cuda.synchronize()
    model.close()
    del cache, cv
    out_o, sub_o, _ = O.kraken_decode(f64(Xn), _StandinCache(w, lens, seed, 2.0),
                                      oracle_layers(w, seed, "plain"), wconcat(w, seed),
                                      w.n_heads)
    check("out", out, out_o, TOL["bf16"])
    check("sub_out", sub, sub_o, TOL["bf16"])


def test_bench_model_prefill_kv_then_decode_equals_prefill_row():
    # Section 2.1: the decode of token 8191 after a cached prefill of tokens 0..8190 is
    # row 8191 of the 8192-token prefill; the cache's first rows match the oracle's
    w = synth.workload(synth.BENCH_WORKLOAD)
    T, P = 8192, 64
    say(f"[prefill_kv + decode full size] {w.name} T={T} oracle prefix {P}")
    model = build_model(w, T, 0, "plain")
    X = synth.gen_hidden(w, T, 0, DEV)
    out_full, sub_full = model.prefill(X, [0, T], sub_out=True)
    cache = model.new_kv_cache(1, T)
    model.prefill_kv(X[:T - 1], [0, T - 1], cache)
    out_d, sub_d = model.decode(X[T - 1:], [T - 1], cache, sub_out=True)
    torch.cuda.synchronize()
    check("decode vs prefill row out", out_d[0], f64(out_full[T - 1]), TOL["bf16"])
    check("decode vs prefill row sub_out", sub_d[:, 0], f64(sub_full[:, T - 1]), TOL["bf16"])
    cv = cache.view(model.cfg)
    _, _, kv = O.kraken_prefill(f64(X[:P]), [0, P], oracle_layers(w, 0, "plain"),
                                wconcat(w), w.n_heads, return_kv=True)
    worst = 0.0
    for j in range(w.n_layers):
        for i in range(w.n_sub):
            for kvi in range(2):
                e = rel_err(f64(cache_rows(cv, j, i, kvi, 0, P)), kv[j][i][kvi])
                worst = max(worst, e)
    say(f"    cache rows 0..{P - 1} vs oracle: max|err|/rms {worst:.3e}")
    assert worst <= TOL["bf16"]
    model.close()
