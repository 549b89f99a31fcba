"""The allocation-free decode attention, kraken_op_decode_attention_noalloc, against the
entry point it varies, kraken_op_decode_attention.

Given a work buffer of KRAKEN_NOALLOC_SCRATCH_FLOATS floats the existing entry point
splits the keys exactly as the static scratch does, so the two must agree bit for bit.
Two calls in a row, the second smaller (the scratch keeps the first call's partials),
each also checked against the oracle's cached attention under the kernel's elementwise
bound."""

import numpy as np
import pytest
import torch

from oracle import kraken_oracle as O

pytestmark = pytest.mark.gpu

DEV = "cuda"


def K():
    from paper_2408_07802_amd import kraken
    return kraken


def f64(t):
    return t.detach().double().cpu().numpy()


def make_inputs(n, d, H, Hkv, lens, max_seqs, cap, dt, seed):
    hd, B = d // H, len(lens)
    dkv = Hkv * hd
    g = torch.Generator(device="cpu").manual_seed(seed)
    qk = (torch.randn((n, B, d + dkv), generator=g) * 2.0).to(dt)
    cache = torch.zeros((n, 2, max_seqs, Hkv, cap, hd), dtype=dt)
    rows = []
    for i in range(n):
        per = []
        for b in range(B):
            k = (torch.randn((lens[b] + 1, dkv), generator=g) * 2.0).to(dt)
            v = torch.randn((lens[b] + 1, dkv), generator=g).to(dt)
            cache[i, 0, b, :, :lens[b] + 1] = k.view(-1, Hkv, hd).transpose(0, 1)
            cache[i, 1, b, :, :lens[b] + 1] = v.view(-1, Hkv, hd).transpose(0, 1)
            per.append((f64(k), f64(v)))
        rows.append(per)
    return qk, cache, rows


def check_oracle(out, qk, rows, n, d, H, Hkv, dtype):
    q64 = f64(qk)
    u = {torch.bfloat16: 2.0 ** -8, torch.float16: 2.0 ** -11, torch.float32: 0.0}[dtype]
    for i in range(n):
        B = len(rows[i])
        k_new = np.stack([rows[i][b][0][-1] for b in range(B)])
        v_new = np.stack([rows[i][b][1][-1] for b in range(B)])
        K_c = [rows[i][b][0][:-1] for b in range(B)]
        V_c = [rows[i][b][1][:-1] for b in range(B)]
        ref = O.cached_attention(q64[i][:, :d], k_new, v_new, K_c, V_c, H, Hkv)
        wabs = O.cached_attention(q64[i][:, :d], k_new, np.abs(v_new), K_c,
                                  [np.abs(x) for x in V_c], H, Hkv)
        bound = u * np.abs(ref) + 2.0 ** -16 * wabs + 1e-6 * np.sqrt(np.mean(ref ** 2))
        got = f64(out[i])
        assert np.all(np.isfinite(got))
        assert np.all(np.abs(got - ref) <= bound), (i, float(np.max(np.abs(got - ref) - bound)))


@pytest.mark.parametrize("dtype", [torch.float16, torch.float32])
def test_noalloc_decode_attention_matches_the_work_buffer_entry_point(dtype):
    calls = [  # (n, d, H, Hkv, lens, max_seqs, capacity): the second call is smaller
        (2, 256, 2, 2, [5000, 17, 0, 900], 4, 5001),
        (1, 128, 4, 2, [3, 200], 2, 300),
    ]
    work = torch.empty(K().NOALLOC_SCRATCH_FLOATS, dtype=torch.float32, device=DEV)
    for c, (n, d, H, Hkv, lens, max_seqs, cap) in enumerate(calls):
        print(f"[no-alloc decode attention] call {c}: n={n} d={d} H={H} Hkv={Hkv} lens={lens}",
              flush=True)
        qk, cache, rows = make_inputs(n, d, H, Hkv, lens, max_seqs, cap, dtype, 100 + c)
        qk, cache = qk.to(DEV), cache.to(DEV)
        B = len(lens)
        out_ref = torch.full((n, B, d), float("nan"), dtype=dtype, device=DEV)
        out = torch.full((n, B, d), float("nan"), dtype=dtype, device=DEV)
        K().op_decode_attention(qk, cache, out_ref, n, d, H, lens, max_seqs, cap, work,
                                n_kv_heads=Hkv)
        K().op_decode_attention_noalloc(qk, cache, out, n, d, H, lens, max_seqs, cap,
                                        n_kv_heads=Hkv)
        torch.cuda.synchronize()
        assert torch.equal(out, out_ref), c
        check_oracle(out, qk, rows, n, d, H, Hkv, dtype)


def test_noalloc_decode_attention_rejects_sizes_past_its_scratch():
    # 16 sub-layers x 256 sequences x 32 heads x (64 + 2) floats per key chunk > 8 Mi floats
    # (the host rejects the sizes before any launch: no buffer is read)
    n, d, H, B = 16, 2048, 32, 256
    qk = torch.zeros(16, dtype=torch.float16, device=DEV)
    with pytest.raises(K().KrakenError) as ei:
        K().op_decode_attention_noalloc(qk, qk, qk, n, d, H, [0] * B, B, 1)
    assert ei.value.status == K().ERR_UNSUPPORTED
    assert b"KRAKEN_NOALLOC_SCRATCH_FLOATS" in K().lib().kraken_last_error()
