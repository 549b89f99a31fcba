"""Throughput benchmark of the Kraken prefill on one MI355X.

One step = one kraken_prefill over the whole stack (L layers x N sub-layers, then
W_concat) for one batch of synthetic input already resident in HBM.  Prints one
JSON line: tokens/s and TTFT, the whole-path MFMA utilisation, a roofline entry for
the dominant kernel (algorithmic FLOPs per launch over its average launch duration,
from HIP events recorded around every launch on the prefill's stream during the
timed steps), and the fp64 oracle timed on a bounded sample on the host.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--compute f16|bf16] [--no-cpu-baseline]
       python bench.py --pmc-probe      (one prefill + one 1 GiB device copy, untimed:
                                          the command the HBM counter runs profile)
       python bench.py --phase decode [--batch B] [--context C]
                                        (one decode step of B sequences of C cached
                                          tokens each: decode tokens/s and an HBM
                                          roofline of its dominant kernel)
       python bench.py --graph          (the timed steps replay the prefill captured
                                          once as a HIP graph)
       python bench.py --share G        (one GPU's part of a G-way split: N/G
                                          sub-layers per layer, no exchange)
       python bench.py --engine MODEL --arch ARCH --ctx C
                                        (the paper's TTFT engines, Section 4.3: the whole
                                          model, tokens to the first token's logits, for
                                          MODEL in 1.3b 6.7b 13b 65b 175b and ARCH in gpt
                                          parallel kraken4 kraken8; one C-token prompt)
"""

import argparse
import dataclasses
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MFMA_PEAK_TFLOPS = {"f16": 2500.0, "bf16": 2500.0, "f32": 157.3}   # MI355X dense
COPY_PROBE_BYTES = 1 << 30

# HBM bytes per launch of the dominant kernel, from two rocprofv3 --pmc runs of
# `python bench.py --pmc-probe` (FETCH_SIZE, then WRITE_SIZE), each scaled by what the
# same counter reads for the probe's 1 GiB device copy.  Valid only for the kernel source
# they were taken on; bench.py reports null once that file changes.
TRAFFIC = {
    "attention": {
        "source": "paper_2408_07802_amd/csrc/attention.hip",
        "source_sha256": "d36a3271213cc855a692f8cbe52ca89e197b506421157266e20b90d46b78bc18",
        "read_bytes": 3262133080, "write_bytes": 269231327,
        "algorithmic_bytes": 4 * 8 * 8192 * 2048 * 2,
        "profile": "profiles/hbm_traffic_n8_l24_d2048_t8192.md",
    },
    # FFN up projection with the GELU epilogue (A: LN2 output, B: W1, C: the activation)
    "gemm_up": {
        "source": "paper_2408_07802_amd/csrc/gemm.hip",
        "source_sha256": "e3b5be6adeb3c4bc7aa9a2404ce5950c6ec763f2b666b5b3039215acb20837bb",
        "read_bytes": 3224425359, "write_bytes": 1074040672,
        "algorithmic_bytes": 2 * (8 * 8192 * 2048 * 2 + 8 * 8192 * 8192) + 8 * 8192 * 4,
        "profile": "profiles/hbm_traffic_n8_l24_d2048_t8192.md",
    },
    # decode step, one sequence of 8192 cached tokens: the attention class is the split-key
    # kernel plus its chunk merge
    "decode_attention_b1_ctx8192": {
        "source": "paper_2408_07802_amd/csrc/decode.hip",
        "source_sha256": "df9a080c2d386a595471223a32068cc34f39fdf729f5379a6d1d5b8a6b132629",
        "read_bytes": 537726597, "write_bytes": 450560,
        "algorithmic_bytes": 537034752,
        "profile": "profiles/hbm_traffic_decode_n8_l24_d2048_ctx8192.md",
    },
}
METRIC = "prefill tokens/s + TTFT ms (all N sub-layers, 1 MI355X); MFMA util %"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def cpu_baseline(w, T, seed=0):
    """The oracle on one sub-layer of one layer at the full sequence length.

    All N x L sub-layers of a stack cost the same, so the stack's oracle time is the
    sample's time x N x L (W_concat, 0.3% of the work, is left out of the sample).
    """
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    from oracle import kraken_oracle as O
    from paper_2408_07802_amd import synth

    p = {k: v.double().numpy() for k, v in synth.gen_sub_layer(w, 1, 0, seed, "cpu").items()}
    x = synth.gen_hidden(w, T, seed, "cpu").double().numpy()
    y = x * float(w.n_sub)          # any combine input: the cost does not depend on it
    cu = [0, T]
    t0 = time.perf_counter()
    O.sub_layer_forward(x, y, p, cu, w.n_heads, n_kv_heads=w.kv_heads)
    dt = time.perf_counter() - t0
    stack_s = dt * w.n_sub * w.n_layers
    blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = max([i.get("num_threads", 1) for i in blas] or [1])
    return {"value": T / stack_s, "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"1 of {w.n_sub} sub-layers x 1 of {w.n_layers} layers at the full "
                      f"{T}-token length ({dt:.1f} s, fp64 numpy), extrapolated x"
                      f"{w.n_sub * w.n_layers}",
            "blas": [{"library": i.get("internal_api"), "version": i.get("version"),
                      "threads": i.get("num_threads"), "arch": i.get("architecture")}
                     for i in blas],
            "host_cpus": len(os.sched_getaffinity(0))}


def step_stats(per_step_ms):
    """TTFT statistics over the timed steps (HIP event pairs around each step)."""
    v = sorted(per_step_ms)
    n = len(v)
    return {"median": v[n // 2] if n % 2 else 0.5 * (v[n // 2 - 1] + v[n // 2]),
            "min": v[0], "p90": v[min(n - 1, int(math.ceil(0.9 * n)) - 1)], "max": v[-1]}


def traffic_of(kernel):
    """Measured HBM traffic of `kernel` per launch: (read + write bytes, detail), or
    (None, None) when no counter run exists for the current source of the kernel."""
    t = TRAFFIC.get(kernel)
    if not t:
        return None, None
    with open(os.path.join(ROOT, t["source"]), "rb") as f:
        if hashlib.sha256(f.read()).hexdigest() != t["source_sha256"]:
            return None, None
    return t["read_bytes"] + t["write_bytes"], {
        "unit": "bytes/launch", "read": t["read_bytes"], "write": t["write_bytes"],
        "algorithmic": t["algorithmic_bytes"], "profile": t["profile"]}


HBM_PEAK_GBS = 8000.0   # MI355X HBM3E


def copy_probe(dev):
    """One device copy of COPY_PROBE_BYTES: the calibration of the HBM byte counters."""
    import torch
    src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()


def decode_class_bytes(w, es, B, ctx):
    """Algorithmic HBM bytes of one decode step per kernel class: every weight matrix
    read once in the operand type (es bytes), each sequence's cached keys and values
    of ctx + 1 positions read once, the new keys and values written once, fp32
    activations of the B rows read and written once per kernel."""
    N, L, d, F, dkv = w.n_sub, w.n_layers, w.d_model, w.d_ff, w.kv_width
    act = lambda cols: B * cols * 4
    return {
        "ln1": L * (act(N * d) + B * N * d * es),
        "gemm_qk": L * N * ((d + dkv) * d * es + B * d * es + B * (d + dkv) * es),
        "gemm_vt": L * N * (dkv * d * es + B * d * es + B * dkv * es),
        "kv_cache": L * N * B * 2 * dkv * es * 2,
        "attention": L * N * (B * (ctx + 1) * 2 * dkv * es + B * (d + dkv) * es + B * d * es),
        "gemm_o": L * N * (d * d * es + B * d * es + 2 * act(d)),
        "combine_ln2": L * (2 * N * act(d) + N * B * d * es),
        "gemm_up": L * N * (F * d * es + B * d * es + B * F * es),
        "gemm_down": L * N * (d * F * es + B * F * es + 2 * act(d)),
        "w_concat": N * d * d * es + 2 * N * act(d) + act(d),
    }


def bench_decode(args, w, compute):
    """One decode step of B sequences, each with `context` cached tokens (stand-in
    values ~ N(0, 1) in the cache; the step's cost does not depend on them)."""
    import torch

    from paper_2408_07802_amd import kraken, synth

    B, ctx = args.batch, args.context
    dev = "cuda:0"
    torch.cuda.set_device(0)
    cfg = kraken.Config(n_sub=w.n_sub, n_layers=w.n_layers, d_model=w.d_model,
                        n_heads=w.n_heads, d_ff=w.d_ff, max_tokens=max(B, 8192), dtype=w.dtype,
                        compute=w.compute, n_kv_heads=w.n_kv_heads)
    log(f"[bench decode] {w.name} B={B} context={ctx} compute={compute}")
    model = kraken.Kraken(cfg)
    blob = kraken.pack_weights((synth.gen_layer(w, j, 0, dev) for j in range(w.n_layers)),
                               synth.gen_w_concat(w, 0, dev), cfg, device=dev)
    model.load_weights(blob)
    torch.cuda.synchronize()
    del blob
    torch.cuda.empty_cache()
    log("[bench decode] weights loaded; filling the cache")
    cache = model.new_kv_cache(B, ctx + 1)
    flat = cache.buf.view(synth.compute_dtype(w))
    g = torch.Generator(device=dev)
    g.manual_seed(1234)
    step = 1 << 28
    for o in range(0, flat.numel(), step):
        flat[o:o + step].normal_(generator=g)
    torch.cuda.synchronize()
    log(f"[bench decode] cache of {cache.buf.numel()} bytes filled")
    X = synth.gen_hidden(w, B, 0, dev)
    out = torch.empty((B, w.d_model), dtype=torch.float32, device=dev)
    lens = [ctx] * B
    if args.pmc_probe:
        model.decode(X, lens, cache, out=out)
        torch.cuda.synchronize()
        copy_probe(dev)
        log(f"[bench decode] probe done: 1 decode step, then a {COPY_PROBE_BYTES}-byte copy")
        model.close()
        return
    for _ in range(args.warmup):
        model.decode(X, lens, cache, out=out)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        model.decode(X, lens, cache, out=out)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_per_step = ev0.elapsed_time(ev1) / args.steps
    log(f"[bench decode] {args.steps} steps: {ms_per_step:.3f} ms/step")

    model.profile_reset()
    model.profile_enable(True)
    for _ in range(args.steps):
        model.decode(X, lens, cache, out=out)
    torch.cuda.synchronize()
    prof = model.profile_read()
    model.profile_enable(False)
    model.close()

    es = 4 if compute == "f32" else 2
    cb = decode_class_bytes(w, es, B, ctx)
    kernels = {}
    for name, (ms, n) in prof.items():
        if n == 0:
            continue
        by = cb.get(name)
        per_launch = by / (n / args.steps) if by else None
        kernels[name] = {"ms_per_step": ms / args.steps, "launches_per_step": n // args.steps,
                         "avg_launch_ms": ms / n,
                         "gbs": per_launch / (ms / n * 1e-3) / 1e9 if by else None}
    dominant = max((k for k in kernels if kernels[k]["gbs"] is not None),
                   key=lambda k: kernels[k]["ms_per_step"])
    dk = kernels[dominant]
    total_bytes = sum(cb.values())
    result = {
        "metric": "decode tokens/s (one new token per sequence, all N sub-layers, 1 MI355X)",
        "value": B / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": compute,
        "data": "synthetic",
        "config": {"workload": w.name + "-decode", "batch": B, "context": ctx,
                   "n_sub": w.n_sub, "n_layers": w.n_layers, "d_model": w.d_model,
                   "n_heads": w.n_heads, "n_kv_heads": w.kv_heads, "d_ff": w.d_ff,
                   "storage_dtype": w.dtype, "mfma_operands": compute,
                   "kv_cache_bytes": cache.buf.numel()},
        "hbm_bytes_per_step": total_bytes,
        "hbm_util_pct": 100.0 * total_bytes / (ms_per_step * 1e-3) / (HBM_PEAK_GBS * 1e9),
        "roofline": {"bound": "hbm", "kernel": dominant, "achieved": dk["gbs"],
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": dk["gbs"] / HBM_PEAK_GBS,
                     "traffic": traffic_of(f"decode_{dominant}_b{B}_ctx{ctx}")[0],
                     "traffic_detail": traffic_of(f"decode_{dominant}_b{B}_ctx{ctx}")[1],
                     "avg_launch_ms": dk["avg_launch_ms"],
                     "launches_per_step": dk["launches_per_step"]},
        "kernels": kernels,
        "wall_ms_per_step": wall / args.steps * 1e3,
    }
    print(json.dumps(result), flush=True)


def bench_engine(args):
    """The whole model of one of the paper's TTFT engines (Section 4.3): token ids of one
    prompt in, the first generated token's logits out (embeddings, every layer, W_concat
    for Kraken, final LayerNorm, unembedding over 51,200 tokens), fp16, random weights."""
    import torch

    from paper_2408_07802_amd import kraken, synth

    w = synth.engine_workload(args.engine, args.arch, args.ctx)
    if args.layers:
        w = dataclasses.replace(w, n_layers=args.layers, name=f"{w.name}-l{args.layers}")
    dev = "cuda:0"
    torch.cuda.set_device(0)
    cfg = kraken.Config(n_sub=w.n_sub, n_layers=w.n_layers, d_model=w.d_model,
                        n_heads=w.n_heads, d_ff=w.d_ff, max_tokens=args.ctx, dtype=w.dtype,
                        compute=w.compute, arch=w.arch, head_dim=w.head_size, vocab=w.vocab,
                        max_positions=w.max_positions)
    log(f"[bench engine] {w.name}: N={w.n_sub} L={w.n_layers} d={w.d_model} H={w.n_heads} "
        f"hd={w.head_dim} F={w.d_ff} V={w.vocab}")
    model = kraken.Kraken(cfg)
    blob = kraken.pack_weights((synth.gen_layer(w, j, 0, dev) for j in range(w.n_layers)),
                               synth.gen_w_concat(w, 0, dev) if w.arch == "kraken" else None,
                               cfg, device=dev, embeddings=synth.gen_embeddings(w, 0, dev))
    model.load_weights(blob)
    torch.cuda.synchronize()
    del blob
    torch.cuda.empty_cache()
    ids = synth.gen_tokens(w, args.ctx, 0)
    cu = [0, args.ctx]
    logits = torch.empty((1, w.vocab), dtype=torch.float32, device=dev)
    for _ in range(args.warmup):
        model.forward_tokens(ids, cu, logits=logits)
    model.sync()
    stream = torch.cuda.current_stream()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(stream)
    for k in range(args.steps):
        model.forward_tokens(ids, cu, logits=logits)
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    model.sync()
    per = [evs[k].elapsed_time(evs[k + 1]) for k in range(args.steps)]
    flops = sum(kraken.class_flops(cfg, k, cu) for k in range(kraken.K_COUNT))
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    model.close()
    print(json.dumps({
        "metric": "TTFT ms (whole model, one prompt, 1 MI355X)", "value": ms, "unit": "ms",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "ttft_ms_stats": step_stats(per), "higher_is_better": False, "scaling": "strong",
        "vs_baseline": None, "dtype": w.compute if w.compute != "storage" else w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "engine": args.engine, "arch": args.arch, "ctx": args.ctx,
                   "n_sub": w.n_sub, "n_layers": w.n_layers, "d_model": w.d_model,
                   "n_heads": w.n_heads, "head_dim": w.head_dim, "d_ff": w.d_ff,
                   "vocab": w.vocab},
        "mfma_util_pct": 100.0 * flops / (ms * 1e-3) / (MFMA_PEAK_TFLOPS["f16"] * 1e12),
        "algorithmic_tflop_per_step": flops / 1e12}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--compute", default=None, help="MFMA operand type (default: workload's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pmc-probe", action="store_true",
                    help="one prefill (decode step with --phase decode) and one 1 GiB "
                         "device copy, untimed (for HBM counters)")
    ap.add_argument("--phase", choices=["prefill", "decode"], default="prefill")
    ap.add_argument("--batch", type=int, default=1, help="decode: sequences per step")
    ap.add_argument("--context", type=int, default=8192, help="decode: cached tokens each")
    ap.add_argument("--share", type=int, default=1,
                    help="run one GPU's share of a G-way split: N/G sub-layers per layer")
    ap.add_argument("--engine", default=None, help="a TTFT engine of the paper's table")
    ap.add_argument("--arch", default="kraken4", help="with --engine: gpt, parallel, kraken4, "
                                                      "kraken8")
    ap.add_argument("--ctx", type=int, default=2048, help="with --engine: prompt length")
    ap.add_argument("--layers", type=int, default=0, help="with --engine: layer count "
                                                          "(0: the engine's)")
    ap.add_argument("--graph", action="store_true",
                    help="time the prefill as one captured HIP graph (replayed per step)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(over G GPUs each would own N/G complete sub-layer chains, with one all-reduce "
              "of the partial N-way sum per layer)",
              file=sys.stderr)
        sys.exit(2)

    if args.engine:
        bench_engine(args)
        return

    import torch

    from paper_2408_07802_amd import kraken, synth

    w = synth.workload(args.workload or synth.BENCH_WORKLOAD)
    if args.compute:
        w = dataclasses.replace(w, compute=args.compute)
    if args.share > 1:
        # one GPU's part of a G-way Kraken (Section 3.1: the N sub-layers split over G
        # devices): N/G sub-layers at the full depth, width and length.  The exchange of the
        # per-layer partial sums is not run, so each layer's combine sums the local
        # sub-layers only; the arithmetic per GPU is the sharded model's.
        if w.n_sub % args.share:
            raise SystemExit(f"--share {args.share} does not divide N = {w.n_sub}")
        w = dataclasses.replace(w, name=f"{w.name}-share1of{args.share}",
                                n_sub=w.n_sub // args.share)
    compute = w.dtype if w.compute == "storage" else w.compute
    if args.phase == "decode":
        bench_decode(args, w, compute)
        return
    lens = synth.seq_lens(w)
    cu = synth.cu_seqlens(lens)
    T = cu[-1]
    dev = "cuda:0"
    torch.cuda.set_device(0)

    cfg = kraken.Config(n_sub=w.n_sub, n_layers=w.n_layers, d_model=w.d_model,
                        n_heads=w.n_heads, d_ff=w.d_ff, max_tokens=T, dtype=w.dtype,
                        compute=w.compute, n_kv_heads=w.n_kv_heads)
    log(f"[bench] workload {w.name} T={T} compute={compute}: generating weights on device")
    model = kraken.Kraken(cfg)
    blob = kraken.pack_weights((synth.gen_layer(w, j, 0, dev) for j in range(w.n_layers)),
                               synth.gen_w_concat(w, 0, dev), cfg, device=dev)
    model.load_weights(blob)
    torch.cuda.synchronize()
    del blob
    torch.cuda.empty_cache()
    X = synth.gen_hidden(w, T, 0, dev)
    out = torch.empty((T, w.d_model), dtype=torch.float32, device=dev)
    log("[bench] weights loaded; warming up")
    if args.pmc_probe:
        model.prefill(X, cu, out=out)
        torch.cuda.synchronize()
        copy_probe(dev)
        log(f"[bench] probe done: 1 prefill, then a {COPY_PROBE_BYTES}-byte device copy")
        model.close()
        return

    for _ in range(args.warmup):
        model.prefill(X, cu, out=out)
    torch.cuda.synchronize()
    step = lambda: model.prefill(X, cu, out=out)
    if args.graph:
        # the whole prefill recorded once as a HIP graph (on a side stream, as capture
        # requires) and replayed per step on the current stream: the same kernels and
        # arguments, without the host's per-launch cost
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.graph(graph, stream=side):
            model.prefill(X, cu, out=out)
        torch.cuda.synchronize()
        step = graph.replay
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()

    # ---- timed region: K steps, no instrumentation (an event between steps: the per-step
    # TTFT distribution; events on the prefill's stream cost nothing measurable)
    stream = torch.cuda.current_stream()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    ev0, ev1 = evs[0], evs[-1]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(stream)
    for k in range(args.steps):
        step()
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_per_step = ev0.elapsed_time(ev1) / args.steps
    ttft = step_stats([evs[k].elapsed_time(evs[k + 1]) for k in range(args.steps)])
    log(f"[bench] {args.steps} steps: {ms_per_step:.3f} ms/step (wall {wall / args.steps * 1e3:.3f})")

    # ---- per-kernel durations: the same K steps with HIP events around every launch
    model.profile_reset()
    model.profile_enable(True)
    ev0.record(stream)
    for _ in range(args.steps):
        model.prefill(X, cu, out=out)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_instr = ev0.elapsed_time(ev1) / args.steps
    prof = model.profile_read()
    model.profile_enable(False)

    peak = MFMA_PEAK_TFLOPS[compute]
    total_flops = sum(kraken.class_flops(cfg, k, cu) for k in range(kraken.K_COUNT))
    kernels = {}
    for k, name in enumerate(kraken.KERNEL_CLASS_NAMES):
        ms, n = prof[name]
        if n == 0:
            continue
        fl = kraken.class_flops(cfg, k, cu)
        per_launch = fl / (n / args.steps) if fl else 0.0
        avg_ms = ms / n
        kernels[name] = {"ms_per_step": ms / args.steps, "launches_per_step": n // args.steps,
                         "avg_launch_ms": avg_ms,
                         "tflops": (per_launch / (avg_ms * 1e-3) / 1e12) if fl else None}
    dominant = max((k for k in kernels if kernels[k]["tflops"] is not None),
                   key=lambda k: kernels[k]["ms_per_step"])
    dk = kernels[dominant]
    gemm_names = ["gemm_qk", "gemm_vt", "gemm_o", "gemm_up", "gemm_down", "w_concat"]
    gemm_ms = sum(kernels[k]["ms_per_step"] for k in gemm_names if k in kernels)
    gemm_fl = sum(kraken.class_flops(cfg, kraken.KERNEL_CLASS_NAMES.index(k), cu)
                  for k in gemm_names)
    attn_ms = kernels["attention"]["ms_per_step"]
    attn_fl = kraken.class_flops(cfg, kraken.K_ATTN, cu)

    result = {
        "metric": METRIC,
        "value": T / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ttft_ms": ms_per_step,
        "ttft_ms_stats": ttft,
        "higher_is_better": True,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": compute,
        "data": "synthetic",
        "config": {"workload": w.name, "n_sub": w.n_sub, "n_layers": w.n_layers,
                   "d_model": w.d_model, "n_heads": w.n_heads, "n_kv_heads": w.kv_heads,
                   "d_ff": w.d_ff, "seq_lens": lens, "tokens": T, "storage_dtype": w.dtype,
                   "mfma_operands": compute, "accumulate": "f32",
                   "launch": "hip_graph" if args.graph else "stream"},
        "mfma_util_pct": 100.0 * total_flops / (ms_per_step * 1e-3) / (peak * 1e12),
        "phase_mfma_util_pct": {
            "gemm": 100.0 * gemm_fl / (gemm_ms * 1e-3) / (peak * 1e12),
            "attention": 100.0 * attn_fl / (attn_ms * 1e-3) / (peak * 1e12)},
        "algorithmic_tflop_per_step": total_flops / 1e12,
        "roofline": {"bound": "mfma", "kernel": dominant,
                     "achieved": dk["tflops"], "peak": peak, "unit": "TFLOP/s",
                     "frac": dk["tflops"] / peak, "traffic": traffic_of(dominant)[0],
                     "traffic_detail": traffic_of(dominant)[1],
                     "avg_launch_ms": dk["avg_launch_ms"],
                     "launches_per_step": dk["launches_per_step"]},
        "kernels": kernels,
        "instrumented_ms_per_step": ms_instr,
        "wall_ms_per_step": wall / args.steps * 1e3,
    }
    model.close()
    del X, out
    torch.cuda.empty_cache()

    if not args.no_cpu_baseline:
        log("[bench] timing the oracle on its sample")
        result["cpu_baseline"] = cpu_baseline(w, T)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
