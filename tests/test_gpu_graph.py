"""A prefill captured as a HIP graph and replayed: every replay must give the eager call's
bits, with eager work on the stream between replays and with new input contents."""

import numpy as np
import pytest
import torch

from paper_2408_07802_amd import kraken as K, synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(msg):
    print(msg, flush=True)


def build(w, T, seed=0):
    cfg = K.Config(n_sub=w.n_sub, n_layers=w.n_layers, d_model=w.d_model, n_heads=w.n_heads,
                   d_ff=w.d_ff, max_tokens=T, dtype=w.dtype, compute=w.compute,
                   n_kv_heads=w.n_kv_heads)
    model = K.Kraken(cfg)
    model.load_weights(K.pack_weights((synth.gen_layer(w, j, seed, DEV)
                                       for j in range(w.n_layers)),
                                      synth.gen_w_concat(w, seed, DEV), cfg, device=DEV))
    return model


CASES = [("kraken-n2-l2-d128-h4-s64-f32", None),
         ("kraken-n4-l12-d768-h12-s2048-bf16", [700, 1, 1347])]


@pytest.mark.parametrize("name,lens", CASES, ids=[c[0] for c in CASES])
def test_prefill_graph_replays_are_bit_identical(name, lens):
    w = synth.workload(name)
    lens = lens or synth.seq_lens(w)
    cu = synth.cu_seqlens(lens)
    T = cu[-1]
    say(f"[graph] {name} lens={lens}")
    torch.cuda.set_device(0)
    model = build(w, T)
    X = synth.gen_hidden(w, T, 0, DEV)
    out_e, sub_e = model.prefill(X, cu, sub_out=True)
    torch.cuda.synchronize()

    out_g = torch.empty_like(out_e)
    sub_g = torch.empty_like(sub_e)
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(graph, stream=side):
        model.prefill(X, cu, out=out_g, sub_out=sub_g)
    torch.cuda.synchronize()
    for r in range(3):
        out_g.fill_(float("nan"))              # eager work between the replays
        sub_g.fill_(float("nan"))
        model.poison_workspace()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_g, out_e), f"replay {r}: out differs"
        assert torch.equal(sub_g, sub_e), f"replay {r}: sub_out differs"
    # the graph reads the input buffer's current contents
    X2 = synth.gen_hidden(w, T, 1, DEV)
    out_e2, sub_e2 = model.prefill(X2, cu, sub_out=True)
    X.copy_(X2)
    graph.replay()
    torch.cuda.synchronize()
    model.sync()
    model.close()
    assert torch.equal(out_g, out_e2) and torch.equal(sub_g, sub_e2)
    assert not torch.equal(out_e2, out_e)
    say("    3 replays and a replay on new input equal the eager calls bit for bit")
