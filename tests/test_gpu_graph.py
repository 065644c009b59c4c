"""The verify step under HIP stream capture: acespec_verify_tree enqueues only kernel
launches on the caller's stream (no allocation, no memset, no synchronisation, no events
while timing is off), so a caller may capture it once into a graph and replay it.  Every
replay, with eager work and synchronisations of the program's own between replays and new
inputs written into the captured buffers, must give exactly the eager step's outputs."""
import pytest
import torch

import synth
from paper_2609_02514_amd.acespec import Verifier
from tests import harness as hz
from tests.test_gpu_parity import small_bf16

pytestmark = pytest.mark.gpu


def _outs_equal(a, b):
    for k, t in a.items():
        if t is not None:
            assert torch.equal(t, b[k]), k


@pytest.mark.parametrize("name", ["small", "1b-bf16"])
def test_graph_replays_equal_eager_steps(name):
    w = small_bf16(B=4) if name == "small" else synth.get("1b-bf16")
    W = synth.make_weights(w, "cuda")
    seeds = hz.parity_seeds(w, 3)
    caps = [synth.make_batch(w, "cuda", sd).cap for sd in seeds]
    cap = max(caps)      # one cache capacity for every batch the graph sees
    batches = [synth.make_batch(w, "cuda", sd, extra_cap=cap - c) for sd, c in zip(seeds, caps)]
    live = synth.make_batch(w, "cuda", seeds[0], extra_cap=cap - caps[0])
    assert all(b.cap == cap for b in batches + [live])
    v = Verifier.for_workload(w)
    ws = v.weights_struct(W)
    B, n1 = batches[0].tokens.shape
    outs = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, "cuda", True)

    def load(bt):
        # new inputs into the buffers the graph was captured with
        for f in ("tokens", "parents", "prefix_len", "kv_k", "kv_v", "q", "u"):
            getattr(live, f).copy_(getattr(bt, f))

    def step():
        v.verify_tree(ws, live.kv_k, live.kv_v, live.cap, live.prefix_len, live.tokens,
                      live.parents, live.q, live.u, w.T, w.top_p, w.top_k, outs)

    eager = []
    for bt in batches:
        load(bt)
        step()
        torch.cuda.synchronize()
        eager.append({k: (t.clone() if t is not None else None) for k, t in outs.items()})
    hz.log(f"{name}: eager steps done; capturing")
    load(batches[0])
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()                      # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for rep in range(2):
        for i, bt in enumerate(batches):
            load(bt)
            for t in outs.values():
                if t is not None:
                    t.fill_(-3)         # eager work between replays
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            _outs_equal(eager[i], outs)
            hz.log(f"{name}: replay {rep} batch {i} equals the eager step")
    del g
    v.close()
