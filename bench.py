"""Throughput of the tree-verify step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 8b-bf16]

A step is one acespec_verify_tree call over a batch of drafted trees (embedding, all
decoder layers with tree attention, LM head, fused vocabulary verify, path walk), on
synthetic inputs already resident in HBM.  Prints one JSON line: verified tree tokens/s
(sessions x drafted nodes / step time), the roofline of the dominant kernel from the
library's own HIP-event timing over the timed steps, and the float64 oracle timed on the
host cores on a bounded sample (cpu_baseline).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_MFMA_TFLOPS = 2500.0   # MI355X dense fp16 / bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def kernel_work(w, B, n1, P, S_tot):
    """Algorithmic work per launch of each kernel kind: (flops, bytes)."""
    R = B * n1
    d, H, Hkv, hd, F, V = w.d, w.H, w.Hkv, w.hd, w.F, w.V
    qkvn = (H + 2 * Hkv) * hd
    wb = 2  # bf16 weights
    return {
        "gemm_qkv": (2.0 * R * qkvn * d, qkvn * d * wb),
        "gemm_o": (2.0 * R * d * H * hd, d * H * hd * wb),
        "gemm_gate_up": (2.0 * R * 2 * F * d, 2 * F * d * wb),
        "gemm_down": (2.0 * R * d * F, d * F * wb),
        "gemm_lm_head": (2.0 * R * V * d, V * d * wb + R * V * 4),
        # K and V of every session's prefix and tree slots, read once
        "tree_attention": (4.0 * w.G * n1 * hd * S_tot * Hkv, 2.0 * S_tot * Hkv * hd * 2),
        # logits of every row once, draft distribution of every parent row once
        "vocab_verify": (0.0, 4.0 * R * V + 4.0 * P * V),
    }


def cpu_baseline(w, W, batch, n_sessions):
    """The oracle as it stands on n_sessions whole sessions: the tree forward through every
    layer, the verify stage of every row and the walk."""
    import numpy as np
    from oracle import model as om
    from oracle import verify as ov
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    sess = list(range(min(n_sessions, batch.tokens.shape[0])))
    # host copies of everything the sample reads, taken before the oracle clock starts
    Wh = type(W)(W.embed.cpu(), [{k: v.cpu() for k, v in lw.items()} for lw in W.layers],
                 W.final_norm.cpu(), W.lm_head.cpu())
    S = {b: int(batch.prefix_len[b]) for b in sess}
    kv = {(l, b): (om.k_prefix(batch.kv_k, l, b, S[b]), om.v_prefix(batch.kv_v, l, b, S[b]))
          for l in range(w.L) for b in sess}
    toks, pars = batch.tokens.cpu(), batch.parents.cpu()
    q = batch.q[: len(sess)].cpu().numpy().astype(np.float64)
    u = batch.u[: len(sess)].cpu().numpy().astype(np.float64)
    t0 = time.perf_counter()
    z = om.forward_tree_batch(Wh, om.dims_of(w), toks, pars, batch.prefix_len.cpu(),
                              lambda l, b: kv[(l, b)], sess)
    for i, b in enumerate(sess):
        tk = [int(t) for t in toks[b]]
        pr = [int(p) for p in pars[b]]
        res = ov.verify_session(z[i], q[i], tk, pr, u[i], w.T, w.top_p, w.top_k)
        ov.walk(tk, pr, res)
    t = time.perf_counter() - t0
    n_tok = len(sess) * (toks.shape[1] - 1)
    return {"value": n_tok / t, "unit": "verified tree tokens/s", "cores": int(cores),
            "kind": "oracle",
            "sample": (f"{len(sess)} of {batch.tokens.shape[0]} sessions of {w.name} "
                       f"({n_tok} drafted nodes): full float64 forward through all {w.L} "
                       f"layers, verify stage of every row, walk; {t:.1f} s")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="8b-bf16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sessions", type=int, default=2)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); the verify step "
              "shards by session with no collectives, see the design notes", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2609_02514_amd.acespec import (Verifier, acespec_timing_enable,
                                              acespec_timing_read)

    torch.cuda.set_device(0)
    w = synth.get(args.workload)
    if w.tree == "tail":
        raise SystemExit("bench.py times the full tree-verify step; pick a tree workload")
    log(f"generating {w.name} on the GPU")
    W = synth.make_weights(w, "cuda")
    batch = synth.make_batch(w, "cuda")
    B, n1 = batch.tokens.shape
    parents = synth.tree_parents(w)
    P = sum(1 for c in synth.children_lists(parents) if c) * B
    S_tot = int(batch.prefix_len.sum().item()) + B * n1
    v = Verifier.for_workload(w)
    ws = v.weights_struct(W)
    outs = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, "cuda", False)

    def step():
        v.verify_tree(ws, batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len, batch.tokens,
                      batch.parents, batch.q, batch.u, w.T, w.top_p, w.top_k, outs)

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    acespec_timing_enable(v.ctx, True)
    acespec_timing_read(v.ctx)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    t_wall = time.perf_counter()
    for i in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_total = e0.elapsed_time(e1)
    per_kernel = acespec_timing_read(v.ctx)
    acespec_timing_enable(v.ctx, False)
    ms_step = ms_total / args.steps
    tokens = B * (n1 - 1)
    value = tokens / (ms_step / 1e3)
    log(f"{args.steps} steps: {ms_step:.3f} ms/step (wall {t_wall / args.steps * 1e3:.3f}), "
        f"{value:.0f} tok/s; status {outs['status'].tolist()[:4]}...")

    work = kernel_work(w, B, n1, P, S_tot)
    kernels = {}
    for name, (ms, cnt) in per_kernel.items():
        avg = ms / max(cnt, 1)
        ent = {"ms_per_step": round(ms / args.steps, 4), "avg_launch_ms": round(avg, 5),
               "launches_per_step": cnt // args.steps}
        if name in work:
            fl, by = work[name]
            if fl and name.startswith("gemm"):
                ent["tflops"] = round(fl / (avg / 1e3) / 1e12, 1)
                ent["mfma_frac"] = round(ent["tflops"] / PEAK_MFMA_TFLOPS, 4)
            if by:
                ent["gbs"] = round(by / (avg / 1e3) / 1e9, 1)
                ent["hbm_frac"] = round(ent["gbs"] / PEAK_HBM_GBS, 4)
        kernels[name] = ent
    dom = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
    dk = kernels[dom]
    if dom.startswith("gemm"):
        roof = {"kernel": dom, "bound": "mfma", "achieved": dk["tflops"],
                "peak": PEAK_MFMA_TFLOPS, "unit": "TFLOP/s", "frac": dk["mfma_frac"],
                "traffic": None}
    else:
        roof = {"kernel": dom, "bound": "hbm", "achieved": dk["gbs"], "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": dk["hbm_frac"], "traffic": None}

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the oracle on the host (bounded sample)")
        cpu = cpu_baseline(w, W, batch, args.cpu_sessions)
        log(f"oracle: {cpu['value']:.3f} tok/s on {cpu['cores']} threads")

    line = {
        "metric": "verified tree tokens/s on 1 MI355X (8B shape)",
        "value": round(value, 1),
        "unit": "verified tree tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 weights/KV, fp16 activations on f16 MFMA, fp32 accumulate",
        "data": "synthetic (seeded random-init weights, KV prefix, drafted trees, draft q)",
        "config": {"workload": w.name, "layers": w.L, "d_model": w.d, "heads": w.H,
                   "kv_heads": w.Hkv, "head_dim": w.hd, "d_ff": w.F, "vocab": w.V,
                   "sessions": B, "prefix_len": w.S, "drafted_nodes": n1 - 1,
                   "temperature": w.T, "top_p": w.top_p, "top_k": w.top_k},
        "roofline": roof,
        "cpu_baseline": cpu,
        "kernels": kernels,
    }
    print(json.dumps(line), flush=True)
    v.close()


if __name__ == "__main__":
    main()
