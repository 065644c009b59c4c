"""Seeded synthetic inputs for the tree-verify step.

This module is shared by the CPU oracle and the GPU path and holds none of the
verification arithmetic: it only draws the model weights, the KV prefix, the
drafted trees, the draft distributions and the uniforms that the method
consumes as inputs.

Recipe (the paper evaluates on GSM8K / HumanEval / Alpaca with Qwen and LLaMA
pairs; none of those datasets or weights are used, these synthetic inputs
stand in for them):

* Every tensor is drawn with ``torch.Generator`` seeded per (master seed,
  sub-stream, tensor index), on the device that consumes it.  The oracle
  receives a host copy of the very same tensors, so both sides always see
  identical bytes.  Sub-streams: 0 weights, 1 KV prefix, 2 tree tokens,
  3 draft logits, 4 uniforms, 5 hidden states (LM-head tail), 6 noise.
* Weights ~ N(0, 0.02) drawn in fp32 and rounded once (RNE) to the model
  dtype; RMSNorm gains are 1.0 unless ``random_gains`` is set.
* KV prefix ~ N(0, 1), already rotated (keys are stored post-RoPE), in the
  model dtype.  No prefill is run.  Cache layout: keys [L, B, Hkv, cap, hd], values
  head-dim-major [L, B, Hkv, hd, cap]; cap is a multiple of 64.
* Draft distributions q = softmax(g / T_q) with g ~ N(0, q_std) per row.
* Trees follow the drafter of the paper (Section III-C): at each parent the
  main child is sampled from q of that parent and the siblings are the top-F
  tokens of q excluding the main token.  Rows are in breadth-first order with
  the main child first; row 0 is the root (the last committed token).
* Uniforms are (k + 1/2) / 2^23 with k uniform in [0, 2^23): exactly
  representable in fp32 and strictly inside (0, 1).
* LM-head tail workload: hidden ~ N(0, 1); q = softmax(z / T + eps) with
  z = hidden . W_lm^T (taken from torch's own matmul) and eps ~ N(0, 1).
"""
from __future__ import annotations

import copy
import math
from dataclasses import dataclass, field, replace
from typing import List, Optional

import torch

UNIFORM_BITS = 23

# --------------------------------------------------------------------------------------
# Workload definitions
# --------------------------------------------------------------------------------------


@dataclass
class Workload:
    name: str
    dtype: str            # "f32" or "bf16"
    L: int                # layers (0 = LM-head tail only)
    d: int
    H: int
    Hkv: int
    hd: int
    F: int
    V: int
    B: int                # sessions
    S: int                # KV prefix length per session
    tree: str             # "chain_sib", "widths_2455", "tail"
    depth: int = 0        # main-chain depth
    sib: int = 0          # siblings per depth (chain_sib)
    q_std: float = 2.0
    q_T: float = 1.0
    T: float = 1.0
    top_p: float = 0.9
    top_k: int = 16
    tokens: str = "draft"  # "uniform" or "draft"
    rope_base: float = 10000.0
    rms_eps: float = 1e-5
    chain_len: int = 16    # tail only
    rows: int = 0          # tail only: total rows
    ragged: bool = False   # per-session prefix lengths in [S/2, S]
    random_gains: bool = False
    seed_base: int = 0
    fanout: tuple = ()     # "fanout" trees: alternatives per rejection depth (F_0, F_1, ...)

    @property
    def N(self) -> int:
        """Drafted nodes per session (the root row is not counted)."""
        return len(tree_parents(self)) - 1 if self.tree != "tail" else 0

    @property
    def G(self) -> int:
        return self.H // self.Hkv

    def scaled(self, **kw) -> "Workload":
        return replace(copy.deepcopy(self), **kw)


WORKLOADS = {
    "tiny-fp32": Workload("tiny-fp32", "f32", L=2, d=256, H=4, Hkv=4, hd=64, F=1024, V=4096,
                          B=1, S=128, tree="chain_sib", depth=4, sib=1, q_std=2.0, q_T=0.8,
                          T=0.8, top_p=0.9, top_k=16, tokens="uniform", seed_base=1235),
    "1b-bf16": Workload("1b-bf16", "bf16", L=16, d=2048, H=32, Hkv=8, hd=64, F=8192, V=32000,
                        B=16, S=1024, tree="chain_sib", depth=8, sib=1, q_std=2.0, q_T=0.7,
                        T=0.7, top_p=0.95, top_k=32, seed_base=1236),
    "8b-bf16": Workload("8b-bf16", "bf16", L=32, d=4096, H=32, Hkv=8, hd=128, F=14336,
                        V=128256, B=64, S=2048, tree="widths_2455", depth=4, q_std=3.0,
                        q_T=0.8, T=0.8, top_p=0.9, top_k=32, seed_base=1237),
    "8b-long-wide": Workload("8b-long-wide", "bf16", L=32, d=4096, H=32, Hkv=8, hd=128,
                             F=14336, V=128256, B=8, S=16384, tree="chain_sib", depth=8, sib=7,
                             q_std=3.0, q_T=1.0, T=1.0, top_p=0.9, top_k=64, seed_base=1238),
    "8b-lmhead-tail": Workload("8b-lmhead-tail", "bf16", L=0, d=4096, H=0, Hkv=1, hd=0, F=0,
                               V=128256, B=256, S=0, tree="tail", T=0.6, top_p=0.8, top_k=8,
                               chain_len=16, rows=4096, seed_base=1239),
    # The 8B model with a paper-shaped tree: budget B* = 32 nodes, a main chain of 8 and
    # B_alloc = 24 alternatives spread by the geometric decay of Section IV (alpha 0.8,
    # beta 1), rounded by largest remainders.
    "8b-geometric": Workload("8b-geometric", "bf16", L=32, d=4096, H=32, Hkv=8, hd=128,
                             F=14336, V=128256, B=64, S=2048, tree="fanout", depth=8,
                             fanout=(4, 4, 3, 3, 3, 3, 2, 2), q_std=3.0, q_T=0.8, T=0.8,
                             top_p=0.9, top_k=32, seed_base=1242),
    # The paper's cloud targets (Section V-A: Qwen-32B and LLaMA-70B classes) at the batch
    # and tree shape of the 8B workload; the 70B weights (140 GB bf16) and KV cache (89 GB)
    # fit one 288 GB GPU.
    "32b-bf16": Workload("32b-bf16", "bf16", L=64, d=5120, H=40, Hkv=8, hd=128, F=27648,
                         V=152064, B=64, S=2048, tree="widths_2455", depth=4, q_std=3.0,
                         q_T=0.8, T=0.8, top_p=0.9, top_k=32, seed_base=1240),
    "70b-bf16": Workload("70b-bf16", "bf16", L=80, d=8192, H=64, Hkv=8, hd=128, F=28672,
                         V=128256, B=64, S=2048, tree="widths_2455", depth=4, q_std=3.0,
                         q_T=0.8, T=0.8, top_p=0.9, top_k=32, seed_base=1241),
}


def get(name: str) -> Workload:
    return copy.deepcopy(WORKLOADS[name])


# --------------------------------------------------------------------------------------
# Tree shapes
# --------------------------------------------------------------------------------------


def tree_parents(w: Workload) -> List[int]:
    """Parent index per row (row 0 is the root, parent -1), breadth-first, main child first.

    chain_sib: a main chain of ``depth`` nodes; at each depth ``sib`` extra siblings of
    the main node (leaves).  widths_2455: two children at the first two levels, one
    below, plus one extra leaf sibling on the main chain at depths 3 and 4 (16 nodes).
    """
    if w.tree == "chain_sib":
        parents = [-1]
        main_prev = 0
        for _ in range(w.depth):
            main_row = len(parents)
            parents.append(main_prev)
            for _ in range(w.sib):
                parents.append(main_prev)
            main_prev = main_row
        return parents
    if w.tree == "widths_2455":
        parents = [-1]
        # depth 1: two children of the root
        d1 = [1, 2]
        parents += [0, 0]
        # depth 2: two children of each depth-1 node
        d2 = []
        for p in d1:
            for _ in range(2):
                d2.append(len(parents))
                parents.append(p)
        # depth 3: one child per depth-2 node, plus an extra sibling under the main chain
        d3 = []
        for i, p in enumerate(d2):
            d3.append(len(parents))
            parents.append(p)
            if i == 0:
                parents.append(p)          # extra leaf sibling on the main chain
        # depth 4: same rule
        for i, p in enumerate(d3):
            parents.append(p)
            if i == 0:
                parents.append(p)
        return parents
    if w.tree == "chain":
        return [-1] + list(range(w.depth))
    if w.tree == "fanout":
        # main chain of len(fanout) nodes; at each depth k+1 the main child comes first,
        # then fanout[k] alternative leaves under the same parent (Section III-C)
        parents = [-1]
        main_prev = 0
        for fk in w.fanout:
            main_row = len(parents)
            parents.extend([main_prev] * (1 + fk))
            main_prev = main_row
        return parents
    raise ValueError(w.tree)


def children_lists(parents: List[int]) -> List[List[int]]:
    ch = [[] for _ in parents]
    for r, p in enumerate(parents):
        if p >= 0:
            ch[p].append(r)
    return ch


# --------------------------------------------------------------------------------------
# Random streams
# --------------------------------------------------------------------------------------


def _gen(device, seed: int, stream: int, index: int = 0) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1_000_003 + stream * 10_007 + index) & 0x7FFF_FFFF_FFFF_FFFF)
    return g


def _torch_dtype(w: Workload):
    return torch.float32 if w.dtype == "f32" else torch.bfloat16


def normal(shape, std, dtype, device, seed, stream, index=0):
    """N(0, std) drawn in fp32 and rounded once to ``dtype``."""
    g = _gen(device, seed, stream, index)
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t.to(dtype)


def uniforms(shape, device, seed, stream=4, index=0) -> torch.Tensor:
    g = _gen(device, seed, stream, index)
    k = torch.randint(0, 1 << UNIFORM_BITS, shape, generator=g, device=device, dtype=torch.int64)
    return ((k.to(torch.float64) + 0.5) / float(1 << UNIFORM_BITS)).to(torch.float32)


# --------------------------------------------------------------------------------------
# Model weights
# --------------------------------------------------------------------------------------


@dataclass
class Weights:
    embed: Optional[torch.Tensor]
    layers: List[dict]
    final_norm: Optional[torch.Tensor]
    lm_head: torch.Tensor

    def to(self, device) -> "Weights":
        mv = lambda t: None if t is None else t.to(device)
        return Weights(mv(self.embed), [{k: mv(v) for k, v in l.items()} for l in self.layers],
                       mv(self.final_norm), mv(self.lm_head))


def make_weights(w: Workload, device="cpu", seed: Optional[int] = None,
                 progress=None) -> Weights:
    """Random-init weights of ``w``; progress(msg), if given, hears every 8th layer."""
    seed = w.seed_base if seed is None else seed
    dt = _torch_dtype(w)
    std = 0.02

    def gain(idx):
        if w.random_gains:
            return (1.0 + normal((w.d,), 0.1, torch.float32, device, seed, 0, idx)).to(dt)
        return torch.ones(w.d, dtype=dt, device=device)

    idx = 0
    layers = []
    qkv_rows = (w.H + 2 * w.Hkv) * w.hd
    for l in range(w.L):
        base = 16 * (l + 1)
        layers.append(dict(
            attn_norm=gain(base + 0),
            wqkv=normal((qkv_rows, w.d), std, dt, device, seed, 0, base + 1),
            wo=normal((w.d, w.H * w.hd), std, dt, device, seed, 0, base + 2),
            mlp_norm=gain(base + 3),
            w_gate_up=normal((2 * w.F, w.d), std, dt, device, seed, 0, base + 4),
            w_down=normal((w.d, w.F), std, dt, device, seed, 0, base + 5),
        ))
        if progress is not None and ((l + 1) % 8 == 0 or l + 1 == w.L):
            progress(f"weights: {l + 1}/{w.L} layers")
    embed = normal((w.V, w.d), std, dt, device, seed, 0, 1) if w.L > 0 else None
    final_norm = gain(2) if w.L > 0 else None
    lm_head = normal((w.V, w.d), std, dt, device, seed, 0, 3)
    return Weights(embed, layers, final_norm, lm_head)


# --------------------------------------------------------------------------------------
# KV prefix, trees, draft distributions, uniforms
# --------------------------------------------------------------------------------------


@dataclass
class Batch:
    tokens: torch.Tensor          # [B, N+1] int32
    parents: torch.Tensor         # [B, N+1] int32
    prefix_len: torch.Tensor      # [B] int32
    kv_k: Optional[torch.Tensor]  # [L, B, Hkv, cap, hd]
    kv_v: Optional[torch.Tensor]  # [L, B, Hkv, hd, cap]
    q: torch.Tensor               # [B, N+1, V] fp32
    u: torch.Tensor               # [B, N+1, 3] fp32
    cap: int = 0
    hidden: Optional[torch.Tensor] = None  # tail only: [R, d]
    draft_tokens: Optional[torch.Tensor] = None  # tail only: [R]


def prefix_lengths(w: Workload, seed: int) -> List[int]:
    if not w.ragged:
        return [w.S] * w.B
    g = _gen("cpu", seed, 1, 999)
    lo = max(1, w.S // 2)
    return [int(x) for x in torch.randint(lo, w.S + 1, (w.B,), generator=g)]


def make_kv(w: Workload, device, seed: int, cap: int, progress=None):
    dt = _torch_dtype(w)
    kshape = (w.L, w.B, w.Hkv, cap, w.hd)
    vshape = (w.L, w.B, w.Hkv, w.hd, cap)
    k = torch.empty(kshape, dtype=dt, device=device)
    v = torch.empty(vshape, dtype=dt, device=device)
    for l in range(w.L):   # per layer, to bound the fp32 staging memory
        k[l].copy_(normal(kshape[1:], 1.0, dt, device, seed, 1, 2 * l))
        v[l].copy_(normal(vshape[1:], 1.0, dt, device, seed, 1, 2 * l + 1))
        if progress is not None and ((l + 1) % 8 == 0 or l + 1 == w.L):
            progress(f"KV cache: {l + 1}/{w.L} layers")
    return k, v


def draft_q(w: Workload, rows_shape, device, seed: int) -> torch.Tensor:
    g = normal(tuple(rows_shape) + (w.V,), w.q_std, torch.float32, device, seed, 3)
    return torch.softmax(g / w.q_T, dim=-1)


def make_batch(w: Workload, device="cpu", seed: Optional[int] = None,
               weights: Optional[Weights] = None, extra_cap: int = 0, progress=None) -> Batch:
    """Draw one batch of drafted trees (or tail rows) for workload ``w``; progress(msg), if
    given, hears every 8th layer of the KV cache."""
    seed = w.seed_base if seed is None else seed
    if w.tree == "tail":
        return _make_tail(w, device, seed, weights)
    parents = tree_parents(w)
    n1 = len(parents)
    ch = children_lists(parents)
    par = torch.tensor(parents, dtype=torch.int32).repeat(w.B, 1)
    q = draft_q(w, (w.B, n1), device, seed)
    u = uniforms((w.B, n1, 3), device, seed)
    gtok = _gen(device, seed, 2)
    root = torch.randint(0, w.V, (w.B,), generator=gtok, device=device)
    if w.tokens == "uniform":
        tok = torch.randint(0, w.V, (w.B, n1), generator=gtok, device=device)
        tok[:, 0] = root
    else:
        tok = torch.zeros((w.B, n1), dtype=torch.int64, device=device)
        tok[:, 0] = root
        for r in range(n1):
            if not ch[r]:
                continue
            qr = q[:, r, :]
            main = torch.multinomial(qr, 1, generator=gtok).squeeze(1)
            tok[:, ch[r][0]] = main
            nsib = len(ch[r]) - 1
            if nsib:
                masked = qr.scatter(1, main[:, None], -1.0)
                sib = torch.topk(masked, nsib, dim=1).indices
                for j, c in enumerate(ch[r][1:]):
                    tok[:, c] = sib[:, j]
    S_list = prefix_lengths(w, seed)
    cap = (max(S_list) + n1 + extra_cap + 63) // 64 * 64
    kv_k, kv_v = make_kv(w, device, seed, cap, progress)
    return Batch(tokens=tok.to(torch.int32), parents=par.to(device),
                 prefix_len=torch.tensor(S_list, dtype=torch.int32, device=device),
                 kv_k=kv_k, kv_v=kv_v, q=q, u=u, cap=cap)


def _make_tail(w: Workload, device, seed: int, weights: Optional[Weights]) -> Batch:
    R = w.rows
    dt = _torch_dtype(w)
    hidden = normal((R, w.d), 1.0, dt, device, seed, 5)
    if weights is None:
        weights = make_weights(w, device, seed)
    # Draft q tracks the target: q = softmax(z / T + eps); z from torch's own matmul.
    q = torch.empty((R, w.V), dtype=torch.float32, device=device)
    chunk = 512
    for i in range(0, R, chunk):
        z = hidden[i:i + chunk].float() @ weights.lm_head.float().t()
        eps = normal(z.shape, 1.0, torch.float32, device, seed, 6, i // chunk)
        q[i:i + chunk] = torch.softmax(z / w.T + eps, dim=-1)
    gtok = _gen(device, seed, 2)
    draft = torch.multinomial(q, 1, generator=gtok).squeeze(1).to(torch.int32)
    u = uniforms((R, 3), device, seed)
    return Batch(tokens=draft.view(-1, 1), parents=torch.full((R, 1), -1, dtype=torch.int32,
                 device=device), prefix_len=torch.zeros(0, dtype=torch.int32, device=device),
                 kv_k=None, kv_v=None, q=q, u=u, hidden=hidden, draft_tokens=draft)
