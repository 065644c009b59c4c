"""Oracle forward pass (float64) -- test infrastructure only.

The verify step runs the target model once over every drafted tree (Section
III-B: the cloud processes the received tokens in a single forward pass).
All drafted nodes of a session are packed into that one pass; each node may
attend to the verified context and to its own ancestral sequence only
(Section III-C, tree attention mask: shared prefix block, main-path branch
block, suffix diagonal block).

The decoder itself is not specified by the paper beyond the families it uses
(Qwen, LLaMA; Section V-A).  Reading used here: Llama-style pre-norm blocks,
RMSNorm with gains, rotate-half RoPE, grouped-query attention with scale
1/sqrt(hd), SwiGLU MLP, no biases, untied LM head.  Tree node positions are
prefix_len + depth (siblings share a position); node keys and values occupy
distinct cache slots prefix_len + row.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, List, Sequence

import numpy as np


def to_f64(t) -> np.ndarray:
    """Exact upcast of a torch tensor (fp32 / bf16) or numpy array to float64."""
    if isinstance(t, np.ndarray):
        return t.astype(np.float64)
    import torch
    return t.detach().to("cpu").to(torch.float64).numpy()


@dataclass
class Dims:
    L: int
    d: int
    H: int
    Hkv: int
    hd: int
    F: int
    V: int
    rope_base: float = 10000.0
    rms_eps: float = 1e-5

    @property
    def G(self) -> int:
        return self.H // self.Hkv


def dims_of(w) -> Dims:
    return Dims(w.L, w.d, w.H, w.Hkv, w.hd, w.F, w.V, w.rope_base, w.rms_eps)


class F64Weights:
    """Lazy float64 view of a weight set, converted one tensor at a time."""

    def __init__(self, weights):
        self._w = weights
        self._cache = {}

    def get(self, name: str, layer: int = -1) -> np.ndarray:
        key = (name, layer)
        if key not in self._cache:
            src = getattr(self._w, name) if layer < 0 else self._w.layers[layer][name]
            self._cache[key] = to_f64(src)
        return self._cache[key]

    def drop_layer(self, layer: int):
        for k in [k for k in self._cache if k[1] == layer]:
            del self._cache[k]

    def embed_rows(self, ids: Sequence[int]) -> np.ndarray:
        return to_f64(self._w.embed[list(ids)])


# ----------------------------------------------------------------------------------------
# Building blocks
# ----------------------------------------------------------------------------------------


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gain, over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * gain


def rope_cos_sin(pos: np.ndarray, hd: int, base: float):
    """Angles pos * base^(-2i/hd) for i < hd/2; returns (cos, sin) of shape [n, hd/2]."""
    inv_freq = base ** (-(2.0 * np.arange(hd // 2, dtype=np.float64)) / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate-half RoPE on x[n, heads, hd]: pair (i, i + hd/2) is rotated by angle i."""
    h = x.shape[-1] // 2
    x1, x2 = x[..., :h], x[..., h:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax_rows(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def tree_depths(parents: Sequence[int]) -> List[int]:
    """depth(0) = 0, depth(r) = depth(parent(r)) + 1 (requires parent(r) < r)."""
    depth = [0] * len(parents)
    for r in range(1, len(parents)):
        depth[r] = depth[parents[r]] + 1
    return depth


def ancestor_matrix(parents: Sequence[int]) -> np.ndarray:
    """anc[r, j] = True iff node j is r itself or an ancestor of r (root included)."""
    n = len(parents)
    anc = np.zeros((n, n), dtype=bool)
    for r in range(n):
        j = r
        while j >= 0:
            anc[r, j] = True
            j = parents[j]
    return anc


def validate_tree(parents: Sequence[int], tokens: Sequence[int], V: int) -> bool:
    if len(parents) == 0 or parents[0] != -1:
        return False
    for r in range(1, len(parents)):
        if not (0 <= parents[r] < r):
            return False
    return all(0 <= t < V for t in tokens)


# ----------------------------------------------------------------------------------------
# Tree forward: all nodes of one session in one pass under the ancestor mask
# ----------------------------------------------------------------------------------------


def tree_layer(W: F64Weights, dims: Dims, l: int, x: np.ndarray, kpre: np.ndarray,
               vpre: np.ndarray, cos: np.ndarray, sin: np.ndarray, anc: np.ndarray,
               S: int, kv_sink: list = None) -> np.ndarray:
    """One decoder layer over the n rows of one tree.  kpre / vpre: [Hkv, S, hd] prefix
    (keys post-RoPE).  Row r attends to the S prefix slots and to rows j with anc[r, j].
    kv_sink, if given, receives this layer's tree-row keys (post-RoPE) and values, each
    [n, Hkv, hd]."""
    n = x.shape[0]
    H, Hkv, hd, G = dims.H, dims.Hkv, dims.hd, dims.G
    scale = 1.0 / np.sqrt(hd)
    a = rms_norm(x, W.get("attn_norm", l), dims.rms_eps)
    qkv = a @ W.get("wqkv", l).T
    q = qkv[:, : H * hd].reshape(n, H, hd)
    k = qkv[:, H * hd: (H + Hkv) * hd].reshape(n, Hkv, hd)
    v = qkv[:, (H + Hkv) * hd:].reshape(n, Hkv, hd)
    q = apply_rope(q, cos, sin)
    k = apply_rope(k, cos, sin)
    if kv_sink is not None:
        kv_sink.append((k.copy(), v.copy()))
    o = np.zeros((n, H, hd))
    visible = np.concatenate([np.ones((n, S), dtype=bool), anc], axis=1)
    for h in range(H):
        g = h // G
        keys = np.concatenate([kpre[g], k[:, g, :]], axis=0)      # [S + n, hd]
        vals = np.concatenate([vpre[g], v[:, g, :]], axis=0)
        s = (q[:, h, :] @ keys.T) * scale                          # [n, S + n]
        s = np.where(visible, s, -np.inf)
        o[:, h, :] = softmax_rows(s) @ vals
    x = x + o.reshape(n, H * hd) @ W.get("wo", l).T
    b = rms_norm(x, W.get("mlp_norm", l), dims.rms_eps)
    gu = b @ W.get("w_gate_up", l).T
    return x + (silu(gu[:, : dims.F]) * gu[:, dims.F:]) @ W.get("w_down", l).T


def final_logits(W: F64Weights, dims: Dims, x: np.ndarray) -> np.ndarray:
    return rms_norm(x, W.get("final_norm"), dims.rms_eps) @ W.get("lm_head").T


def forward_tree_session(W: F64Weights, dims: Dims, kpre: List[np.ndarray],
                         vpre: List[np.ndarray], tokens: Sequence[int],
                         parents: Sequence[int], S: int, kv_sink: list = None) -> np.ndarray:
    """Logits z[r] (float64, [n, V]) for every row of one drafted tree.

    kpre / vpre: per layer, the session's cache prefix [Hkv, S, hd] (keys post-RoPE).
    kv_sink, if given, receives per layer the tree rows' (keys, values) [n, Hkv, hd].
    """
    depth = np.array(tree_depths(parents))
    anc = ancestor_matrix(parents)
    cos, sin = rope_cos_sin(S + depth, dims.hd, dims.rope_base)
    x = W.embed_rows(tokens)
    for l in range(dims.L):
        x = tree_layer(W, dims, l, x, kpre[l], vpre[l], cos, sin, anc, S, kv_sink)
    return final_logits(W, dims, x)


# ----------------------------------------------------------------------------------------
# Plain-definition twin: causal decode along one root-to-node path
# ----------------------------------------------------------------------------------------


def forward_causal_path(W: F64Weights, dims: Dims, kpre: List[np.ndarray],
                        vpre: List[np.ndarray], path_tokens: Sequence[int],
                        S: int, return_cache: bool = False):
    """Logits at the last token of [prefix; path_tokens], decoding one token at a time.

    Token i of the path sits at position S + i and sees the whole prefix and the
    path tokens before it: an ordinary causal language-model pass.  The tree
    forward must reproduce, for every row, this quantity evaluated on the
    row's root-to-node path.  With return_cache, also returns the cache this decode
    builds: per layer, keys and values [Hkv, S + len(path_tokens), hd].
    """
    H, Hkv, hd, G = dims.H, dims.Hkv, dims.hd, dims.G
    ks = [[kpre[l][g].copy() for g in range(Hkv)] for l in range(dims.L)]
    vs = [[vpre[l][g].copy() for g in range(Hkv)] for l in range(dims.L)]
    logits = None
    for i, t in enumerate(path_tokens):
        pos = S + i
        cos, sin = rope_cos_sin(np.array([pos]), hd, dims.rope_base)
        x = W.embed_rows([t])[0]
        for l in range(dims.L):
            a = rms_norm(x[None, :], W.get("attn_norm", l), dims.rms_eps)[0]
            qkv = W.get("wqkv", l) @ a
            q = apply_rope(qkv[: H * hd].reshape(1, H, hd), cos, sin)[0]
            k = apply_rope(qkv[H * hd: (H + Hkv) * hd].reshape(1, Hkv, hd), cos, sin)[0]
            v = qkv[(H + Hkv) * hd:].reshape(Hkv, hd)
            for g in range(Hkv):
                ks[l][g] = np.vstack([ks[l][g], k[g][None, :]])
                vs[l][g] = np.vstack([vs[l][g], v[g][None, :]])
            o = np.zeros((H, hd))
            for h in range(H):
                g = h // G
                s = ks[l][g] @ q[h] / np.sqrt(hd)
                w = np.exp(s - s.max())
                o[h] = (w / w.sum()) @ vs[l][g]
            x = x + W.get("wo", l) @ o.reshape(-1)
            b = rms_norm(x[None, :], W.get("mlp_norm", l), dims.rms_eps)[0]
            gu = W.get("w_gate_up", l) @ b
            x = x + W.get("w_down", l) @ (silu(gu[: dims.F]) * gu[dims.F:])
        if i == len(path_tokens) - 1:
            xn = rms_norm(x[None, :], W.get("final_norm"), dims.rms_eps)[0]
            logits = W.get("lm_head") @ xn
    if return_cache:
        return logits, ([np.stack(ks[l]) for l in range(dims.L)],
                        [np.stack(vs[l]) for l in range(dims.L)])
    return logits


def commit_path(k_cache: np.ndarray, v_cache: np.ndarray, S: int, path: Sequence[int]):
    """COMPACT_KV of Algorithm 1 on one session's cache.

    k_cache [L, Hkv, cap, hd] and v_cache [L, Hkv, hd, cap] (values head-dim-major, the
    cache layout) hold the tree rows' entries at slots S + row after a verify step.  The
    cloud keeps the root (row 0) and the accepted rows `path` (root-first) and discards
    the rest: their entries move, in path order, to slots S, S + 1, ...  Returns the new
    arrays and the new prefix length S + 1 + len(path)."""
    rows = [0] + [int(r) for r in path]
    src = [S + r for r in rows]
    k, v = k_cache.copy(), v_cache.copy()
    k[:, :, S: S + len(rows), :] = k_cache[:, :, src, :]
    v[:, :, :, S: S + len(rows)] = v_cache[:, :, :, src]
    return k, v, S + len(rows)


def path_to(parents: Sequence[int], r: int) -> List[int]:
    """Rows on the root-to-r path, root first."""
    p = []
    while r >= 0:
        p.append(r)
        r = parents[r]
    return p[::-1]


# ----------------------------------------------------------------------------------------
# Batch helpers
# ----------------------------------------------------------------------------------------


def k_prefix(kv_k, l: int, b: int, S: int) -> np.ndarray:
    """Keys of session b at layer l, slots [0, S): cache [L, B, Hkv, cap, hd] -> [Hkv, S, hd]."""
    return to_f64(kv_k[l, b, :, :S])


def v_prefix(kv_v, l: int, b: int, S: int) -> np.ndarray:
    """Values of session b at layer l, slots [0, S): the value cache is head-dim-major,
    [L, B, Hkv, hd, cap] -> [Hkv, S, hd]."""
    return np.ascontiguousarray(to_f64(kv_v[l, b, :, :, :S]).transpose(0, 2, 1))


def session_prefix(kv_k, kv_v, b: int, S: int):
    """Per-layer float64 copies of session b's cache prefix [Hkv, S, hd]."""
    L = kv_k.shape[0]
    return ([k_prefix(kv_k, l, b, S) for l in range(L)],
            [v_prefix(kv_v, l, b, S) for l in range(L)])


def forward_tree_batch(weights, dims: Dims, tokens, parents, prefix_len, kv_prefix,
                       sessions: Sequence[int], progress: Callable[[str], None] = None,
                       drop_layers: bool = True) -> np.ndarray:
    """Logits [len(sessions), N+1, V] for the chosen sessions.

    kv_prefix(l, b) -> (K [Hkv, S_b, hd], V [Hkv, S_b, hd]) gives session b's cache prefix
    at layer l.  Layers run outermost so each layer's weights are converted once for all
    sessions and can be dropped afterwards (the 8B shapes do not fit in fp64 at once).
    """
    W = weights if isinstance(weights, F64Weights) else F64Weights(weights)
    st = []
    for b in sessions:
        S = int(prefix_len[b])
        toks = [int(t) for t in tokens[b]]
        pars = [int(p) for p in parents[b]]
        depth = np.array(tree_depths(pars))
        cos, sin = rope_cos_sin(S + depth, dims.hd, dims.rope_base)
        st.append(dict(b=b, S=S, anc=ancestor_matrix(pars), cos=cos, sin=sin,
                       x=W.embed_rows(toks)))
    for l in range(dims.L):
        for s in st:
            kp, vp = kv_prefix(l, s["b"])
            s["x"] = tree_layer(W, dims, l, s["x"], kp, vp, s["cos"], s["sin"], s["anc"],
                                s["S"])
        if drop_layers:
            W.drop_layer(l)
        if progress:
            progress(f"oracle layer {l + 1}/{dims.L} done")
    return np.stack([final_logits(W, dims, s["x"]) for s in st])


def lm_head_tail(weights, hidden, final_norm: bool = False, eps: float = 1e-5) -> np.ndarray:
    """z = W_lm . h (optionally RMSNorm'd with the final gain) for tail rows."""
    W = weights if isinstance(weights, F64Weights) else F64Weights(weights)
    h = to_f64(hidden)
    if final_norm:
        h = rms_norm(h, W.get("final_norm"), eps)
    return h @ W.get("lm_head").T
