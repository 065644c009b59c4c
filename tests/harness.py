"""Parity harness: runs the HIP path through the C ABI and the oracle on the same seeded
inputs, and classifies every disagreement.

Tolerances (from the target stated for this hot path):
  * logits: per row, max |z_gpu - z_ref| / max |z_ref| <= 2e-2 (bf16 weights and
    activations; fp32 path and LM-head-only runs are held to tighter bounds by the tests);
  * decisions (accept, acc_prefix_len, resample, bonus, top-k ids): compared with the
    oracle's verify stage run on the GPU's own logits, identical on >= 99.9 % of nodes,
    every mismatch explained by a boundary case:
      accept      |p/q - u| < 1e-3
      inv. CDF    |C_j / S - u| < 1e-3 at the chosen or a neighbouring id
      top-p       |C_m - top_p| < 1e-4 (the nucleus edge moves)
      top-k       |p_a - p_b| <= 1e-4 p_a (tie)
    and the walk is re-derived from the GPU's own per-node decisions exactly.
"""
from __future__ import annotations

import sys
import time
from dataclasses import dataclass, field
from typing import Dict, List, Sequence

import numpy as np
import torch

import synth
from oracle import model as om
from oracle import verify as ov


def log(msg: str):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


def host(t):
    return t.detach().to("cpu")


# ---------------------------------------------------------------------------------------
# GPU runs
# ---------------------------------------------------------------------------------------


@dataclass
class TreeRun:
    w: synth.Workload
    W: synth.Weights          # device weights
    batch: synth.Batch        # device inputs
    outs: Dict                # host copies of the outputs
    host_in: Dict             # host copies of the inputs the oracle needs
    sessions: List[int]


def run_tree(w: synth.Workload, seed=None, sessions: Sequence[int] = None, device="cuda",
             weights=None, keep_logits=True, verifier=None) -> TreeRun:
    from paper_2609_02514_amd.acespec import Verifier
    seed = w.seed_base if seed is None else seed
    log(f"gen {w.name} seed={seed} L={w.L} d={w.d} V={w.V} B={w.B} S={w.S} tree={w.tree}")
    W = weights or synth.make_weights(w, device, seed)
    batch = synth.make_batch(w, device, seed)
    B, n1 = batch.tokens.shape
    sessions = list(range(B)) if sessions is None else list(sessions)
    # host copies BEFORE the HIP path runs (it writes the tree slots of the cache)
    hin = dict(tokens=host(batch.tokens), parents=host(batch.parents),
               prefix_len=host(batch.prefix_len), q=host(batch.q), u=host(batch.u),
               kv={(l, b): (om.k_prefix(batch.kv_k, l, b, int(batch.prefix_len[b])),
                            om.v_prefix(batch.kv_v, l, b, int(batch.prefix_len[b])))
                   for l in range(w.L) for b in sessions})
    v = verifier or Verifier.for_workload(w)
    ws = v.weights_struct(W)
    outs = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, device, keep_logits)
    log(f"verify_tree B={B} N={n1 - 1} cap={batch.cap}")
    v.verify_tree(ws, batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len, batch.tokens,
                  batch.parents, batch.q, batch.u, w.T, w.top_p, w.top_k, outs)
    torch.cuda.synchronize()
    log("verify_tree done")
    ho = {k: (host(t) if t is not None else None) for k, t in outs.items()}
    if verifier is None:
        v.close()
    return TreeRun(w, W, batch, ho, hin, sessions)


def oracle_tree_logits(run: TreeRun) -> np.ndarray:
    w = run.w
    hin = run.host_in
    return om.forward_tree_batch(run.W, om.dims_of(w), hin["tokens"], hin["parents"],
                                 hin["prefix_len"], lambda l, b: hin["kv"][(l, b)],
                                 run.sessions, progress=log)


# ---------------------------------------------------------------------------------------
# Comparisons
# ---------------------------------------------------------------------------------------


def logits_rel_err(z_gpu: np.ndarray, z_ref: np.ndarray) -> np.ndarray:
    """Per row: max |z_gpu - z_ref| / max |z_ref|."""
    return np.abs(z_gpu - z_ref).max(axis=-1) / np.abs(z_ref).max(axis=-1)


@dataclass
class Report:
    nodes: int = 0
    mismatches: List[str] = field(default_factory=list)
    unexplained: List[str] = field(default_factory=list)

    def ok(self, rate=1e-3) -> bool:
        allowed = max(1, int(rate * self.nodes))
        return not self.unexplained and len(self.mismatches) <= allowed

    def __str__(self):
        return (f"nodes={self.nodes} mismatches={len(self.mismatches)} "
                f"unexplained={self.unexplained[:5]} first={self.mismatches[:5]}")


def _cdf_boundary(w: np.ndarray, u: float, j_a: int, j_b: int, eps=1e-3) -> bool:
    c = np.cumsum(w) / w.sum()
    lo, hi = min(j_a, j_b), max(j_a, j_b)
    cand = [c[j] for j in range(max(0, lo - 1), min(len(c), hi + 1))]
    return any(abs(x - u) < eps for x in cand)


def _topp_boundary(pt: np.ndarray, top_p: float, eps=1e-4) -> bool:
    order = ov.sorted_order(pt)
    cs = np.cumsum(pt[order])
    m = int(np.searchsorted(cs, top_p))
    near = [cs[j] for j in range(max(0, m - 1), min(len(cs), m + 2))]
    return any(abs(x - top_p) < eps for x in near)


def compare_row_decisions(rep: Report, tag: str, z: np.ndarray, q_par: np.ndarray,
                          children: List[int], tok: Sequence[int], u: np.ndarray,
                          T: float, top_p: float, k: int, g: Dict, row_g: int,
                          child_g: Dict[int, int]):
    """Oracle verify of one parent row on the GPU's logits vs the GPU's decisions.

    g: host GPU outputs; row_g: index of this row in the GPU outputs; child_g maps local
    child -> GPU output index.  u rows are indexed by local row."""
    pt = ov.tempered_softmax(z, T)
    p, order, m = ov.nucleus(pt, top_p)
    topp_edge = _topp_boundary(pt, top_p)
    ids, probs = ov.topk_payload(p, order, k)
    rep.nodes += 1
    gid = g["topk_ids"][row_g].numpy()
    if not np.array_equal(gid, ids):
        msg = f"{tag}: topk ids"
        # ids may differ only through exact or near ties of p
        diff = [i for i in range(k) if gid[i] != ids[i]]
        tie = all(abs(pt[gid[i]] - pt[ids[i]]) <= 1e-4 * pt[ids[i]] for i in diff)
        rep.mismatches.append(msg)
        if not tie:
            rep.unexplained.append(msg)
    else:
        gp = g["topk_probs"][row_g].numpy().astype(np.float64)
        if np.abs(gp - probs).max() > 1e-4 and not topp_edge:
            rep.mismatches.append(f"{tag}: topk probs {np.abs(gp - probs).max():.2e}")
            rep.unexplained.append(rep.mismatches[-1])
    j = ov.inverse_cdf(p, float(u[2]) if u.ndim == 1 else float(u[row_g, 2]))
    gb = int(g["bonus_token"][row_g])
    ub = float(u[2]) if u.ndim == 1 else float(u[row_g, 2])
    if gb != j:
        msg = f"{tag}: bonus {gb} vs {j}"
        rep.mismatches.append(msg)
        if not (_cdf_boundary(p, ub, gb, j) or topp_edge):
            rep.unexplained.append(msg)


def compare_child(rep: Report, tag: str, z: np.ndarray, qrow: np.ndarray, x: int, u0: float,
                  u1: float, T: float, top_p: float, g_acc: int, g_res: int):
    pt = ov.tempered_softmax(z, T)
    p, order, m = ov.nucleus(pt, top_p)
    topp_edge = _topp_boundary(pt, top_p)
    rep.nodes += 1
    acc = ov.accept_token(p, qrow, x, u0)
    res = ov.residual_sample(p, qrow, u1)
    if bool(g_acc) != acc:
        msg = f"{tag}: accept {g_acc} vs {int(acc)} (p/q={p[x] / max(qrow[x], 1e-300):.6f} u={u0:.6f})"
        rep.mismatches.append(msg)
        ratio = p[x] / qrow[x] if qrow[x] > 0 else np.inf
        if not (abs(ratio - u0) < 1e-3 or topp_edge):
            rep.unexplained.append(msg)
    if g_res != res:
        msg = f"{tag}: resample {g_res} vs {res}"
        rep.mismatches.append(msg)
        rho = np.maximum(p - qrow, 0.0)
        wv = rho if rho.sum() > 0 else p
        if not (_cdf_boundary(wv, u1, g_res, res) or topp_edge):
            rep.unexplained.append(msg)


def check_tree_decisions(run: TreeRun, z_gpu_rows: Dict[int, np.ndarray]) -> Report:
    """Oracle verify stage on the GPU's logits for the sampled sessions."""
    w = run.w
    hin, g = run.host_in, run.outs
    B, n1 = hin["tokens"].shape
    rep = Report()
    for b in run.sessions:
        toks = [int(t) for t in hin["tokens"][b]]
        pars = [int(p) for p in hin["parents"][b]]
        ch = ov.children_of(pars)
        q = hin["q"][b].numpy().astype(np.float64)
        u = hin["u"][b].numpy().astype(np.float64)
        for r in range(n1):
            gi = b * n1 + r
            z = z_gpu_rows[gi]
            compare_row_decisions(rep, f"b{b}r{r}", z, q[r], ch[r], toks, u[r], w.T, w.top_p,
                                  w.top_k, g, gi, {})
            for c in ch[r]:
                compare_child(rep, f"b{b}c{c}", z, q[r], toks[c], float(u[c, 0]),
                              float(u[c, 1]), w.T, w.top_p, int(g["accept"][b * n1 + c]),
                              int(g["resample_token"][b * n1 + c]))
        # the walk and prefix lengths follow exactly from the GPU's own decisions
        res = ov.RowResult(accept=g["accept"][b * n1:(b + 1) * n1].numpy(), acc_prefix_len=None,
                           resample=g["resample_token"][b * n1:(b + 1) * n1].numpy(),
                           bonus=g["bonus_token"][b * n1:(b + 1) * n1].numpy(), topk_ids=None,
                           topk_probs=None, nucleus_size=None)
        wr = ov.walk(toks, pars, res)
        gl = int(g["path_len"][b])
        gp = g["path"][b].numpy().tolist()
        assert gl == len(wr.path), (b, gl, wr.path)
        assert gp[:gl] == wr.path and all(x == -1 for x in gp[gl:]), (b, gp, wr.path)
        assert int(g["next_token"][b]) == wr.next_token, (b, int(g["next_token"][b]), wr)
        assert int(g["sibling_hit"][b]) == int(wr.sibling_hit)
        # acc_prefix_len from the GPU accept bits
        depth = om.tree_depths(pars)
        acc = [0] * n1
        for r in range(1, n1):
            p_ = pars[r]
            acc[r] = acc[p_] + 1 if (acc[p_] == depth[p_] and res.accept[r]) else acc[p_]
        assert g["acc_prefix_len"][b * n1:(b + 1) * n1].tolist() == acc
        assert int(g["accept"][b * n1]) == 1 and int(g["resample_token"][b * n1]) == -1
        assert int(g["status"][b]) == 0
    return rep
