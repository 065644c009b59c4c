"""Oracle vocabulary stage and path walk (float64) -- test infrastructure only.

Per tree row r (its logits z_r), the cloud reduces the target distribution to
what the downlink carries (Section III-B; Algorithm 1, RECEIVE_WAIT returns the
rejection index and a sparse target distribution), and per drafted child n of
r it runs the speculative acceptance test of Chen et al. (cited in Section II:
the output law stays that of the target model):

  V1  p~ = softmax(z_r / T)                     (temperature, T > 0)
  V2  sigma = ids sorted by (p~ desc, id asc); m = first index where the
      running sum reaches top_p; nucleus = sigma[0..m] (crossing token kept);
      p_r = p~ renormalised on the nucleus, 0 elsewhere          (top-p)
  V3  top-k payload: ids sigma[0..k-1], probs p_r(ids) / sum p_r(ids)
  V4  bonus[r] = inverse CDF of p_r in id order at u[r, 2]
  V5  child n (token x, draft distribution Q = q[r]):
      accept[n] = u[n, 0] * Q(x) < p_r(x)   (i.e. u < min(1, p/q));
      resample[n] = inverse CDF of max(0, p_r - Q) at u[n, 1]
      (of p_r itself if that residual has no mass)
  V6  acc_prefix_len[n] = leading accepted nodes on the root-to-n path

Walk (Algorithm 1, after verification): from the root follow the main (lowest-index)
child while accepted; on a rejection the resampled token is looked up among
the other children (w = (pi, x_resampled) in dom(T)); a hit continues down
that sibling, a miss ends the path with the resampled token; a node without
children ends with its bonus token.

Inverse CDF: the smallest id j with C_j > u * S, C_j the running sum in id
order and S the total, so ids of zero mass are never chosen.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence

import numpy as np


# ----------------------------------------------------------------------------------------
# Per-row distribution
# ----------------------------------------------------------------------------------------


def tempered_softmax(z: np.ndarray, T: float) -> np.ndarray:
    """V1: softmax(z / T), max-subtracted, float64."""
    l = np.asarray(z, dtype=np.float64) / T
    e = np.exp(l - l.max())
    return e / e.sum()


def sorted_order(pt: np.ndarray) -> np.ndarray:
    """Ids by probability descending, ties by id ascending."""
    ids = np.arange(pt.shape[0])
    return np.lexsort((ids, -pt))


def nucleus(pt: np.ndarray, top_p: float, order: np.ndarray = None):
    """V2: returns (p_r, order, m) with p_r renormalised on the top-p nucleus."""
    if order is None:
        order = sorted_order(pt)
    cs = np.cumsum(pt[order])
    hit = np.nonzero(cs >= top_p)[0]
    m = int(hit[0]) if hit.size else pt.shape[0] - 1
    keep = order[: m + 1]
    p = np.zeros_like(pt)
    p[keep] = pt[keep] / pt[keep].sum()
    return p, order, m


def topk_payload(p: np.ndarray, order: np.ndarray, k: int):
    """V3: the k most probable ids (sigma order) and their renormalised probs."""
    ids = order[:k]
    head = p[ids]
    return ids.astype(np.int64), head / head.sum()


def inverse_cdf(w: np.ndarray, u: float) -> int:
    """Smallest j with C_j > u * sum(w), C the running sum of w in id order."""
    c = np.cumsum(np.asarray(w, dtype=np.float64))
    j = int(np.searchsorted(c, u * c[-1], side="right"))
    return min(j, w.shape[0] - 1)


def accept_token(p: np.ndarray, q: np.ndarray, x: int, u: float) -> bool:
    """V5: accept x ~ q with probability min(1, p(x)/q(x)), decided by u."""
    return bool(u * q[x] < p[x])


def residual_sample(p: np.ndarray, q: np.ndarray, u: float) -> int:
    """V5: inverse CDF of the normalised residual max(0, p - q) (of p if it has no mass)."""
    rho = np.maximum(p - q, 0.0)
    if rho.sum() > 0.0:
        return inverse_cdf(rho, u)
    return inverse_cdf(p, u)


# ----------------------------------------------------------------------------------------
# One session: all rows, then the walk
# ----------------------------------------------------------------------------------------


@dataclass
class RowResult:
    accept: np.ndarray          # [n] uint8
    acc_prefix_len: np.ndarray  # [n] int
    resample: np.ndarray        # [n] int (-1 on the root)
    bonus: np.ndarray           # [n] int
    topk_ids: np.ndarray        # [n, k]
    topk_probs: np.ndarray      # [n, k]
    nucleus_size: np.ndarray    # [n]


def children_of(parents: Sequence[int]) -> List[List[int]]:
    ch = [[] for _ in parents]
    for r, p in enumerate(parents):
        if p >= 0:
            ch[p].append(r)
    return ch


def verify_session(logits: np.ndarray, q: np.ndarray, tokens: Sequence[int],
                   parents: Sequence[int], u: np.ndarray, T: float, top_p: float,
                   k: int, rows: Sequence[int] = None) -> RowResult:
    """V1-V6 for one tree.  logits [n, V], q [n, V] (row r = draft dist of r's children),
    u [n, 3] = (accept, residual, bonus) uniforms.  ``rows`` limits which rows get their
    distribution computed (their children are still decided); default all."""
    n, V = logits.shape
    ch = children_of(parents)
    accept = np.zeros(n, dtype=np.uint8)
    accept[0] = 1
    resample = np.full(n, -1, dtype=np.int64)
    bonus = np.full(n, -1, dtype=np.int64)
    tk_ids = np.full((n, k), -1, dtype=np.int64)
    tk_probs = np.zeros((n, k))
    nsize = np.zeros(n, dtype=np.int64)
    rows = range(n) if rows is None else rows
    for r in rows:
        pt = tempered_softmax(logits[r], T)
        p, order, m = nucleus(pt, top_p)
        nsize[r] = m + 1
        tk_ids[r], tk_probs[r] = topk_payload(p, order, k)
        bonus[r] = inverse_cdf(p, float(u[r, 2]))
        for c in ch[r]:
            x = int(tokens[c])
            accept[c] = accept_token(p, q[r], x, float(u[c, 0]))
            resample[c] = residual_sample(p, q[r], float(u[c, 1]))
    acc = np.zeros(n, dtype=np.int64)
    depth = np.zeros(n, dtype=np.int64)
    for r in range(1, n):
        pr = parents[r]
        depth[r] = depth[pr] + 1
        full = acc[pr] == depth[pr]
        acc[r] = acc[pr] + 1 if (full and accept[r]) else acc[pr]
    return RowResult(accept, acc, resample, bonus, tk_ids, tk_probs, nsize)


@dataclass
class WalkResult:
    path: List[int]        # drafted rows kept, root-first (root itself not listed)
    next_token: int
    sibling_hit: bool


def walk(tokens: Sequence[int], parents: Sequence[int], res: RowResult) -> WalkResult:
    """The walk of Algorithm 1 on the GPU-side verification results of one tree."""
    ch = children_of(parents)
    cur, path, hit = 0, [], False
    while True:
        if not ch[cur]:
            return WalkResult(path, int(res.bonus[cur]), hit)
        c0 = ch[cur][0]
        if res.accept[c0]:
            cur = c0
            path.append(c0)
            continue
        r_star = int(res.resample[c0])
        sib = [c for c in ch[cur][1:] if int(tokens[c]) == r_star]
        if sib:
            cur = sib[0]
            hit = True
            path.append(cur)
            continue
        return WalkResult(path, r_star, hit)


# ----------------------------------------------------------------------------------------
# LM-head tail: each row is the parent of one drafted token, chains of chain_len rows
# ----------------------------------------------------------------------------------------


def verify_tail(logits: np.ndarray, q: np.ndarray, draft: Sequence[int], u: np.ndarray,
                T: float, top_p: float, k: int, chain_len: int, rows: Sequence[int] = None):
    """Per row: accept / resample of its one drafted token, bonus, top-k.
    Per chain of ``chain_len`` rows: kept length (leading accepts) and the next token
    (the resample at the first rejection; -1 when the whole chain is accepted, since the
    bonus then needs the row after the chain)."""
    R, V = logits.shape
    accept = np.zeros(R, dtype=np.uint8)
    resample = np.full(R, -1, dtype=np.int64)
    bonus = np.full(R, -1, dtype=np.int64)
    tk_ids = np.full((R, k), -1, dtype=np.int64)
    tk_probs = np.zeros((R, k))
    rows = range(R) if rows is None else rows
    for r in rows:
        pt = tempered_softmax(logits[r], T)
        p, order, m = nucleus(pt, top_p)
        tk_ids[r], tk_probs[r] = topk_payload(p, order, k)
        bonus[r] = inverse_cdf(p, float(u[r, 2]))
        x = int(draft[r])
        accept[r] = accept_token(p, q[r], x, float(u[r, 0]))
        resample[r] = residual_sample(p, q[r], float(u[r, 1]))
    return dict(accept=accept, resample=resample, bonus=bonus, topk_ids=tk_ids,
                topk_probs=tk_probs)


def walk_tail(accept: np.ndarray, resample: np.ndarray, chain_len: int):
    R = accept.shape[0]
    nb = R // chain_len
    path_len = np.zeros(nb, dtype=np.int64)
    nxt = np.full(nb, -1, dtype=np.int64)
    for b in range(nb):
        i = 0
        while i < chain_len and accept[b * chain_len + i]:
            i += 1
        path_len[b] = i
        nxt[b] = resample[b * chain_len + i] if i < chain_len else -1
    return path_len, nxt


# ---------------------------------------------------------------------------------------
# The paper's own protocol: scalar q-hat uplink, sparse downlink, edge-side resampling
# ---------------------------------------------------------------------------------------


def accept_scalar(p: np.ndarray, x: int, q_hat: float, u0: float) -> bool:
    """Acceptance of a drafted token from its draft probability alone (the uplink carries
    q(x) per drafted token, Algorithm 1): accept iff u0 * q_hat < p(x)."""
    return bool(u0 * q_hat < p[x])


def edge_resample(ids, probs, q: np.ndarray, u: float, rejected: bool = True) -> int:
    """RESAMPLE(P_hat, Q) of Algorithm 1 on the edge, from the cloud's k-sparse payload.

    After a rejection the corrected token follows max(0, P_hat - Q) over the payload's ids
    (P_hat if that is all zero); after full acceptance it follows P_hat.  Inverse CDF in
    ascending id order, first running mass strictly above u times the total."""
    pairs = sorted(zip([int(i) for i in ids], [float(p) for p in probs]))
    weights = []
    for i, p in pairs:
        weights.append(max(p - float(q[i]), 0.0) if rejected else p)
    if sum(weights) <= 0.0:
        weights = [p for _, p in pairs]
    total = sum(weights)
    run = 0.0
    for (i, _), w in zip(pairs, weights):
        run += w
        if w > 0.0 and run > u * total:
            return i
    return [i for (i, _), w in zip(pairs, weights) if w > 0.0][-1]


def exact_residual_law(p: np.ndarray, q: np.ndarray) -> np.ndarray:
    """The law of the exact residual resample over the whole vocabulary."""
    r = np.maximum(p - q, 0.0)
    return r / r.sum() if r.sum() > 0 else p / p.sum()
