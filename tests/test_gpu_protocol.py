"""GPU parity of the paper's own protocol (scalar q-hat uplink, no cloud-side sampling,
edge-side resampling from the k-sparse payload; Section III-B, Algorithm 1)."""
import numpy as np
import pytest
import torch

import synth
from oracle import verify as ov
from paper_2609_02514_amd import edge
from tests import harness as hz
from tests.test_gpu_parity import small_bf16

pytestmark = pytest.mark.gpu


def _q_hat(batch):
    """q_hat[b, r] = draft probability of row r's token under its parent's distribution
    (the uplink's one float per drafted node); row 0 unused."""
    B = batch.tokens.shape[0]
    par = batch.parents.long().clamp(min=0)
    tok = batch.tokens.long()
    qpar = batch.q[torch.arange(B, device=batch.q.device)[:, None], par]        # [B, n1, V]
    q_hat = qpar.gather(2, tok.unsqueeze(-1)).squeeze(-1).contiguous()
    q_hat[:, 0] = 0.0
    return q_hat


def _scalar_run(w, seed=None):
    """Dense and scalar-q-hat verify steps on the same seeded inputs."""
    from paper_2609_02514_amd.acespec import Verifier
    seed = w.seed_base if seed is None else seed
    W = synth.make_weights(w, "cuda", seed)
    batch = synth.make_batch(w, "cuda", seed)
    B, n1 = batch.tokens.shape
    q_hat = _q_hat(batch)
    v = Verifier.for_workload(w)
    ws = v.weights_struct(W)
    od = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, "cuda", True)
    osq = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, "cuda", True)
    hz.log(f"dense and scalar-q verify {w.name} B={B} N={n1 - 1} seed={seed}")
    v.verify_tree(ws, batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len, batch.tokens,
                  batch.parents, batch.q, batch.u, w.T, w.top_p, w.top_k, od)
    v.verify_tree_scalar_q(ws, batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len,
                           batch.tokens, batch.parents, q_hat, batch.u, w.T, w.top_p, w.top_k,
                           osq)
    torch.cuda.synchronize()
    gd = {k: hz.host(t) for k, t in od.items()}
    gs = {k: hz.host(t) for k, t in osq.items()}
    v.close()
    hin = dict(tokens=hz.host(batch.tokens), parents=hz.host(batch.parents),
               prefix_len=hz.host(batch.prefix_len), q=hz.host(batch.q), u=hz.host(batch.u))
    run = hz.TreeRun(w, W, batch, gs, hin, [])
    return run, gd, gs, hz.host(q_hat).numpy().astype(np.float64)


def _check_scalar_against_oracle(run, gs, q_hat):
    """Scalar mode's accept (u0 q_hat < p(x)), top-k payload and walk against the oracle's
    accept_scalar / nucleus / topk_payload on the GPU's logits (Section III-B; Algorithm 1):
    every row of every session; no cloud-side samples (resample, bonus, next token -1)."""
    w = run.w
    B, n1 = run.host_in["tokens"].shape
    zl = gs["logits_out"].numpy()
    g = {k: t.numpy() for k, t in gs.items()}
    rep = hz.check_rows(hz.tree_jobs(run, lambda b: zl[b * n1:(b + 1) * n1], range(B),
                                     q_hat=q_hat), g, w.T, w.top_p, w.top_k, scalar=True)
    hz.log(f"scalar-q decisions vs oracle (all {B} sessions): {rep}")
    assert rep.ok(), str(rep)
    hz.check_tree_walk(run, range(B), scalar=True)
    assert (gs["resample_token"] == -1).all() and (gs["bonus_token"] == -1).all()
    assert (gs["next_token"] == -1).all() and (gs["sibling_hit"] == 0).all()


def test_scalar_q_decisions_and_edge_resample():
    w = small_bf16(B=6, ragged=True)
    run, gd, gs, q_hat = _scalar_run(w)
    _check_scalar_against_oracle(run, gs, q_hat)
    # the same forward: identical logits and payload, and (q_hat being the dense row's own
    # float) identical accept bits to the dense mode
    for k in ("logits_out", "accept", "acc_prefix_len", "topk_ids", "topk_probs", "status"):
        assert torch.equal(gd[k], gs[k]), k
    B, n1 = run.host_in["tokens"].shape
    q_h, u_h = run.host_in["q"], run.host_in["u"]
    tvs = []
    for b in range(B):
        toks = run.host_in["tokens"][b].tolist()
        pars = run.host_in["parents"][b].tolist()
        res = ov.RowResult(accept=gs["accept"][b * n1:(b + 1) * n1].numpy(), acc_prefix_len=None,
                           resample=gs["resample_token"][b * n1:(b + 1) * n1].numpy(),
                           bonus=gs["bonus_token"][b * n1:(b + 1) * n1].numpy(), topk_ids=None,
                           topk_probs=None, nucleus_size=None)
        wr = ov.walk(toks, pars, res)
        # edge: resample at the row where the walk stopped
        cur = wr.path[-1] if wr.path else 0
        kids = ov.children_of(pars)[cur]
        rejected = bool(kids)
        u = float(u_h[b, kids[0], 1]) if rejected else float(u_h[b, cur, 2])
        row = b * n1 + cur
        ids, probs = gs["topk_ids"][row].numpy(), gs["topk_probs"][row].numpy()
        qrow = q_h[b, cur].numpy().astype(np.float64)
        t_edge = edge.resample(ids, probs, qrow, u, rejected)
        assert t_edge == ov.edge_resample(ids, probs.astype(np.float64), qrow, u, rejected)
        # gap to the exact residual (informational; zero when the payload covers the nucleus)
        pt = ov.tempered_softmax(gs["logits_out"][row].numpy().astype(np.float64), w.T)
        p, _, _ = ov.nucleus(pt, w.top_p)
        exact = ov.exact_residual_law(p, qrow) if rejected else p / p.sum()
        sid, sw = edge.residual_law(ids, probs, qrow, rejected)
        sparse = np.zeros_like(exact)
        sparse[sid] = sw
        tvs.append(0.5 * np.abs(sparse - exact).sum())
    hz.log(f"edge resample vs exact residual: total variation mean {np.mean(tvs):.3f} "
           f"max {np.max(tvs):.3f} (top-k {w.top_k} of vocab {w.V})")
    assert all(0.0 <= t <= 1.0 + 1e-9 for t in tvs)


@pytest.mark.timeout(900)
def test_scalar_q_8b_full_size():
    """The scalar-q-hat protocol at the 8B workload's full size: every row of all 64
    sessions against the oracle (its forward is covered by the dense-mode parity tests on
    the same seeds: both modes share the forward, checked identical here)."""
    w = synth.get("8b-bf16")
    run, gd, gs, q_hat = _scalar_run(w)
    for k in ("logits_out", "topk_ids", "topk_probs", "status"):
        assert torch.equal(gd[k], gs[k]), k
    _check_scalar_against_oracle(run, gs, q_hat)
