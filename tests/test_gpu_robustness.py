"""Data errors found on the device are reported per session and leave the other sessions
untouched (bitwise): NaN / infinite / negative draft probabilities (ACESPEC_EBADDRAFT),
and target logits that are not finite (ACESPEC_ENONFINITE) -- an activation that left the
fp16 range it is handed on in, or NaN/inf in the caller's cache or hidden states."""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from paper_2609_02514_amd import acespec as A
from tests import harness as hz
from tests.test_gpu_parity import small_bf16

pytestmark = pytest.mark.gpu


def _verify(v, ws, batch, w, q=None, kv_v=None, scalar_q=None):
    B, n1 = batch.tokens.shape
    outs = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, "cuda", True)
    args = (ws, batch.kv_k, batch.kv_v if kv_v is None else kv_v, batch.cap, batch.prefix_len,
            batch.tokens, batch.parents)
    if scalar_q is None:
        v.verify_tree(*args, batch.q if q is None else q, batch.u, w.T, w.top_p, w.top_k, outs)
    else:
        v.verify_tree_scalar_q(*args, scalar_q, batch.u, w.T, w.top_p, w.top_k, outs)
    torch.cuda.synchronize()
    return {k: (t.cpu() if t is not None else None) for k, t in outs.items()}


def _same_sessions(a, b, sessions, n1):
    """Every output of the given sessions is bitwise identical in the two runs."""
    for s in sessions:
        rows = slice(s * n1, (s + 1) * n1)
        for k in ("accept", "acc_prefix_len", "resample_token", "bonus_token", "topk_ids",
                  "topk_probs", "logits_out"):
            assert torch.equal(a[k][rows], b[k][rows]), (s, k)
        for k in ("path", "path_len", "next_token", "sibling_hit", "status"):
            assert torch.equal(a[k][s], b[k][s]), (s, k)


def _setup(**kw):
    w = small_bf16(B=4, ragged=False, **kw)
    W = synth.make_weights(w, "cuda")
    batch = synth.make_batch(w, "cuda")
    v = A.Verifier.for_workload(w)
    return w, W, batch, v, v.weights_struct(W)


def test_bad_draft_distribution_flags_only_its_session():
    w, W, batch, v, ws = _setup()
    B, n1 = batch.tokens.shape
    ch = synth.children_lists(batch.parents[0].tolist())
    leaf = next(r for r in range(n1) if not ch[r])
    clean = _verify(v, ws, batch, w)
    assert clean["status"].tolist() == [0] * B
    q = batch.q.clone()
    q[1, 0, 5] = float("nan")         # the root row's draft distribution: read
    q[2, 1, 7] = -0.25                # a parent row: read
    q[3, leaf, 9] = float("nan")      # a leaf row: never read, nothing to report
    bad = _verify(v, ws, batch, w, q=q)
    hz.log(f"status {bad['status'].tolist()}")
    assert bad["status"].tolist() == [0, A.ACESPEC_EBADDRAFT, A.ACESPEC_EBADDRAFT, 0]
    _same_sessions(clean, bad, [0, 3], n1)
    q = batch.q.clone()
    q[0, 0, 11] = float("inf")
    assert _verify(v, ws, batch, w, q=q)["status"].tolist() == [A.ACESPEC_EBADDRAFT, 0, 0, 0]
    v.close()


def test_bad_scalar_q_hat_flags_only_its_session():
    w, W, batch, v, ws = _setup()
    B, n1 = batch.tokens.shape
    q_hat = torch.full((B, n1), 0.25, dtype=torch.float32, device="cuda")
    clean = _verify(v, ws, batch, w, scalar_q=q_hat)
    assert clean["status"].tolist() == [0] * B
    q_hat[1, 3] = 1.5
    q_hat[2, 4] = float("nan")
    bad = _verify(v, ws, batch, w, scalar_q=q_hat)
    assert bad["status"].tolist() == [0, A.ACESPEC_EBADDRAFT, A.ACESPEC_EBADDRAFT, 0]
    _same_sessions(clean, bad, [0, 3], n1)
    v.close()


def test_nonfinite_cache_entry_flags_only_its_session():
    """A value of 1e6 in one session's bf16 cache prefix has no fp16 counterpart (max
    65504): its attention output, and from there every logit of the session, is not
    finite.  The session reports ACESPEC_ENONFINITE, the others are unchanged."""
    w, W, batch, v, ws = _setup()
    B, n1 = batch.tokens.shape
    clean = _verify(v, ws, batch, w)
    kv_v = batch.kv_v.clone()
    kv_v[0, 2, 0, 5, 17] = 1.0e6      # layer 0, session 2, kv head 0, head dim 5, slot 17
    bad = _verify(v, ws, batch, w, kv_v=kv_v)
    hz.log(f"status {bad['status'].tolist()}")
    assert bad["status"].tolist() == [0, 0, A.ACESPEC_ENONFINITE, 0]
    _same_sessions(clean, bad, [0, 1, 3], n1)
    # the flagged session's rows carry no decisions
    rows = slice(2 * n1, 3 * n1)
    assert (bad["bonus_token"][rows] == -1).all() and (bad["topk_ids"][rows] == -1).all()
    assert (bad["accept"][2 * n1 + 1:3 * n1] == 0).all()
    v.close()


def test_activation_overflow_flags_every_session():
    """RMSNorm gains of 1e5 push the normalised activations past the fp16 range in every
    row: every session reports ACESPEC_ENONFINITE (and no decision is taken on them)."""
    w, W, batch, v, _ = _setup()
    layers = [dict(l) for l in W.layers]
    layers[0]["attn_norm"] = (layers[0]["attn_norm"].float() * 1e5).to(torch.bfloat16)
    ws = v.weights_struct(dataclasses.replace(W, layers=layers))
    bad = _verify(v, ws, batch, w)
    assert bad["status"].tolist() == [A.ACESPEC_ENONFINITE] * w.B
    v.close()


def test_tail_hidden_overflow_flags_only_its_chain():
    """LM-head tail without a final norm: bf16 hidden values beyond the fp16 range (here
    1e5) in one chain flag that chain; with a final norm the rows are normalised first and
    stay finite."""
    w = synth.get("8b-lmhead-tail").scaled(name="tail-ovf", d=256, V=5004, rows=64,
                                          chain_len=8, top_k=16)
    W = synth.make_weights(w, "cuda")
    batch = synth.make_batch(w, "cuda", weights=W)
    v = A.Verifier.for_workload(w)
    R, nch = w.rows, w.rows // w.chain_len

    def tail(hidden, final_norm=None):
        outs = v.alloc_outputs(R, nch, w.chain_len, w.top_k, w.V, "cuda", True)
        v.verify_tail(W.lm_head, final_norm, hidden, batch.draft_tokens, batch.q, batch.u,
                      w.chain_len, w.T, w.top_p, w.top_k, outs)
        torch.cuda.synchronize()
        return {k: (t.cpu() if t is not None else None) for k, t in outs.items()}

    clean = tail(batch.hidden)
    hidden = batch.hidden.clone()
    hidden[3 * w.chain_len + 2, 10] = 1.0e5
    bad = tail(hidden)
    assert bad["status"].tolist() == [0, 0, 0, A.ACESPEC_ENONFINITE] + [0] * (nch - 4)
    for c in [0, 1, 2, 4, 5, 6, 7]:
        rows = slice(c * w.chain_len, (c + 1) * w.chain_len)
        for k in ("accept", "resample_token", "bonus_token", "topk_ids", "logits_out"):
            assert torch.equal(clean[k][rows], bad[k][rows]), (c, k)
    normed = tail(hidden, final_norm=torch.ones(w.d, dtype=torch.bfloat16, device="cuda"))
    assert normed["status"].tolist() == [0] * nch
    v.close()
