"""Pins for the CPU oracle: each test checks it against something other than itself.

* forward: an independent library implementation of a Llama decoder (transformers'
  LlamaForCausalLM, eager attention, fed the ancestor mask as a 4D attention mask and
  the KV prefix as its cache), torch's RMSNorm, the complex-number form of RoPE, and
  the token-by-token causal twin (tree mask on a chain == causal mask; every tree row ==
  a causal decode of its root-to-node path, Section III-C).
* verify: hand vectors (tests/golden/hand_vectors.json), brute force on tiny vocabularies,
  numpy's searchsorted, the exactness theorem of speculative sampling (output law == the
  target law, Chen et al., cited in Section II) driven through the oracle's own code on
  a midpoint grid, and a Monte Carlo law check of the walk with sibling hits
  (Algorithm 1).
"""
import json
import os

import numpy as np
import pytest
import torch

import synth
from oracle import model as om
from oracle import verify as ov

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_vectors.json")))


def tiny_workload(**kw):
    base = dict(name="pin", dtype="f32", L=2, d=64, H=4, Hkv=2, hd=16, F=96, V=50, B=2, S=7,
                tree="chain_sib", depth=3, sib=1, q_std=2.0, q_T=0.8, T=0.8, top_p=0.9,
                top_k=8, tokens="uniform", random_gains=True, seed_base=77)
    base.update(kw)
    return synth.Workload(**base)


# ---------------------------------------------------------------------------------------
# Building blocks
# ---------------------------------------------------------------------------------------


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 32))
    g = rng.standard_normal(32)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (32,), torch.tensor(g), eps=1e-5)
    np.testing.assert_allclose(om.rms_norm(x, g, 1e-5), ref.numpy(), rtol=1e-13, atol=1e-13)


def test_rope_complex_form_and_relative_position():
    rng = np.random.default_rng(1)
    hd, base = 16, 10000.0
    x = rng.standard_normal((3, 2, hd))
    pos = np.array([0, 5, 1234])
    cos, sin = om.rope_cos_sin(pos, hd, base)
    y = om.apply_rope(x, cos, sin)
    # complex form: z_i = x_i + j x_{i+hd/2} multiplied by exp(j pos theta_i)
    h = hd // 2
    theta = base ** (-np.arange(h) * 2.0 / hd)
    z = (x[..., :h] + 1j * x[..., h:]) * np.exp(1j * pos[:, None, None] * theta[None, None, :])
    np.testing.assert_allclose(y[..., :h], z.real, atol=1e-12)
    np.testing.assert_allclose(y[..., h:], z.imag, atol=1e-12)
    # position 0 is the identity; dot products depend on the position difference only
    np.testing.assert_allclose(y[0], x[0], atol=1e-15)
    q, k = rng.standard_normal((1, 1, hd)), rng.standard_normal((1, 1, hd))

    def dot(m, n):
        cm, sm = om.rope_cos_sin(np.array([m]), hd, base)
        cn, sn = om.rope_cos_sin(np.array([n]), hd, base)
        return float(np.sum(om.apply_rope(q, cm, sm) * om.apply_rope(k, cn, sn)))

    assert abs(dot(10, 3) - dot(110, 103)) < 1e-10


def test_tree_helpers():
    parents = [-1, 0, 0, 1, 1, 3]
    assert om.tree_depths(parents) == [0, 1, 1, 2, 2, 3]
    anc = om.ancestor_matrix(parents)
    assert anc[5].tolist() == [True, True, False, True, False, True]
    assert om.path_to(parents, 5) == [0, 1, 3, 5]
    assert om.validate_tree(parents, [0] * 6, 10)
    assert not om.validate_tree([-1, 0, 2], [0] * 3, 10)      # forward reference
    assert not om.validate_tree([-1, 0, 1], [0, 0, 10], 10)   # token out of range
    assert not om.validate_tree([0, 0, 1], [0] * 3, 10)       # root with a parent


# ---------------------------------------------------------------------------------------
# Forward: tree mask semantics
# ---------------------------------------------------------------------------------------


def _session(w, b=0, seed=None):
    W = synth.make_weights(w, "cpu", seed)
    batch = synth.make_batch(w, "cpu", seed)
    S = int(batch.prefix_len[b])
    kp, vp = om.session_prefix(batch.kv_k, batch.kv_v, b, S)
    toks = [int(t) for t in batch.tokens[b]]
    pars = [int(p) for p in batch.parents[b]]
    return W, batch, S, kp, vp, toks, pars


def test_chain_tree_equals_causal_decode():
    w = tiny_workload(tree="chain", depth=5)
    W, batch, S, kp, vp, toks, pars = _session(w)
    dims = om.dims_of(w)
    F = om.F64Weights(W)
    z = om.forward_tree_session(F, dims, kp, vp, toks, pars, S)
    for r in range(len(toks)):
        ref = om.forward_causal_path(F, dims, kp, vp, toks[: r + 1], S)
        np.testing.assert_allclose(z[r], ref, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("tree,depth,sib", [("chain_sib", 3, 2), ("widths_2455", 4, 0)])
def test_tree_rows_equal_per_path_decode(tree, depth, sib):
    w = tiny_workload(tree=tree, depth=depth, sib=sib, tokens="draft")
    W, batch, S, kp, vp, toks, pars = _session(w, b=1)
    dims = om.dims_of(w)
    F = om.F64Weights(W)
    z = om.forward_tree_session(F, dims, kp, vp, toks, pars, S)
    for r in range(len(toks)):
        path = om.path_to(pars, r)
        ref = om.forward_causal_path(F, dims, kp, vp, [toks[i] for i in path], S)
        np.testing.assert_allclose(z[r], ref, rtol=1e-11, atol=1e-12)


def _hf_model(w, W):
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(vocab_size=w.V, hidden_size=w.d, intermediate_size=w.F,
                      num_hidden_layers=w.L, num_attention_heads=w.H,
                      num_key_value_heads=w.Hkv, head_dim=w.hd, rms_norm_eps=w.rms_eps,
                      rope_theta=w.rope_base, max_position_embeddings=4096,
                      tie_word_embeddings=False, attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "eager"
    m = LlamaForCausalLM(cfg).to(torch.float64).eval()
    Hd, KVd = w.H * w.hd, w.Hkv * w.hd
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(W.embed.double())
        for l, lw in enumerate(W.layers):
            blk = m.model.layers[l]
            wqkv = lw["wqkv"].double()
            blk.self_attn.q_proj.weight.copy_(wqkv[:Hd])
            blk.self_attn.k_proj.weight.copy_(wqkv[Hd:Hd + KVd])
            blk.self_attn.v_proj.weight.copy_(wqkv[Hd + KVd:])
            blk.self_attn.o_proj.weight.copy_(lw["wo"].double())
            blk.input_layernorm.weight.copy_(lw["attn_norm"].double())
            blk.post_attention_layernorm.weight.copy_(lw["mlp_norm"].double())
            gu = lw["w_gate_up"].double()
            blk.mlp.gate_proj.weight.copy_(gu[: w.F])
            blk.mlp.up_proj.weight.copy_(gu[w.F:])
            blk.mlp.down_proj.weight.copy_(lw["w_down"].double())
        m.model.norm.weight.copy_(W.final_norm.double())
        m.lm_head.weight.copy_(W.lm_head.double())
    return m


@pytest.mark.parametrize("tree,depth,sib", [("chain_sib", 3, 1), ("widths_2455", 4, 0)])
def test_tree_forward_matches_transformers_llama(tree, depth, sib):
    """Library pin: HF Llama with a 4D ancestor mask, positions S+depth and the prefix cache."""
    from transformers import DynamicCache
    w = tiny_workload(tree=tree, depth=depth, sib=sib, tokens="draft")
    W, batch, S, kp, vp, toks, pars = _session(w)
    dims = om.dims_of(w)
    z = om.forward_tree_session(om.F64Weights(W), dims, kp, vp, toks, pars, S)
    m = _hf_model(w, W)
    n = len(toks)
    cache = DynamicCache()
    for l in range(w.L):
        cache.update(torch.tensor(kp[l])[None], torch.tensor(vp[l])[None], l)
    anc = torch.tensor(om.ancestor_matrix(pars))
    allowed = torch.cat([torch.ones(n, S, dtype=torch.bool), anc], dim=1)
    mask = torch.zeros(1, 1, n, S + n, dtype=torch.float64)
    mask[0, 0][~allowed] = float("-inf")
    pos = torch.tensor([[S + d for d in om.tree_depths(pars)]])
    with torch.no_grad():
        out = m(torch.tensor([toks]), past_key_values=cache, position_ids=pos,
                attention_mask=mask, use_cache=False).logits[0].numpy()
    # transformers evaluates RoPE angles, RMSNorm and the softmax in fp32 internally
    err = np.abs(out - z).max() / np.abs(z).max()
    assert err < 2e-5, err


# ---------------------------------------------------------------------------------------
# Verify stage
# ---------------------------------------------------------------------------------------


def test_top_p_hand_vectors():
    for key in ("top_p", "top_p_ties"):
        g = GOLD[key]
        pt = ov.tempered_softmax(np.log(g["p_tilde"]), 1.0)
        p, order, m = ov.nucleus(pt, g["top_p"])
        np.testing.assert_allclose(p, g["expect_p"], atol=1e-12)
    # a running sum that lands exactly on top_p closes the nucleus there
    g = GOLD["top_p_exact_boundary"]
    p, order, m = ov.nucleus(np.array(g["p_tilde"]), g["top_p"])
    np.testing.assert_allclose(p, g["expect_p"], atol=1e-15)


def test_temperature_hand_vectors():
    """The logits are divided by T before the softmax (Section III-B): at T = 1/2 the
    tempered distribution is the square of the untempered one renormalised, at T = 2 its
    square root; the nucleus and the top-k payload follow from the tempered values."""
    g = GOLD["temperature"]
    z = np.array(g["z"])
    for c in g["cases"]:
        pt = ov.tempered_softmax(z, c["T"])
        np.testing.assert_allclose(pt, c["expect_p_tilde"], rtol=1e-12)
        p, order, m = ov.nucleus(pt, c["top_p"])
        np.testing.assert_allclose(p, c["expect_p"], rtol=1e-12, atol=1e-15)
        ids, probs = ov.topk_payload(p, order, 2)
        assert ids.tolist() == [0, 1]
        np.testing.assert_allclose(probs, np.array(c["expect_p"])[:2], rtol=1e-12)


def test_accept_residual_hand_vector():
    g = GOLD["accept_residual"]
    p, q = np.array(g["p"]), np.array(g["q"])
    M = 1000
    grid = (np.arange(M) + 0.5) / M
    for x in range(4):
        frac = np.mean([ov.accept_token(p, q, x, u) for u in grid])
        assert abs(frac - g["accept_prob"][x]) <= 1.0 / M
    res = [ov.residual_sample(p, q, u) for u in grid]
    np.testing.assert_allclose(np.bincount(res, minlength=4) / M, g["residual"], atol=1e-12)
    assert abs(np.minimum(p, q).sum() - g["beta"]) < 1e-12


def test_inverse_cdf_hand_vector_and_searchsorted():
    g = GOLD["inverse_cdf"]
    for u, j in g["cases"]:
        assert ov.inverse_cdf(np.array(g["w"]), u) == j
    rng = np.random.default_rng(3)
    for _ in range(200):
        w = rng.random(17) * (rng.random(17) < 0.6)
        if w.sum() == 0:
            continue
        u = rng.random()
        j = ov.inverse_cdf(w, u)
        assert w[j] > 0
        assert j == np.searchsorted(np.cumsum(w), u * w.sum(), side="right")


def _brute_nucleus(pt, top_p):
    idx = sorted(range(len(pt)), key=lambda i: (-pt[i], i))
    acc, keep = 0.0, []
    for i in idx:
        keep.append(i)
        acc += pt[i]
        if acc >= top_p:
            break
    return idx, keep


def test_nucleus_and_topk_brute_force():
    rng = np.random.default_rng(4)
    for trial in range(300):
        V = int(rng.integers(2, 12))
        z = np.round(rng.standard_normal(V) * 2, 1)          # coarse values -> exact ties
        T = float(rng.choice([0.5, 1.0, 1.7]))
        top_p = float(rng.choice([0.3, 0.8, 0.95, 1.0]))
        k = int(rng.integers(1, V + 1))
        pt = ov.tempered_softmax(z, T)
        p, order, m = ov.nucleus(pt, top_p)
        idx, keep = _brute_nucleus(list(pt), top_p)
        assert list(order) == idx
        assert sorted(np.nonzero(p)[0].tolist()) == sorted(keep)
        assert abs(p.sum() - 1.0) < 1e-12
        ids, probs = ov.topk_payload(p, order, k)
        assert list(ids) == idx[:k]
        head = p[ids]
        np.testing.assert_allclose(probs, head / head.sum(), atol=1e-14)
        if top_p == 1.0:
            # without truncation the payload is the renormalised head of the full distribution
            np.testing.assert_allclose(probs, pt[ids] / pt[ids].sum(), atol=1e-12)
        # the top-k ids are the k largest logits
        assert set(np.argsort(-z, kind="stable")[:k]) == set(ids.tolist()) or \
            len(set(np.round(z, 6))) < V


def test_speculative_sampling_is_exact_on_vocab8():
    """Output law of accept-or-resample equals the target: the oracle's own accept and
    residual code, integrated on a midpoint grid of M uniforms, is within 2/M of p."""
    rng = np.random.default_rng(5)
    M = 400
    grid = (np.arange(M) + 0.5) / M
    for trial in range(10):
        z = rng.standard_normal(8) * 2
        p, _, _ = ov.nucleus(ov.tempered_softmax(z, 0.8), 0.9)
        q = rng.dirichlet(np.ones(8) * 0.7)
        q[rng.integers(0, 8)] = 0.0   # a token the draft never proposes
        q /= q.sum()
        acc = np.array([np.mean([ov.accept_token(p, q, x, u) for u in grid]) for x in range(8)])
        res = np.bincount([ov.residual_sample(p, q, u) for u in grid], minlength=8) / M
        out = np.zeros(8)
        for x in range(8):
            out[x] += q[x] * acc[x]
            out += q[x] * (1 - acc[x]) * res
        assert np.abs(out - p).max() <= 2.0 / M, (out, p)
        # exact closed form of the same law
        a = np.minimum(1.0, np.divide(p, q, out=np.ones(8), where=q > 0))
        rho = np.maximum(p - q, 0)
        exact = q * a + (q * (1 - a)).sum() * rho / rho.sum()
        np.testing.assert_allclose(exact, p, atol=1e-12)


def test_rejected_resample_never_equals_draft_token():
    rng = np.random.default_rng(6)
    for _ in range(500):
        V = 10
        p, _, _ = ov.nucleus(ov.tempered_softmax(rng.standard_normal(V) * 2, 1.0), 0.9)
        q = rng.dirichlet(np.ones(V))
        x = int(rng.choice(V, p=q))
        u0, u1 = rng.random(2)
        if not ov.accept_token(p, q, x, u0):
            assert ov.residual_sample(p, q, u1) != x
            assert p[x] < q[x]


def test_acceptance_rate_matches_sum_min():
    rng = np.random.default_rng(7)
    V = 30
    p, _, _ = ov.nucleus(ov.tempered_softmax(rng.standard_normal(V) * 1.5, 0.8), 0.9)
    q = rng.dirichlet(np.ones(V))
    n = 40000
    xs = rng.choice(V, size=n, p=q)
    us = rng.random(n)
    rate = np.mean([ov.accept_token(p, q, int(x), u) for x, u in zip(xs, us)])
    beta = np.minimum(p, q).sum()
    assert abs(rate - beta) < 4 * np.sqrt(beta * (1 - beta) / n)


def test_walk_with_sibling_hits_reproduces_target_law():
    """Monte Carlo over drafted trees and uniforms: the first two emitted tokens follow the
    target's joint law even though sibling hits reuse drafted branches."""
    rng = np.random.default_rng(8)
    V = 5
    p0 = rng.dirichlet(np.ones(V))                       # target at the root
    p1 = rng.dirichlet(np.ones(V), size=V)               # target after token a
    q0 = rng.dirichlet(np.ones(V))                       # draft at the root
    q1 = rng.dirichlet(np.ones(V), size=V)
    parents = [-1, 0, 0, 0, 1, 1, 2]                      # root: main + 2 siblings; two subtrees
    ch = ov.children_of(parents)
    n_trials = 30000
    first = np.zeros(V)
    second = np.zeros((V, V))
    hits = 0
    for t in range(n_trials):
        tok = [0] * len(parents)
        main = int(rng.choice(V, p=q0))
        sibs = [i for i in np.argsort(-q0, kind="stable") if i != main][:2]
        tok[1], tok[2], tok[3] = main, int(sibs[0]), int(sibs[1])
        for r in (1, 2):
            a = tok[r]
            c = ch[r]
            m2 = int(rng.choice(V, p=q1[a]))
            tok[c[0]] = m2
            for cc, s in zip(c[1:], [i for i in np.argsort(-q1[a], kind="stable") if i != m2]):
                tok[cc] = int(s)
        logits = np.zeros((len(parents), V))
        q = np.zeros((len(parents), V))
        logits[0], q[0] = np.log(p0), q0
        for r in range(1, len(parents)):
            if om.tree_depths(parents)[r] == 1:
                logits[r], q[r] = np.log(p1[tok[r]]), q1[tok[r]]
            else:
                logits[r], q[r] = np.log(np.full(V, 1.0 / V)), np.full(V, 1.0 / V)
        u = rng.random((len(parents), 3))
        res = ov.verify_session(logits, q, tok, parents, u, T=1.0, top_p=1.0, k=2)
        wr = ov.walk(tok, parents, res)
        emitted = [tok[r] for r in wr.path] + [wr.next_token]
        hits += wr.sibling_hit
        first[emitted[0]] += 1
        if len(emitted) >= 2:
            second[emitted[0], emitted[1]] += 1
    f = first / n_trials
    tol = 5 * np.sqrt(p0 * (1 - p0) / n_trials) + 1e-3
    assert np.all(np.abs(f - p0) < tol), (f, p0)
    for a in range(V):
        na = second[a].sum()
        if na < 2000:
            continue
        emp = second[a] / na
        tol = 5 * np.sqrt(p1[a] * (1 - p1[a]) / na) + 1e-3
        assert np.all(np.abs(emp - p1[a]) < tol), (a, emp, p1[a])
    assert hits > 0.05 * n_trials


def test_acc_prefix_len_and_walk_on_hand_tree():
    parents = [-1, 0, 0, 1, 1, 3]
    tokens = [9, 1, 2, 3, 4, 5]
    res = ov.RowResult(accept=np.array([1, 1, 0, 0, 1, 1], dtype=np.uint8),
                       acc_prefix_len=None, resample=np.array([-1, 7, 7, 4, 8, 8]),
                       bonus=np.array([11, 12, 13, 14, 15, 16]), topk_ids=None,
                       topk_probs=None, nucleus_size=None)
    wr = ov.walk(tokens, parents, res)
    # root -> main child 1 accepted; at 1 main child 3 rejected, resample 4 == token of
    # sibling 4 -> hit; node 4 has no children -> bonus of 4
    assert wr.path == [1, 4] and wr.next_token == 15 and wr.sibling_hit
    # acc_prefix_len through verify_session on a contrived distribution
    V = 6
    logits = np.log(np.full((6, V), 1.0 / V))
    q = np.full((6, V), 1.0 / V)
    u = np.full((6, 3), 0.5)
    r = ov.verify_session(logits, q, [0, 1, 2, 3, 4, 5], parents, u, 1.0, 1.0, 3)
    assert r.accept.tolist() == [1] * 6           # p == q accepts everything
    assert r.acc_prefix_len.tolist() == [0, 1, 1, 2, 2, 3]


def test_tail_equals_chain_session():
    rng = np.random.default_rng(9)
    V, n = 40, 6
    logits = rng.standard_normal((n, V)) * 2
    q = rng.dirichlet(np.ones(V), size=n)
    draft = [int(rng.choice(V, p=q[i])) for i in range(n)]
    u = rng.random((n, 3))
    tail = ov.verify_tail(logits, q, draft, u, 0.8, 0.9, 5, chain_len=n)
    parents = [-1] + list(range(n))
    toks = [0] + draft
    lg = np.vstack([logits, np.zeros((1, V))])
    qq = np.vstack([q, np.full((1, V), 1.0 / V)])
    # the session's child i+1 uses u[i+1, 0:2]; its row i bonus uses u[i, 2]
    us = np.zeros((n + 1, 3))
    us[1:, 0:2] = u[:, 0:2]
    us[:n, 2] = u[:, 2]
    sess = ov.verify_session(lg, qq, toks, parents, us, 0.8, 0.9, 5)
    assert sess.accept[1:].tolist() == tail["accept"].tolist()
    assert sess.resample[1:].tolist() == tail["resample"].tolist()
    assert sess.bonus[:n].tolist() == tail["bonus"].tolist()
    pl, nx = ov.walk_tail(tail["accept"], tail["resample"], n)
    wr = ov.walk(toks, parents, sess)
    assert pl[0] == len(wr.path)
    if pl[0] < n:
        assert nx[0] == wr.next_token


# ---------------------------------------------------------------------------------------
# Generator
# ---------------------------------------------------------------------------------------


def test_synth_determinism_and_shapes():
    w = tiny_workload(tokens="draft", ragged=True, B=3)
    a = synth.make_batch(w, "cpu")
    b = synth.make_batch(w, "cpu")
    c = synth.make_batch(w, "cpu", seed=w.seed_base + 1)
    for f in ("tokens", "parents", "prefix_len", "kv_k", "kv_v", "q", "u"):
        assert torch.equal(getattr(a, f), getattr(b, f)), f
    assert not torch.equal(a.q, c.q)
    assert float(a.u.min()) > 0 and float(a.u.max()) < 1
    assert torch.all(a.prefix_len >= w.S // 2) and torch.all(a.prefix_len <= w.S)
    # siblings are the top-F draft tokens excluding the main token (Section III-C)
    ch = synth.children_lists(synth.tree_parents(w))
    for bb in range(w.B):
        for r, c_ in enumerate(ch):
            if len(c_) > 1:
                main = int(a.tokens[bb, c_[0]])
                qr = a.q[bb, r].clone()
                qr[main] = -1
                expect = torch.topk(qr, len(c_) - 1).indices.tolist()
                assert [int(a.tokens[bb, x]) for x in c_[1:]] == expect


@pytest.mark.parametrize("name,N,P", [("tiny-fp32", 8, 4), ("1b-bf16", 16, 8),
                                      ("8b-bf16", 16, 11), ("8b-long-wide", 64, 8),
                                      ("32b-bf16", 16, 11), ("70b-bf16", 16, 11)])
def test_workload_tree_shapes(name, N, P):
    w = synth.get(name)
    parents = synth.tree_parents(w)
    assert len(parents) - 1 == N
    ch = synth.children_lists(parents)
    assert sum(1 for c in ch if c) == P
    depths = om.tree_depths(parents)
    assert max(depths) == w.depth


# ---------------------------------------------------------------------------------------
# KV commit (Algorithm 1, COMPACT_KV)
# ---------------------------------------------------------------------------------------


def test_commit_hand_vector():
    """Entries are labelled by their slot; path [2, 4] keeps slots S+0, S+2, S+4 and moves
    them to S, S+1, S+2 (Algorithm 1: the cloud keeps the accepted prefix only)."""
    cap, S = 8, 2
    k = np.zeros((1, 1, cap, 2))
    v = np.zeros((1, 1, 2, cap))
    for s in range(cap):
        k[0, 0, s] = [s, 10 + s]
        v[0, 0, :, s] = [100 + s, 200 + s]
    k2, v2, n = om.commit_path(k, v, S, [2, 4])
    assert n == 5
    assert k2[0, 0, :, 0].tolist() == [0, 1, 2, 4, 6, 5, 6, 7]
    assert k2[0, 0, :, 1].tolist() == [10, 11, 12, 14, 16, 15, 16, 17]
    assert v2[0, 0, 0].tolist() == [100, 101, 102, 104, 106, 105, 106, 107]
    assert v2[0, 0, 1].tolist() == [200, 201, 202, 204, 206, 205, 206, 207]
    k3, v3, n3 = om.commit_path(k, v, S, [])        # nothing accepted: the root stays
    assert n3 == S + 1 and np.array_equal(k3, k) and np.array_equal(v3, v)


@pytest.mark.parametrize("path", [[1, 3, 5], [2], [1, 4], []])
def test_commit_equals_causal_decode_cache(path):
    """After a tree verify pass and the commit of a kept path, the cache equals the one a
    plain causal decode of [prefix; root, kept tokens] builds (positions S + depth)."""
    w = tiny_workload(tree="chain_sib", depth=3, sib=1, tokens="draft")
    W, batch, S, kp, vp, toks, pars = _session(w, b=0)
    # the kept rows must form a root-first chain of the tree
    for a, b_ in zip([0] + path, path):
        assert pars[b_] == a
    dims = om.dims_of(w)
    F = om.F64Weights(W)
    sink = []
    om.forward_tree_session(F, dims, kp, vp, toks, pars, S, kv_sink=sink)
    n1, cap = len(toks), S + len(toks) + 3
    kc = np.full((w.L, w.Hkv, cap, w.hd), np.nan)
    vc = np.full((w.L, w.Hkv, w.hd, cap), np.nan)
    for l in range(w.L):
        kc[l, :, :S] = kp[l]
        vc[l, :, :, :S] = vp[l].transpose(0, 2, 1)
        kt, vt = sink[l]                                   # [n1, Hkv, hd]
        kc[l, :, S:S + n1] = kt.transpose(1, 0, 2)
        vc[l, :, :, S:S + n1] = vt.transpose(1, 2, 0)
    k2, v2, n = om.commit_path(kc, vc, S, path)
    assert n == S + 1 + len(path)
    _, (kref, vref) = om.forward_causal_path(F, dims, kp, vp, [toks[r] for r in [0] + path], S,
                                             return_cache=True)
    for l in range(w.L):
        np.testing.assert_allclose(k2[l, :, :n], kref[l], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(v2[l, :, :, :n], vref[l].transpose(0, 2, 1), rtol=1e-12,
                                   atol=1e-12)
