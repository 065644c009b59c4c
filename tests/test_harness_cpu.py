"""The parity harness's decision check, on the CPU: outputs produced by the oracle's own
verify stage pass with zero mismatches, and planted disagreements are found and given the
right boundary class (or none)."""
import numpy as np
import torch

import synth
from oracle import verify as ov
from tests import harness as hz


def _fake_run(seed=7):
    w = synth.Workload("harness-cpu", "f32", L=0, d=64, H=0, Hkv=1, hd=0, F=0, V=512, B=3,
                       S=0, tree="widths_2455", depth=4, q_std=2.0, q_T=0.8, T=0.8,
                       top_p=0.9, top_k=8, seed_base=seed)
    parents = synth.tree_parents(w)
    n1 = len(parents)
    rng = np.random.default_rng(seed)
    z = rng.normal(0, 2.0, (w.B * n1, w.V)).astype(np.float32)
    q = rng.dirichlet(np.ones(w.V), (w.B, n1)).astype(np.float32)
    u = rng.uniform(0.001, 0.999, (w.B, n1, 3)).astype(np.float32)
    tok = rng.integers(0, w.V, (w.B, n1)).astype(np.int32)
    par = np.tile(np.array(parents, dtype=np.int32), (w.B, 1))
    g = dict(accept=np.zeros(w.B * n1, np.uint8), acc_prefix_len=np.zeros(w.B * n1, np.int32),
             resample_token=np.zeros(w.B * n1, np.int32),
             bonus_token=np.zeros(w.B * n1, np.int32),
             topk_ids=np.zeros((w.B * n1, w.top_k), np.int32),
             topk_probs=np.zeros((w.B * n1, w.top_k), np.float32),
             path=np.full((w.B, n1), -1, np.int32), path_len=np.zeros(w.B, np.int32),
             next_token=np.zeros(w.B, np.int32), sibling_hit=np.zeros(w.B, np.uint8),
             status=np.zeros(w.B, np.int32), logits_out=z)
    for b in range(w.B):
        sl = slice(b * n1, (b + 1) * n1)
        res = ov.verify_session(z[sl].astype(np.float64), q[b].astype(np.float64), tok[b],
                                parents, u[b].astype(np.float64), float(np.float32(w.T)),
                                float(np.float32(w.top_p)), w.top_k)
        for k, src in (("accept", res.accept), ("acc_prefix_len", res.acc_prefix_len),
                       ("resample_token", res.resample), ("bonus_token", res.bonus),
                       ("topk_ids", res.topk_ids), ("topk_probs", res.topk_probs)):
            g[k][sl] = src
        wr = ov.walk(tok[b], parents, res)
        g["path_len"][b] = len(wr.path)
        g["path"][b, :len(wr.path)] = wr.path
        g["next_token"][b] = wr.next_token
        g["sibling_hit"][b] = wr.sibling_hit
    hin = dict(tokens=torch.from_numpy(tok), parents=torch.from_numpy(par),
               prefix_len=torch.zeros(w.B, dtype=torch.int32), q=torch.from_numpy(q),
               u=torch.from_numpy(u))
    outs = {k: torch.from_numpy(np.ascontiguousarray(v)) for k, v in g.items()}
    return hz.TreeRun(w, None, None, outs, hin, []), n1


def test_oracle_outputs_pass_with_no_mismatch():
    run, n1 = _fake_run()
    rep = hz.check_tree_decisions(run)
    assert rep.nodes == run.w.B * (2 * n1 - 1)   # every row + every child
    assert rep.mismatches == [] and rep.ok()


def test_planted_disagreements_are_classified():
    run, n1 = _fake_run()
    g = run.outs
    # a wrong bonus far from any CDF boundary: unexplained
    j = int(g["bonus_token"][n1 + 2])
    g["bonus_token"][n1 + 2] = (j + 200) % run.w.V
    # a swapped pair of top-k ids that are not tied: unexplained
    g["topk_ids"][2 * n1 + 1, [0, 1]] = g["topk_ids"][2 * n1 + 1, [1, 0]]
    rep = hz.check_rows(hz.tree_jobs(run, lambda b: g["logits_out"].numpy()[b * n1:(b + 1) * n1],
                                     range(run.w.B)),
                        {k: v.numpy() for k, v in g.items()}, run.w.T, run.w.top_p,
                        run.w.top_k)
    assert len(rep.mismatches) == 2 and len(rep.unexplained) == 2 and not rep.ok()


def test_accept_flip_at_the_boundary_is_explained():
    """A child whose p/q sits within 1e-3 of its uniform: flipping the GPU's accept bit is
    a boundary case; flipping one far from its uniform is not."""
    run, n1 = _fake_run()
    g = {k: v.numpy() for k, v in run.outs.items()}
    z = g["logits_out"]
    jobs = hz.tree_jobs(run, lambda b: z[b * n1:(b + 1) * n1], range(run.w.B))
    job = next(j for j in jobs if j.children)
    ci, x, u0, u1, _ = job.children[0]
    pt = ov.tempered_softmax(job.z.astype(np.float64), float(np.float32(run.w.T)))
    p, _, _ = ov.nucleus(pt, float(np.float32(run.w.top_p)))
    ratio = p[x] / float(job.q[x])
    for u_new, cls in ((ratio * (1 - 2e-4), "accept_boundary"), (0.5 * ratio, "unexplained")):
        if not 0.0 < u_new < 1.0:
            continue
        j2 = hz.RowJob(job.tag, job.gi, job.z, job.q, job.u_bonus,
                       [(ci, x, u_new, u1, None)] + job.children[1:])
        g2 = dict(g)
        g2["accept"] = g["accept"].copy()
        g2["accept"][ci] = 0 if ov.accept_token(p, job.q.astype(np.float64), x, u_new) else 1
        rep = hz.check_rows([j2], g2, run.w.T, run.w.top_p, run.w.top_k)
        assert [m.cls for m in rep.mismatches if "accept" in m.what] == [cls]


def test_walk_check_catches_a_wrong_path():
    run, n1 = _fake_run()
    run.outs["next_token"][1] = run.outs["next_token"][1] + 1
    try:
        hz.check_tree_walk(run, range(run.w.B))
    except AssertionError:
        return
    raise AssertionError("a wrong next token went unnoticed")
