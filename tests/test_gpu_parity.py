"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on the same
seeded inputs.  Logits are compared element by element; decisions are compared with the
oracle's verify stage run on the GPU's own logits, every mismatch classified."""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import model as om
from oracle import verify as ov
from tests import harness as hz

pytestmark = pytest.mark.gpu


def small_bf16(**kw):
    base = dict(name="small-bf16", dtype="bf16", L=2, d=320, H=8, Hkv=2, hd=64, F=576, V=5000,
                B=3, S=150, tree="widths_2455", depth=4, q_std=2.5, q_T=0.8, T=0.8,
                top_p=0.9, top_k=24, ragged=True, random_gains=True, seed_base=4242)
    base.update(kw)
    return synth.Workload(**base)


def _check_tree(run, tol):
    """Logits of the forward-sampled sessions against the oracle's float64 forward;
    decisions of EVERY row of every session against the oracle's verify stage on the GPU's
    logits; the walk of every session from the GPU's decisions."""
    z_ref = hz.oracle_tree_logits(run)
    n1 = run.host_in["tokens"].shape[1]
    zg = np.stack([run.outs["logits_out"][b * n1:(b + 1) * n1].numpy() for b in run.sessions])
    err = hz.logits_rel_err(zg.astype(np.float64), z_ref)
    hz.log(f"logits max rel err {err.max():.3e} over {len(run.sessions)} sessions (tol {tol})")
    assert err.max() <= tol, err.max()
    rep = hz.check_tree_decisions(run)
    hz.log(f"decisions (all {run.host_in['tokens'].shape[0]} sessions): {rep}")
    info = hz.agreement_on_oracle_logits(run, z_ref)
    hz.log(f"informational, on the oracle's own logits: {info}")
    assert rep.ok(), str(rep)
    return err, rep


@pytest.mark.parametrize("seed", hz.parity_seeds(synth.get("tiny-fp32"), 10))
def test_tree_tiny_fp32_full_config(seed):
    """The tiny fp32 workload at its full size (2 layers, d=256, vocab 4096, 8-node tree),
    ten parity seeds."""
    w = synth.get("tiny-fp32")
    run = hz.run_tree(w, seed=seed)
    _check_tree(run, tol=1e-4)


@pytest.mark.parametrize("variant", [
    dict(),                                                    # hd 64, G 4, 16-node tree
    dict(hd=128, H=4, Hkv=1, d=256, tree="chain_sib", depth=6, sib=2, V=4100),
    dict(hd=128, H=8, Hkv=8, tree="chain", depth=9, B=2, S=64, ragged=False, V=2048),
    dict(hd=64, H=8, Hkv=2, tree="chain_sib", depth=8, sib=7, B=2, S=700, top_k=64),
    # 8 query heads per kv head under a 64-node tree: 520 query rows, two query groups
    dict(hd=64, H=16, Hkv=2, d=256, tree="chain_sib", depth=8, sib=7, B=2, S=300, top_k=32),
    dict(hd=128, H=8, Hkv=1, d=256, tree="chain_sib", depth=8, sib=7, B=3, S=200, V=3000),
    # 8 query heads under a 36-node tree: 296 rows in two query groups of 148, i.e. four
    # 32-row tiles and a 20-row remainder, which is a padded 32-row tile of its own
    dict(hd=64, H=16, Hkv=2, d=256, tree="chain_sib", depth=4, sib=8, B=2, S=1024, V=3000),
    dict(hd=128, H=16, Hkv=2, d=256, tree="chain_sib", depth=4, sib=8, B=2, S=600, V=3000),
])
def test_tree_small_bf16(variant):
    w = small_bf16(**variant)
    run = hz.run_tree(w)
    _check_tree(run, tol=2e-2)


@pytest.mark.parametrize("variant", [
    dict(),
    dict(hd=128, H=4, Hkv=1, d=256, tree="chain_sib", depth=6, sib=2, V=4112),
    dict(hd=64, H=16, Hkv=2, d=256, tree="chain_sib", depth=8, sib=7, B=2, S=300, top_k=32,
         V=4096),
])
def test_tree_small_bf16_packed_weights(variant):
    """The same forward with the dense matrices in the packed layout
    (acespec_pack_weight): every GEMM takes its weight operands straight from the packed
    copy."""
    w = small_bf16(**dict(dict(V=5008), **variant))
    run = hz.run_tree(w, packed=True)
    _check_tree(run, tol=2e-2)


def test_pack_weight_layout_matches_its_definition():
    """acespec_pack_weight against the layout written out on the host: 16-byte unit
    u = (nb * cols/32 + kt) * 64 + l holds row nb*16 + l%16, columns kt*32 + (l/16)*8 .. +8,
    widened to fp16."""
    from paper_2609_02514_amd.acespec import Verifier, acespec_pack_weight
    rows, cols = 48, 96
    g = torch.Generator().manual_seed(7)
    src = (torch.randn(rows, cols, generator=g) * 0.05).to(torch.bfloat16)
    dst = torch.empty(rows * cols, dtype=torch.float16, device="cuda")
    srcd = src.cuda()
    acespec_pack_weight(srcd.data_ptr(), dst.data_ptr(), rows, cols, Verifier._stream())
    torch.cuda.synchronize()
    got = dst.cpu().numpy().reshape(rows // 16, cols // 32, 64, 8)
    ref = np.empty_like(got)
    s16 = src.to(torch.float16).numpy()
    for nb in range(rows // 16):
        for kt in range(cols // 32):
            for l in range(64):
                r, c = nb * 16 + l % 16, kt * 32 + (l // 16) * 8
                ref[nb, kt, l] = s16[r, c:c + 8]
    assert np.array_equal(got.view(np.uint16), ref.view(np.uint16))


def test_tree_empty_tree_and_long_ragged_prefix():
    """N = 0 (root only: bonus and top-k only) and prefixes that end mid-chunk."""
    w = small_bf16(tree="chain", depth=0, B=5, S=1000, ragged=True)
    run = hz.run_tree(w)
    _check_tree(run, tol=2e-2)
    assert run.outs["path_len"].tolist() == [0] * 5


@pytest.mark.timeout(900)
@pytest.mark.parametrize("seed", hz.parity_seeds(synth.get("1b-bf16"), 4))
def test_tree_1b_full_size(seed):
    """1B-class workload at full size, all 16 sessions through the oracle's forward."""
    w = synth.get("1b-bf16")
    # even seeds with packed weights (the benchmark's layout), odd ones row-major
    packed = (seed - w.seed_base) // 100 % 2 == 0
    run = hz.run_tree(w, seed=seed, packed=packed)
    _check_tree(run, tol=2e-2)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("seed", hz.parity_seeds(synth.get("8b-bf16"), 3))
def test_tree_8b_full_size(seed):
    """8B-class workload at full size: the oracle's forward on 4 sessions spread over the
    batch, decisions on all 64 sessions' 1088 rows."""
    w = synth.get("8b-bf16")
    i = (seed - w.seed_base) // 100
    run = hz.run_tree(w, seed=seed, sessions=[5 + i, 21 + i, 37 + i, 63 - i],
                      packed=i % 2 == 0)
    _check_tree(run, tol=2e-2)


@pytest.mark.timeout(900)
def test_tree_8b_geometric_tree():
    """A paper-shaped tree: main chain of 8 with 24 alternatives allocated by the geometric
    decay of Section IV (32 drafted nodes per session)."""
    w = synth.get("8b-geometric")
    run = hz.run_tree(w, sessions=[0, 23])
    _check_tree(run, tol=2e-2)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("seed", hz.parity_seeds(synth.get("8b-long-wide"), 3))
def test_tree_8b_long_wide(seed):
    """Long-context wide-tree workload at full size (16k-token prefixes, 64-node trees):
    the first seed runs the oracle's forward on all 8 sessions, the others on two."""
    w = synth.get("8b-long-wide")
    i = (seed - w.seed_base) // 100
    sessions = list(range(8)) if i == 0 else [2 * i, 7 - i]
    run = hz.run_tree(w, seed=seed, sessions=sessions, packed=i % 2 == 0)
    _check_tree(run, tol=2e-2)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["32b-bf16", "70b-bf16"])
def test_tree_paper_scale_widths(name):
    """The paper's cloud-target shapes (Qwen-32B / LLaMA-70B classes: d 5120 / 8192, G 5 / 8,
    vocab 152064 / 128256) at their full widths and batch, two layers deep: every kernel
    runs the launch configuration of the full-depth model (depth changes only the layer
    loop), and the float64 oracle stays within seconds per session."""
    w = synth.get(name).scaled(L=2)
    run = hz.run_tree(w, sessions=[11, 50], packed=name == "70b-bf16")
    _check_tree(run, tol=2e-2)


@pytest.mark.timeout(900)
def test_tree_70b_widths_64_node_tree():
    """The 70B-class widths (8 query heads per kv head) under the long-context workload's
    64-node tree: 520 query rows per kv head, more than one attention workgroup holds."""
    w = synth.get("70b-bf16").scaled(L=2, B=4, S=1024, tree="chain_sib", depth=8, sib=7,
                                     top_k=64, T=1.0, q_T=1.0, name="70b-wide")
    run = hz.run_tree(w, sessions=[1, 3], packed=True)
    _check_tree(run, tol=2e-2)


# ---------------------------------------------------------------------------------------
# LM-head tail
# ---------------------------------------------------------------------------------------


def _run_tail(w, W=None, rows_check=None, tol=1e-4, final_norm=False, seed=None,
              packed=False):
    """LM-head tail through the C ABI: logits of rows_check (default all) against the
    oracle's float64 LM head; decisions of EVERY row against the oracle's verify stage on
    the GPU's logits; the chain walk from the GPU's accept bits.  packed: the LM head in
    the packed layout (acespec_pack_weight), the oracle on the row-major matrix."""
    from paper_2609_02514_amd.acespec import Verifier
    dev = "cuda"
    seed = w.seed_base if seed is None else seed
    W = W or synth.make_weights(w, dev, seed)
    batch = synth.make_batch(w, dev, seed, weights=W)
    R = w.rows
    q_h, u_h, d_h = hz.host(batch.q), hz.host(batch.u), hz.host(batch.draft_tokens)
    v = Verifier.for_workload(w)
    outs = v.alloc_outputs(R, R // w.chain_len, w.chain_len, w.top_k, w.V, dev, True)
    hz.log(f"verify_tail R={R} V={w.V} seed={seed} packed={packed}")
    lm = v.pack_weights(W).lm_head if packed else W.lm_head
    v.verify_tail(lm, W.final_norm if final_norm else None, batch.hidden,
                  batch.draft_tokens, batch.q, batch.u, w.chain_len, w.T, w.top_p, w.top_k, outs,
                  packed=packed)
    torch.cuda.synchronize()
    del lm
    g = {k: (hz.host(t) if t is not None else None) for k, t in outs.items()}
    v.close()
    rows = list(range(R)) if rows_check is None else rows_check
    z_ref = om.lm_head_tail(W, batch.hidden[rows], final_norm=final_norm, eps=w.rms_eps)
    zg = g["logits_out"].numpy()
    err = hz.logits_rel_err(zg[rows].astype(np.float64), z_ref)
    hz.log(f"tail logits max rel err {err.max():.3e} over {len(rows)} rows")
    assert err.max() <= tol
    gn = {k: (t.numpy() if t is not None else None) for k, t in g.items()}
    rep = hz.check_rows(hz.tail_jobs(zg, q_h.numpy(), d_h.numpy(), u_h.numpy(), range(R),
                                     z_row_of=lambda r: r), gn, w.T, w.top_p, w.top_k)
    hz.log(f"tail decisions (all {R} rows): {rep}")
    info = hz.check_rows(hz.tail_jobs(z_ref, q_h.numpy(), d_h.numpy(), u_h.numpy(), rows),
                         gn, w.T, w.top_p, w.top_k)
    hz.log(f"informational, on the oracle's own logits ({len(rows)} rows): {info}")
    assert rep.ok(), str(rep)
    # chain walk from the GPU's own accept bits
    pl, nx = ov.walk_tail(g["accept"].numpy(), g["resample_token"].numpy(), w.chain_len)
    assert g["path_len"].tolist() == pl.tolist()
    assert g["next_token"].tolist() == nx.tolist()
    assert g["status"].tolist() == [0] * (R // w.chain_len)
    return g


def test_tail_small():
    w = synth.get("8b-lmhead-tail").scaled(name="tail-small", d=256, V=5004, rows=96,
                                          chain_len=8, top_k=16)
    _run_tail(w)


def test_tail_small_packed_lm_head():
    """The LM head in the packed layout (a vocabulary that is a multiple of 16), with a
    final norm: the same decisions as row-major against the oracle."""
    w = synth.get("8b-lmhead-tail").scaled(name="tail-packed", d=256, V=5008, rows=96,
                                          chain_len=8, top_k=16)
    W = synth.make_weights(w, "cuda")
    gain = 1.0 + synth.normal((w.d,), 0.1, torch.float32, "cuda", w.seed_base, 0, 2)
    W = dataclasses.replace(W, final_norm=gain.to(torch.bfloat16))
    _run_tail(w, W=W, tol=2e-3, final_norm=True, packed=True)


def test_tail_with_final_norm():
    """A non-NULL final_norm: the tail rows are RMS-normalised with the gain (rounded to
    fp16 for the LM head) before the product; the oracle normalises in float64."""
    w = synth.get("8b-lmhead-tail").scaled(name="tail-norm", d=256, V=5004, rows=64,
                                          chain_len=8, top_k=16)
    W = synth.make_weights(w, "cuda")
    gain = 1.0 + synth.normal((w.d,), 0.1, torch.float32, "cuda", w.seed_base, 0, 2)
    W = dataclasses.replace(W, final_norm=gain.to(torch.bfloat16))
    _run_tail(w, W=W, tol=2e-3, final_norm=True)


def test_tail_fp32_model_with_final_norm():
    """The fp32 model's tail (reference-precision kernels) with a final RMSNorm gain."""
    w = synth.get("8b-lmhead-tail").scaled(name="tail-f32", dtype="f32", d=192, V=3000,
                                          rows=48, chain_len=6, top_k=24)
    W = synth.make_weights(w, "cuda")
    gain = 1.0 + synth.normal((w.d,), 0.1, torch.float32, "cuda", w.seed_base, 0, 2)
    W = dataclasses.replace(W, final_norm=gain)
    _run_tail(w, W=W, tol=1e-4, final_norm=True)


@pytest.mark.parametrize("packed", [False, True])
def test_tail_exact_logit_ties(packed):
    """Duplicated LM-head rows give exactly equal logits (in either layout: every output
    column sums its products in the same order): ties must be broken by token id in the
    nucleus, the top-k payload and the inverse CDFs."""
    w = synth.get("8b-lmhead-tail").scaled(name="tail-ties", d=128, V=4096, rows=64,
                                          chain_len=4, top_k=32, T=1.0, top_p=0.5)
    W = synth.make_weights(w, "cuda")
    W.lm_head = W.lm_head[torch.arange(w.V, device="cuda") // 8].contiguous()
    _run_tail(w, W=W, packed=packed)


@pytest.mark.parametrize("T,top_p,top_k", [
    (1.0, 1.0, 256),    # whole vocabulary in the nucleus, the largest payload
    (0.05, 0.9, 1),     # near-greedy target, a one-token payload
    (4.0, 0.3, 8),      # flat target, a nucleus of a small mass fraction
    (0.8, 0.999, 200),  # nucleus boundary deep in the tail
])
def test_tail_parameter_extremes(T, top_p, top_k):
    """Section III-B's sampling parameters at the ends of their ranges (temperature,
    nucleus mass, payload size), on the same decisions as the other tail tests."""
    w = synth.get("8b-lmhead-tail").scaled(name="tail-extremes", d=256, V=5004, rows=64,
                                          chain_len=4, top_k=top_k, T=T, top_p=top_p)
    _run_tail(w)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("seed", hz.parity_seeds(synth.get("8b-lmhead-tail"), 3))
def test_tail_8b_full_size(seed):
    """The LM-head tail at full size (4096 rows, vocab 128256): decisions on all rows,
    the float64 LM head on 512 sampled rows; even seeds with the packed LM head (the
    benchmark's layout), odd ones row-major."""
    w = synth.get("8b-lmhead-tail")
    rng = np.random.default_rng(seed)
    rows = sorted(rng.choice(w.rows, 512, replace=False).tolist())
    packed = (seed - w.seed_base) // 100 % 2 == 0
    g = _run_tail(w, rows_check=rows, tol=1e-4, seed=seed, packed=packed)
    rate = float(g["accept"].float().mean())
    hz.log(f"tail acceptance rate {rate:.3f}")
    assert 0.3 < rate < 0.95


# ---------------------------------------------------------------------------------------
# ABI behaviour on the device
# ---------------------------------------------------------------------------------------


def test_bad_trees_flag_only_their_session():
    from paper_2609_02514_amd.acespec import Verifier
    w = small_bf16(B=4, ragged=False)
    W = synth.make_weights(w, "cuda")
    batch = synth.make_batch(w, "cuda")
    par = batch.parents.clone()
    tok = batch.tokens.clone()
    par[1, 5] = 7          # forward reference
    tok[2, 3] = w.V + 3    # token outside the vocabulary
    plen = batch.prefix_len.clone()
    plen[3] = batch.cap    # prefix leaves no room for the tree
    v = Verifier.for_workload(w)
    B, n1 = tok.shape
    outs = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, "cuda", False)
    v.verify_tree(v.weights_struct(W), batch.kv_k, batch.kv_v, batch.cap, plen, tok, par,
                  batch.q, batch.u, w.T, w.top_p, w.top_k, outs)
    torch.cuda.synchronize()
    assert outs["status"].tolist() == [0, -5, -5, -5]
    v.close()


def test_argument_errors_are_synchronous():
    from paper_2609_02514_amd import acespec as A
    w = small_bf16(B=2)
    W = synth.make_weights(w, "cuda")
    batch = synth.make_batch(w, "cuda")
    v = A.Verifier.for_workload(w)
    B, n1 = batch.tokens.shape
    outs = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, "cuda", False)
    ws = v.weights_struct(W)
    for T, top_p, k, code in [(0.0, 0.9, 8, -1), (0.8, 0.0, 8, -1), (0.8, 1.5, 8, -1),
                              (0.8, 0.9, 0, -1), (0.8, 0.9, 300, -1)]:
        with pytest.raises(A.AcespecError) as e:
            v.verify_tree(ws, batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len,
                          batch.tokens, batch.parents, batch.q, batch.u, T, top_p, k, outs)
        assert e.value.code == code
    with pytest.raises(A.AcespecError):   # more sessions than the context holds
        big = batch.tokens.repeat(3, 1)
        v.verify_tree(ws, batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len, big,
                      batch.parents.repeat(3, 1), batch.q, batch.u, 0.8, 0.9, 8, outs)
    v.close()
    with pytest.raises(A.AcespecError) as e:
        A.Verifier(1, 256, 4, 4, 96, 512, 1000, "bf16", 2, 4)   # head_dim 96
    assert e.value.code == -2


def test_run_to_run_bitwise_determinism():
    from paper_2609_02514_amd.acespec import Verifier
    w = small_bf16(B=2)
    W = synth.make_weights(w, "cuda")
    batch = synth.make_batch(w, "cuda")
    v = Verifier.for_workload(w)
    B, n1 = batch.tokens.shape
    ws = v.weights_struct(W)
    res = []
    for _ in range(2):
        outs = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, "cuda", True)
        v.verify_tree(ws, batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len, batch.tokens,
                      batch.parents, batch.q, batch.u, w.T, w.top_p, w.top_k, outs)
        torch.cuda.synchronize()
        res.append({k: t.clone() for k, t in outs.items() if t is not None})
    for k in res[0]:
        assert torch.equal(res[0][k], res[1][k]), k
    v.close()


def test_timing_selection():
    """acespec_timing_only restricts the recorded kernels to one kind; unknown kinds are
    rejected synchronously; NULL restores every kind."""
    from paper_2609_02514_amd import acespec as A
    w = small_bf16(B=2)
    W = synth.make_weights(w, "cuda")
    batch = synth.make_batch(w, "cuda")
    v = A.Verifier.for_workload(w)
    B, n1 = batch.tokens.shape
    ws = v.weights_struct(W)
    outs = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, "cuda", False)

    def step():
        v.verify_tree(ws, batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len, batch.tokens,
                      batch.parents, batch.q, batch.u, w.T, w.top_p, w.top_k, outs)

    A.acespec_timing_enable(v.ctx, True)
    A.acespec_timing_only(v.ctx, "gemm_gate_up")
    A.acespec_timing_read(v.ctx)
    step()
    got = A.acespec_timing_read(v.ctx)
    assert list(got) == ["gemm_gate_up"] and got["gemm_gate_up"][1] == w.L
    with pytest.raises(A.AcespecError) as e:
        A.acespec_timing_only(v.ctx, "no_such_kernel")
    assert e.value.code == -1
    A.acespec_timing_only(v.ctx, None)
    step()
    got = A.acespec_timing_read(v.ctx)
    assert {"gemm_gate_up", "tree_attention", "vocab_verify", "path_walk"} <= set(got)
    A.acespec_timing_enable(v.ctx, False)
    v.close()
