"""GPU parity of the KV commit (Algorithm 1, COMPACT_KV) through the C ABI: bit-exact
against the oracle's gather on the same post-verify cache, and end to end against the cache
a causal decode of the accepted tokens builds."""
import numpy as np
import pytest
import torch

import synth
from oracle import model as om
from tests import harness as hz
from tests.test_gpu_parity import small_bf16

pytestmark = pytest.mark.gpu


def _main_chain(parents, n):
    """Root-first chain of lowest-index children, at most n rows."""
    ch = synth.children_lists(parents)
    path, r = [], 0
    while ch[r] and len(path) < n:
        r = ch[r][0]
        path.append(r)
    return path


def _verify(w):
    from paper_2609_02514_amd.acespec import Verifier
    W = synth.make_weights(w, "cuda")
    batch = synth.make_batch(w, "cuda")
    v = Verifier.for_workload(w)
    B, n1 = batch.tokens.shape
    outs = v.alloc_outputs(B * n1, B, n1, w.top_k, w.V, "cuda", False)
    hz.log(f"verify {w.name} B={B} N={n1 - 1}")
    v.verify_tree(v.weights_struct(W), batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len,
                  batch.tokens, batch.parents, batch.q, batch.u, w.T, w.top_p, w.top_k, outs)
    torch.cuda.synchronize()
    return v, W, batch, outs


def _host(t):
    return t.detach().to("cpu").to(torch.float64).numpy()


@pytest.mark.parametrize("name", ["small", "tiny-fp32"])
def test_commit_matches_oracle_gather(name):
    w = small_bf16(B=5, ragged=True) if name == "small" else synth.get("tiny-fp32")
    v, W, batch, outs = _verify(w)
    B, n1 = batch.tokens.shape
    parents = [int(p) for p in batch.parents[0].tolist()]
    path, plen, status = outs["path"].clone(), outs["path_len"].clone(), outs["status"].clone()
    chain = _main_chain(parents, n1)
    path[0, :] = -1
    path[0, :len(chain)] = torch.tensor(chain, dtype=torch.int32)
    plen[0] = len(chain)                  # the deepest chain of the tree
    if B > 1:
        plen[1] = 0                       # nothing accepted: the root only
    if B > 3:
        status[2] = -5                    # a flagged session is not committed
        plen[3] = n1                      # an impossible path length
    kh, vh = _host(batch.kv_k), _host(batch.kv_v)
    pre = batch.prefix_len.tolist()
    new_len = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    hz.log(f"commit_kv B={B}")
    v.commit_kv(batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len, path, plen, status, new_len)
    torch.cuda.synchronize()
    k2, v2 = _host(batch.kv_k), _host(batch.kv_v)
    got = new_len.tolist()
    for b in range(B):
        S = pre[b]
        if (B > 3 and b in (2, 3)):
            assert got[b] == -1
            assert np.array_equal(k2[:, b], kh[:, b]) and np.array_equal(v2[:, b], vh[:, b])
            continue
        kp = path[b, :int(plen[b])].tolist()
        ek, ev, n = om.commit_path(kh[:, b], vh[:, b], S, kp)
        assert got[b] == n, (b, got[b], n)
        assert np.array_equal(k2[:, b], ek), b
        assert np.array_equal(v2[:, b], ev), b
    v.close()


def test_commit_after_verify_equals_causal_decode_cache():
    """The committed slots hold the keys (post-RoPE) and values that a plain causal decode
    of [prefix; root, kept tokens] computes (bf16 storage: within 2e-2 of the row scale)."""
    w = small_bf16(B=2, ragged=False, tree="chain_sib", depth=5, sib=1)
    v, W, batch, outs = _verify(w)
    B, n1 = batch.tokens.shape
    b = 1
    S = int(batch.prefix_len[b])
    toks = batch.tokens[b].tolist()
    parents = batch.parents[b].tolist()
    chain = _main_chain(parents, n1)
    kp, vp = om.session_prefix(batch.kv_k, batch.kv_v, b, S)   # prefix is never written
    path = torch.full((B, n1), -1, dtype=torch.int32, device="cuda")
    path[b, :len(chain)] = torch.tensor(chain, dtype=torch.int32)
    plen = torch.tensor([0, len(chain)], dtype=torch.int32, device="cuda")
    new_len = torch.empty(B, dtype=torch.int32, device="cuda")
    v.commit_kv(batch.kv_k, batch.kv_v, batch.cap, batch.prefix_len, path, plen, None, new_len)
    torch.cuda.synchronize()
    n = S + 1 + len(chain)
    assert new_len.tolist()[b] == n
    dims = om.dims_of(w)
    _, (kref, vref) = om.forward_causal_path(om.F64Weights(W), dims, kp, vp,
                                             [toks[r] for r in [0] + chain], S,
                                             return_cache=True)
    for l in range(w.L):
        kg = _host(batch.kv_k[l, b, :, S:n])                      # [Hkv, n - S, hd]
        vg = _host(batch.kv_v[l, b, :, :, S:n]).transpose(0, 2, 1)
        for got, ref in ((kg, kref[l][:, S:n]), (vg, vref[l][:, S:n])):
            err = np.abs(got - ref).max() / np.abs(ref).max()
            hz.log(f"layer {l}: committed cache rel err {err:.2e}")
            assert err < 2e-2
    v.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_convert_v_cache_is_an_exact_transpose_both_ways(dtype):
    """acespec_convert_v_cache against torch's transpose, bit for bit: a slot-major value
    cache [planes, cap, hd] becomes the head-dim-major [planes, hd, cap] the verify step
    reads, and back.  Ragged head_dim (40: a partial 32-wide tile) and a capacity of 3 x 64
    slots check the tile edges; NaN and inf bit patterns must survive."""
    from paper_2609_02514_amd import acespec as A
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    adt = A.ACESPEC_BF16 if dtype == "bf16" else A.ACESPEC_F32
    for planes, cap, hd in ((3, 192, 40), (64, 128, 128)):
        hz.log(f"convert_v_cache {dtype} planes={planes} cap={cap} hd={hd}")
        g = torch.Generator(device="cpu").manual_seed(planes * 1000 + cap + hd)
        slot_major = torch.randn(planes, cap, hd, generator=g).to(tdt)
        slot_major[0, 5, 3] = float("nan")
        slot_major[-1, -1, -1] = float("inf")
        slot_major = slot_major.cuda()
        hd_major = torch.empty(planes, hd, cap, dtype=tdt, device="cuda")
        back = torch.empty_like(slot_major)
        stream = torch.cuda.current_stream().cuda_stream
        A.acespec_convert_v_cache(slot_major.data_ptr(), hd_major.data_ptr(), planes, cap, hd,
                                  adt, A.ACESPEC_V_TO_HEAD_DIM_MAJOR, stream)
        A.acespec_convert_v_cache(hd_major.data_ptr(), back.data_ptr(), planes, cap, hd, adt,
                                  A.ACESPEC_V_TO_SLOT_MAJOR, stream)
        torch.cuda.synchronize()
        iview = torch.int16 if dtype == "bf16" else torch.int32
        want = slot_major.transpose(1, 2).contiguous()
        assert torch.equal(hd_major.view(iview), want.view(iview))
        assert torch.equal(back.view(iview), slot_major.view(iview))
