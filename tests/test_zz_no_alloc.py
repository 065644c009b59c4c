"""The allocation-free LM-head verify (acespec_verify_tail_noalloc) through the C ABI
against acespec_verify_tail on the same inputs: every output bitwise equal, on two calls
in a row, the second with fewer rows (the shared scratch keeps the first call's data).

The first call's 2048 rows leave no room in the 48 MiB scratch for the vocabulary
kernel's per-row candidate lists, so its threshold refinement re-reads each logit row;
the second call's 256 rows, and the context path, keep the candidates instead.  Bitwise
equality therefore also pins the re-read path against the candidate path."""
import pytest
import torch

import synth
from paper_2609_02514_amd import acespec as A
from tests import harness as hz

pytestmark = pytest.mark.gpu


def _outs(R, w):
    return A.Verifier.alloc_outputs(R, R // w.chain_len, w.chain_len, w.top_k, w.V, "cuda", True)


@pytest.mark.parametrize("final_norm,packed", [(False, False), (True, False), (False, True)])
def test_noalloc_tail_equals_context_tail(final_norm, packed):
    w = synth.get("8b-lmhead-tail").scaled(name="tail-noalloc", rows=2048, chain_len=16)
    W = synth.make_weights(w, "cuda")
    batch = synth.make_batch(w, "cuda", weights=W)
    gain = (1.0 + synth.normal((w.d,), 0.1, torch.float32, "cuda", w.seed_base, 0, 2)).to(
        torch.bfloat16) if final_norm else None
    v = A.Verifier.for_workload(w)
    lm = v.pack_weights(W).lm_head if packed else W.lm_head
    layout = A.ACESPEC_LAYOUT_PACKED if packed else A.ACESPEC_LAYOUT_ROWS
    stream = torch.cuda.current_stream().cuda_stream
    # scratch layout of the entry point: row flags, LM-head maxima per 128-column tile and
    # the widened hidden states, then 4096 candidate keys a row if they still fit
    def cand_fits(R):
        al = lambda n: (n + 255) // 256 * 256
        need = al(4 * R) + al(4 * R * ((w.V + 127) // 128)) + al(2 * R * w.d)
        return need + al(4 * R * 4096) <= 48 << 20
    assert not cand_fits(2048) and cand_fits(256)
    for R in (2048, 256):                 # second call: fewer rows
        ref = _outs(R, w)
        v.verify_tail(lm, gain, batch.hidden[:R], batch.draft_tokens[:R], batch.q[:R],
                      batch.u[:R], w.chain_len, w.T, w.top_p, w.top_k, ref, packed=packed)
        got = _outs(R, w)
        for t in got.values():
            if t is not None:
                t.fill_(-7)
        A.acespec_verify_tail_noalloc(v.desc, lm.data_ptr(), layout,
                                      gain.data_ptr() if gain is not None else None,
                                      batch.hidden[:R].data_ptr(),
                                      batch.draft_tokens[:R].data_ptr(), batch.q[:R].data_ptr(),
                                      batch.u[:R].data_ptr(), R, w.chain_len,
                                      A.Params(w.T, w.top_p, w.top_k),
                                      A.Verifier.outputs_struct(got), stream)
        torch.cuda.synchronize()
        for k, t in ref.items():
            if t is not None:
                assert torch.equal(t, got[k]), (R, k)
        assert got["status"].tolist() == [0] * (R // w.chain_len)
        hz.log(f"no-alloc tail R={R} final_norm={final_norm} packed={packed}: every output "
               f"equals verify_tail")
    v.close()


def test_noalloc_rejects_rows_beyond_its_scratch():
    w = synth.get("8b-lmhead-tail")
    desc = A.ModelDesc(0, w.d, 0, 1, 0, 0, w.V, 10000.0, 1e-5, A.ACESPEC_BF16)
    R = 8192
    fake = A.Outputs(*([0x1000] * 12))
    with pytest.raises(A.AcespecError) as e:
        A.acespec_verify_tail_noalloc(desc, 0x1000, A.ACESPEC_LAYOUT_ROWS, None, 0x1000, 0x1000,
                                      0x1000, 0x1000, R, 16,
                                      A.Params(0.6, 0.8, 8), fake,
                                      torch.cuda.current_stream().cuda_stream)
    assert e.value.code == A.ACESPEC_EINVAL and "scratch" in str(e.value)
