"""ctypes binding of libacespec.so: the C entry points under the same names, plus a thin
marshalling helper (``Verifier``) that passes torch device tensors' pointers and the current
torch stream.  Every step of the verify path runs in the library's HIP kernels; this module
only moves pointers and sizes across the boundary.  Importing it fails loudly if the
library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, List, Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libacespec.so")

ACESPEC_OK, ACESPEC_EINVAL, ACESPEC_EUNSUPPORTED = 0, -1, -2
ACESPEC_ENOMEM, ACESPEC_EHIP, ACESPEC_EBADTREE = -3, -4, -5
ACESPEC_EBADDRAFT, ACESPEC_ENONFINITE = -6, -7
ACESPEC_F32, ACESPEC_BF16 = 0, 1

EXPORTED = ["acespec_create", "acespec_destroy", "acespec_verify_tree",
            "acespec_verify_tree_scalar_q", "acespec_verify_tail", "acespec_commit_kv",
            "acespec_last_error", "acespec_timing_enable", "acespec_timing_read",
            "acespec_timing_only", "acespec_verify_tail_noalloc", "acespec_pack_weight",
            "acespec_convert_v_cache"]


class ModelDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int), ("d_model", C.c_int), ("n_heads", C.c_int),
                ("n_kv_heads", C.c_int), ("head_dim", C.c_int), ("d_ff", C.c_int),
                ("vocab", C.c_int), ("rope_base", C.c_float), ("rms_eps", C.c_float),
                ("dtype", C.c_int)]


class LayerWeights(C.Structure):
    _fields_ = [("attn_norm", C.c_void_p), ("wqkv", C.c_void_p), ("wo", C.c_void_p),
                ("mlp_norm", C.c_void_p), ("w_gate_up", C.c_void_p), ("w_down", C.c_void_p)]


ACESPEC_LAYOUT_ROWS, ACESPEC_LAYOUT_PACKED = 0, 1
ACESPEC_V_TO_HEAD_DIM_MAJOR, ACESPEC_V_TO_SLOT_MAJOR = 0, 1


class Weights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("layers", C.POINTER(LayerWeights)),
                ("final_norm", C.c_void_p), ("lm_head", C.c_void_p), ("layout", C.c_int)]


class KVCache(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("capacity", C.c_int),
                ("prefix_len", C.c_void_p)]


class Params(C.Structure):
    _fields_ = [("temperature", C.c_float), ("top_p", C.c_float), ("top_k", C.c_int)]


class Outputs(C.Structure):
    _fields_ = [("accept", C.c_void_p), ("acc_prefix_len", C.c_void_p),
                ("resample_token", C.c_void_p), ("bonus_token", C.c_void_p),
                ("topk_ids", C.c_void_p), ("topk_probs", C.c_void_p), ("path", C.c_void_p),
                ("path_len", C.c_void_p), ("next_token", C.c_void_p),
                ("sibling_hit", C.c_void_p), ("status", C.c_void_p),
                ("logits_out", C.c_void_p)]


_lib = None


def load(path: str = LIB_PATH) -> C.CDLL:
    """Loads the HIP library (raises if it is missing: there is no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2609_02514_amd.build`")
    lib = C.CDLL(path)
    lib.acespec_create.argtypes = [C.POINTER(ModelDesc), C.c_int, C.c_int,
                                   C.POINTER(C.c_void_p)]
    lib.acespec_create.restype = C.c_int
    lib.acespec_destroy.argtypes = [C.c_void_p]
    lib.acespec_destroy.restype = None
    lib.acespec_verify_tree.argtypes = [C.c_void_p, C.POINTER(Weights), C.POINTER(KVCache),
                                        C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                        C.c_int, C.c_int, C.POINTER(Params),
                                        C.POINTER(Outputs), C.c_void_p]
    lib.acespec_verify_tree.restype = C.c_int
    lib.acespec_verify_tree_scalar_q.argtypes = lib.acespec_verify_tree.argtypes
    lib.acespec_verify_tree_scalar_q.restype = C.c_int
    lib.acespec_verify_tail.argtypes = [C.c_void_p, C.c_void_p, C.c_int, C.c_void_p,
                                        C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                        C.c_int, C.c_int, C.POINTER(Params),
                                        C.POINTER(Outputs), C.c_void_p]
    lib.acespec_verify_tail.restype = C.c_int
    lib.acespec_verify_tail_noalloc.argtypes = [C.POINTER(ModelDesc), C.c_void_p, C.c_int,
                                                C.c_void_p, C.c_void_p, C.c_void_p,
                                                C.c_void_p, C.c_void_p, C.c_int, C.c_int,
                                                C.POINTER(Params), C.POINTER(Outputs),
                                                C.c_void_p]
    lib.acespec_verify_tail_noalloc.restype = C.c_int
    lib.acespec_commit_kv.argtypes = [C.c_void_p, C.POINTER(KVCache), C.c_void_p, C.c_void_p,
                                      C.c_void_p, C.c_int, C.c_int, C.c_void_p, C.c_void_p]
    lib.acespec_commit_kv.restype = C.c_int
    lib.acespec_pack_weight.argtypes = [C.c_void_p, C.c_void_p, C.c_int, C.c_int, C.c_void_p]
    lib.acespec_pack_weight.restype = C.c_int
    lib.acespec_convert_v_cache.argtypes = [C.c_void_p, C.c_void_p, C.c_int, C.c_int, C.c_int,
                                            C.c_int, C.c_int, C.c_void_p]
    lib.acespec_convert_v_cache.restype = C.c_int
    lib.acespec_last_error.argtypes = []
    lib.acespec_last_error.restype = C.c_char_p
    lib.acespec_timing_enable.argtypes = [C.c_void_p, C.c_int]
    lib.acespec_timing_enable.restype = C.c_int
    lib.acespec_timing_read.argtypes = [C.c_void_p, C.POINTER(C.c_char_p),
                                        C.POINTER(C.c_double), C.POINTER(C.c_int), C.c_int]
    lib.acespec_timing_read.restype = C.c_int
    lib.acespec_timing_only.argtypes = [C.c_void_p, C.c_char_p]
    lib.acespec_timing_only.restype = C.c_int
    _lib = lib
    return lib


# --------------------------------------------------------------------------------------
# The C entry points, same names
# --------------------------------------------------------------------------------------


def acespec_last_error() -> str:
    return load().acespec_last_error().decode()


class AcespecError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"acespec error {code}: {msg}")
        self.code = code


def _check(rc: int) -> int:
    if rc < 0:
        raise AcespecError(rc, acespec_last_error())
    return rc


def acespec_create(desc: ModelDesc, max_batch: int, max_nodes: int) -> C.c_void_p:
    ctx = C.c_void_p()
    _check(load().acespec_create(C.byref(desc), max_batch, max_nodes, C.byref(ctx)))
    return ctx


def acespec_destroy(ctx) -> None:
    load().acespec_destroy(ctx)


def acespec_verify_tree(ctx, weights: Weights, kv: KVCache, tree_tokens: int, parent_idx: int,
                        draft_q: int, uniforms: int, B: int, N: int, params: Params,
                        outputs: Outputs, stream: int) -> int:
    return _check(load().acespec_verify_tree(ctx, C.byref(weights), C.byref(kv), tree_tokens,
                                             parent_idx, draft_q, uniforms, B, N,
                                             C.byref(params), C.byref(outputs), stream))


def acespec_verify_tree_scalar_q(ctx, weights: Weights, kv: KVCache, tree_tokens: int,
                                 parent_idx: int, q_hat: int, uniforms: int, B: int, N: int,
                                 params: Params, outputs: Outputs, stream: int) -> int:
    return _check(load().acespec_verify_tree_scalar_q(ctx, C.byref(weights), C.byref(kv),
                                                      tree_tokens, parent_idx, q_hat, uniforms,
                                                      B, N, C.byref(params), C.byref(outputs),
                                                      stream))


def acespec_verify_tail(ctx, lm_head: int, lm_head_layout: int, final_norm: Optional[int],
                        hidden: int, draft_tokens: int, draft_q: int, uniforms: int, R: int,
                        chain_len: int, params: Params, outputs: Outputs, stream: int) -> int:
    return _check(load().acespec_verify_tail(ctx, lm_head, lm_head_layout, final_norm, hidden,
                                             draft_tokens, draft_q, uniforms, R, chain_len,
                                             C.byref(params), C.byref(outputs), stream))


def acespec_verify_tail_noalloc(desc: ModelDesc, lm_head: int, lm_head_layout: int,
                                final_norm: Optional[int], hidden: int, draft_tokens: int,
                                draft_q: int, uniforms: int, R: int, chain_len: int,
                                params: Params, outputs: Outputs, stream: int) -> int:
    return _check(load().acespec_verify_tail_noalloc(C.byref(desc), lm_head, lm_head_layout,
                                                     final_norm, hidden, draft_tokens, draft_q,
                                                     uniforms, R, chain_len, C.byref(params),
                                                     C.byref(outputs), stream))


def acespec_commit_kv(ctx, kv: KVCache, path: int, path_len: int, status: Optional[int], B: int,
                      N: int, new_prefix_len: int, stream: int) -> int:
    return _check(load().acespec_commit_kv(ctx, C.byref(kv), path, path_len, status, B, N,
                                           new_prefix_len, stream))


def acespec_pack_weight(src: int, dst: int, rows: int, cols: int, stream: int) -> int:
    return _check(load().acespec_pack_weight(src, dst, rows, cols, stream))


def acespec_convert_v_cache(src: int, dst: int, planes: int, capacity: int, head_dim: int,
                            dtype: int, direction: int, stream: int) -> int:
    return _check(load().acespec_convert_v_cache(src, dst, planes, capacity, head_dim, dtype,
                                                 direction, stream))


def acespec_timing_enable(ctx, enable: bool) -> None:
    _check(load().acespec_timing_enable(ctx, 1 if enable else 0))


def acespec_timing_only(ctx, kind: Optional[str]) -> None:
    _check(load().acespec_timing_only(ctx, kind.encode() if kind else None))


def acespec_timing_read(ctx) -> Dict[str, tuple]:
    n = 32
    names = (C.c_char_p * n)()
    ms = (C.c_double * n)()
    cnt = (C.c_int * n)()
    k = _check(load().acespec_timing_read(ctx, names, ms, cnt, n))
    return {names[i].decode(): (ms[i], cnt[i]) for i in range(k)}


# --------------------------------------------------------------------------------------
# Marshalling helper over torch device tensors
# --------------------------------------------------------------------------------------


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


class Verifier:
    """Owns a context for one model shape and turns torch tensors into ABI structs."""

    def __init__(self, L, d, H, Hkv, hd, F, V, dtype: str, max_batch: int, max_nodes: int,
                 rope_base=10000.0, rms_eps=1e-5):
        self.desc = ModelDesc(L, d, H, Hkv, hd, F, V, rope_base, rms_eps,
                              ACESPEC_BF16 if dtype == "bf16" else ACESPEC_F32)
        self.V = V
        self.ctx = acespec_create(self.desc, max_batch, max_nodes)
        self._keep: List = []

    @classmethod
    def for_workload(cls, w, max_batch=None, max_nodes=None):
        import synth
        n = 0 if w.tree == "tail" else len(synth.tree_parents(w)) - 1
        mb = max_batch or (w.rows if w.tree == "tail" else w.B)
        return cls(w.L, w.d, w.H, w.Hkv, w.hd, w.F, w.V, w.dtype, mb,
                   n if max_nodes is None else max_nodes, w.rope_base, w.rms_eps)

    def close(self):
        if self.ctx:
            acespec_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    DENSE = ("wqkv", "wo", "w_gate_up", "w_down")

    def pack_weights(self, W, drop_source=False):
        """A copy of W whose dense matrices (the DENSE ones of every layer and the LM head)
        are in the packed layout (acespec_pack_weight); the embedding and the norm gains
        are shared with W.  The result carries `packed = True` for weights_struct.
        drop_source: release each row-major matrix of W once it is packed (W's entries
        become None), so that a model only slightly smaller than the device fits."""
        import copy
        import torch

        def pk(t):
            out = torch.empty(t.numel(), dtype=torch.float16, device=t.device)
            acespec_pack_weight(_ptr(t), _ptr(out), t.shape[0], t.shape[1], self._stream())
            return out

        P = copy.copy(W)
        P.layers = []
        for lw in W.layers:
            P.layers.append(dict(lw, **{k: pk(lw[k]) for k in self.DENSE}))
            if drop_source:
                for k in self.DENSE:
                    lw[k] = None
        P.lm_head = pk(W.lm_head)
        if drop_source:
            W.lm_head = None
        P.packed = True
        return P

    def weights_struct(self, W) -> Weights:
        layers = (LayerWeights * max(1, len(W.layers)))()
        for i, lw in enumerate(W.layers):
            layers[i] = LayerWeights(_ptr(lw["attn_norm"]), _ptr(lw["wqkv"]), _ptr(lw["wo"]),
                                     _ptr(lw["mlp_norm"]), _ptr(lw["w_gate_up"]),
                                     _ptr(lw["w_down"]))
        self._keep.append(layers)
        layout = ACESPEC_LAYOUT_PACKED if getattr(W, "packed", False) else ACESPEC_LAYOUT_ROWS
        return Weights(_ptr(W.embed), layers, _ptr(W.final_norm), _ptr(W.lm_head), layout)

    @staticmethod
    def alloc_outputs(rows: int, sessions: int, n1: int, k: int, V: int, device,
                      keep_logits: bool = False) -> Dict:
        import torch
        i32 = dict(dtype=torch.int32, device=device)
        return dict(
            accept=torch.zeros(rows, dtype=torch.uint8, device=device),
            acc_prefix_len=torch.zeros(rows, **i32),
            resample_token=torch.zeros(rows, **i32),
            bonus_token=torch.zeros(rows, **i32),
            topk_ids=torch.zeros(rows, k, **i32),
            topk_probs=torch.zeros(rows, k, dtype=torch.float32, device=device),
            path=torch.zeros(sessions, n1, **i32),
            path_len=torch.zeros(sessions, **i32),
            next_token=torch.zeros(sessions, **i32),
            sibling_hit=torch.zeros(sessions, dtype=torch.uint8, device=device),
            status=torch.zeros(sessions, **i32),
            logits_out=(torch.zeros(rows, V, dtype=torch.float32, device=device)
                        if keep_logits else None),
        )

    @staticmethod
    def outputs_struct(o: Dict) -> Outputs:
        return Outputs(*[_ptr(o[f]) for f, _ in Outputs._fields_])

    @staticmethod
    def _stream() -> int:
        import torch
        return torch.cuda.current_stream().cuda_stream

    def verify_tree(self, wstruct: Weights, kv_k, kv_v, capacity: int, prefix_len, tokens,
                    parents, q, u, T: float, top_p: float, k: int, outs: Dict) -> int:
        B, n1 = tokens.shape
        kv = KVCache(_ptr(kv_k), _ptr(kv_v), capacity, _ptr(prefix_len))
        return acespec_verify_tree(self.ctx, wstruct, kv, _ptr(tokens), _ptr(parents), _ptr(q),
                                   _ptr(u), B, n1 - 1, Params(T, top_p, k),
                                   self.outputs_struct(outs), self._stream())

    def verify_tree_scalar_q(self, wstruct: Weights, kv_k, kv_v, capacity: int, prefix_len,
                             tokens, parents, q_hat, u, T: float, top_p: float, k: int,
                             outs: Dict) -> int:
        B, n1 = tokens.shape
        kv = KVCache(_ptr(kv_k), _ptr(kv_v), capacity, _ptr(prefix_len))
        return acespec_verify_tree_scalar_q(self.ctx, wstruct, kv, _ptr(tokens), _ptr(parents),
                                            _ptr(q_hat), _ptr(u), B, n1 - 1, Params(T, top_p, k),
                                            self.outputs_struct(outs), self._stream())

    def commit_kv(self, kv_k, kv_v, capacity: int, prefix_len, path, path_len, status,
                  new_prefix_len) -> int:
        B, n1 = path.shape
        kv = KVCache(_ptr(kv_k), _ptr(kv_v), capacity, _ptr(prefix_len))
        return acespec_commit_kv(self.ctx, kv, _ptr(path), _ptr(path_len), _ptr(status), B,
                                 n1 - 1, _ptr(new_prefix_len), self._stream())

    def verify_tail(self, lm_head, final_norm, hidden, draft, q, u, chain_len: int, T: float,
                    top_p: float, k: int, outs: Dict, packed: bool = False) -> int:
        """packed: lm_head is the flat output of pack_weights (acespec_pack_weight)."""
        R = hidden.shape[0]
        return acespec_verify_tail(self.ctx, _ptr(lm_head),
                                   ACESPEC_LAYOUT_PACKED if packed else ACESPEC_LAYOUT_ROWS,
                                   _ptr(final_norm), _ptr(hidden), _ptr(draft), _ptr(q),
                                   _ptr(u), R, chain_len, Params(T, top_p, k),
                                   self.outputs_struct(outs), self._stream())
