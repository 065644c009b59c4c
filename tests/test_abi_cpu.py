"""C ABI checks that need no GPU: the library loads and exports every entry point that
include/acespec.h declares (no compute call is made here)."""
import ctypes
import os
import re

import paper_2609_02514_amd.acespec as A

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "acespec.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(acespec_[a-z_]+)\s*\(", src)))


def test_header_declares_the_bound_entry_points():
    assert declared_symbols() == sorted(A.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(A.LIB_PATH)
    for name in declared_symbols():
        assert hasattr(lib, name), name


def test_struct_layouts_match_the_header():
    # sizes of the plain structs as laid out by the C compiler on x86-64
    assert ctypes.sizeof(A.ModelDesc) == 40
    assert ctypes.sizeof(A.LayerWeights) == 48
    assert ctypes.sizeof(A.Weights) == 40
    assert A.Weights.layout.offset == 32
    assert ctypes.sizeof(A.KVCache) == 32
    assert ctypes.sizeof(A.Params) == 12
    assert ctypes.sizeof(A.Outputs) == 96


def test_last_error_starts_empty():
    assert A.acespec_last_error() == ""


def test_status_codes_match_the_header():
    src = open(os.path.join(ROOT, "include", "acespec.h")).read()
    enum = dict((k, int(v)) for k, v in re.findall(r"\b(ACESPEC_E[A-Z]+)\s*=\s*(-?\d+)", src))
    assert enum == {"ACESPEC_EINVAL": -1, "ACESPEC_EUNSUPPORTED": -2, "ACESPEC_ENOMEM": -3,
                    "ACESPEC_EHIP": -4, "ACESPEC_EBADTREE": -5, "ACESPEC_EBADDRAFT": -6,
                    "ACESPEC_ENONFINITE": -7}
    for k, v in enum.items():
        assert getattr(A, k) == v, k


def test_commit_rejects_new_prefix_len_aliasing_prefix_len():
    """acespec_commit_kv's workgroups read prefix_len[b] while one of them writes
    new_prefix_len[b], so overlapping arrays are refused before anything is launched (no
    device memory is touched: the pointers below are never dereferenced)."""
    lib = A.load()
    base = 0x7F0000001000
    B, N = 4, 16
    for new_ptr in (base, base + 8, base - 12):   # same array, inside it, straddling it
        kv = A.KVCache(0x1000, 0x2000, 64, base)
        rc = lib.acespec_commit_kv(None, ctypes.byref(kv), 0x3000, 0x4000, None, B, N, new_ptr,
                                   None)
        assert rc == A.ACESPEC_EINVAL
        assert "overlaps" in A.acespec_last_error()
    # disjoint arrays pass the check and stop at the missing context instead
    kv = A.KVCache(0x1000, 0x2000, 64, base)
    rc = lib.acespec_commit_kv(None, ctypes.byref(kv), 0x3000, 0x4000, None, B, N, base + 16,
                               None)
    assert rc == A.ACESPEC_EINVAL and "ctx is NULL" in A.acespec_last_error()


def test_pack_weight_rejects_bad_shapes_and_overlap_before_launching():
    """acespec_pack_weight checks its arguments before anything is enqueued (the pointers
    below are never dereferenced)."""
    lib = A.load()
    src, dst = 0x7F0000100000, 0x7F0000900000
    for rows, cols in ((0, 64), (15, 64), (16, 48), (24, 64), (16, 0)):
        assert lib.acespec_pack_weight(src, dst, rows, cols, None) == A.ACESPEC_EINVAL
        assert "multiple of 16" in A.acespec_last_error()
    assert lib.acespec_pack_weight(None, dst, 16, 32, None) == A.ACESPEC_EINVAL
    assert lib.acespec_pack_weight(src, None, 16, 32, None) == A.ACESPEC_EINVAL
    # dst starting inside src's 16 x 32 x 2 = 1024 bytes
    assert lib.acespec_pack_weight(src, src + 512, 16, 32, None) == A.ACESPEC_EINVAL
    assert "overlap" in A.acespec_last_error()


def test_convert_v_cache_rejects_bad_arguments_before_launching():
    """acespec_convert_v_cache checks its arguments before anything is enqueued (the
    pointers below are never dereferenced)."""
    lib = A.load()
    src, dst = 0x7F0000100000, 0x7F0010000000
    to_hd = A.ACESPEC_V_TO_HEAD_DIM_MAJOR

    def conv(s=src, d=dst, planes=4, cap=128, hd=64, dt=A.ACESPEC_BF16, direction=to_hd):
        return lib.acespec_convert_v_cache(s, d, planes, cap, hd, dt, direction, None)

    assert conv(s=None) == A.ACESPEC_EINVAL and "NULL" in A.acespec_last_error()
    assert conv(d=None) == A.ACESPEC_EINVAL
    assert conv(dt=7) == A.ACESPEC_EINVAL and "dtype" in A.acespec_last_error()
    assert conv(direction=2) == A.ACESPEC_EINVAL and "direction" in A.acespec_last_error()
    for planes, cap, hd in ((0, 128, 64), (4, 100, 64), (4, 0, 64), (4, 128, 0)):
        assert conv(planes=planes, cap=cap, hd=hd) == A.ACESPEC_EINVAL
        assert "multiple of 64" in A.acespec_last_error()
    # 2^30 planes of 2 x 2 tiles: more than one launch holds
    assert conv(planes=1 << 30, cap=64, hd=64) == A.ACESPEC_EINVAL
    assert "in parts" in A.acespec_last_error()
    # dst starting inside src's 4 x 128 x 64 x 2 = 64 KB; fp32 doubles the extent
    assert conv(d=src + 60000) == A.ACESPEC_EINVAL and "overlap" in A.acespec_last_error()
    assert conv(d=src + 100000, dt=A.ACESPEC_F32) == A.ACESPEC_EINVAL
    assert "overlap" in A.acespec_last_error()


def test_header_declares_the_v_cache_directions():
    src = open(os.path.join(ROOT, "include", "acespec.h")).read()
    enum = dict((k, int(v)) for k, v in re.findall(r"\b(ACESPEC_V_TO_[A-Z_]+)\s*=\s*(\d+)", src))
    assert enum == {"ACESPEC_V_TO_HEAD_DIM_MAJOR": A.ACESPEC_V_TO_HEAD_DIM_MAJOR,
                    "ACESPEC_V_TO_SLOT_MAJOR": A.ACESPEC_V_TO_SLOT_MAJOR}


def test_header_declares_the_weight_layouts():
    src = open(os.path.join(ROOT, "include", "acespec.h")).read()
    enum = dict((k, int(v)) for k, v in re.findall(r"\b(ACESPEC_LAYOUT_[A-Z]+)\s*=\s*(\d+)", src))
    assert enum == {"ACESPEC_LAYOUT_ROWS": A.ACESPEC_LAYOUT_ROWS,
                    "ACESPEC_LAYOUT_PACKED": A.ACESPEC_LAYOUT_PACKED}


def test_noalloc_tail_checks_the_lm_head_layout_before_launching():
    """acespec_verify_tail_noalloc validates lm_head_layout before touching a device (the
    pointers below are never dereferenced): an unknown value is ACESPEC_EINVAL, a packed
    head of an fp32 model or of a vocabulary that is not a multiple of 16 is
    ACESPEC_EUNSUPPORTED."""
    lib = A.load()
    p = 0x7F0000100000
    params = A.Params(0.8, 0.9, 8)
    outs = A.Outputs(*([p] * 12))

    def call(dtype, vocab, layout):
        desc = A.ModelDesc(0, 256, 0, 1, 0, 0, vocab, 10000.0, 1e-5, dtype)
        return lib.acespec_verify_tail_noalloc(A.C.byref(desc), p, layout, None, p, p, p, p,
                                               16, 16, A.C.byref(params), A.C.byref(outs), None)

    assert call(A.ACESPEC_BF16, 5008, 7) == A.ACESPEC_EINVAL
    assert "layout" in A.acespec_last_error()
    assert call(A.ACESPEC_F32, 5008, A.ACESPEC_LAYOUT_PACKED) == A.ACESPEC_EUNSUPPORTED
    assert call(A.ACESPEC_BF16, 5004, A.ACESPEC_LAYOUT_PACKED) == A.ACESPEC_EUNSUPPORTED
    assert "multiple of 16" in A.acespec_last_error()
