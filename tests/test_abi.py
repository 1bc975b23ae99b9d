"""The C-ABI library loads without a GPU, exports every declared entry point, and
rejects bad arguments before touching the device (no compute calls here)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2609_34814_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wavealign.h")


def _lib():
    if not os.path.exists(L.LIB_PATH):
        pytest.skip("library not built (run python -m paper_2609_34814_amd.build)")
    return L.load()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wa_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    _lib()
    out = subprocess.run(["nm", "-D", "--defined-only", L.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (wa_[a-z0-9_]+)$", out, flags=re.M))
    declared = _declared()
    assert declared, "no declarations parsed"
    assert set(declared) <= exported, set(declared) - exported
    assert set(_declared()) == set(L._SIGNATURES)   # the binding declares exactly the ABI


def test_version_and_strings():
    lib = _lib()
    assert lib.wa_abi_version() == 3
    for code in (0, -1, -2, -3, -4, -6):
        assert lib.wa_status_string(code)
    p = L.WaSkipProfile()
    assert lib.wa_default_skip_profile(ctypes.byref(p)) == 0
    assert p.cache_bytes == 96 * 1024 * 1024 and p.j_max == 0.2 and p.eta_min == 0.05
    # the library's built-in profile is the oracle's default, field for field
    from oracle import skip as S
    ref = S.SkipProfile()
    for name, _ in L.WaSkipProfile._fields_:
        assert getattr(p, name) == getattr(ref, name), name
    assert lib.wa_default_skip_profile(None) == L.WA_ERR_INVALID_ARG


def test_status_bits_match_the_header():
    """The status-word bits the binding names are the header's."""
    text = open(HEADER).read()
    for name in ("WA_ATTN_BAD_PERM", "WA_ATTN_BAD_KV_INDEX", "WA_PRODUCE_WAIT_EXPIRED"):
        m = re.search(rf"\b{name}\s*=\s*(\d+)", text)
        assert m, name
        assert int(m.group(1)) == getattr(L, name), name


FAKE = ctypes.c_void_p(1 << 20)   # never dereferenced: every call below fails validation first


def _shape(**kw):
    d = dict(batch=1, heads=2, seq_len=4096, head_dim=64, block=64)
    d.update(kw)
    return L.WaShape(**d)


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=96), L.WA_ERR_UNSUPPORTED),
    (dict(block=32), L.WA_ERR_UNSUPPORTED),
    (dict(seq_len=0), L.WA_ERR_INVALID_ARG),
    (dict(heads=0), L.WA_ERR_INVALID_ARG),
    (dict(seq_len=64 * 4097), L.WA_ERR_UNSUPPORTED),
    (dict(batch=200, heads=300, seq_len=128 * 200, block=128), L.WA_ERR_UNSUPPORTED),
])
def test_shape_validation(kw, code):
    lib = _lib()
    n = ctypes.c_size_t(0)
    assert lib.wa_attn_workspace_size(ctypes.byref(_shape(**kw)), ctypes.byref(n)) == code
    assert lib.wa_last_error()
    assert lib.wa_perm_workspace_size(ctypes.byref(_shape(**kw)), ctypes.byref(n)) == code
    assert lib.wa_attn_workspace_size(None, ctypes.byref(n)) == L.WA_ERR_INVALID_ARG


def test_workspace_sizes():
    lib = _lib()
    n = ctypes.c_size_t(0)
    s = _shape()
    assert lib.wa_attn_workspace_size(ctypes.byref(s), ctypes.byref(n)) == 0
    assert n.value >= 2 * 65 * 4 + 2 * 64 * 64 * 4
    assert lib.wa_perm_workspace_size(ctypes.byref(s), ctypes.byref(n)) == 0
    assert n.value >= 2 * 2 * 64 * 8


def test_sparse_attn_validation():
    lib = _lib()
    s = _shape()
    ws_n = ctypes.c_size_t(0)
    lib.wa_attn_workspace_size(ctypes.byref(s), ctypes.byref(ws_n))
    args = dict(q=FAKE, k=FAKE, v=FAKE, mask=FAKE, perm=None, o=FAKE, ws=ctypes.c_void_p(1 << 24), n_xcd=8,
                ws_bytes=ws_n.value)

    def call(**kw):
        a = dict(args)
        a.update(kw)
        return lib.wa_sparse_attn(a["q"], a["k"], a["v"], a["mask"], a["perm"], None, ctypes.byref(s), 0.0,
                                  a["n_xcd"], a["o"], None, a.get("status"), a["ws"], a["ws_bytes"], None)

    assert call(q=None) == L.WA_ERR_INVALID_ARG
    assert call(o=None) == L.WA_ERR_INVALID_ARG
    assert call(mask=None) == L.WA_ERR_INVALID_ARG
    assert call(k=ctypes.c_void_p((1 << 20) + 2)) == L.WA_ERR_ALIGNMENT
    assert call(n_xcd=0) == L.WA_ERR_INVALID_ARG
    assert call(n_xcd=65) == L.WA_ERR_INVALID_ARG
    assert call(ws=None) == L.WA_ERR_INVALID_ARG
    assert call(ws=ctypes.c_void_p((1 << 24) + 64)) == L.WA_ERR_ALIGNMENT
    assert call(ws_bytes=ws_n.value - 1) == L.WA_ERR_WORKSPACE
    assert b"workspace" in lib.wa_last_error()
    assert call(status=ctypes.c_void_p((1 << 20) + 2)) == L.WA_ERR_ALIGNMENT
    assert lib.wa_sparse_attn_csr(FAKE, FAKE, FAKE, None, FAKE, None, None, ctypes.byref(s), 0.0, 8, FAKE, None,
                                  None, ctypes.c_void_p(1 << 24), ws_n.value, None) == L.WA_ERR_INVALID_ARG
    assert lib.wa_sparse_attn_csr(FAKE, FAKE, FAKE, FAKE, FAKE, None, None, ctypes.byref(s), 0.0, 8, FAKE, None,
                                  None, ctypes.c_void_p(1 << 24), 256, None) == L.WA_ERR_WORKSPACE


def test_sparse_attn_vt_validation():
    lib = _lib()
    s = _shape()
    n_full, n_vt = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert lib.wa_attn_workspace_size(ctypes.byref(s), ctypes.byref(n_full)) == 0
    assert lib.wa_attn_vt_workspace_size(ctypes.byref(s), ctypes.byref(n_vt)) == 0
    # the V^T copy is not part of this call's workspace: at least B*H*d*M_B*block*2 bytes smaller
    assert n_vt.value + 1 * 2 * 64 * 64 * 64 * 2 <= n_full.value
    assert n_vt.value % 256 == 0 and n_vt.value >= 4 * (64 + 64 * 3 + 2 * 64)
    opts = L.WaAttnOptions(0.0, 8, L.WA_HEADS_IN_ORDER)
    ws = ctypes.c_void_p(1 << 24)

    def call(o=None, **kw):
        a = dict(q=FAKE, k=FAKE, vt=FAKE, rp=FAKE, ci=FAKE, out=FAKE, status=None, ws=ws, ws_bytes=n_vt.value)
        a.update(kw)
        return lib.wa_sparse_attn_vt(a["q"], a["k"], a["vt"], a["rp"], a["ci"], None, None, ctypes.byref(s),
                                     ctypes.byref(o) if o is not None else None, a["out"], None, a["status"], a["ws"],
                                     a["ws_bytes"], None)

    assert call(None) == L.WA_ERR_INVALID_ARG
    assert call(opts, vt=None) == L.WA_ERR_INVALID_ARG
    assert call(opts, rp=None) == L.WA_ERR_INVALID_ARG
    assert call(opts, vt=ctypes.c_void_p((1 << 20) + 4)) == L.WA_ERR_ALIGNMENT
    assert call(opts, status=ctypes.c_void_p((1 << 20) + 1)) == L.WA_ERR_ALIGNMENT
    assert call(L.WaAttnOptions(0.0, 0, 0)) == L.WA_ERR_INVALID_ARG
    assert call(L.WaAttnOptions(0.0, 8, 2)) == L.WA_ERR_INVALID_ARG
    assert b"head_order" in lib.wa_last_error()
    assert call(opts, ws_bytes=n_vt.value - 1) == L.WA_ERR_WORKSPACE
    assert lib.wa_transpose_v(None, ctypes.byref(s), FAKE, None) == L.WA_ERR_INVALID_ARG
    assert lib.wa_transpose_v(FAKE, ctypes.byref(s), ctypes.c_void_p((1 << 20) + 2), None) == L.WA_ERR_ALIGNMENT
    assert lib.wa_transpose_v(FAKE, ctypes.byref(_shape(head_dim=96)), FAKE, None) == L.WA_ERR_UNSUPPORTED


def test_produce_block_mask_validation():
    lib = _lib()
    s = _shape()
    ws_n = ctypes.c_size_t(0)
    assert lib.wa_mask_producer_workspace_size(ctypes.byref(s), ctypes.byref(ws_n)) == 0
    b, h, mb, d = s.batch, s.heads, -(-s.seq_len // s.block), s.head_dim
    assert ws_n.value >= 2 * b * h * mb * d * 5
    args = dict(q=FAKE, k=FAKE, keep=8, mask=FAKE, codes=None, status=None, ws=ctypes.c_void_p(1 << 24),
                ws_bytes=ws_n.value)

    def call(**kw):
        a = dict(args)
        a.update(kw)
        return lib.wa_produce_block_mask(a["q"], a["k"], ctypes.byref(s), a["keep"], 1, a["mask"], a["codes"],
                                         a["status"], a["ws"], a["ws_bytes"], None)

    assert call(q=None) == L.WA_ERR_INVALID_ARG
    assert call(k=None) == L.WA_ERR_INVALID_ARG
    assert call(mask=None) == L.WA_ERR_INVALID_ARG
    assert call(keep=-1) == L.WA_ERR_INVALID_ARG
    assert call(q=ctypes.c_void_p((1 << 20) + 2)) == L.WA_ERR_ALIGNMENT
    assert call(codes=ctypes.c_void_p((1 << 20) + 8)) == L.WA_ERR_ALIGNMENT
    assert call(status=ctypes.c_void_p((1 << 20) + 2)) == L.WA_ERR_ALIGNMENT
    assert call(ws=None) == L.WA_ERR_INVALID_ARG
    assert call(ws_bytes=ws_n.value - 1) == L.WA_ERR_WORKSPACE
    bad = L.WaShape(1, 1, 100, 96, 64)
    assert lib.wa_produce_block_mask(FAKE, FAKE, ctypes.byref(bad), 4, 1, FAKE, None, None, ctypes.c_void_p(1 << 24),
                                     1 << 30, None) == L.WA_ERR_UNSUPPORTED


def test_check_perm_validation():
    lib = _lib()
    s = _shape()
    n = ctypes.c_size_t(0)
    assert lib.wa_check_perm_workspace_size(ctypes.byref(s), ctypes.byref(n)) == 0 and n.value >= 4
    ws = ctypes.c_void_p(1 << 24)
    assert lib.wa_check_perm(None, ctypes.byref(s), None, ws, n.value, None) == L.WA_ERR_INVALID_ARG
    assert lib.wa_check_perm(FAKE, ctypes.byref(s), None, ws, 0, None) == L.WA_ERR_WORKSPACE
    assert lib.wa_check_perm(FAKE, ctypes.byref(s), None, None, n.value, None) == L.WA_ERR_INVALID_ARG
    assert lib.wa_status_string(L.WA_ERR_INVALID_PERM) == b"not a permutation"


def test_build_permutation_validation():
    lib = _lib()
    s = _shape()
    ws_n = ctypes.c_size_t(0)
    lib.wa_perm_workspace_size(ctypes.byref(s), ctypes.byref(ws_n))
    ws = ctypes.c_void_p(1 << 24)

    def call(params, mask=FAKE, perm=FAKE, wsb=ws_n.value, wsp=ws):
        return lib.wa_build_permutation(mask, ctypes.byref(s), ctypes.byref(params) if params else None, perm,
                                        None, None, None, None, wsp, wsb, None)

    good = dict(wave_per_xcd=64, n_xcd=8, iters=10, skip_mode=0, seed=0, profile=None)

    def P(**kw):
        d = dict(good)
        d.update(kw)
        return L.WaPermParams(**d)

    assert call(None) == L.WA_ERR_INVALID_ARG
    assert call(P(), mask=None) == L.WA_ERR_INVALID_ARG
    assert call(P(), perm=None) == L.WA_ERR_INVALID_ARG
    assert call(P(n_xcd=0)) == L.WA_ERR_INVALID_ARG
    assert call(P(iters=0)) == L.WA_ERR_INVALID_ARG
    assert call(P(iters=65)) == L.WA_ERR_INVALID_ARG
    assert call(P(skip_mode=3)) == L.WA_ERR_INVALID_ARG
    assert call(P(wave_per_xcd=-1)) == L.WA_ERR_INVALID_ARG
    assert call(P(), wsb=ws_n.value - 8) == L.WA_ERR_WORKSPACE
    assert call(P(), wsp=ctypes.c_void_p((1 << 24) + 8)) == L.WA_ERR_ALIGNMENT
    assert lib.wa_compact_mask(None, ctypes.byref(s), FAKE, FAKE, None) == L.WA_ERR_INVALID_ARG
    assert lib.wa_mask_stats(FAKE, ctypes.byref(s), None, FAKE, FAKE, ws, ws_n.value, None) == L.WA_ERR_INVALID_ARG
    assert lib.wa_fp64_probe(None, FAKE, FAKE, FAKE, 4, None) == L.WA_ERR_INVALID_ARG
    assert lib.wa_xcc_probe(None, 4, None) == L.WA_ERR_INVALID_ARG
    out = ctypes.c_int32(0)
    assert lib.wa_wave_size(96, 128, ctypes.byref(out)) == L.WA_ERR_UNSUPPORTED
    assert lib.wa_wave_size(128, 128, None) == L.WA_ERR_INVALID_ARG


def test_product_path_fails_loudly_without_library(tmp_path):
    with pytest.raises(ImportError):
        L._LIB_SAVED = L._LIB
        try:
            L._LIB = None
            L.load(str(tmp_path / "missing.so"))
        finally:
            L._LIB = L._LIB_SAVED


# ------------------------------------------------------------------------------------------------
# the Python binding rejects mismatched shapes and dtypes before any device work (CPU tensors here:
# the shape checks come before the placement check)
# ------------------------------------------------------------------------------------------------
def _cpu_args(b=1, h=2, n=300, d=64, blk=64):
    import torch
    mb = -(-n // blk)
    q = torch.zeros((b, h, n, d), dtype=torch.bfloat16)
    return dict(q=q, k=q.clone(), v=q.clone(), mask=torch.zeros((b, h, mb, mb), dtype=torch.uint8),
                perm=torch.zeros((b, h, mb), dtype=torch.int32), seg=torch.zeros((b, h, 9), dtype=torch.int32),
                rp=torch.zeros((b, h, mb + 1), dtype=torch.int32), ci=torch.zeros(b * h * mb * mb, dtype=torch.int32),
                vt=torch.zeros((b, h, d, mb * blk), dtype=torch.bfloat16), mb=mb, blk=blk, n=n, d=d)


@pytest.mark.parametrize("case,match", [
    ("mask_shape", "mask must have shape"),
    ("mask_dtype", "mask must be uint8"),
    ("perm_shape", "perm must have shape"),
    ("perm_dtype", "perm must be torch.int32"),
    ("seg_for_other_n_xcd", "seg must have shape"),
    ("n_xcd", "n_xcd"),
    ("out_shape", "out must have shape"),
    ("status_dtype", "status must be torch.int32"),
    ("not_on_device", "must be a device tensor"),
])
def test_binding_rejects_bad_sparse_attn_arguments(case, match):
    import torch
    _lib()
    import paper_2609_34814_amd as W
    a = _cpu_args()
    kw = dict(block=a["blk"], n_xcd=8)
    mask, perm, seg = a["mask"], a["perm"], a["seg"]
    if case == "mask_shape":
        mask = torch.zeros((1, 2, a["mb"], a["mb"] + 1), dtype=torch.uint8)
    elif case == "mask_dtype":
        mask = mask.to(torch.int32)
    elif case == "perm_shape":
        perm = torch.zeros((1, 2, a["mb"] + 1), dtype=torch.int32)
    elif case == "perm_dtype":
        perm = perm.to(torch.int64)
    elif case == "seg_for_other_n_xcd":
        seg = torch.zeros((1, 2, 2), dtype=torch.int32)    # built with n_xcd = 1, passed with 8
    elif case == "n_xcd":
        kw["n_xcd"] = 65
    elif case == "out_shape":
        kw["out"] = torch.zeros((1, 2, a["n"] - 1, a["d"]), dtype=torch.bfloat16)
    elif case == "status_dtype":
        kw["status"] = torch.zeros(1, dtype=torch.int64)
    with pytest.raises(ValueError, match=match):
        W.sparse_attn(a["q"], a["k"], a["v"], mask, perm, seg, **kw)


@pytest.mark.parametrize("case,match", [
    ("row_ptr_shape", "row_ptr must have shape"),
    ("row_ptr_dtype", "row_ptr must be torch.int32"),
    ("col_idx_small", "col_idx must hold at least"),
    ("vt_shape", "vt must have shape"),
    ("head_order", "head_order"),
])
def test_binding_rejects_bad_list_and_vt_arguments(case, match):
    import torch
    _lib()
    import paper_2609_34814_amd as W
    a = _cpu_args()
    rp, ci, vt = a["rp"], a["ci"], a["vt"]
    kw = dict(block=a["blk"], n_xcd=8)
    if case == "row_ptr_shape":
        rp = torch.zeros((1, 2, a["mb"]), dtype=torch.int32)
    elif case == "row_ptr_dtype":
        rp = rp.to(torch.int64)
    elif case == "col_idx_small":
        ci = ci[:-1]
    elif case == "vt_shape":
        vt = torch.zeros((1, 2, a["d"], a["n"]), dtype=torch.bfloat16)   # not padded to whole blocks
    elif case == "head_order":
        kw["head_order"] = "by-xcd"
    with pytest.raises(ValueError, match=match):
        if case in ("vt_shape", "head_order"):
            W.sparse_attn_vt(a["q"], a["k"], vt, rp, ci, **kw)
        else:
            W.sparse_attn_csr(a["q"], a["k"], a["v"], rp, ci, **kw)
    if case in ("row_ptr_shape", "row_ptr_dtype", "col_idx_small"):
        with pytest.raises(ValueError, match=match):
            W.sparse_attn_vt(a["q"], a["k"], a["vt"], rp, ci, **kw)


def test_binding_rejects_bad_permutation_outputs():
    import torch
    _lib()
    import paper_2609_34814_amd as W
    a = _cpu_args()
    with pytest.raises(ValueError, match="seg_out must have shape"):
        W.build_permutation(a["mask"], seq_len=a["n"], block=a["blk"], head_dim=a["d"], n_xcd=1,
                            seg_out=torch.zeros((1, 2, 9), dtype=torch.int32))
    with pytest.raises(ValueError, match="mask must have shape"):
        W.build_permutation(a["mask"], seq_len=a["n"] + a["blk"], block=a["blk"], head_dim=a["d"])
    with pytest.raises(ValueError, match="skip must be one of"):
        W.build_permutation(a["mask"], seq_len=a["n"], block=a["blk"], head_dim=a["d"], skip="sometimes")
    with pytest.raises(ValueError, match="row_ptr must have shape"):
        W.compact_mask(a["mask"], seq_len=a["n"], block=a["blk"], row_ptr=torch.zeros(3, dtype=torch.int32))


def test_noalloc_rejects_state_beyond_its_static_scratch():
    """20,000 heads of 64 blocks need a 5 MB scheduler state, more than the static scratch: the call
    fails before anything is enqueued (the device pointers here are never dereferenced)."""
    lib = _lib()
    s = L.WaShape(1, 20000, 64 * 64, 64, 64)
    opts = L.WaAttnOptions(0.0, 1, L.WA_HEADS_IN_ORDER)
    assert lib.wa_sparse_attn_vt_noalloc(FAKE, FAKE, FAKE, FAKE, FAKE, None, None, ctypes.byref(s),
                                         ctypes.byref(opts), FAKE, None, None, None) == L.WA_ERR_WORKSPACE
    assert b"static scratch" in lib.wa_last_error()
    assert lib.wa_sparse_attn_vt_noalloc(FAKE, FAKE, FAKE, FAKE, FAKE, None, None, ctypes.byref(s), None, FAKE,
                                         None, None, None) == L.WA_ERR_INVALID_ARG
    assert L.WA_NOALLOC_SCRATCH_BYTES == 4 * 1024 * 1024
