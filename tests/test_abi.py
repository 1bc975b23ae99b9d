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
    assert lib.wa_abi_version() == 1
    for code in (0, -1, -2, -3, -4, -6):
        assert lib.wa_status_string(code)
    p = L.WaSkipProfile()
    assert lib.wa_default_skip_profile(ctypes.byref(p)) == 0
    assert p.cache_bytes == 96 * 1024 * 1024 and p.j_max == 0.2 and p.eta_min == 0.05
    assert lib.wa_default_skip_profile(None) == L.WA_ERR_INVALID_ARG


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
                                  a["n_xcd"], a["o"], None, a["ws"], a["ws_bytes"], None)

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
    assert lib.wa_sparse_attn_csr(FAKE, FAKE, FAKE, None, FAKE, None, None, ctypes.byref(s), 0.0, 8, FAKE, None,
                                  ctypes.c_void_p(1 << 24), ws_n.value, None) == L.WA_ERR_INVALID_ARG
    assert lib.wa_sparse_attn_csr(FAKE, FAKE, FAKE, FAKE, FAKE, None, None, ctypes.byref(s), 0.0, 8, FAKE, None,
                                  ctypes.c_void_p(1 << 24), 256, None) == L.WA_ERR_WORKSPACE


def test_produce_block_mask_validation():
    lib = _lib()
    s = _shape()
    ws_n = ctypes.c_size_t(0)
    assert lib.wa_mask_producer_workspace_size(ctypes.byref(s), ctypes.byref(ws_n)) == 0
    b, h, mb, d = s.batch, s.heads, -(-s.seq_len // s.block), s.head_dim
    assert ws_n.value >= 2 * b * h * mb * d * 5
    args = dict(q=FAKE, k=FAKE, keep=8, mask=FAKE, codes=None, ws=ctypes.c_void_p(1 << 24), ws_bytes=ws_n.value)

    def call(**kw):
        a = dict(args)
        a.update(kw)
        return lib.wa_produce_block_mask(a["q"], a["k"], ctypes.byref(s), a["keep"], 1, a["mask"], a["codes"],
                                         a["ws"], a["ws_bytes"], None)

    assert call(q=None) == L.WA_ERR_INVALID_ARG
    assert call(k=None) == L.WA_ERR_INVALID_ARG
    assert call(mask=None) == L.WA_ERR_INVALID_ARG
    assert call(keep=-1) == L.WA_ERR_INVALID_ARG
    assert call(q=ctypes.c_void_p((1 << 20) + 2)) == L.WA_ERR_ALIGNMENT
    assert call(codes=ctypes.c_void_p((1 << 20) + 8)) == L.WA_ERR_ALIGNMENT
    assert call(ws=None) == L.WA_ERR_INVALID_ARG
    assert call(ws_bytes=ws_n.value - 1) == L.WA_ERR_WORKSPACE
    bad = L.WaShape(1, 1, 100, 96, 64)
    assert lib.wa_produce_block_mask(FAKE, FAKE, ctypes.byref(bad), 4, 1, FAKE, None, ctypes.c_void_p(1 << 24),
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
