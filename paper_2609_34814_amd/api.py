"""Python binding of the block-sparse attention path (argument marshalling only).

Every computation runs in the HIP kernels of libwavealign.so; torch supplies
device memory and the current HIP stream.
"""
from __future__ import annotations

import ctypes
import math
from typing import Optional

import torch

from . import _lib as L

_SKIP = {"auto": L.WA_SKIP_AUTO, "never": L.WA_SKIP_NEVER, "always": L.WA_SKIP_ALWAYS}
_HEAD_ORDER = {"in-order": L.WA_HEADS_IN_ORDER, "interleaved": L.WA_HEADS_INTERLEAVED}


def _stream() -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dev(t: torch.Tensor, name: str) -> None:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _mask_u8(mask: torch.Tensor, shape=None) -> torch.Tensor:
    """The mask as uint8, checked against the expected [B][H][M_B][N_B] shape (if given) before
    its placement, so that a mismatch is reported the same way on any device."""
    if mask.dtype not in (torch.bool, torch.uint8):
        raise ValueError("mask must be uint8 or bool")
    if mask.dim() != 4 or (shape is not None and tuple(mask.shape) != tuple(shape)):
        want = "[B][H][M_B][N_B]" if shape is None else str(tuple(shape))
        raise ValueError(f"mask must have shape {want}, got {tuple(mask.shape)}")
    if mask.shape[2] != mask.shape[3]:
        raise ValueError(f"mask must be square per head (M_B = N_B), got {tuple(mask.shape)}")
    return mask.view(torch.uint8) if mask.dtype == torch.bool else mask


def _check(t: Optional[torch.Tensor], name: str, dtype, shape=None, numel_min: Optional[int] = None) -> None:
    """dtype and shape (or minimum element count) of an optional tensor argument."""
    if t is None:
        return
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if numel_min is not None and t.numel() < numel_min:
        raise ValueError(f"{name} must hold at least {numel_min} elements, got {t.numel()}")


def _on_device(**tensors) -> None:
    """Placement and layout, checked once every shape is known to be right."""
    for name, t in tensors.items():
        if t is not None:
            _dev(t, name)


def _mask_dims(mask: torch.Tensor, seq_len: int, block: int):
    b, h = mask.shape[0], mask.shape[1]
    mb = -(-seq_len // block)
    return b, h, mb


def shape_of(batch: int, heads: int, seq_len: int, head_dim: int, block: int) -> L.WaShape:
    return L.WaShape(batch, heads, seq_len, head_dim, block)


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def wave_size(head_dim: int, block: int) -> int:
    lib = L.load()
    out = ctypes.c_int32(0)
    L.check(lib.wa_wave_size(head_dim, block, ctypes.byref(out)))
    return out.value


def default_skip_profile() -> L.WaSkipProfile:
    lib = L.load()
    p = L.WaSkipProfile()
    L.check(lib.wa_default_skip_profile(ctypes.byref(p)))
    return p


def perm_workspace_size(shape: L.WaShape) -> int:
    lib = L.load()
    n = ctypes.c_size_t(0)
    L.check(lib.wa_perm_workspace_size(ctypes.byref(shape), ctypes.byref(n)))
    return n.value


def attn_workspace_size(shape: L.WaShape) -> int:
    lib = L.load()
    n = ctypes.c_size_t(0)
    L.check(lib.wa_attn_workspace_size(ctypes.byref(shape), ctypes.byref(n)))
    return n.value


def mask_stats(mask: torch.Tensor, *, seq_len: int, block: int, head_dim: int = 128):
    """(row_nnz [B][H][M_B], col_cnt [B][H][N_B], head_stats [B][H][6]) as device tensors."""
    lib = L.load()
    b, h, mb = _mask_dims(mask, seq_len, block)
    mask = _mask_u8(mask, (b, h, mb, mb))
    _on_device(mask=mask)
    shape = shape_of(b, h, seq_len, head_dim, block)
    dev = mask.device
    row_nnz = torch.empty((b, h, mb), dtype=torch.int32, device=dev)
    col_cnt = torch.empty((b, h, mb), dtype=torch.int32, device=dev)
    stats = torch.empty((b, h, 6), dtype=torch.int64, device=dev)
    ws = _workspace(perm_workspace_size(shape), dev)
    L.check(lib.wa_mask_stats(_ptr(mask), ctypes.byref(shape), _ptr(row_nnz), _ptr(col_cnt), _ptr(stats),
                              _ptr(ws), ws.numel(), _stream()))
    return row_nnz, col_cnt, stats


def build_permutation(mask: torch.Tensor, *, seq_len: int, block: int, head_dim: int, wave: Optional[int] = None,
                      n_xcd: int = 8, iters: int = 10, seed: int = 0, skip: str = "auto",
                      profile: Optional[L.WaSkipProfile] = None, workspace: Optional[torch.Tensor] = None,
                      return_info: bool = False, out: Optional[torch.Tensor] = None,
                      flags_out: Optional[torch.Tensor] = None, seg_out: Optional[torch.Tensor] = None,
                      stage1_out: Optional[torch.Tensor] = None):
    """(perm int32 [B][H][M_B], seg_start int32 [B][H][n_xcd+1], head flags uint8 [B][H])
    (plus embedding and Stage-1 order if asked; stage1_out, if given, receives the Stage-1 order)."""
    lib = L.load()
    b, h, mb = _mask_dims(mask, seq_len, block)
    mask = _mask_u8(mask, (b, h, mb, mb))
    if skip not in _SKIP:
        raise ValueError(f"skip must be one of {sorted(_SKIP)}")
    _check(out, "out", torch.int32, (b, h, mb))
    _check(flags_out, "flags_out", torch.uint8, (b, h))
    _check(seg_out, "seg_out", torch.int32, (b, h, n_xcd + 1))
    _check(stage1_out, "stage1_out", torch.int32, (b, h, mb))
    _check(workspace, "workspace", torch.uint8)
    _on_device(mask=mask, out=out, flags_out=flags_out, seg_out=seg_out, stage1_out=stage1_out, workspace=workspace)
    shape = shape_of(b, h, seq_len, head_dim, block)
    dev = mask.device
    perm = torch.empty((b, h, mb), dtype=torch.int32, device=dev) if out is None else out
    flags = torch.empty((b, h), dtype=torch.uint8, device=dev) if flags_out is None else flags_out
    seg = torch.empty((b, h, n_xcd + 1), dtype=torch.int32, device=dev) if seg_out is None else seg_out
    emb = torch.empty((b, h, mb, 2), dtype=torch.int32, device=dev) if return_info else None
    s1 = torch.empty((b, h, mb), dtype=torch.int32, device=dev) if return_info and stage1_out is None else stage1_out
    params = L.WaPermParams(0 if wave is None else int(wave), int(n_xcd), int(iters), _SKIP[skip],
                            int(seed) & ((1 << 64) - 1),
                            ctypes.pointer(profile) if profile is not None else None)
    need = perm_workspace_size(shape)
    if workspace is None or workspace.numel() < need:
        workspace = _workspace(need, dev)
    L.check(lib.wa_build_permutation(_ptr(mask), ctypes.byref(shape), ctypes.byref(params), _ptr(perm), _ptr(seg),
                                     _ptr(flags), _ptr(emb), _ptr(s1), _ptr(workspace), workspace.numel(),
                                     _stream()))
    if return_info:
        return perm, seg, flags, emb, s1
    return perm, seg, flags


def compact_mask(mask: torch.Tensor, *, seq_len: int, block: int, head_dim: int = 128,
                 row_ptr: Optional[torch.Tensor] = None, col_idx: Optional[torch.Tensor] = None):
    """CSR lists: row_ptr int32 [B][H][M_B+1] (head-local offsets), col_idx int32 [B*H*M_B*N_B]."""
    lib = L.load()
    b, h, mb = _mask_dims(mask, seq_len, block)
    mask = _mask_u8(mask, (b, h, mb, mb))
    _check(row_ptr, "row_ptr", torch.int32, (b, h, mb + 1))
    _check(col_idx, "col_idx", torch.int32, numel_min=b * h * mb * mb)
    _on_device(mask=mask, row_ptr=row_ptr, col_idx=col_idx)
    shape = shape_of(b, h, seq_len, head_dim, block)
    if row_ptr is None:
        row_ptr = torch.empty((b, h, mb + 1), dtype=torch.int32, device=mask.device)
    if col_idx is None:
        col_idx = torch.empty((b * h * mb * mb,), dtype=torch.int32, device=mask.device)
    L.check(lib.wa_compact_mask(_ptr(mask), ctypes.byref(shape), _ptr(row_ptr), _ptr(col_idx), _stream()))
    return row_ptr, col_idx


def mask_producer_workspace_size(shape: L.WaShape) -> int:
    lib = L.load()
    n = ctypes.c_size_t(0)
    L.check(lib.wa_mask_producer_workspace_size(ctypes.byref(shape), ctypes.byref(n)))
    return n.value


def produce_block_mask(q: torch.Tensor, k: torch.Tensor, *, block: int, keep: int, diagonal: bool = True,
                       out: Optional[torch.Tensor] = None, codes_out: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None, status: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Pooled-score top-k block mask uint8 [B][H][M_B][M_B] from q, k bf16 [B][H][N][d]. ``status``: an int32
    device tensor of one element the call zeroes and sets WA_PRODUCE_WAIT_EXPIRED in (nullable)."""
    lib = L.load()
    for t, nm in ((q, "q"), (k, "k")):
        _dev(t, nm)
        if t.dtype != torch.bfloat16:
            raise ValueError(f"{nm} must be bfloat16")
    if q.shape != k.shape or q.dim() != 4:
        raise ValueError("q and k must share one [B][H][N][d] shape")
    b, h, n, d = q.shape
    shape = shape_of(b, h, n, d, block)
    mb = -(-n // block)
    mask = torch.empty((b, h, mb, mb), dtype=torch.uint8, device=q.device) if out is None else out
    if mask.dtype != torch.uint8 or mask.numel() < b * h * mb * mb:
        raise ValueError("out must be a uint8 tensor of B*H*M_B*M_B elements")
    if codes_out is not None and (codes_out.dtype != torch.int8 or codes_out.numel() < 2 * b * h * mb * d):
        raise ValueError("codes_out must be an int8 tensor of 2*B*H*M_B*d elements")
    if status is not None and (status.dtype != torch.int32 or status.numel() < 1):
        raise ValueError("status must be an int32 tensor of at least one element")
    need = mask_producer_workspace_size(shape)
    if workspace is None or workspace.numel() < need:
        workspace = _workspace(need, q.device)
    L.check(lib.wa_produce_block_mask(_ptr(q), _ptr(k), ctypes.byref(shape), int(keep), 1 if diagonal else 0,
                                      _ptr(mask), _ptr(codes_out), _ptr(status), _ptr(workspace), workspace.numel(),
                                      _stream()))
    return mask


def check_perm(perm: torch.Tensor, *, seq_len: int, block: int, head_dim: int = 128,
               head_ok: Optional[torch.Tensor] = None) -> bool:
    """True if every perm[b][h] is a permutation of 0..M_B-1 (synchronises the current stream)."""
    lib = L.load()
    _dev(perm, "perm")
    if perm.dtype != torch.int32 or perm.dim() != 3:
        raise ValueError("perm must be an int32 [B][H][M_B] tensor")
    b, h, mb = perm.shape
    shape = shape_of(b, h, seq_len, head_dim, block)
    if -(-seq_len // block) != mb:
        raise ValueError("perm's last dimension must be ceil(seq_len / block)")
    n = ctypes.c_size_t(0)
    L.check(lib.wa_check_perm_workspace_size(ctypes.byref(shape), ctypes.byref(n)))
    ws = _workspace(n.value, perm.device)
    st = lib.wa_check_perm(_ptr(perm.contiguous()), ctypes.byref(shape), _ptr(head_ok), _ptr(ws), ws.numel(),
                           _stream())
    if st == L.WA_ERR_INVALID_PERM:
        return False
    L.check(st)
    return True


def _attn_args(q, k, v, block, v_transposed=False):
    """Shape of the call from q, k, v (checked before their placement); v may be the transposed
    [B][H][d][M_B*block] layout."""
    for t, nm in ((q, "q"), (k, "k"), (v, "v")):
        if t.dtype != torch.bfloat16:
            raise ValueError(f"{nm} must be bfloat16")
    if q.dim() != 4 or q.shape != k.shape:
        raise ValueError("q and k must share one [B][H][N][d] shape")
    b, h, n, d = q.shape
    if v_transposed:
        want = (b, h, d, -(-n // block) * block)
        if tuple(v.shape) != want:
            raise ValueError(f"vt must have shape {want} ([B][H][d][M_B*block]), got {tuple(v.shape)}")
    elif v.shape != q.shape:
        raise ValueError("q, k, v must share one [B][H][N][d] shape")
    return shape_of(b, h, n, d, block)


def _attn_outputs(q, out, status, return_lse):
    _check(out, "out", torch.bfloat16, tuple(q.shape))
    _check(status, "status", torch.int32, numel_min=1)
    if out is None or return_lse:
        _on_device(q=q)
    o = torch.empty_like(q) if out is None else out
    lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device) if return_lse else None
    return o, lse


def _order_args(q, block, perm, seg, n_xcd):
    b, h, n, _ = q.shape
    mb = -(-n // block)
    if not 1 <= int(n_xcd) <= 64:
        raise ValueError("n_xcd must lie in 1..64")
    _check(perm, "perm", torch.int32, (b, h, mb))
    _check(seg, "seg", torch.int32, (b, h, int(n_xcd) + 1))
    return b, h, mb


def _csr_args(row_ptr, col_idx, b, h, mb):
    if row_ptr is None or col_idx is None:
        raise ValueError("row_ptr and col_idx are required")
    _check(row_ptr, "row_ptr", torch.int32, (b, h, mb + 1))
    _check(col_idx, "col_idx", torch.int32, numel_min=b * h * mb * mb)


def sparse_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, mask: torch.Tensor,
                perm: Optional[torch.Tensor] = None, seg: Optional[torch.Tensor] = None, *, block: int,
                scale: Optional[float] = None,
                n_xcd: int = 8, return_lse: bool = False, out: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None, status: Optional[torch.Tensor] = None):
    """O = block-sparse softmax attention of q over the kept KV blocks, in the original row order.
    `status` (int32, device) receives the call's WA_ATTN_* bits."""
    lib = L.load()
    shape = _attn_args(q, k, v, block)
    b, h, mb = _order_args(q, block, perm, seg, n_xcd)
    mask = _mask_u8(mask, (b, h, mb, mb))
    _check(workspace, "workspace", torch.uint8)
    o, lse = _attn_outputs(q, out, status, return_lse)
    _on_device(q=q, k=k, v=v, mask=mask, perm=perm, seg=seg, out=o, status=status, workspace=workspace)
    need = attn_workspace_size(shape)
    if workspace is None or workspace.numel() < need:
        workspace = _workspace(need, q.device)
    L.check(lib.wa_sparse_attn(_ptr(q), _ptr(k), _ptr(v), _ptr(mask), _ptr(perm), _ptr(seg), ctypes.byref(shape),
                               float(scale or 0.0), int(n_xcd), _ptr(o), _ptr(lse), _ptr(status), _ptr(workspace),
                               workspace.numel(), _stream()))
    return (o, lse) if return_lse else o


def sparse_attn_csr(q, k, v, row_ptr, col_idx, perm=None, seg=None, *, block: int, scale: Optional[float] = None,
                    n_xcd: int = 8, return_lse: bool = False, out: Optional[torch.Tensor] = None,
                    workspace: Optional[torch.Tensor] = None, status: Optional[torch.Tensor] = None):
    """As sparse_attn, from the lists of compact_mask."""
    lib = L.load()
    shape = _attn_args(q, k, v, block)
    b, h, mb = _order_args(q, block, perm, seg, n_xcd)
    _csr_args(row_ptr, col_idx, b, h, mb)
    _check(workspace, "workspace", torch.uint8)
    o, lse = _attn_outputs(q, out, status, return_lse)
    _on_device(q=q, k=k, v=v, row_ptr=row_ptr, col_idx=col_idx, perm=perm, seg=seg, out=o, status=status,
               workspace=workspace)
    need = attn_workspace_size(shape)
    if workspace is None or workspace.numel() < need:
        workspace = _workspace(need, q.device)
    L.check(lib.wa_sparse_attn_csr(_ptr(q), _ptr(k), _ptr(v), _ptr(row_ptr), _ptr(col_idx), _ptr(perm), _ptr(seg),
                                   ctypes.byref(shape), float(scale or 0.0), int(n_xcd), _ptr(o), _ptr(lse),
                                   _ptr(status), _ptr(workspace), workspace.numel(), _stream()))
    return (o, lse) if return_lse else o


def transpose_v(v: torch.Tensor, *, block: int, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """V [B][H][N][d] -> V^T [B][H][d][M_B*block], zero past the last token (the layout of sparse_attn_vt)."""
    lib = L.load()
    if v.dtype != torch.bfloat16 or v.dim() != 4:
        raise ValueError("v must be a bfloat16 [B][H][N][d] tensor")
    b, h, n, d = v.shape
    want = (b, h, d, -(-n // block) * block)
    _check(out, "out", torch.bfloat16, want)
    _on_device(v=v, out=out)
    vt = torch.empty(want, dtype=torch.bfloat16, device=v.device) if out is None else out
    shape = shape_of(b, h, n, d, block)
    L.check(lib.wa_transpose_v(_ptr(v), ctypes.byref(shape), _ptr(vt), _stream()))
    return vt


def attn_vt_workspace_size(shape: L.WaShape) -> int:
    lib = L.load()
    n = ctypes.c_size_t(0)
    L.check(lib.wa_attn_vt_workspace_size(ctypes.byref(shape), ctypes.byref(n)))
    return n.value


def sparse_attn_vt(q, k, vt, row_ptr, col_idx, perm=None, seg=None, *, block: int, scale: Optional[float] = None,
                   n_xcd: int = 8, head_order: str = "in-order", return_lse: bool = False,
                   out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                   status: Optional[torch.Tensor] = None):
    """As sparse_attn_csr with V given as V^T (transpose_v's layout); head_order is "in-order" (heads one
    after another in every queue) or "interleaved" (round-robin over the heads)."""
    lib = L.load()
    if head_order not in _HEAD_ORDER:
        raise ValueError(f"head_order must be one of {sorted(_HEAD_ORDER)}")
    shape = _attn_args(q, k, vt, block, v_transposed=True)
    b, h, mb = _order_args(q, block, perm, seg, n_xcd)
    _csr_args(row_ptr, col_idx, b, h, mb)
    _check(workspace, "workspace", torch.uint8)
    o, lse = _attn_outputs(q, out, status, return_lse)
    _on_device(q=q, k=k, vt=vt, row_ptr=row_ptr, col_idx=col_idx, perm=perm, seg=seg, out=o, status=status,
               workspace=workspace)
    need = attn_vt_workspace_size(shape)
    if workspace is None or workspace.numel() < need:
        workspace = _workspace(need, q.device)
    opts = L.WaAttnOptions(float(scale or 0.0), int(n_xcd), _HEAD_ORDER[head_order])
    L.check(lib.wa_sparse_attn_vt(_ptr(q), _ptr(k), _ptr(vt), _ptr(row_ptr), _ptr(col_idx), _ptr(perm), _ptr(seg),
                                  ctypes.byref(shape), ctypes.byref(opts), _ptr(o), _ptr(lse), _ptr(status),
                                  _ptr(workspace), workspace.numel(), _stream()))
    return (o, lse) if return_lse else o


def sparse_attn_vt_noalloc(q, k, vt, row_ptr, col_idx, perm=None, seg=None, *, block: int,
                           scale: Optional[float] = None, n_xcd: int = 8, head_order: str = "in-order",
                           lse: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                           status: Optional[torch.Tensor] = None) -> torch.Tensor:
    """As sparse_attn_vt, for callers that cannot allocate: the library keeps the scheduler state in
    its static per-GPU scratch, so `out` (and `lse`, if wanted) must be given. Calls that overlap on
    one GPU race."""
    lib = L.load()
    if head_order not in _HEAD_ORDER:
        raise ValueError(f"head_order must be one of {sorted(_HEAD_ORDER)}")
    if out is None:
        raise ValueError("out is required (this entry point allocates nothing)")
    shape = _attn_args(q, k, vt, block, v_transposed=True)
    b, h, mb = _order_args(q, block, perm, seg, n_xcd)
    _csr_args(row_ptr, col_idx, b, h, mb)
    _check(out, "out", torch.bfloat16, tuple(q.shape))
    _check(lse, "lse", torch.float32, tuple(q.shape[:3]))
    _check(status, "status", torch.int32, numel_min=1)
    _on_device(q=q, k=k, vt=vt, row_ptr=row_ptr, col_idx=col_idx, perm=perm, seg=seg, out=out, lse=lse,
               status=status)
    opts = L.WaAttnOptions(float(scale or 0.0), int(n_xcd), _HEAD_ORDER[head_order])
    L.check(lib.wa_sparse_attn_vt_noalloc(_ptr(q), _ptr(k), _ptr(vt), _ptr(row_ptr), _ptr(col_idx), _ptr(perm),
                                          _ptr(seg), ctypes.byref(shape), ctypes.byref(opts), _ptr(out), _ptr(lse),
                                          _ptr(status), _stream()))
    return out


def fp64_probe(a: torch.Tensor, b: torch.Tensor, c: torch.Tensor) -> torch.Tensor:
    lib = L.load()
    out = torch.empty((a.numel(), 6), dtype=torch.float64, device=a.device)
    L.check(lib.wa_fp64_probe(_ptr(a), _ptr(b), _ptr(c), _ptr(out), a.numel(), _stream()))
    return out


def xcc_probe(n_wg: int, device="cuda") -> torch.Tensor:
    lib = L.load()
    out = torch.full((n_wg,), -1, dtype=torch.int32, device=device)
    L.check(lib.wa_xcc_probe(_ptr(out), int(n_wg), _stream()))
    return out


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)
