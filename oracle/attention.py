"""fp64 block-sparse attention: the plain definition (test infrastructure only).

Definition followed (Sec. II-B, II-C): the sequence of N tokens is cut into
blocks of ``blk`` consecutive tokens; block j holds tokens
[j*blk, min((j+1)*blk, N)). Query block i attends only to the key/value blocks j
with M[i, j] = 1. For a query token q in block i the output is

    O_q = sum_k softmax_k(scale * <Q_q, K_k>) V_k,   k over tokens of kept blocks,

with the usual scale 1/sqrt(d) (the paper does not state one). A query block
with no kept block produces O = 0 and log-sum-exp -inf (the paper is silent;
this is our reading). Reordering query rows does not change any O_q
(Sec. IV-A): each row's result depends only on its own mask row.

Inputs are bf16 bit patterns (uint16); they are widened exactly to fp64.
"""
from __future__ import annotations

import math
from typing import Iterable, Optional

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def block_token_range(j: int, blk: int, n: int):
    return j * blk, min((j + 1) * blk, n)


def attend_block_row(qb: np.ndarray, kf: np.ndarray, vf: np.ndarray, mask_row: np.ndarray,
                     blk: int, scale: float):
    """O and LSE (natural log) for one query block ``qb`` [rows][d] against its kept KV blocks."""
    n = kf.shape[0]
    cols = np.nonzero(mask_row)[0]
    rows, d = qb.shape
    if cols.size == 0:
        return np.zeros((rows, d)), np.full(rows, -np.inf)
    keys = np.concatenate([np.arange(*block_token_range(int(j), blk, n)) for j in cols])
    s = (qb @ kf[keys].T) * scale
    mx = s.max(axis=1, keepdims=True)
    p = np.exp(s - mx)
    den = p.sum(axis=1, keepdims=True)
    o = (p @ vf[keys]) / den
    lse = mx[:, 0] + np.log(den[:, 0])
    return o, lse


def block_sparse_attention(q, k, v, mask, blk: int, scale: Optional[float] = None):
    """Full fp64 result. q,k,v: bf16 bits [B][H][N][d]; mask: [B][H][M_B][N_B] (nonzero = keep).

    Returns (O [B][H][N][d] fp64, LSE [B][H][N] fp64).
    """
    b_, h_, n, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    mb = -(-n // blk)
    assert mask.shape == (b_, h_, mb, mb), (mask.shape, (b_, h_, mb, mb))
    o = np.zeros((b_, h_, n, d))
    lse = np.zeros((b_, h_, n))
    for b in range(b_):
        for h in range(h_):
            qf, kf, vf = bf16_to_f64(q[b, h]), bf16_to_f64(k[b, h]), bf16_to_f64(v[b, h])
            for i in range(mb):
                lo, hi = block_token_range(i, blk, n)
                o[b, h, lo:hi], lse[b, h, lo:hi] = attend_block_row(qf[lo:hi], kf, vf, mask[b, h, i], blk, scale)
    return o, lse


def block_sparse_attention_rows(q, k, v, mask, blk: int, picks: Iterable, scale: Optional[float] = None):
    """fp64 result for selected query blocks only: ``picks`` is an iterable of (b, h, i).

    Returns {(b, h, i): (O_block [rows][d], LSE [rows])}. Used on sizes where the
    full oracle would take too long; each block is computed exactly as above.
    """
    b_, h_, n, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = {}
    by_head = {}
    for b, h, i in picks:
        by_head.setdefault((int(b), int(h)), []).append(int(i))
    for (b, h), rows in by_head.items():
        kf, vf = bf16_to_f64(k[b, h]), bf16_to_f64(v[b, h])
        for i in rows:
            lo, hi = block_token_range(i, blk, n)
            qb = bf16_to_f64(q[b, h, lo:hi])
            out[(b, h, i)] = attend_block_row(qb, kf, vf, mask[b, h, i], blk, scale)
    return out


def dense_attention(q, k, v, scale: Optional[float] = None):
    """Textbook full softmax attention in fp64 for one head: q,k,v bf16 bits [N][d]."""
    qf, kf, vf = bf16_to_f64(q), bf16_to_f64(k), bf16_to_f64(v)
    if scale is None:
        scale = 1.0 / math.sqrt(qf.shape[1])
    s = qf @ kf.T * scale
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    return (p / p.sum(axis=1, keepdims=True)) @ vf


def token_masked_attention(q, k, v, mask, blk: int, scale: Optional[float] = None):
    """Brute force for one head: expand the block mask to tokens and use -inf scores.

    Rows whose every score is -inf produce 0. Only for tiny inputs.
    """
    qf, kf, vf = bf16_to_f64(q), bf16_to_f64(k), bf16_to_f64(v)
    n, d = qf.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    tok = np.arange(n) // blk
    allowed = np.asarray(mask, dtype=bool)[tok[:, None], tok[None, :]]
    s = np.where(allowed, qf @ kf.T * scale, -np.inf)
    o = np.zeros((n, d))
    for r in range(n):
        if not allowed[r].any():
            continue
        e = np.exp(s[r] - s[r].max())
        o[r] = (e / e.sum()) @ vf
    return o
