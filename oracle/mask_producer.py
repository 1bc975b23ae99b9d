"""Pooled-score top-k block mask from Q and K (test infrastructure only).

A content-dependent producer of the binary block mask that the path consumes.
The paper describes the dynamic sparse-attention methods that produce such
masks at run time from online attention statistics, one of them predicting
block relevance from pooled Q/K features (Sec. II-B, "Sparse Attention for
Long-Video Generation"). It prints no formula; this reading:

  1. pooling: for block i (tokens [i*blk, min((i+1)*blk, N)), c_i of them)
        qbar_i[c] = fl32( fl32-sum_t Q[t][c] / c_i ),
     where fl32-sum adds the tokens in ascending order in IEEE float32, each
     addition rounded (Q is bf16, exact in float32); the division is one
     correctly rounded float32 operation. The same for K.
  2. per-head int8 quantisation: a = max_{i,c} |qbar_i[c]| (exact),
     inv = fl32(127 / a), code = rint(fl32(qbar * inv)) (ties to even),
     clamped to [-127, 127]; a = 0 gives all-zero codes. The same for K with
     its own maximum.
  3. block scores s_ij = sum_c qcode_i[c] * kcode_j[c], an exact integer.
  4. row i keeps the k largest scores (equal scores: smaller j first) and,
     with the diagonal option, block j = i as well.

Every step is exact or a single IEEE float32 rounding in a fixed order, so an
independent implementation produces the identical mask.
"""
from __future__ import annotations

import numpy as np

from .attention import block_token_range


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def pooled_means(x_bits: np.ndarray, blk: int) -> np.ndarray:
    """x_bits bf16 [N][d] -> float32 [M_B][d] block means (step 1)."""
    x = bf16_bits_to_f32(x_bits)
    n, d = x.shape
    mb = -(-n // blk)
    acc = np.zeros((mb, d), dtype=np.float32)
    counts = np.zeros(mb, dtype=np.int64)
    for j in range(mb):
        lo, hi = block_token_range(j, blk, n)
        counts[j] = hi - lo
    # fold position t of every block at once, in ascending t; blocks shorter than t+1 are done
    for t in range(blk):
        live = counts > t
        rows = np.nonzero(live)[0] * blk + t
        acc[live] = (acc[live] + x[rows]).astype(np.float32)
    return (acc / counts.astype(np.float32)[:, None]).astype(np.float32)


def quantize(means: np.ndarray) -> np.ndarray:
    """float32 [M_B][d] -> int8 codes (step 2)."""
    a = np.float32(np.abs(means).max()) if means.size else np.float32(0)
    if a == 0:
        return np.zeros(means.shape, dtype=np.int8)
    inv = np.float32(np.float32(127.0) / a)
    scaled = (means * inv).astype(np.float32)
    return np.clip(np.rint(scaled), -127, 127).astype(np.int8)


def block_scores(qcode: np.ndarray, kcode: np.ndarray) -> np.ndarray:
    """Exact int64 [M_B][M_B] scores (step 3). The float64 product is exact (|s| < 2^22)."""
    return (qcode.astype(np.float64) @ kcode.astype(np.float64).T).astype(np.int64)


def topk_rows(scores: np.ndarray, k: int, diagonal: bool) -> np.ndarray:
    """uint8 [M_B][N_B] mask: the k largest entries of each row (ties: smaller column), plus the
    diagonal if asked (step 4)."""
    m, nb = scores.shape
    kk = min(max(k, 0), nb)
    mask = np.zeros((m, nb), dtype=np.uint8)
    if kk > 0:
        # descending score, then ascending column: sort on (-score, column)
        order = np.lexsort((np.broadcast_to(np.arange(nb), (m, nb)), -scores), axis=1)
        rows = np.repeat(np.arange(m), kk)
        mask[rows, order[:, :kk].reshape(-1)] = 1
    if diagonal:
        d = np.arange(min(m, nb))
        mask[d, d] = 1
    return mask


def produce_head(q_bits: np.ndarray, k_bits: np.ndarray, blk: int, k: int, diagonal: bool = True):
    """One head: (mask u8 [M_B][M_B], scores int64, qcode, kcode)."""
    qc = quantize(pooled_means(q_bits, blk))
    kc = quantize(pooled_means(k_bits, blk))
    s = block_scores(qc, kc)
    return topk_rows(s, k, diagonal), s, qc, kc


def produce_mask(q: np.ndarray, k: np.ndarray, blk: int, keep: int, diagonal: bool = True) -> np.ndarray:
    """q, k bf16 bits [B][H][N][d] -> mask uint8 [B][H][M_B][M_B]."""
    b_, h_, n, _ = q.shape
    mb = -(-n // blk)
    out = np.empty((b_, h_, mb, mb), dtype=np.uint8)
    for b in range(b_):
        for h in range(h_):
            out[b, h] = produce_head(q[b, h], k[b, h], blk, keep, diagonal)[0]
    return out
