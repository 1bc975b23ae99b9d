"""Per-row KV-block index lists (test infrastructure only).

The backend's inner loop visits, for query block i, exactly the KV blocks j with
M[i, j] = 1 (Sec. II-C). The compacted form is a CSR per head:

    row_ptr[b][h][i] = sum_{i' < i} n_{i'}          (exclusive prefix sum of row counts,
                                                     offsets local to the head)
    col_idx[b][h][row_ptr[i] : row_ptr[i+1]] = ascending j with M[i, j] = 1

where n_i = sum_j M[i, j] (Sec. II-B). Head (b, h)'s list occupies the slice
starting at (b*H + h) * M_B * N_B of a buffer sized for a full mask.
"""
from __future__ import annotations

import numpy as np


def compact_head(mask_h: np.ndarray):
    """(row_ptr [M_B+1] int32, col_idx [nnz] int32) for one head."""
    m = mask_h.shape[0]
    row_ptr = np.zeros(m + 1, dtype=np.int64)
    cols = []
    for i in range(m):
        nz = np.nonzero(mask_h[i])[0]
        cols.append(nz)
        row_ptr[i + 1] = row_ptr[i] + nz.size
    col_idx = np.concatenate(cols) if cols else np.zeros(0, dtype=np.int64)
    return row_ptr.astype(np.int32), col_idx.astype(np.int32)


def compact_mask(mask: np.ndarray):
    """CSR of a [B][H][M_B][N_B] mask.

    Returns (row_ptr [B][H][M_B+1] int32, lists) where ``lists[b][h]`` is the
    head's col_idx array (its length is row_ptr[b][h][-1]).
    """
    b_, h_, m, _ = mask.shape
    row_ptr = np.zeros((b_, h_, m + 1), dtype=np.int32)
    lists = [[None] * h_ for _ in range(b_)]
    for b in range(b_):
        for h in range(h_):
            row_ptr[b, h], lists[b][h] = compact_head(mask[b, h])
    return row_ptr, lists
