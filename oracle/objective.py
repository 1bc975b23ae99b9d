"""The row-ordering objective of Eq. 1 (diagnostic; test infrastructure only).

For a permutation of the rows cut into consecutive waves of at most W rows,
Eq. 1 sums, over waves, the squared distances ||S[i] - S[j]||^2 between every
pair of rows of the same wave. For 0/1 rows the squared distance is the size of
the symmetric difference. A good order makes this small.
"""
from __future__ import annotations

import numpy as np


def wave_objective(mask_h: np.ndarray, perm: np.ndarray, wave: int) -> int:
    rows = (np.asarray(mask_h)[np.asarray(perm)] != 0).astype(np.int64)
    total = 0
    for s in range(0, rows.shape[0], wave):
        w = rows[s:s + wave]
        k = w.shape[0]
        # sum_{i,j} ||a_i - a_j||^2 = 2k * sum_i ||a_i||^2 - 2 ||sum_i a_i||^2 (ordered pairs)
        col = w.sum(axis=0)
        total += 2 * k * int(w.sum()) - 2 * int((col * col).sum())
    return total
