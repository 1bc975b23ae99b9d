"""Helpers for the GPU tests: host <-> device conversion and comparison against the oracle."""
import math

import numpy as np
import torch

from oracle import attention as A


def bf16_dev(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def dev_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def u8_dev(mask: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(mask)).cuda()


def rows_of_block(i, blk, n):
    return A.block_token_range(i, blk, n)


def compare_blocks(o_dev: np.ndarray, ref: dict, blk: int, n: int, lse_dev=None):
    """Error statistics of device O (fp64 copy, [B][H][N][d]) over the oracle's sampled blocks."""
    max_abs, sum_abs, cnt, num, den, lse_err = 0.0, 0.0, 0, 0.0, 0.0, 0.0
    for (b, h, i), (ob, lb) in ref.items():
        lo, hi = rows_of_block(i, blk, n)
        d = o_dev[b, h, lo:hi] - ob
        max_abs = max(max_abs, float(np.abs(d).max()))
        sum_abs += float(np.abs(d).sum())
        cnt += d.size
        num += float((d * d).sum())
        den += float((ob * ob).sum())
        if lse_dev is not None:
            fin = np.isfinite(lb)
            if fin.any():
                lse_err = max(lse_err, float(np.abs(lse_dev[b, h, lo:hi][fin] - lb[fin]).max()))
            assert np.all(np.isneginf(lse_dev[b, h, lo:hi][~fin]))
    return dict(max_abs=max_abs, mean_abs=sum_abs / max(cnt, 1),
                rel_rms=math.sqrt(num / den) if den > 0 else math.sqrt(num), lse=lse_err)


def sample_blocks(mask: np.ndarray, count: int, seed: int):
    """(b, h, i) picks: first, last, heaviest, lightest and empty rows of each head plus random rows."""
    b_, h_, mb, _ = mask.shape
    rng = np.random.default_rng(seed)
    picks = set()
    n = mask.sum(-1)
    for b in range(b_):
        for h in range(h_):
            picks.update({(b, h, 0), (b, h, mb - 1), (b, h, int(n[b, h].argmax())), (b, h, int(n[b, h].argmin()))})
    while len(picks) < count + 4 * b_ * h_:
        picks.add((int(rng.integers(b_)), int(rng.integers(h_)), int(rng.integers(mb))))
    return sorted(picks)


def csr_matches_mask(mask_h: np.ndarray, row_ptr: np.ndarray, cols: np.ndarray) -> bool:
    """True if (row_ptr, cols) is exactly the ascending-index CSR of mask_h."""
    m = mask_h.shape[0]
    counts = (mask_h != 0).sum(1)
    if row_ptr[0] != 0 or not np.array_equal(np.diff(row_ptr), counts):
        return False
    rows, cidx = np.nonzero(mask_h)   # row-major, ascending columns within a row
    return np.array_equal(cols[: row_ptr[m]], cidx.astype(cols.dtype))
