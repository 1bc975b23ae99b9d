"""Mask statistics and the adaptive reordering skip (test infrastructure only).

Sec. IV-E names three situations in which reordering cannot repay its cost and
says the decision is taken from a few mask statistics weighed against costs
measured ahead of time on the target; Sec. VI-F shows the rule firing for short
sequences and very sparse masks. The paper prints no formula, so the reading
here is:

  case 1 "fits in cache": the head's distinct K/V blocks fit in the last-level
          cache that all compute units share (the paper's GPU: its L2; on the
          target, the 256 MiB memory-attached last-level cache behind the eight
          per-XCD L2s, which timing on and off showed to absorb the re-reads):
          distinct_h * kv_block_bytes <= cache_bytes
  case 2 "too little work": the expected kernel-time saving does not exceed
          the reordering overhead, both linear models from offline profiles:
          nnz_h * gain_ns_per_block < ovh_ns_fixed + ovh_ns_per_row*m + ovh_ns_per_nnz*nnz_h,
          with a second set of overhead constants (ovh_fused_*) for heads of at
          most fused_max_blocks rows: the implementation builds those in another
          form whose measured cost follows another line
  case 3 "already local": adjacent rows already share most blocks:
          J_h = sum_i |M_i & M_{i+1}| / sum_i |M_i | M_{i+1}| >= j_max,
          or, once the two-stage order P is built, it does not raise that overlap:
          J_h(P) <= J_h, compared exactly as integer cross-products (the order
          cannot make the rows that run together share more blocks than the
          natural order already does)
  case 4 (our addition) "no low-rank structure": the rank-2 embedding keeps too
          little of the centred mask's energy for Stage 1 to group anything:
          eta_h = (lambda_1 + lambda_2) / ||M~||_F^2 < eta_min,
          with lambda_1 + lambda_2 the exact Rayleigh-Ritz trace (Alg. 1) and
          ||M~||_F^2 = (m*nnz - sum_j c_j^2) / m (centring, Eq. 2).

The default constants are offline profiles of the target, taken by timing each
step with and without reordering over sequence length and density (the sweep of
Sec. VI-F): the overhead terms are a least-squares fit of the permutation's time
per head; the gain is the attention time saved per kept block where reordering
paid; cache_bytes is the K/V per head below which it did not pay (the shared
last-level cache holds that much next to the streamed Q, O and V^T); j_max lies
below the adjacent-row overlap of heads whose raster order is already local.

Each floating-point expression below is evaluated in fp64 with one IEEE
rounding per operation in the order written, so that an independent
implementation reaches the same decision.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

FLAG_FITS_CACHE = 1
FLAG_LITTLE_WORK = 2
FLAG_LOCAL = 4
FLAG_UNSTRUCTURED = 8
FLAG_DEGENERATE = 16
FLAG_IDENTITY = 64

SKIP_AUTO, SKIP_NEVER, SKIP_ALWAYS = 0, 1, 2


@dataclass(frozen=True)
class SkipProfile:
    cache_bytes: float = 96.0 * 1024 * 1024
    gain_ns_per_block: float = 0.5
    ovh_ns_fixed: float = -3000.0
    ovh_ns_per_row: float = 11.06
    ovh_ns_per_nnz: float = 0.0
    j_max: float = 0.2
    eta_min: float = 0.05
    fused_max_blocks: float = 1024.0
    ovh_fused_ns_fixed: float = 1184.0
    ovh_fused_ns_per_row: float = 10.50
    ovh_fused_ns_per_nnz: float = 0.0


@dataclass
class HeadStats:
    m: int
    n: int
    row_nnz: np.ndarray      # int32 [m]
    col_cnt: np.ndarray      # int32 [n]
    nnz: int
    distinct: int            # columns with at least one kept entry
    adj_and: int             # sum_i |M_i & M_{i+1}|
    adj_or: int              # sum_i |M_i | M_{i+1}|
    sum_c2: int              # sum_j c_j^2


def head_stats(mask_h: np.ndarray) -> HeadStats:
    mb = np.asarray(mask_h) != 0
    m, n = mb.shape
    rn = mb.sum(axis=1).astype(np.int64)
    cc = mb.sum(axis=0).astype(np.int64)
    a = int((mb[:-1] & mb[1:]).sum()) if m > 1 else 0
    o = int((mb[:-1] | mb[1:]).sum()) if m > 1 else 0
    return HeadStats(m, n, rn.astype(np.int32), cc.astype(np.int32), int(rn.sum()), int((cc > 0).sum()),
                     a, o, int((cc * cc).sum()))


def kv_block_bytes(block: int, head_dim: int) -> int:
    return 2 * block * head_dim * 2   # K and V, bf16


def tier1_flags(st: HeadStats, prof: SkipProfile, block: int, head_dim: int) -> int:
    flags = 0
    if float(st.distinct) * float(kv_block_bytes(block, head_dim)) <= prof.cache_bytes:
        flags |= FLAG_FITS_CACHE
    saving = float(st.nnz) * prof.gain_ns_per_block
    if float(st.m) <= prof.fused_max_blocks:
        c0, c1, c2 = prof.ovh_fused_ns_fixed, prof.ovh_fused_ns_per_row, prof.ovh_fused_ns_per_nnz
    else:
        c0, c1, c2 = prof.ovh_ns_fixed, prof.ovh_ns_per_row, prof.ovh_ns_per_nnz
    cost = c0 + c1 * float(st.m) + c2 * float(st.nnz)
    if saving < cost:
        flags |= FLAG_LITTLE_WORK
    if st.adj_or > 0 and float(st.adj_and) / float(st.adj_or) >= prof.j_max:
        flags |= FLAG_LOCAL
    return flags


def adjacent_overlap(mask_h: np.ndarray, order: np.ndarray) -> tuple[int, int]:
    """(sum_s |M_order[s] & M_order[s+1]|, sum_s |M_order[s] | M_order[s+1]|) over consecutive rows of an order."""
    mb = (np.asarray(mask_h) != 0)[np.asarray(order)]
    if mb.shape[0] < 2:
        return 0, 0
    return int((mb[:-1] & mb[1:]).sum()), int((mb[:-1] | mb[1:]).sum())


def order_not_more_local(st: HeadStats, mask_h: np.ndarray, order: np.ndarray) -> bool:
    """Case 3 against a built order: J(order) <= J(natural order), by exact integer cross-products."""
    a, o = adjacent_overlap(mask_h, order)
    return a * st.adj_or <= st.adj_and * o


def eta(st: HeadStats, trace: int, scale_exp: int) -> float:
    """Share of ||M~||_F^2 captured by the rank-2 embedding."""
    den = float(st.m) * float(st.m * st.nnz - st.sum_c2)
    if den <= 0.0:
        return 0.0
    return math.ldexp(float(trace), scale_exp) / den


def tier2_flags(st: HeadStats, prof: SkipProfile, trace: int, scale_exp: int, degenerate: bool) -> int:
    if degenerate:
        return FLAG_DEGENERATE
    return FLAG_UNSTRUCTURED if eta(st, trace, scale_exp) < prof.eta_min else 0
