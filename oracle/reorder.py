"""Whole-mask permutation driver: skip rule + two-stage reordering (test infrastructure only).

Mirrors the per-head flow of Sec. IV-A and Alg. 2: the adaptive guard first
(cases 1-3 from mask statistics), then Stage 1 and Stage 2; case 4 uses the
Rayleigh-Ritz trace of Stage 1, and case 3 is checked once more against the
built order (it must raise the adjacent-row overlap). A skipped head keeps the
identity order.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from . import permutation as P
from . import skip as S


def build_permutation(mask: np.ndarray, *, block: int, head_dim: int, wave: int, n_xcd: int = 8,
                      iters: int = 10, seed: int = 0, skip_mode: int = S.SKIP_AUTO,
                      profile: Optional[S.SkipProfile] = None):
    """mask u8 [B][H][M_B][N_B] -> (perm int32 [B][H][M_B], flags uint8 [B][H], stage1 info).

    ``flags`` holds the skip-rule bits that fired (S.FLAG_*) and S.FLAG_IDENTITY when the
    identity order was returned. With skip_mode NEVER the rule is still evaluated and
    reported but never applied; with ALWAYS every head returns the identity.
    ``info["seg"][(b, h)]`` is the work-balanced XCD segment table of the returned order.
    """
    profile = profile or S.SkipProfile()
    b_, h_, m, n = mask.shape
    perm = np.empty((b_, h_, m), dtype=np.int32)
    flags = np.zeros((b_, h_), dtype=np.uint8)
    info = {"seg": {}}
    for b in range(b_):
        for h in range(h_):
            hh = b * h_ + h
            st = S.head_stats(mask[b, h])
            f = S.tier1_flags(st, profile, block, head_dim)
            if skip_mode == S.SKIP_ALWAYS or (skip_mode == S.SKIP_AUTO and f != 0):
                perm[b, h] = P.identity_permutation(m)
                flags[b, h] = f | S.FLAG_IDENTITY
                info["seg"][(b, h)] = P.work_segments(perm[b, h], st.row_nnz, n_xcd)
                continue
            s1 = P.stage1(mask[b, h], seed, hh, iters)
            f |= S.tier2_flags(st, profile, s1.trace, s1.scale_exp, s1.degenerate)
            info[(b, h)] = s1
            if skip_mode == S.SKIP_AUTO and (f & S.FLAG_UNSTRUCTURED):
                perm[b, h] = P.identity_permutation(m)
                flags[b, h] = f | S.FLAG_IDENTITY
                info["seg"][(b, h)] = P.work_segments(perm[b, h], st.row_nnz, n_xcd)
                continue
            seg = P.work_segments(s1.order, st.row_nnz, n_xcd)
            built = P.stage2(s1.order, st.row_nnz, n_xcd, wave, seg)
            if skip_mode == S.SKIP_AUTO and S.order_not_more_local(st, mask[b, h], built):
                perm[b, h] = P.identity_permutation(m)
                flags[b, h] = f | S.FLAG_LOCAL | S.FLAG_IDENTITY
                info["seg"][(b, h)] = P.work_segments(perm[b, h], st.row_nnz, n_xcd)
                continue
            perm[b, h] = built
            info["seg"][(b, h)] = seg
            flags[b, h] = f
    return perm, flags, info
