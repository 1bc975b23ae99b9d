"""Pins of the mask statistics, the skip rule and the whole-mask permutation driver."""
import math

import numpy as np
import pytest

from oracle import compaction as C
from oracle import permutation as P
from oracle import reorder as R
from oracle import skip as S
from workloads import CONFIGS, custom, make_mask, make_mask_head


def test_head_stats_brute_force():
    rng = np.random.default_rng(1)
    mask = (rng.random((23, 23)) < 0.3).astype(np.uint8)
    st = S.head_stats(mask)
    m, n = mask.shape
    assert [sum(int(mask[i, j]) for j in range(n)) for i in range(m)] == list(st.row_nnz)
    assert [sum(int(mask[i, j]) for i in range(m)) for j in range(n)] == list(st.col_cnt)
    a = sum(int(mask[i, j] and mask[i + 1, j]) for i in range(m - 1) for j in range(n))
    o = sum(int(mask[i, j] or mask[i + 1, j]) for i in range(m - 1) for j in range(n))
    assert (a, o) == (st.adj_and, st.adj_or)
    assert st.distinct == sum(1 for j in range(n) if any(mask[:, j]))
    # ||M~||_F^2 from the statistics equals the explicitly centred matrix's
    cen = mask - mask.mean(0, keepdims=True)
    assert abs((m * st.nnz - st.sum_c2) / m - (cen ** 2).sum()) < 1e-9


def test_eta_equals_svd_energy_share():
    mask = make_mask_head(CONFIGS["wan1.3b-480p-81f"], 0, 2)
    st = S.head_stats(mask)
    s1 = P.stage1(mask, 0, 2, iters=300)
    cen = mask - mask.mean(0, keepdims=True)
    sv = np.linalg.svd(cen, compute_uv=False)
    ref = (sv[0] ** 2 + sv[1] ** 2) / (sv ** 2).sum()
    assert abs(S.eta(st, s1.trace, s1.scale_exp) / ref - 1) < 1e-6


def test_eta_separates_random_from_structured():
    wl = CONFIGS["skip-d64"]
    for h, lo, hi in ((0, 0.0, 0.05), (20, 0.1, 1.0)):
        mask = make_mask_head(wl, 0, h)
        st = S.head_stats(mask)
        s1 = P.stage1(mask, 0, h, 10)
        assert lo <= S.eta(st, s1.trace, s1.scale_exp) < hi


# A profile under which only the designed case fires on the inputs below: a 4 MiB cache and
# a cheap reordering that saves 1 ns per kept block.
PERMISSIVE = S.SkipProfile(cache_bytes=4 * 1024 * 1024, gain_ns_per_block=1.0, ovh_ns_fixed=2000.0,
                           ovh_ns_per_row=2.0, ovh_ns_per_nnz=0.05, j_max=0.75)


def test_tier1_cases():
    prof = S.SkipProfile()
    tiny = make_mask_head(CONFIGS["tiny"], 0, 0)
    f = S.tier1_flags(S.head_stats(tiny), prof, 64, 64)
    assert f & S.FLAG_FITS_CACHE          # 64 KV blocks of 16 KiB = 1 MiB < 96 MiB
    big = S.head_stats(make_mask_head(CONFIGS["wan14b-720p-81f"], 0, 0))
    # 591 KV blocks of 64 KiB = 37 MiB: below the 96 MiB break-even, not inside one 4 MiB L2;
    # 84K kept blocks save 42 us at 0.5 ns each, more than the 17 us the permutation costs;
    # adjacent rows share 36% of their blocks (raster order is already local)
    assert S.tier1_flags(big, prof, 128, 128) == S.FLAG_FITS_CACHE | S.FLAG_LOCAL
    assert S.tier1_flags(big, PERMISSIVE, 128, 128) == 0
    prof = PERMISSIVE
    # already local: every row equal to its neighbour except one column
    band = np.zeros((100, 100), dtype=np.uint8)
    for i in range(100):
        band[i, max(0, i - 30):i + 30] = 1
    assert S.tier1_flags(S.head_stats(band), prof, 128, 128) & S.FLAG_LOCAL
    # little work: a nearly empty mask
    sparse = np.eye(300, dtype=np.uint8)
    assert S.tier1_flags(S.head_stats(sparse), prof, 128, 128) & S.FLAG_LITTLE_WORK
    # boundary of case 1 is inclusive: exactly one cache of distinct blocks fits
    st = S.head_stats(np.eye(128, dtype=np.uint8))
    exact = S.SkipProfile(cache_bytes=128 * S.kv_block_bytes(128, 128))
    assert S.tier1_flags(st, exact, 128, 128) & S.FLAG_FITS_CACHE
    below = S.SkipProfile(cache_bytes=128 * S.kv_block_bytes(128, 128) - 1)
    assert not (S.tier1_flags(st, below, 128, 128) & S.FLAG_FITS_CACHE)


def test_little_work_uses_the_cost_curve_of_the_form_that_builds_the_head():
    """Case 2 takes the one-workgroup form's overhead line up to fused_max_blocks rows and the sliced
    form's line above: the same statistics flip the decision at the boundary when only one of the
    two lines exceeds the saving."""
    prof = S.SkipProfile(cache_bytes=0.0, gain_ns_per_block=1.0, j_max=2.0, fused_max_blocks=512.0,
                         ovh_ns_fixed=0.0, ovh_ns_per_row=0.0, ovh_ns_per_nnz=0.0,
                         ovh_fused_ns_fixed=1e9, ovh_fused_ns_per_row=0.0, ovh_fused_ns_per_nnz=0.0)
    for m, want in ((512, S.FLAG_LITTLE_WORK), (513, 0)):
        st = S.head_stats(np.eye(m, dtype=np.uint8))
        assert S.tier1_flags(st, prof, 128, 128) == want, m
    # the saving is compared strictly: equal costs keep the reordering (a head of the sliced form)
    st = S.head_stats(np.eye(600, dtype=np.uint8))
    even = S.SkipProfile(cache_bytes=0.0, gain_ns_per_block=1.0, j_max=2.0, ovh_ns_fixed=600.0,
                         ovh_ns_per_row=0.0, ovh_ns_per_nnz=0.0, fused_max_blocks=512.0)
    assert S.tier1_flags(st, even, 128, 128) == 0
    assert S.tier1_flags(st, S.SkipProfile(cache_bytes=0.0, gain_ns_per_block=1.0, j_max=2.0,
                                           ovh_ns_fixed=600.5, ovh_ns_per_row=0.0, ovh_ns_per_nnz=0.0,
                                           fused_max_blocks=512.0),
                         128, 128) == S.FLAG_LITTLE_WORK


def test_default_rule_decides_per_head_on_mixed_heads():
    """Default profile on the 401-frame workload with spatial and temporal heads: the spatial heads are
    already local in raster order (adjacent rows share ~33% of their blocks) and keep it; the temporal
    heads (~6%) are reordered; 178 MiB of K/V per head is above the cache break-even."""
    from workloads.gen import ALL_CONFIGS
    wl = ALL_CONFIGS["long-720p-401f-mixed"]
    prof = S.SkipProfile()
    spatial = S.head_stats(make_mask_head(wl, 0, 0))
    temporal = S.head_stats(make_mask_head(wl, 0, 20))
    assert S.tier1_flags(spatial, prof, wl.block, wl.head_dim) == S.FLAG_LOCAL
    assert S.tier1_flags(temporal, prof, wl.block, wl.head_dim) == 0


def test_driver_modes():
    wl = CONFIGS["skip-d64"]
    mask = make_mask(wl)[:, [0, 1, 20, 21]].copy()
    # head 3: a locality head with its rows shuffled, so that its natural order is not local
    mask[0, 3] = mask[0, 3][np.random.default_rng(7).permutation(wl.mb)]
    kw = dict(block=wl.block, head_dim=wl.head_dim, wave=64, n_xcd=8, iters=10, seed=0)
    p_always, f_always, _ = R.build_permutation(mask, skip_mode=S.SKIP_ALWAYS, **kw)
    assert np.all(p_always == np.arange(wl.mb)) and np.all(f_always & S.FLAG_IDENTITY)
    p_never, f_never, _ = R.build_permutation(mask, skip_mode=S.SKIP_NEVER, **kw)
    for h in range(4):
        ref, _ = P.two_stage_permutation(mask[0, h], seed=0, flat_head=h, wave=64, n_xcd=8, iters=10)
        assert np.array_equal(p_never[0, h], ref)
    assert not np.any(f_never & S.FLAG_IDENTITY)
    # a 4 MiB cache keeps case 1 quiet (11.6 MiB of K/V per head), so the later cases decide
    p_auto, f_auto, _ = R.build_permutation(mask, skip_mode=S.SKIP_AUTO, profile=PERMISSIVE, **kw)
    # random heads: unstructured -> identity; a locality head in raster order: the built order does
    # not raise the adjacent-row overlap (case 3 after the fact) -> identity; the shuffled one: reordered
    assert f_auto[0, 0] & S.FLAG_UNSTRUCTURED and np.all(p_auto[0, 0] == np.arange(wl.mb))
    st2 = S.head_stats(mask[0, 2])
    assert S.order_not_more_local(st2, mask[0, 2], p_never[0, 2])
    assert f_auto[0, 2] == S.FLAG_LOCAL | S.FLAG_IDENTITY and np.all(p_auto[0, 2] == np.arange(wl.mb))
    st3 = S.head_stats(mask[0, 3])
    a3, o3 = S.adjacent_overlap(mask[0, 3], p_never[0, 3])
    assert a3 / o3 > 2 * st3.adj_and / st3.adj_or
    assert f_auto[0, 3] == 0 and np.array_equal(p_auto[0, 3], p_never[0, 3])
    # default profile: every head's K/V fits the shared cache, so case 1 keeps the identity order
    p_def, f_def, _ = R.build_permutation(mask, skip_mode=S.SKIP_AUTO, **kw)
    assert np.all(f_def & S.FLAG_FITS_CACHE) and np.all(f_def & S.FLAG_IDENTITY)
    assert np.all(p_def == np.arange(wl.mb))


def test_adjacent_overlap_brute_force():
    """The overlap of consecutive rows of an order, by sets on a small mask, and case 3 against a built
    order on a band (its natural order is the most local) and on the band with rows shuffled."""
    rng = np.random.default_rng(3)
    m = 40
    band = np.zeros((m, m), np.uint8)
    for i in range(m):
        band[i, max(0, i - 3): i + 4] = 1
    order = rng.permutation(m)
    a, o = S.adjacent_overlap(band, order)
    rows = [set(np.nonzero(band[r])[0]) for r in order]
    assert a == sum(len(rows[s] & rows[s + 1]) for s in range(m - 1))
    assert o == sum(len(rows[s] | rows[s + 1]) for s in range(m - 1))
    st = S.head_stats(band)
    assert (st.adj_and, st.adj_or) == S.adjacent_overlap(band, np.arange(m))
    assert S.order_not_more_local(st, band, order)            # a shuffle only loses locality
    assert S.order_not_more_local(st, band, np.arange(m))     # equal overlap counts as no gain
    shuffled = band[order]
    st_s = S.head_stats(shuffled)
    assert not S.order_not_more_local(st_s, shuffled, np.argsort(order))  # un-shuffling gains


def test_compaction_brute_force():
    wl = custom("c", heads=2, head_dim=64, block=64, grid=(2, 8, 16), rule=dict(kind="empty_rows", p=0.3))
    mask = make_mask(wl)
    row_ptr, lists = C.compact_mask(mask)
    for h in range(2):
        pos = 0
        for i in range(wl.mb):
            cols = [j for j in range(wl.mb) if mask[0, h, i, j]]
            assert row_ptr[0, h, i] == pos
            assert list(lists[0][h][pos:pos + len(cols)]) == cols
            pos += len(cols)
        assert row_ptr[0, h, wl.mb] == pos == len(lists[0][h])
