"""Pins of the reference permutation (Alg. 1 + Alg. 2 under the integer-exact reading).

The paper prints no worked numeric example (its figures are not available), so
the permutation is pinned by: published SplitMix64 outputs; the exact centring
identity of Sec. IV-C (products with the explicitly materialised centred
matrix); the Eckart-Young special case (a textbook SVD); the same iteration in
plain fp64; closed forms (clustered rows, rank one, all ones); atan2 itself for
the exact angle comparator; and a hand-worked Stage-2 example.
"""
import math
import os

import numpy as np
import pytest

from oracle import permutation as P
from oracle import objective as OBJ
from oracle.splitmix import splitmix64_stream
from workloads import CONFIGS, custom, make_mask, make_mask_head

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold_lines(name):
    with open(os.path.join(GOLD, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


def test_splitmix64_published_vectors():
    for row in _gold_lines("splitmix64_vectors.txt"):
        seed, outs = int(row[0]), [int(x) for x in row[1:]]
        assert splitmix64_stream(seed, len(outs)) == outs


def test_random_start_range_and_formula():
    z = P.random_start(5, 11, 2)
    assert z.shape == (5, 2)
    assert np.all(z >= -(1 << 23)) and np.all(z < (1 << 23))
    from oracle.splitmix import splitmix64
    assert z[3, 1] == (splitmix64(11 + 2 * (2 * 5 + 3) + 1) >> 40) - (1 << 23)


def _rand_mask(m, n, p, seed):
    return (np.random.default_rng(seed).random((m, n)) < p).astype(np.uint8)


def test_centred_products_equal_materialised_centring():
    """m*M~^T X and m*M~ Ys computed matrix-free equal the products with (m*M - 1 c^T)."""
    mask = _rand_mask(37, 29, 0.3, 1)
    m = mask.shape[0]
    c = mask.sum(0).astype(np.int64)
    x, _ = P.orth(P.random_start(m, 5, 0))
    zm, sy = P.centred_apply(mask, c, x)
    cen = m * mask.astype(object) - np.outer(np.ones(m, dtype=object), c.astype(object))  # m * M~, exact ints
    ym = cen.T.dot(x.astype(object))
    mx = max(abs(int(v)) for v in ym.flat)
    assert sy == max(0, mx.bit_length() - 30)
    ys = np.array([[int(v) >> sy for v in r] for r in ym], dtype=object)
    ref = cen.dot(ys)
    assert np.array_equal(zm.astype(object), ref)
    # centring removes the all-ones direction: 1^T (m M~) = 0 (Sec. IV-C)
    assert all(int(v) == 0 for v in np.ones(m, dtype=object).dot(cen))


def test_centring_preserves_row_distances_and_eq3():
    mask = _rand_mask(20, 24, 0.4, 2).astype(np.float64)
    m = mask.shape[0]
    cen = mask - mask.mean(0, keepdims=True)
    d_raw = ((mask[:, None] - mask[None]) ** 2).sum(-1)
    d_cen = ((cen[:, None] - cen[None]) ** 2).sum(-1)
    assert np.allclose(d_raw, d_cen)
    u, s, vt = np.linalg.svd(cen)
    d_eq3 = ((s[None, None, :] * (u[:, None, :] - u[None, :, :])) ** 2).sum(-1)
    assert np.allclose(d_cen, d_eq3)
    assert m == 20


def test_orth_columns_orthonormal():
    z = P.random_start(300, 9, 1) * 977
    x, deg = P.orth(z)
    assert not deg
    q = x.astype(np.float64) / 2 ** 30
    assert np.allclose(q.T @ q, np.eye(2), atol=1e-8)
    # span is kept: Z = Q R with R upper triangular -> Z's first column is parallel to Q's
    zf = z.astype(np.float64)
    assert abs(abs(zf[:, 0] @ q[:, 0]) - np.linalg.norm(zf[:, 0])) < 1e-6 * np.linalg.norm(zf[:, 0])


def test_orth_rank_one_and_zero():
    v = np.arange(-5, 7, dtype=np.int64)
    z = np.stack([3 * v, -7 * v], axis=1)
    x, deg = P.orth(z)
    assert not deg and np.all(x[:, 1] == 0)
    x, deg = P.orth(np.zeros((6, 2), dtype=np.int64))
    assert deg


def _svd_top2(mask):
    cen = mask.astype(np.float64) - mask.mean(0, keepdims=True)
    u, s, _ = np.linalg.svd(cen, full_matrices=False)
    return u, s


def _structured_mask(m, seed):
    """Locality-band mask plus noise: a clear spectral gap after centring."""
    rng = np.random.default_rng(seed)
    i = np.arange(m)
    band = (np.abs(i[:, None] - i[None, :]) <= m // 6)
    noise = rng.random((m, m)) < 0.03
    return (band ^ noise).astype(np.uint8)


def test_textbook_svd_special_case():
    """With many iterations the embedding spans the top-2 left singular subspace (Eckart-Young)."""
    mask = _structured_mask(160, 4)
    uu, s = _svd_top2(mask)
    assert s[2] / s[1] <= 0.9 and s[1] / s[0] <= 0.9
    U, deg, rr = P.mfcsi_embedding(mask, seed=3, flat_head=0, iters=200)
    assert not deg
    q = U.astype(np.float64) / 2 ** 30
    q /= np.linalg.norm(q, axis=0, keepdims=True)
    # sine of the angle between each column and the top-2 singular subspace (projection residual)
    top = uu[:, :2]
    sines = np.linalg.norm(q - top @ (top.T @ q), axis=0)
    assert sines.max() < 1e-5
    # each column matches its singular vector up to sign; the sign follows the canonical rule
    for k in range(2):
        ref = uu[:, k]
        i_star = int(np.argmax(np.abs(ref)))
        ref = ref if ref[i_star] > 0 else -ref
        assert np.allclose(q[:, k], ref, atol=1e-6)
    # the Rayleigh-Ritz trace recovers sigma_1^2 + sigma_2^2 through the fixed-point bookkeeping
    m = mask.shape[0]
    tr = math.ldexp(float(rr.trace), rr.scale_exp) / (m * m)
    assert abs(tr / (s[0] ** 2 + s[1] ** 2) - 1) < 1e-6


def _plain_fp64_mfcsi(mask, z0, iters):
    """Alg. 1 in plain fp64 (numpy QR / eigh), same start, no fixed point."""
    mk = mask.astype(np.float64)
    m = mk.shape[0]
    c = mk.sum(0)

    def qr(z):
        q, r = np.linalg.qr(z)
        return q * np.sign(np.diag(r))[None, :]

    def app(x):
        y = mk.T @ x - np.outer(c, x.sum(0)) / m
        return mk @ y - np.outer(np.ones(m), c @ y) / m

    x = qr(z0.astype(np.float64))
    for _ in range(iters):
        x = qr(app(x))
    z = app(x)
    lam, r = np.linalg.eigh(x.T @ z)
    x = x @ r[:, ::-1]
    for k in range(2):
        i_star = int(np.argmax(np.abs(x[:, k])))
        if x[i_star, k] < 0:
            x[:, k] = -x[:, k]
    return x


def _kendall_tau(a, b):
    pos = np.empty_like(b); pos[b] = np.arange(b.size)
    r = pos[a]
    n = r.size
    conc = 0
    for i in range(n):
        conc += int((r[i + 1:] > r[i]).sum())
    tot = n * (n - 1) // 2
    return (2 * conc - tot) / tot


@pytest.mark.parametrize("cfg,head", [("wan1.3b-480p-81f", 0), ("wan14b-720p-81f", 3)])
def test_fixed_point_matches_plain_fp64_iteration(cfg, head):
    wl = CONFIGS[cfg]
    mask = make_mask_head(wl, 0, head)
    m = mask.shape[0]
    z0 = P.random_start(m, 0, head)
    U, deg, _ = P.mfcsi_embedding(mask, seed=0, flat_head=head, iters=10)
    xf = _plain_fp64_mfcsi(mask, z0, 10)
    uq = U.astype(np.float64) / 2 ** 30
    ang_q = np.arctan2(uq[:, 1], uq[:, 0])
    ang_f = np.arctan2(xf[:, 1], xf[:, 0])
    rad = np.hypot(xf[:, 0], xf[:, 1])
    ok = rad > 1e-3 * rad.max()
    diff = np.abs(np.angle(np.exp(1j * (ang_q - ang_f))))[ok]
    assert diff.max() < 1e-5
    order_q = P.stage1(mask, 0, head, 10).order
    order_f = np.lexsort((np.arange(m), ang_f))
    assert _kendall_tau(order_q, order_f) >= 0.999


def test_clustered_rows_are_contiguous():
    rng = np.random.default_rng(8)
    n = 40
    protos = (rng.random((3, n)) < 0.5).astype(np.uint8)
    labels = rng.integers(0, 3, size=30)
    mask = protos[labels]
    s1 = P.stage1(mask, seed=1, flat_head=0, iters=10)
    assert not s1.degenerate
    lab_in_order = labels[s1.order]
    changes = int((lab_in_order[1:] != lab_in_order[:-1]).sum())
    assert changes == 2, lab_in_order
    for lab in range(3):
        rows = s1.order[lab_in_order == lab]
        assert np.all(np.diff(rows) > 0)


def test_two_row_types_split_in_two_groups():
    rng = np.random.default_rng(9)
    protos = (rng.random((2, 25)) < 0.5).astype(np.uint8)
    labels = rng.integers(0, 2, size=21)
    s1 = P.stage1(protos[labels], seed=2, flat_head=1, iters=10)
    assert np.all(s1.embedding[:, 1] == 0)
    lab = labels[s1.order]
    assert int((lab[1:] != lab[:-1]).sum()) == 1


def test_all_ones_and_equal_rows_are_degenerate():
    s1 = P.stage1(np.ones((12, 12), dtype=np.uint8), 0, 0)
    assert s1.degenerate and np.array_equal(s1.order, np.arange(12))
    row = (np.arange(15) % 3 == 0).astype(np.uint8)
    s1 = P.stage1(np.tile(row, (9, 1)), 0, 0)
    assert s1.degenerate


def test_angle_comparator_equals_atan2():
    rng = np.random.default_rng(10)
    pts = rng.integers(-1000, 1000, size=(300, 2))
    pts[:6] = [[5, 0], [0, 0], [-3, 0], [0, 4], [0, -4], [7, 0]]
    pts[6:10] = [[2, 2], [4, 4], [-1, -1], [-3, -3]]   # equal angles -> by index
    order = P.angle_order(pts)
    ang = np.array([math.atan2(float(y), float(x)) for x, y in pts])
    ref = np.lexsort((np.arange(len(pts)), ang))
    # atan2's angle for distinct rational directions differs by far more than fp64 rounding here
    assert np.array_equal(order, ref)


def test_stage2_hand_example():
    lines = _gold_lines("stage2_hand_example.txt")
    order = np.array([int(v) for v in lines[0][1:]])
    nnz = np.array([int(v) for v in lines[1][1:]])
    for ln in lines[2:]:
        n_xcd, w = int(ln[1]), int(ln[2])
        bar = ln.index("|")
        expect = [int(v) for v in ln[4:bar]]
        expect_seg = [int(v) for v in ln[bar + 1:]]
        assert list(P.stage2(order, nnz, n_xcd, w)) == expect
        assert P.work_segments(order, nnz, n_xcd) == expect_seg


@pytest.mark.parametrize("m,n_xcd,w", [(64, 8, 64), (591, 8, 64), (2841, 8, 128), (17, 1, 4), (9, 2, 3), (5, 8, 2)])
def test_stage2_invariants(m, n_xcd, w):
    rng = np.random.default_rng(m)
    order = rng.permutation(m).astype(np.int32)
    nnz = rng.lognormal(2.0, 1.0, size=m).astype(np.int64)
    perm = P.stage2(order, nnz, n_xcd, w)
    assert np.array_equal(np.sort(perm), np.arange(m))
    seg = P.work_segments(order, nnz, n_xcd)
    assert seg[0] == 0 and seg[-1] == m and all(a <= b for a, b in zip(seg, seg[1:]))
    # work balance: every segment's work differs from the even share by less than its heaviest row
    wts = nnz[order] + 1
    share = wts.sum() / n_xcd
    for x in range(n_xcd):
        sw = wts[seg[x]:seg[x + 1]].sum()
        assert sw < share + wts.max() and (seg[x] == seg[x + 1] or sw > share - 2 * wts.max())
    # the equal-count layout used without a schedule
    bounds = P.segment_bounds(m, n_xcd)
    assert bounds[0][0] == 0 and bounds[-1][1] == m
    lens = [b - a for a, b in bounds]
    assert max(lens) - min(lens) <= 1 and lens == sorted(lens, reverse=True)
    for s0, s1 in zip(seg[:-1], seg[1:]):
        for b0 in range(s0, s1, w):
            b1 = min(b0 + w, s1)
            assert sorted(perm[b0:b1]) == sorted(order[b0:b1])
            assert np.all(np.diff(nnz[perm[b0:b1]]) <= 0)


def test_wave_objective_equals_brute_force_pairs_with_a_ragged_last_wave():
    """Eq. 1 summed literally: over consecutive waves of at most W rows of the permuted
    mask, over every ordered pair (i, j) of rows of a wave, the squared distance of the
    two 0/1 rows (the size of their symmetric difference). 23 rows in waves of 5 leave
    a last wave of 3 rows."""
    rng = np.random.default_rng(31)
    m, n, w = 23, 17, 5
    mask = (rng.random((m, n)) < 0.35).astype(np.uint8)
    for perm in (np.arange(m), rng.permutation(m), rng.permutation(m)):
        rows = mask[perm].astype(np.int64)
        brute = 0
        for s in range(0, m, w):
            wave = range(s, min(s + w, m))
            for i in wave:
                for j in wave:
                    brute += int(((rows[i] - rows[j]) ** 2).sum())
        assert OBJ.wave_objective(mask, perm, w) == brute
    # one wave holding every row: the ordering cannot matter
    assert OBJ.wave_objective(mask, rng.permutation(m), m) == OBJ.wave_objective(mask, np.arange(m), m)
    # waves of one row: every term is a row with itself
    assert OBJ.wave_objective(mask, rng.permutation(m), 1) == 0


def test_wave_objective_improves_on_shuffled_clusters():
    rng = np.random.default_rng(12)
    protos = (rng.random((6, 64)) < 0.3).astype(np.uint8)
    labels = rng.integers(0, 6, size=96)
    noise = (rng.random((96, 64)) < 0.02).astype(np.uint8)
    mask = protos[labels] ^ noise
    perm, _ = P.two_stage_permutation(mask, seed=0, flat_head=0, wave=16, n_xcd=1)
    ident = np.arange(96)
    assert OBJ.wave_objective(mask, perm, 16) < 0.7 * OBJ.wave_objective(mask, ident, 16)


def test_planted_row_count_segments_are_caught(monkeypatch):
    def by_rows(order, nnz, n_xcd):
        return [b[0] for b in P.segment_bounds(order.size, n_xcd)] + [order.size]

    monkeypatch.setattr(P, "work_segments", by_rows)
    with pytest.raises(AssertionError):
        test_stage2_hand_example()


def test_golden_permutation_unchanged():
    """Regression against the stored output of tests/golden/make_golden.py (oracle only)."""
    path = os.path.join(GOLD, "perm_small.txt")
    from tests.golden.make_golden import golden_cases, compute_case
    with open(path) as f:
        stored = {ln.split()[0]: [int(v) for v in ln.split()[1:]] for ln in f if ln.strip() and not ln.startswith("#")}
    for key, args in golden_cases():
        assert compute_case(*args) == stored[key], key


# ---- planted mistakes -------------------------------------------------------------------------
def test_planted_missing_centring_is_caught(monkeypatch):
    orig = P.centred_apply

    def no_centre(mask, c, x):
        return orig(mask, np.zeros_like(c), x)

    monkeypatch.setattr(P, "centred_apply", no_centre)
    with pytest.raises(AssertionError):
        test_centred_products_equal_materialised_centring()


def test_planted_swapped_cross_sign_is_caught(monkeypatch):
    real = P.angle_precedes

    def wrong(p, q):
        return real((p[1], p[0], p[2]), (q[1], q[0], q[2]))

    monkeypatch.setattr(P, "angle_precedes", wrong)
    with pytest.raises(AssertionError):
        test_angle_comparator_equals_atan2()


def test_planted_unstable_stage2_is_caught(monkeypatch):
    def unstable(order, nnz, n_xcd, wave, seg_start=None):
        perm = np.empty(order.size, dtype=np.int32)
        seg = P.work_segments(order, nnz, n_xcd)
        for s0, s1 in zip(seg[:-1], seg[1:]):
            for b0 in range(s0, s1, wave):
                b1 = min(b0 + wave, s1)
                bucket = list(order[b0:b1])
                perm[b0:b1] = sorted(bucket, key=lambda r: (-int(nnz[r]), -int(r)))
        return perm

    monkeypatch.setattr(P, "stage2", unstable)
    with pytest.raises(AssertionError):
        test_stage2_hand_example()
