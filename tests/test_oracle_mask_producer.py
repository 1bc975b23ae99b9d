"""Pins of the pooled-score top-k mask producer oracle (CPU)."""
import struct

import numpy as np
import pytest

from oracle import mask_producer as MP
from oracle.attention import bf16_to_f64
from workloads import make_qkv
from workloads.gen import PRODUCER_CONFIGS, _f64_to_bf16_bits


def _f32(x: float) -> float:
    """Round a Python float (fp64) to IEEE float32, nearest even."""
    return struct.unpack("f", struct.pack("f", x))[0]


def _bits(rng, shape, scale=1.0):
    return _f64_to_bf16_bits(rng.standard_normal(shape) * scale)


def test_pooled_means_against_exact_means():
    """Ragged tail counted with its true length; float32 fold error within its a-priori bound."""
    rng = np.random.default_rng(0)
    n, d, blk = 3 * 64 + 17, 8, 64
    x = _bits(rng, (n, d), 3.0)
    got = MP.pooled_means(x, blk).astype(np.float64)
    xf = bf16_to_f64(x)
    for j in range(4):
        lo, hi = j * blk, min((j + 1) * blk, n)
        exact = xf[lo:hi].mean(axis=0)
        bound = (hi - lo) * 2.0 ** -24 * np.abs(xf[lo:hi]).sum(axis=0) / (hi - lo) + 2.0 ** -23 * np.abs(exact)
        assert np.all(np.abs(got[j] - exact) <= bound), j
    assert got.shape == (4, d)


def test_pooled_fold_order_brute_force():
    """The exact float32 result of the ascending fold, recomputed with scalar float32 rounding."""
    rng = np.random.default_rng(1)
    n, d, blk = 2 * 16 + 5, 3, 16
    x = _bits(rng, (n, d), 1e3)   # large spread of magnitudes makes the rounding order visible
    x[::7] = _bits(rng, (len(x[::7]), d), 1e-2)
    got = MP.pooled_means(x, blk)
    xf = bf16_to_f64(x)
    for j in range(3):
        lo, hi = j * blk, min((j + 1) * blk, n)
        for c in range(d):
            acc = 0.0
            for t in range(lo, hi):
                acc = _f32(acc + xf[t, c])
            assert got[j, c] == np.float32(_f32(acc / (hi - lo))), (j, c)


def test_quantize_range_and_scale():
    rng = np.random.default_rng(2)
    m = rng.standard_normal((50, 16)).astype(np.float32)
    m[7, 3] = -5.0                           # the largest magnitude is negative
    q = MP.quantize(m)
    assert q.dtype == np.int8 and q.min() >= -127 and q.max() <= 127
    assert q[7, 3] == -127
    # within one step of the fp64 quantisation
    ref = m.astype(np.float64) * 127.0 / 5.0
    assert np.all(np.abs(q - ref) <= 0.5 + 1e-5)
    # powers of two cancel exactly
    assert np.array_equal(MP.quantize(m * np.float32(8.0)), q)
    assert not MP.quantize(np.zeros((3, 4), np.float32)).any()


def test_scores_are_the_integer_products():
    rng = np.random.default_rng(3)
    qc = rng.integers(-127, 128, size=(9, 12)).astype(np.int8)
    kc = rng.integers(-127, 128, size=(11, 12)).astype(np.int8)
    s = MP.block_scores(qc, kc)
    for i in range(9):
        for j in range(11):
            assert s[i, j] == sum(int(qc[i, c]) * int(kc[j, c]) for c in range(12))


@pytest.mark.parametrize("k,diag", [(1, False), (3, True), (5, False), (11, True), (20, True)])
def test_topk_brute_force(k, diag):
    rng = np.random.default_rng(4 + k)
    s = rng.integers(-3, 4, size=(8, 11)).astype(np.int64)   # many ties
    got = MP.topk_rows(s, k, diag)
    for i in range(8):
        ranked = sorted(range(11), key=lambda j: (-s[i, j], j))
        want = set(ranked[:min(k, 11)])
        if diag and i < 11:
            want.add(i)
        assert set(np.nonzero(got[i])[0]) == want, i


def test_row_counts_and_diagonal():
    wl = PRODUCER_CONFIGS["produced-tiny"]
    q, k, _ = make_qkv(wl)
    keep = 7
    mask = MP.produce_mask(q, k, wl.block, keep, diagonal=True)
    for h in range(wl.heads):
        _, s, _, _ = MP.produce_head(q[0, h], k[0, h], wl.block, keep)
        for i in range(wl.mb):
            thr = np.sort(s[i])[::-1][keep - 1]
            in_top = s[i, i] > thr or (s[i, i] == thr and np.sum(s[i, :i] == thr) + np.sum(s[i] > thr) < keep)
            assert mask[0, h, i].sum() == keep + (0 if in_top else 1)
            assert mask[0, h, i, i] == 1


def test_masks_follow_the_positional_structure():
    """Spatial heads keep blocks near in time; temporal heads keep blocks across all frames at about
    the same in-frame position. A transposed or misindexed score would destroy both."""
    wl = PRODUCER_CONFIGS["produced-tiny"]
    q, k, _ = make_qkv(wl)
    mask = MP.produce_mask(q, k, wl.block, 8, diagonal=False)
    per_frame = wl.frame_tokens // wl.block
    frame = np.arange(wl.mb) // per_frame
    inframe = np.arange(wl.mb) % per_frame
    rng = np.random.default_rng(5)
    rand = np.zeros_like(mask[0, 0])
    for i in range(wl.mb):
        rand[i, rng.choice(wl.mb, 8, replace=False)] = 1
    def mean_dist(m, key):
        i, j = np.nonzero(m)
        return np.abs(key[i] - key[j]).mean()
    spatial, temporal = mask[0, 0], mask[0, 1]
    assert mean_dist(spatial, frame) < 0.5 * mean_dist(rand, frame)
    assert mean_dist(temporal, inframe) < 0.5 * mean_dist(rand, inframe)
    assert mean_dist(temporal, frame) > mean_dist(spatial, frame)


def test_planted_ragged_count_is_caught(monkeypatch):
    def by_blk(x_bits, blk):
        x = MP.bf16_bits_to_f32(x_bits)
        n, d = x.shape
        mb = -(-n // blk)
        pad = np.zeros((mb * blk, d), np.float32)
        pad[:n] = x
        return (pad.reshape(mb, blk, d).sum(axis=1) / np.float32(blk)).astype(np.float32)
    monkeypatch.setattr(MP, "pooled_means", by_blk)
    with pytest.raises(AssertionError):
        test_pooled_means_against_exact_means()


def test_planted_signed_max_is_caught(monkeypatch):
    def signed(means):
        a = np.float32(means.max())
        inv = np.float32(np.float32(127.0) / a)
        return np.clip(np.rint((means * inv).astype(np.float32)), -127, 127).astype(np.int8)
    monkeypatch.setattr(MP, "quantize", signed)
    with pytest.raises(AssertionError):
        test_quantize_range_and_scale()


def test_planted_transposed_scores_are_caught(monkeypatch):
    orig = MP.block_scores
    monkeypatch.setattr(MP, "block_scores", lambda qc, kc: orig(qc, kc).T)
    with pytest.raises((AssertionError, IndexError)):
        test_scores_are_the_integer_products()
