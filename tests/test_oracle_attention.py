"""Pins of the fp64 attention oracle against what the definition fixes.

Each test ties the block-sparse oracle to something other than itself: a
library dense attention, a brute-force token-level mask, closed forms, and the
row-permutation invariance the paper relies on (Sec. IV-A). The last tests plant
plausible mistakes in the oracle and check that a pin catches each one.
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as A
from workloads import custom, make_mask, make_tensor


def _qkv(wl):
    return tuple(make_tensor(wl, s) for s in (0, 1, 2))


def _wl(n=None, heads=2, d=32, blk=16, grid=(2, 4, 8), rule=None, seed=3):
    return custom("pin", heads=heads, head_dim=d, block=blk, grid=grid, rule=rule, seed=seed, seq_len=n)


def _bf16_closed_form(b: int) -> float:
    """Value of bf16 bit pattern b from the format's definition: sign bit, 8-bit biased
    exponent (bias 127), 7-bit fraction; exponent 0 is subnormal, 255 infinity / NaN."""
    sign = -1.0 if b >> 15 else 1.0
    e, f = (b >> 7) & 0xFF, b & 0x7F
    if e == 255:
        return sign * math.inf if f == 0 else math.nan
    if e == 0:
        return sign * math.ldexp(f, -126 - 7)
    return sign * math.ldexp(128 + f, e - 127 - 7)


def test_bf16_widening_matches_torch_and_the_format_on_every_pattern():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = A.bf16_to_f64(bits)
    lib = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    form = np.array([_bf16_closed_form(int(b)) for b in bits])
    nan = np.isnan(form)
    assert nan.sum() == 2 * 127                        # 0x7F81..0x7FFF and 0xFF81..0xFFFF
    assert np.array_equal(np.isnan(ours), nan) and np.array_equal(np.isnan(lib), nan)
    assert np.array_equal(ours[~nan], form[~nan]) and np.array_equal(lib[~nan], form[~nan])
    # signed zeros keep their sign
    assert math.copysign(1.0, ours[0x8000]) == -1.0 and math.copysign(1.0, ours[0]) == 1.0


def test_all_ones_equals_dense_and_library_sdpa():
    wl = _wl(rule=dict(kind="ones"))
    q, k, v = _qkv(wl)
    mask = make_mask(wl)
    o, lse = A.block_sparse_attention(q, k, v, mask, wl.block)
    for h in range(wl.heads):
        dense = A.dense_attention(q[0, h], k[0, h], v[0, h])
        assert np.allclose(o[0, h], dense, atol=1e-12, rtol=0)
        qt = torch.from_numpy(A.bf16_to_f64(q[0, h]))[None]
        kt = torch.from_numpy(A.bf16_to_f64(k[0, h]))[None]
        vt = torch.from_numpy(A.bf16_to_f64(v[0, h]))[None]
        lib = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt)[0].numpy()
        assert np.allclose(o[0, h], lib, atol=1e-12, rtol=0)
        s = A.bf16_to_f64(q[0, h]) @ A.bf16_to_f64(k[0, h]).T / math.sqrt(wl.head_dim)
        ref_lse = np.log(np.exp(s - s.max(1, keepdims=True)).sum(1)) + s.max(1)
        assert np.allclose(lse[0, h], ref_lse, atol=1e-12)


@pytest.mark.parametrize("n", [None, 57, 49])   # full blocks, ragged tail of 9, ragged tail of 1
def test_brute_force_token_mask(n):
    wl = _wl(n=n, rule=dict(kind="empty_rows", p=0.35, empty=0.2))
    q, k, v = _qkv(wl)
    mask = make_mask(wl)
    o, _ = A.block_sparse_attention(q, k, v, mask, wl.block)
    for h in range(wl.heads):
        bf = A.token_masked_attention(q[0, h], k[0, h], v[0, h], mask[0, h], wl.block)
        assert np.allclose(o[0, h], bf, atol=1e-12, rtol=0)


def test_row_permutation_invariance():
    wl = _wl(n=61, rule=dict(kind="bernoulli", p=0.4))
    q, k, v = _qkv(wl)
    mask = make_mask(wl)
    blk, mb = wl.block, wl.mb
    o, _ = A.block_sparse_attention(q, k, v, mask, blk)
    rng = np.random.default_rng(0)
    # permute the full query blocks among themselves (the ragged last block stays last)
    perm = np.concatenate([rng.permutation(mb - 1), [mb - 1]])
    tok = np.concatenate([np.arange(i * blk, min((i + 1) * blk, wl.seq_len)) for i in perm])
    q2 = q[:, :, tok]
    m2 = mask[:, :, perm]
    o2, _ = A.block_sparse_attention(q2, k, v, m2, blk)
    back = np.empty_like(o2)
    back[:, :, tok] = o2
    assert np.array_equal(back, o)


def test_closed_forms():
    wl = _wl(n=50, rule=dict(kind="empty_rows", p=0.4, empty=0.3))
    q, k, v = _qkv(wl)
    mask = make_mask(wl)
    blk = wl.block
    # V constant along tokens -> O equals that vector on every non-empty row
    vc = np.broadcast_to(v[:, :, :1], v.shape).copy()
    o, lse = A.block_sparse_attention(q, k, vc, mask, blk)
    vec = A.bf16_to_f64(vc[0, 0, 0])
    for h in range(wl.heads):
        for i in range(wl.mb):
            lo, hi = A.block_token_range(i, blk, wl.seq_len)
            if mask[0, h, i].any():
                assert np.allclose(o[0, h, lo:hi], A.bf16_to_f64(vc[0, h, 0]), atol=1e-12)
            else:
                assert np.all(o[0, h, lo:hi] == 0) and np.all(lse[0, h, lo:hi] == -np.inf)
    assert vec.shape == (wl.head_dim,)
    # Q = 0 -> O is the plain mean of V over the kept tokens
    qz = np.zeros_like(q)
    o, _ = A.block_sparse_attention(qz, k, v, mask, blk)
    vf = A.bf16_to_f64(v[0, 1])
    for i in range(wl.mb):
        lo, hi = A.block_token_range(i, blk, wl.seq_len)
        cols = np.nonzero(mask[0, 1, i])[0]
        if cols.size:
            keys = np.concatenate([np.arange(*A.block_token_range(j, blk, wl.seq_len)) for j in cols])
            assert np.allclose(o[0, 1, lo:hi], vf[keys].mean(0), atol=1e-12)
    # a single kept block -> ordinary softmax over that block's keys
    m1 = np.zeros_like(mask)
    m1[0, 0, 1, 3] = 1
    o, _ = A.block_sparse_attention(q, k, v, m1, blk)
    lo, hi = A.block_token_range(1, blk, wl.seq_len)
    klo, khi = A.block_token_range(3, blk, wl.seq_len)
    ref = A.dense_attention(q[0, 0, lo:hi], k[0, 0, klo:khi], v[0, 0, klo:khi])
    assert np.allclose(o[0, 0, lo:hi], ref, atol=1e-12)


def test_ragged_tail_equals_padded_with_neg_inf():
    wl = _wl(n=53, rule=dict(kind="bernoulli", p=0.5))
    q, k, v = _qkv(wl)
    mask = make_mask(wl)
    blk, n, mb = wl.block, wl.seq_len, wl.mb
    o, _ = A.block_sparse_attention(q, k, v, mask, blk)
    pad = mb * blk
    for h in range(wl.heads):
        qf = np.zeros((pad, wl.head_dim)); qf[:n] = A.bf16_to_f64(q[0, h])
        kf = np.zeros((pad, wl.head_dim)); kf[:n] = A.bf16_to_f64(k[0, h])
        vf = np.zeros((pad, wl.head_dim)); vf[:n] = A.bf16_to_f64(v[0, h])
        tok = np.arange(pad) // blk
        allowed = mask[0, h][tok[:, None], tok[None, :]].astype(bool) & (np.arange(pad) < n)[None, :]
        s = np.where(allowed, qf @ kf.T / math.sqrt(wl.head_dim), -np.inf)
        for r in range(n):
            if allowed[r].any():
                e = np.exp(s[r] - s[r].max())
                assert np.allclose(o[0, h, r], e @ vf / e.sum(), atol=1e-12)


def test_sampled_rows_match_full():
    wl = _wl(n=70, heads=3, rule=dict(kind="bernoulli", p=0.3))
    q, k, v = _qkv(wl)
    mask = make_mask(wl)
    o, lse = A.block_sparse_attention(q, k, v, mask, wl.block)
    picks = [(0, 2, 4), (0, 0, 0), (0, 1, wl.mb - 1)]
    res = A.block_sparse_attention_rows(q, k, v, mask, wl.block, picks)
    for (b, h, i), (ob, lb) in res.items():
        lo, hi = A.block_token_range(i, wl.block, wl.seq_len)
        assert np.array_equal(ob, o[b, h, lo:hi]) and np.array_equal(lb, lse[b, h, lo:hi])


# ---- planted mistakes: each must be caught by one of the pins above -----------------------------
def test_planted_unclipped_tail_is_caught(monkeypatch):
    monkeypatch.setattr(A, "block_token_range", lambda j, blk, n: (j * blk, (j + 1) * blk))
    with pytest.raises(Exception):
        test_brute_force_token_mask(57)


def test_planted_wrong_scale_is_caught(monkeypatch):
    orig = A.attend_block_row
    monkeypatch.setattr(A, "attend_block_row", lambda qb, kf, vf, row, blk, scale: orig(qb, kf, vf, row, blk, scale * 1.01))
    with pytest.raises(AssertionError):
        test_all_ones_equals_dense_and_library_sdpa()


def test_planted_transposed_mask_is_caught(monkeypatch):
    orig = A.attend_block_row
    state = {}

    def wrong(qb, kf, vf, row, blk, scale):
        return orig(qb, kf, vf, state["mt"][state["i"]], blk, scale)

    real = A.block_sparse_attention

    def patched(q, k, v, mask, blk, scale=None):
        out_o = np.zeros(q.shape); out_l = np.zeros(q.shape[:3])
        for h in range(q.shape[1]):
            state["mt"] = mask[0, h].T
            for i in range(mask.shape[2]):
                state["i"] = i
                lo, hi = A.block_token_range(i, blk, q.shape[2])
                out_o[0, h, lo:hi], out_l[0, h, lo:hi] = wrong(
                    A.bf16_to_f64(q[0, h, lo:hi]), A.bf16_to_f64(k[0, h]), A.bf16_to_f64(v[0, h]), None, blk,
                    1 / math.sqrt(q.shape[3]))
        return out_o, out_l

    monkeypatch.setattr(A, "block_sparse_attention", patched)
    with pytest.raises(AssertionError):
        test_brute_force_token_mask(None)
    assert real is not patched
