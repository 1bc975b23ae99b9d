"""GPU parity of the pooled-score top-k mask producer against its oracle, through the C ABI.

Bar: codes and mask bit-exact (every step is exact or one float32 rounding in a fixed order).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from oracle import attention as A          # noqa: E402
from oracle import mask_producer as MP     # noqa: E402
from tests.gpu_util import bf16_dev, compare_blocks, dev_f64, u8_dev  # noqa: E402
from workloads import custom, make_qkv     # noqa: E402
from workloads.gen import PRODUCER_CONFIGS  # noqa: E402


def _w():
    import paper_2609_34814_amd as W
    return W


def _oracle_codes(q, k, blk):
    b_, h_ = q.shape[:2]
    out = []
    for src in (q, k):
        out.append(np.stack([np.stack([MP.quantize(MP.pooled_means(src[b, h], blk)) for h in range(h_)])
                             for b in range(b_)]))
    return np.stack(out)


def _run(q, k, blk, keep, diagonal):
    qd, kd = bf16_dev(q), bf16_dev(k)
    b_, h_, n, d = q.shape
    mb = -(-n // blk)
    codes = torch.empty((2, b_, h_, mb, d), dtype=torch.int8, device="cuda")
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")  # the call clears it
    mask = _w().produce_block_mask(qd, kd, block=blk, keep=keep, diagonal=diagonal, codes_out=codes, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0  # no selection's wait for codes ran out
    return mask.cpu().numpy(), codes.cpu().numpy()


@pytest.mark.parametrize("name,keep,diagonal", [("produced-tiny", 8, True), ("produced-tiny", 1, False),
                                                ("produced-tiny", 0, True), ("produced-tiny", 64, False),
                                                ("produced-tiny", 500, True), ("produced-ragged", 6, True),
                                                ("produced-ragged", 13, False)])
def test_producer_bit_exact(name, keep, diagonal):
    wl = PRODUCER_CONFIGS[name]
    q, k, _ = make_qkv(wl)
    mask, codes = _run(q, k, wl.block, keep, diagonal)
    assert np.array_equal(codes, _oracle_codes(q, k, wl.block))
    assert np.array_equal(mask, MP.produce_mask(q, k, wl.block, keep, diagonal))


def test_producer_ties_and_zero_maximum():
    """All-zero K: every score is 0, so each row keeps the first `keep` blocks; constant Q rows tie too."""
    wl = custom("ties", heads=2, head_dim=64, block=64, grid=(2, 16, 16), seed=21)
    q, k, _ = make_qkv(wl)
    k[:] = 0
    q[0, 1] = q[0, 1, :1]          # one constant row in every block of head 1
    mask, codes = _run(q, k, wl.block, 5, False)
    assert not codes[1].any()
    ref = MP.produce_mask(q, k, wl.block, 5, False)
    assert np.array_equal(mask, ref)
    assert np.all(mask[..., :5] == 1) and not mask[..., 5:].any()


@pytest.mark.parametrize("keep", [5, 30, 50, 64])
def test_producer_partial_ties_at_the_threshold(keep):
    """Every KV block repeats one of three token rows, so each row's scores take three values about 21
    times each: the threshold score is tied and only some of its ties are kept (the first in j)."""
    wl = custom("ties3", heads=2, head_dim=64, block=64, grid=(4, 32, 32), seed=22)
    q, k, _ = make_qkv(wl)
    rng = np.random.default_rng(22)
    mb = wl.mb
    for h in range(wl.heads):
        pats = k[0, h, [0, 1, 2]].copy()
        pick = rng.integers(0, 3, size=mb)
        for j in range(mb):
            k[0, h, j * wl.block:(j + 1) * wl.block] = pats[pick[j]]
    mask, codes = _run(q, k, wl.block, keep, True)
    assert np.array_equal(codes, _oracle_codes(q, k, wl.block))
    assert np.array_equal(mask, MP.produce_mask(q, k, wl.block, keep, True))


@pytest.mark.parametrize("mb,d,keep", [(1500, 128, 75), (4096, 64, 200), (257, 64, 9)])
def test_producer_bit_exact_row_widths(mb, d, keep):
    """Heads of 1,500, 4,096 and 257 blocks (ragged last blocks): every width of the selection's
    per-lane score array, the largest supported head included."""
    wl = custom(f"rows{mb}", heads=1, head_dim=d, block=64, grid=(mb, 8, 8), seq_len=mb * 64 - 33, seed=23 + mb)
    assert wl.mb == mb
    q, k, _ = make_qkv(wl)
    mask, codes = _run(q, k, wl.block, keep, True)
    assert np.array_equal(codes, _oracle_codes(q, k, wl.block))
    assert np.array_equal(mask, MP.produce_mask(q, k, wl.block, keep, True))


def test_producer_bit_exact_head_groups():
    """Two sequences of seven heads of 1,500 blocks: the pipeline takes heads in groups of eight, so
    the launches see a full group, a short last group, and heads of both sequences in one group."""
    wl = custom("groups", batch=2, heads=7, head_dim=64, block=64, grid=(1500, 8, 8), seq_len=1500 * 64 - 17,
                seed=31)
    q, k, _ = make_qkv(wl)
    mask, codes = _run(q, k, wl.block, 60, True)
    assert np.array_equal(codes, _oracle_codes(q, k, wl.block))
    assert np.array_equal(mask, MP.produce_mask(q, k, wl.block, 60, True))


@pytest.mark.parametrize("batch,heads,d,blk,seq,keep", [(3, 37, 64, 64, 300, 2), (2, 100, 128, 128, 100, 1)])
def test_producer_bit_exact_many_short_heads(batch, heads, d, blk, seq, keep):
    """Heads of 5 blocks (ragged) and of a single block: one pooling item of the queue covers the blocks of
    up to 64 heads of one tensor, so one workgroup writes the codes of many heads (64 at once with one
    block per head and d 128, as many as an item holds), and one head group holds every head."""
    wl = custom(f"short{heads}", batch=batch, heads=heads, head_dim=d, block=blk, grid=(1, 1, seq), seq_len=seq,
                seed=40 + heads)
    q, k, _ = make_qkv(wl)
    mask, codes = _run(q, k, wl.block, keep, True)
    assert np.array_equal(codes, _oracle_codes(q, k, wl.block))
    assert np.array_equal(mask, MP.produce_mask(q, k, wl.block, keep, True))


def test_producer_bit_exact_full_size():
    """363,600 tokens, 40 heads, 5% of the blocks per row: every row of every head."""
    wl = PRODUCER_CONFIGS["produced-long-720p-401f"]
    q, k, _ = make_qkv(wl, threads=16)
    keep = round(0.05 * wl.mb)
    mask, codes = _run(q, k, wl.block, keep, True)
    assert np.array_equal(codes, _oracle_codes(q, k, wl.block))
    for h in range(wl.heads):
        ref = MP.produce_head(q[0, h], k[0, h], wl.block, keep, True)[0]
        assert np.array_equal(mask[0, h], ref), h


def test_produced_mask_feeds_the_path():
    """The produced mask through permutation, compaction and attention: sampled rows vs the oracle."""
    wl = PRODUCER_CONFIGS["produced-ragged"]
    q, k, v = make_qkv(wl)
    W = _w()
    qd, kd, vd = bf16_dev(q), bf16_dev(k), bf16_dev(v)
    md = W.produce_block_mask(qd, kd, block=wl.block, keep=6, diagonal=True)
    perm, seg, _ = W.build_permutation(md, seq_len=wl.seq_len, block=wl.block, head_dim=wl.head_dim, skip="never")
    rp, ci = W.compact_mask(md, seq_len=wl.seq_len, block=wl.block, head_dim=wl.head_dim)
    o, lse = W.sparse_attn_csr(qd, kd, vd, rp, ci, perm, seg, block=wl.block, return_lse=True)
    torch.cuda.synchronize()
    mask = md.cpu().numpy()
    assert np.array_equal(mask, MP.produce_mask(q, k, wl.block, 6, True))
    picks = [(b, h, i) for b in range(wl.batch) for h in range(wl.heads) for i in (0, 17, wl.mb - 1)]
    ref = A.block_sparse_attention_rows(q, k, v, mask, wl.block, picks)
    st = compare_blocks(dev_f64(o), ref, wl.block, wl.seq_len, lse.cpu().numpy().astype(np.float64))
    assert st["max_abs"] <= 1e-2 and st["mean_abs"] <= 1e-3 and st["lse"] <= 1e-3, st
