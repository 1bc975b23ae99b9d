"""The attention entry point that allocates nothing, through the C ABI: on two calls in a row, the
second with a smaller input, its O, LSE and status equal those of the workspace entry point
(wa_sparse_attn_vt) bit for bit."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from tests.gpu_util import bf16_dev, u8_dev   # noqa: E402
from workloads import CONFIGS, make_mask, make_qkv   # noqa: E402


def _case(W, wl, n_xcd, head_order, reorder):
    q, k, v = (bf16_dev(x) for x in make_qkv(wl, threads=16))
    md = u8_dev(make_mask(wl, threads=16))
    rp, ci = W.compact_mask(md, seq_len=wl.seq_len, block=wl.block, head_dim=wl.head_dim)
    vt = W.transpose_v(v, block=wl.block)
    perm = seg = None
    if reorder:
        perm, seg, _ = W.build_permutation(md, seq_len=wl.seq_len, block=wl.block, head_dim=wl.head_dim,
                                           n_xcd=n_xcd, skip="never")
    ref, ref_lse = W.sparse_attn_vt(q, k, vt, rp, ci, perm, seg, block=wl.block, n_xcd=n_xcd,
                                    head_order=head_order, return_lse=True)
    out = torch.full_like(q, float("nan"))
    lse = torch.full(q.shape[:3], float("nan"), dtype=torch.float32, device="cuda")
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    W.sparse_attn_vt_noalloc(q, k, vt, rp, ci, perm, seg, block=wl.block, n_xcd=n_xcd, head_order=head_order,
                             lse=lse, out=out, status=status)
    torch.cuda.synchronize()
    print(f"no-alloc call: {wl.name}, n_xcd {n_xcd}, {head_order}, reordered {reorder}", flush=True)
    assert int(status.item()) == 0
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), ref_lse.view(torch.int32))


def test_noalloc_matches_workspace_entry_on_two_calls_second_smaller():
    import paper_2609_34814_amd as W
    # 40 heads x 591 blocks (per-XCD queues, two-stage order), then 2 heads x 64 blocks (one queue,
    # heads interleaved): the second call reuses the GPU's scratch the first one left behind
    _case(W, CONFIGS["wan14b-720p-81f"], 8, "in-order", True)
    _case(W, CONFIGS["tiny"], 1, "interleaved", False)
