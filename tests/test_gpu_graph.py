"""The whole path captured in one graph (torch.cuda.CUDAGraph on the HIP runtime) and replayed.

Mask producer -> permutation -> compaction -> V transpose -> attention. Once their outputs and workspaces
are given, none of these calls allocates, synchronises or records a memset (the scheduler state is
cleared by a kernel), so the sequence can be captured. Every replay, with the outputs overwritten and
other eager work run in between, must give the same bytes as the eager calls.
"""
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from tests.gpu_util import bf16_dev                  # noqa: E402
from workloads import custom, make_qkv               # noqa: E402
from workloads.gen import PRODUCER_CONFIGS           # noqa: E402


def _w():
    import paper_2609_34814_amd as W
    return W


CASES = {
    # one head group in the producer, the one-workgroup permutation
    "produced-ragged": PRODUCER_CONFIGS["produced-ragged"],
    # two head groups in the producer pipeline, the sliced permutation (1,500 blocks per head)
    "groups-sliced": custom("graph-groups", batch=2, heads=7, head_dim=64, block=64, grid=(1500, 8, 8),
                            seq_len=1500 * 64 - 17, seed=41),
}


@pytest.mark.parametrize("name", list(CASES))
def test_path_graph_replays_match_eager(name):
    W = _w()
    wl = CASES[name]
    q, k, v = make_qkv(wl)
    qd, kd, vd = bf16_dev(q), bf16_dev(k), bf16_dev(v)
    b, h, n, d, blk, mb = wl.batch, wl.heads, wl.seq_len, wl.head_dim, wl.block, wl.mb
    shape = W.shape_of(b, h, n, d, blk)
    keep = max(1, mb // 10)
    u8, i32 = torch.uint8, torch.int32
    mask = torch.empty((b, h, mb, mb), dtype=u8, device="cuda")
    pws = torch.empty(W.mask_producer_workspace_size(shape), dtype=u8, device="cuda")
    perm = torch.empty((b, h, mb), dtype=i32, device="cuda")
    flags = torch.empty((b, h), dtype=u8, device="cuda")
    seg = torch.empty((b, h, 9), dtype=i32, device="cuda")
    perm_ws = torch.empty(W.perm_workspace_size(shape), dtype=u8, device="cuda")
    row_ptr = torch.empty((b, h, mb + 1), dtype=i32, device="cuda")
    col_idx = torch.empty((b * h * mb * mb,), dtype=i32, device="cuda")
    vt = torch.empty((b, h, d, mb * blk), dtype=torch.bfloat16, device="cuda")
    o = torch.empty_like(qd)
    status = torch.empty((1,), dtype=i32, device="cuda")
    attn_ws = torch.empty(W.attn_vt_workspace_size(shape), dtype=u8, device="cuda")

    def path():
        W.produce_block_mask(qd, kd, block=blk, keep=keep, diagonal=True, out=mask, workspace=pws)
        W.build_permutation(mask, seq_len=n, block=blk, head_dim=d, skip="never", out=perm, flags_out=flags,
                            seg_out=seg, workspace=perm_ws)
        W.compact_mask(mask, seq_len=n, block=blk, head_dim=d, row_ptr=row_ptr, col_idx=col_idx)
        W.transpose_v(vd, block=blk, out=vt)
        _, lse = W.sparse_attn_vt(qd, kd, vt, row_ptr, col_idx, perm, seg, block=blk, return_lse=True, out=o,
                                  workspace=attn_ws, status=status)
        return lse

    def snapshot(lse):
        # each head's list starts at (b H + h) M_B^2; the entries past its end are not written
        ends = row_ptr[..., -1].reshape(-1).cpu().tolist()
        lists = torch.cat([col_idx[x * mb * mb: x * mb * mb + e] for x, e in enumerate(ends)])
        return {"mask": mask.clone(), "perm": perm.clone(), "flags": flags.clone(), "seg": seg.clone(),
                "row_ptr": row_ptr.clone(), "col_idx": lists.clone(),
                "vt": vt.view(torch.int16).clone(), "o": o.view(torch.int16).clone(),
                "lse": lse.view(torch.int32).clone(), "status": status.clone()}

    lse_e = path()
    torch.cuda.synchronize()
    ref = snapshot(lse_e)
    assert int(ref["status"].item()) == 0
    assert int(ref["mask"].sum().item()) >= b * h * mb * keep  # keep blocks per row (+ the diagonal)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # a warm-up on the capture stream's side, as torch recommends
        path()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lse_g = path()
    torch.cuda.synchronize()

    rng = torch.Generator(device="cuda").manual_seed(7)
    for rep in range(3):
        # overwrite every output, run unrelated eager work, then replay
        for t in (mask, flags):
            t.fill_(0xAB)
        for t in (perm, seg, row_ptr, col_idx, status):
            t.fill_(-7)
        vt.fill_(float("nan"))
        o.fill_(float("nan"))
        lse_g.fill_(float("nan"))
        x = torch.randn((512, 512), device="cuda", generator=rng)
        (x @ x).sum().item()
        g.replay()
        torch.cuda.synchronize()
        got = snapshot(lse_g)
        for key, want in ref.items():
            assert torch.equal(got[key], want), (name, rep, key)
