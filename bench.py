"""Benchmark of the block-sparse attention path with cache-aware row reordering on one MI355X.

A step is one pass of the whole path over the workload, inputs resident in HBM:
  build_permutation (mask scans, subspace iteration, polar sort, wave buckets, Stage 2)
  -> compact_mask (per-row KV-block lists) -> sparse attention (bf16 MFMA).
The headline value is effective TFLOP/s = 4 * block^2 * d * sum(nnz) / step time,
i.e. the FLOPs of the kept blocks over the whole step (reordering overhead included).

Prints one JSON line. Default workload: the 720p / 401-frame long-video shape
(40 heads, d = 128, 363,600 tokens, 128-token blocks, ~5% mean density).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from workloads import CONFIGS, make_mask, make_qkv  # noqa: E402

MFMA_BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
HBM_PEAK_GBS = 8000.0
ATTN_SRC = os.path.join(ROOT, "paper_2609_34814_amd", "csrc", "attn_fwd.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_traffic.json")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    with open(ATTN_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def load_traffic(workload: str, variant: str):
    """HBM bytes per attention launch from the committed rocprofv3 counter summary, if it is current."""
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    entry = data.get(workload, {}).get(variant)
    if not entry or entry.get("kernel_sha") != kernel_source_hash():
        return None
    return entry.get("hbm_bytes_per_launch")


def _pmc_means(csv_path: str, kernel_substr: str):
    import csv
    vals = {}
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            if kernel_substr in r["Kernel_Name"]:
                vals.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in vals.items()}, max((len(v) for v in vals.values()), default=0)


def summarize_pmc(root: str, workload: str, out_json: str, out_md: str, command_note: str) -> None:
    """Turn rocprofv3 --pmc CSV passes into the traffic figure and a text summary.

    Expects <root>/<variant>_{A,B,C}/run_counter_collection.csv for the attention kernel
    (A: TCC_HIT_sum TCC_MISS_sum SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CYCLES
    GRBM_GUI_ACTIVE; B: FETCH_SIZE; C: WRITE_SIZE TCC_EA0_RDREQ_DRAM_sum) and copy_{B,C} for a plain
    1 GiB device copy, whose FETCH_SIZE / WRITE_SIZE give the byte-scaling factors.
    """
    cb, _ = _pmc_means(os.path.join(root, "copy_B", "run_counter_collection.csv"), "copyBuffer")
    cc, _ = _pmc_means(os.path.join(root, "copy_C", "run_counter_collection.csv"), "copyBuffer")
    copy_bytes = float(1 << 30)
    f_fetch = copy_bytes / (cb["FETCH_SIZE"] * 1024.0)
    f_write = copy_bytes / (cc["WRITE_SIZE"] * 1024.0)
    sha = kernel_source_hash()
    try:
        with open(out_json) as f:
            data = json.load(f)
    except (OSError, ValueError):
        data = {}
    lines = [f"# attention kernel counters, workload {workload}", "", f"Command: {command_note}", "",
             f"Copy calibration (1 GiB device copy): FETCH_SIZE x {f_fetch:.3f}, WRITE_SIZE x {f_write:.3f}", "",
             "| variant | dispatches | L2 hit % | L2->fabric read GB/launch (scaled) | write GB/launch (scaled) | "
             "DRAM read req | MFMA FLOP (MOPS x 512) | MFMA busy % |",
             "|---|---|---|---|---|---|---|---|"]
    entry = data.setdefault(workload, {})
    variants = sorted({d.rsplit("_", 1)[0] for d in os.listdir(root) if d.endswith("_A")})
    for v in variants:
        a, na = _pmc_means(os.path.join(root, f"{v}_A", "run_counter_collection.csv"), "attn_fwd")
        b, _ = _pmc_means(os.path.join(root, f"{v}_B", "run_counter_collection.csv"), "attn_fwd")
        c, _ = _pmc_means(os.path.join(root, f"{v}_C", "run_counter_collection.csv"), "attn_fwd")
        hit = a["TCC_HIT_sum"] / (a["TCC_HIT_sum"] + a["TCC_MISS_sum"])
        fetch = b["FETCH_SIZE"] * 1024.0 * f_fetch
        write = c["WRITE_SIZE"] * 1024.0 * f_write
        cycles = a["GRBM_GUI_ACTIVE"] / 8.0          # summed over the 8 XCDs
        busy = a["SQ_VALU_MFMA_BUSY_CYCLES"] / (256 * 4 * cycles)
        entry[v] = {"kernel_sha": sha, "hbm_bytes_per_launch": fetch + write, "fetch_bytes": fetch,
                    "write_bytes": write, "l2_hit": hit, "dram_read_requests": c["TCC_EA0_RDREQ_DRAM_sum"],
                    "mfma_flop": a["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512, "mfma_busy": busy}
        lines.append(f"| {v} | {na} | {100 * hit:.2f} | {fetch / 1e9:.1f} | {write / 1e9:.2f} | "
                     f"{c['TCC_EA0_RDREQ_DRAM_sum']:.4g} | {a['SQ_INSTS_VALU_MFMA_MOPS_BF16'] * 512:.4g} | "
                     f"{100 * busy:.1f} |")
    with open(out_json, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def cpu_baseline(wl, q, k, v, mask, total_flop, budget_s: float):
    """The oracle, as it stands, timed on a bounded sample of the workload on the host cores."""
    from oracle import attention as A
    from oracle import permutation as P
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count() or 1
    rng = np.random.default_rng(7)
    # attention oracle on random query blocks until the budget is spent
    t0 = time.perf_counter()
    flop_done, blocks = 0.0, 0
    blk, d = wl.block, wl.head_dim
    while time.perf_counter() - t0 < budget_s * 0.7:
        h = int(rng.integers(wl.heads))
        i = int(rng.integers(wl.mb))
        A.block_sparse_attention_rows(q, k, v, mask, blk, [(0, h, i)])
        flop_done += 4.0 * blk * blk * d * float(mask[0, h, i].sum())
        blocks += 1
    t_attn = time.perf_counter() - t0
    # permutation oracle on one head
    t1 = time.perf_counter()
    P.two_stage_permutation(mask[0, 0], seed=0, flat_head=0, wave=64, n_xcd=8, iters=10)
    t_perm_head = time.perf_counter() - t1
    est_step = t_attn / max(flop_done, 1.0) * total_flop + t_perm_head * wl.batch * wl.heads
    return {
        "value": total_flop / est_step / 1e12,
        "unit": "TFLOP/s",
        "cores": int(cores),
        "kind": "oracle",
        "sample": (f"fp64 oracle attention on {blocks} random query blocks ({flop_done / 1e9:.1f} GFLOP, "
                   f"{t_attn:.1f} s) plus the permutation oracle on 1 of {wl.batch * wl.heads} heads "
                   f"({t_perm_head:.1f} s); step time extrapolated by FLOPs and head count "
                   f"(est. {est_step:.0f} s per step)"),
    }


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="long-720p-401f", choices=sorted(CONFIGS))
    ap.add_argument("--variants", default="reordered,natural",
                    help="comma list of: reordered (two-stage order, work-balanced XCD segments, skip never), "
                         "natural (identity order, equal row-count XCD segments), auto (adaptive skip), "
                         "naive (identity, plain dispatch order), reordered-rowseg (two-stage order, equal "
                         "row-count segments), natural-balanced (identity order, work-balanced segments)")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of this many MiB (3 times), to calibrate the HBM counters")
    ap.add_argument("--summarize-pmc", metavar="DIR", help="summarize rocprofv3 counter passes found in DIR "
                    "into profiles/attn_traffic.json and a markdown table (no GPU needed)")
    ap.add_argument("--pmc-command", default="", help="command line recorded in the counter summary")
    args = ap.parse_args()

    if args.summarize_pmc:
        md = os.path.join(ROOT, "profiles", f"attn_fwd_{args.config}_counters.md")
        summarize_pmc(args.summarize_pmc, args.config, TRAFFIC_FILE, md, args.pmc_command)
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the path is a single-GPU kernel pipeline "
              "(see DESIGN.md for how it would shard across GPUs)", file=sys.stderr)
        return 2

    import torch
    import paper_2609_34814_amd as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_calibration:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 3}))
        return 0
    wl = CONFIGS[args.config]
    t0 = time.perf_counter()
    mask = make_mask(wl, threads=16)
    q, k, v = make_qkv(wl, threads=16)
    log(f"generated {wl.name} in {time.perf_counter() - t0:.1f} s")

    def dev(bits):
        return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()

    qd, kd, vd = dev(q), dev(k), dev(v)
    md = torch.from_numpy(mask).cuda()
    nnz = int(mask.sum(dtype=np.int64))
    flop = 4.0 * wl.block * wl.block * wl.head_dim * nnz
    b_, h_, mb = wl.batch, wl.heads, wl.mb
    shape = W.shape_of(b_, h_, wl.seq_len, wl.head_dim, wl.block)
    perm_ws = torch.empty(W.perm_workspace_size(shape), dtype=torch.uint8, device="cuda")
    perm = torch.empty((b_, h_, mb), dtype=torch.int32, device="cuda")
    row_ptr = torch.empty((b_, h_, mb + 1), dtype=torch.int32, device="cuda")
    col_idx = torch.empty((b_ * h_ * mb * mb,), dtype=torch.int32, device="cuda")
    o = torch.empty_like(qd)
    flags = torch.empty((b_, h_), dtype=torch.uint8, device="cuda")
    seg = torch.empty((b_, h_, 9), dtype=torch.int32, device="cuda")
    attn_ws = torch.empty(W.attn_workspace_size(shape), dtype=torch.uint8, device="cuda")
    wave = W.wave_size(wl.head_dim, wl.block)
    stream = torch.cuda.current_stream()
    log(f"uploaded; nnz={nnz} density={nnz / (b_ * h_ * mb * mb):.4f} wave_per_xcd={wave}")

    def make_step(variant):
        skip = {"reordered": "never", "auto": "auto", "reordered-rowseg": "never",
                "natural-balanced": "always"}.get(variant)
        n_xcd = 1 if variant == "naive" else 8
        use_seg = variant in ("reordered", "auto", "natural-balanced")

        def step(ev=None):
            p = None
            if skip is not None:
                W.build_permutation(md, seq_len=wl.seq_len, block=wl.block, head_dim=wl.head_dim,
                                    wave=wave, n_xcd=8, skip=skip, workspace=perm_ws, out=perm, flags_out=flags,
                                    seg_out=seg)
                p = perm
            rp, ci = W.compact_mask(md, seq_len=wl.seq_len, block=wl.block, head_dim=wl.head_dim,
                                    row_ptr=row_ptr, col_idx=col_idx)
            if ev is not None:
                ev[0].record(stream)
            W.sparse_attn_csr(qd, kd, vd, rp, ci, p, seg if use_seg else None, block=wl.block, n_xcd=n_xcd,
                              out=o, workspace=attn_ws)
            if ev is not None:
                ev[1].record(stream)
        return step

    results = {}
    for variant in [s.strip() for s in args.variants.split(",") if s.strip()]:
        step = make_step(variant)
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        start.record(stream)
        for i in range(args.steps):
            step(evs[i])
        end.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        ms_step = start.elapsed_time(end) / args.steps
        attn_ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
        results[variant] = dict(ms_per_step=ms_step, wall_ms_per_step=wall * 1e3 / args.steps, attn_ms=attn_ms,
                                tflops_step=flop / (ms_step * 1e-3) / 1e12,
                                tflops_attn=flop / (attn_ms * 1e-3) / 1e12)
        log(f"{variant}: step {ms_step:.2f} ms, attention kernel {attn_ms:.2f} ms "
            f"({results[variant]['tflops_attn']:.1f} TFLOP/s)")

    head = "reordered" if "reordered" in results else next(iter(results))
    r = results[head]
    traffic = load_traffic(wl.name, head)
    roof = {
        "bound": "mfma",
        "achieved": r["tflops_attn"],
        "peak": MFMA_BF16_PEAK_TFLOPS,
        "unit": "TFLOP/s",
        "frac": r["tflops_attn"] / MFMA_BF16_PEAK_TFLOPS,
        "traffic": traffic,
    }
    out = {
        "metric": "sparse-attn effective TFLOP/s (reordered path incl. reordering overhead)",
        "value": r["tflops_step"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": b_, "heads": h_, "seq_len": wl.seq_len, "head_dim": wl.head_dim,
                   "block": wl.block, "kept_blocks": nnz, "density": nnz / (b_ * h_ * mb * mb),
                   "flop_per_step": flop, "variant": head, "wave_per_xcd": wave},
        "roofline": roof,
        "variants": results,
    }
    if "natural" in results and "reordered" in results:
        out["speedup_reordered_vs_natural"] = {
            "step": results["natural"]["ms_per_step"] / results["reordered"]["ms_per_step"],
            "attention_kernel": results["natural"]["attn_ms"] / results["reordered"]["attn_ms"],
        }
    if not args.no_cpu_baseline:
        log("timing the oracle on the host")
        out["cpu_baseline"] = cpu_baseline(wl, q, k, v, mask, flop, args.cpu_budget)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
