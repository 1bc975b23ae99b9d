"""Benchmark of the block-sparse attention path with cache-aware row reordering on one MI355X.

A step is one pass of the whole path over the workload, inputs resident in HBM:
  build_permutation (mask scans, subspace iteration, polar sort, wave buckets, Stage 2)
  -> compact_mask (per-row KV-block lists) -> sparse attention (bf16 MFMA).
The headline value is effective TFLOP/s = 4 * block^2 * d * sum(nnz) / step time,
i.e. the FLOPs of the kept blocks over the whole step (reordering overhead included), of the
method as the paper defines it: the adaptive skip rule decides per head whether the two-stage
order is built or the identity order kept (variant `auto`). The same line reports every timed
variant (by default also `reordered`, the two-stage order on every head, and `natural`), their
speedups over natural order, and the L2 hit ratio and L2-to-fabric read bytes of each from the
committed counter summary while it matches the kernel source.

Prints one JSON line. Default workload: the 720p / 401-frame long-video shape
(40 heads, d = 128, 363,600 tokens, 128-token blocks, ~5% mean density).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from workloads import ALL_CONFIGS, make_mask, make_qkv  # noqa: E402

MFMA_BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
HBM_PEAK_GBS = 8000.0
ATTN_SRC = os.path.join(ROOT, "paper_2609_34814_amd", "csrc", "attn_fwd.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_traffic.json")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


_CODE_TOKENS = re.compile(r'"(?:\\.|[^"\\\n])*"|//[^\n]*|/\*.*?\*/', re.S)


def kernel_source_hash() -> str:
    """Hash of the attention source's code: comments removed and whitespace runs collapsed, so that a
    counter summary stays attached to the kernel it measured when only its comments change."""
    with open(ATTN_SRC, encoding="utf-8") as f:
        text = f.read()
    code = _CODE_TOKENS.sub(lambda m: m.group(0) if m.group(0).startswith('"') else " ", text)
    return hashlib.sha256(" ".join(code.split()).encode()).hexdigest()[:16]


def load_traffic(workload: str, variant: str):
    """HBM bytes per attention launch from the committed rocprofv3 counter summary, if it is current."""
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    entry = data.get(workload, {}).get(variant)
    if not entry or entry.get("kernel_sha") != kernel_source_hash() or entry.get("variant_spec") != VARIANTS[variant]:
        return None
    return entry.get("hbm_bytes_per_launch")


def load_counters(workload: str, variant: str):
    """L2 hit ratio, L2-to-fabric read bytes, MFMA busy and clock of one variant's attention launch, from
    the committed rocprofv3 counter summary while it matches the kernel source (else None)."""
    try:
        with open(TRAFFIC_FILE) as f:
            entry = json.load(f).get(workload, {}).get(variant)
    except (OSError, ValueError):
        return None
    if not entry or entry.get("kernel_sha") != kernel_source_hash() or entry.get("variant_spec") != VARIANTS[variant]:
        return None
    return {"l2_hit": entry.get("l2_hit"), "l2_fabric_read_bytes": entry.get("fetch_bytes"),
            "dram_addressed_read_bytes": entry.get("dram_read_bytes"), "mfma_busy": entry.get("mfma_busy"),
            "clock_ghz": entry.get("clock_ghz"), "source": "profiles/attn_traffic.json"}


def _pmc_dispatches(csv_path: str, kernel_substr: str):
    """Counters of every matching dispatch, in launch order: [(name, duration ns, {counter: value})]."""
    import csv
    rows = {}
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            if kernel_substr not in r["Kernel_Name"]:
                continue
            d = rows.setdefault(int(r["Dispatch_Id"]), [r["Kernel_Name"],
                                                       int(r["End_Timestamp"]) - int(r["Start_Timestamp"]), {}])
            d[2][r["Counter_Name"]] = d[2].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return [tuple(rows[k]) for k in sorted(rows)]


def _mean_counters(disp):
    out = {}
    for _, _, c in disp:
        for k, v in c.items():
            out[k] = out.get(k, 0.0) + v / len(disp)
    out["duration_ns"] = sum(d for _, d, _ in disp) / len(disp)
    return out


# rocprofv3 --pmc passes (one run each; every pass stays within one run's counter limits: at most
# 4 TCC, 8 SQ, 4 TCP, 2 GRBM counters)
PMC_PASSES = {
    "A": "TCC_HIT_sum TCC_MISS_sum SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CYCLES GRBM_GUI_ACTIVE",
    "B": "FETCH_SIZE",
    "C": "WRITE_SIZE",
    "D": "TCP_TCC_READ_REQ_sum TCP_TCC_READ_REQ_LATENCY_sum TCC_EA0_RDREQ_sum TCC_EA0_RDREQ_LEVEL_sum",
    "E": "TCC_EA0_RDREQ_sum TCC_EA0_RDREQ_32B_sum TCC_BUBBLE_sum TCC_EA0_RDREQ_DRAM_sum",
}


def _read_bytes_e(c):
    """L2 read bytes to the fabric from pass E (128-, 64- and 32-byte requests), and the share of them
    addressed to DRAM: on MI355X those go through the 256 MiB last-level cache on the way, and no
    counter of this pool tells its hits from HBM reads."""
    rd, r32, bub, dram = (c["TCC_EA0_RDREQ_sum"], c["TCC_EA0_RDREQ_32B_sum"], c["TCC_BUBBLE_sum"],
                          c["TCC_EA0_RDREQ_DRAM_sum"])
    total = bub * 128.0 + (rd - bub - r32) * 64.0 + r32 * 32.0
    return total, (dram / rd if rd else 0.0)


def summarize_pmc(root: str, workload: str, variants, warmup: int, steps: int, bench_json: str, out_json: str,
                  out_md: str, command_note: str) -> None:
    """Counter tables of one workload from rocprofv3 --pmc passes of ONE bench.py run per pass.

    <root>/<pass>/run_counter_collection.csv holds the attention kernel's dispatches of
    `bench.py --variants v1,v2,... --warmup W --steps K` in launch order: variant i owns dispatches
    [i (W+K), (i+1)(W+K)), of which the last K are averaged. <root>/copy_{B,C,E} hold a plain 1 GiB
    device copy, whose FETCH_SIZE, WRITE_SIZE and pass-E read bytes give the byte-scaling factors.
    bench_json is the line of an unprofiled run of the same variants (flushed median call times,
    effective TFLOP/s, order statistics)."""
    def copy_pass(p):
        # the 1 GiB copies only (the run also holds the small kernel that fills the source)
        d = _pmc_dispatches(os.path.join(root, "copy_" + p, "run_counter_collection.csv"), "copyBuffer")
        if not d:
            raise RuntimeError(f"copy pass {p}: no copy dispatches")
        return _mean_counters(d)

    copy_bytes = float(1 << 30)
    f_fetch = copy_bytes / (copy_pass("B")["FETCH_SIZE"] * 1024.0)
    f_write = copy_bytes / (copy_pass("C")["WRITE_SIZE"] * 1024.0)
    f_e = copy_bytes / _read_bytes_e(copy_pass("E"))[0]
    with open(bench_json) as f:
        line = json.loads([ln for ln in f.read().splitlines() if ln.startswith("{")][-1])
    per = warmup + steps
    passes = {}
    for p in PMC_PASSES:
        path = os.path.join(root, p, "run_counter_collection.csv")
        if not os.path.exists(path):
            continue
        disp = _pmc_dispatches(path, "attn_fwd_kernel")
        if len(disp) != per * len(variants):
            raise RuntimeError(f"pass {p}: {len(disp)} attention dispatches, expected {per * len(variants)}")
        passes[p] = {v: _mean_counters(disp[i * per + warmup:(i + 1) * per]) for i, v in enumerate(variants)}
    sha = kernel_source_hash()
    try:
        with open(out_json) as f:
            data = json.load(f)
    except (OSError, ValueError):
        data = {}
    entry = data.setdefault(workload, {})
    alg = line["algorithmic_bytes"]
    kv_global = alg["kv_compulsory"]
    xcd = alg.get("kv_compulsory_per_xcd", {})
    ost = line.get("order_stats", {})
    cfg = line["config"]
    lines = [f"# attention kernel counters, workload {workload}", "",
             f"{cfg['heads']} heads x {cfg['seq_len']} tokens, d {cfg['head_dim']}, {cfg['block']}-token blocks, "
             f"density {100 * cfg['density']:.2f}% ({cfg['kept_blocks']} kept blocks, "
             f"{cfg['flop_per_step']:.4g} FLOP per call); compulsory K/V {kv_global / 1e9:.3f} GB, Q+O "
             f"{alg['q_and_o'] / 1e9:.3f} GB.", "",
             "Commands (one rocprofv3 run per pass, each running the variants below in this order):", ""]
    run = ("cd /tmp && export TMPDIR=/tmp && cd $GRAFT_REPO_ROOT && timeout -s KILL 300 rocprofv3 --pmc {ctr} "
           "--kernel-include-regex {kre} --output-format csv -d {root}/{p} -o run -- {cmd}")
    bench_cmd = (f"python bench.py --config {workload} --steps {steps} --warmup {warmup} --no-cpu-baseline "
                 f"--no-gemm-reference --no-order-stats --variants {','.join(variants)}")
    for p, ctr in PMC_PASSES.items():
        lines.append(f"* pass {p}: `" + run.format(ctr=ctr, kre="attn_fwd", root=root, p=p, cmd=bench_cmd) + "`")
    for p in ("B", "C", "E"):
        lines.append(f"* copy pass {p}: `" + run.format(ctr=PMC_PASSES[p], kre="'copy|elementwise'", root=root,
                                                      p="copy_" + p, cmd="python bench.py --copy-calibration 1024")
                     + "`")
    lines += [f"* timings and order statistics: `python bench.py --config {workload} --steps 10 --warmup 2 "
              f"--no-cpu-baseline --no-gemm-reference --variants {','.join(variants)}`"]
    if command_note:
        lines += ["", f"Driver: {command_note}"]
    lines += ["",
              "Columns. call ms / TFLOP/s: the unprofiled run, median over steps each started after a 1 GiB cache "
              "flush; frac = TFLOP/s / 2500 (dense bf16 peak). kernel ms: the profiled dispatches. L2 hit % = "
              "TCC_HIT / (TCC_HIT + TCC_MISS). fabric rd GB = FETCH_SIZE x copy factor: what the eight L2s read "
              "from the fabric, i.e. from the 256 MiB last-level cache and HBM together. DRAM rd GB = pass E's "
              "read bytes (128/64/32-byte requests) x copy factor x TCC_EA0_RDREQ_DRAM / TCC_EA0_RDREQ: the reads "
              "addressed to DRAM, which still includes last-level-cache hits (this pool exposes no counter that "
              "separates them, so true HBM read bytes cannot be measured here). K/V xcd GB: compulsory K/V if each "
              "XCD fetches every block its own rows need once (per-XCD model, see bench.py). MFMA busy % = "
              "SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE / 8), against the clock the chip ran at "
              "(= GRBM_GUI_ACTIVE / 8 / kernel time). J: adjacent-row overlap of the executed order; Eq. 1: the "
              "paper's objective over chip-wide waves, relative to natural order (lower is better). L2 lat / "
              "fabric lat: cycles per L2 request from a CU / per fabric read in flight.", "",
              f"Copy calibration (1 GiB device copy): FETCH_SIZE x {f_fetch:.3f}, WRITE_SIZE x {f_write:.3f}, "
              f"pass E x {f_e:.3f}.", "",
              "| variant | call ms | TFLOP/s | frac | kernel ms | clock GHz | L2 hit % | fabric rd GB | DRAM rd GB | "
              "K/V xcd GB | write GB | MFMA busy % | J | Eq. 1 | L2 lat | fabric lat |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    nan = float("nan")
    for v in variants:
        a, b, c = passes["A"][v], passes["B"][v], passes["C"][v]
        e = passes.get("E", {}).get(v)
        dd = passes.get("D", {}).get(v, {})
        hit = a["TCC_HIT_sum"] / (a["TCC_HIT_sum"] + a["TCC_MISS_sum"])
        fetch = b["FETCH_SIZE"] * 1024.0 * f_fetch
        write = c["WRITE_SIZE"] * 1024.0 * f_write
        cycles = a["GRBM_GUI_ACTIVE"] / 8.0
        busy = a["SQ_VALU_MFMA_BUSY_CYCLES"] / (256 * 4 * cycles)
        clock = cycles / a["duration_ns"]
        dram = None
        if e:
            tot, share = _read_bytes_e(e)
            dram = tot * f_e * share
        bv = line["variants"].get(v, {})
        entry[v] = {"kernel_sha": sha, "variant_spec": VARIANTS.get(v), "hbm_bytes_per_launch": fetch + write,
                    "fetch_bytes": fetch, "write_bytes": write, "dram_read_bytes": dram, "l2_hit": hit,
                    "mfma_flop": a["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512, "mfma_busy": busy, "clock_ghz": clock,
                    "kernel_ms": a["duration_ns"] / 1e6}
        l2_lat = (f"{dd['TCP_TCC_READ_REQ_LATENCY_sum'] / dd['TCP_TCC_READ_REQ_sum']:.0f}"
                  if dd.get("TCP_TCC_READ_REQ_sum") else "-")
        fab_lat = f"{dd['TCC_EA0_RDREQ_LEVEL_sum'] / dd['TCC_EA0_RDREQ_sum']:.0f}" if dd.get("TCC_EA0_RDREQ_sum") else "-"
        o = ost.get(v, {})
        xb = xcd.get(v, {}).get("bytes")
        eq1 = o.get("eq1_vs_natural")
        tf = bv.get("tflops_attn", nan)
        lines.append(
            f"| {v} | {bv.get('attn_ms', nan):.3f} | {tf:.1f} | {tf / MFMA_BF16_PEAK_TFLOPS:.3f} | "
            f"{a['duration_ns'] / 1e6:.3f} | {clock:.3f} | {100 * hit:.2f} | {fetch / 1e9:.2f} | "
            f"{'-' if dram is None else f'{dram / 1e9:.2f}'} | {'-' if xb is None else f'{xb / 1e9:.2f}'} | "
            f"{write / 1e9:.3f} | {100 * busy:.1f} | {o.get('adj_jaccard', nan):.3f} | "
            f"{'-' if eq1 is None else f'{eq1:.3f}'} | {l2_lat} | {fab_lat} |")
    with open(out_json, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_trace(stats_csv: str, bench_json: str, out_md: str, command_note: str) -> None:
    """Turn a rocprofv3 --kernel-trace --stats kernel table (and the bench line of the same run) into a
    text summary: per-kernel calls and durations, and the attention kernel's average next to the
    duration bench.py measured with HIP events in the same run."""
    import csv
    rows = list(csv.DictReader(open(stats_csv)))
    with open(bench_json) as f:
        line = json.loads([ln for ln in f.read().splitlines() if ln.startswith("{")][-1])
    if line.get("mode") == "producer":
        return summarize_producer_trace(rows, line, out_md, command_note)
    lines = [f"# kernel trace: {line['config']['workload']}, variant {line['config']['variant']}", "",
             f"Command: `{command_note}`", "",
             "Kernels of the library (torch's fill and sum of the 1 GiB cache flush before every step are left "
             "out; the warm-up launches are included).", "",
             "| kernel | calls | average ms | min ms | max ms | share % |", "|---|---|---|---|---|---|"]
    attn_avg = None
    for r in rows:
        name = r["Name"]
        short = name.replace("(anonymous namespace)::", "").replace("void ", "").split("(")[0]
        avg = float(r["AverageNs"]) / 1e6
        if "attn_fwd_kernel" in name:
            attn_avg = avg
        if short.startswith("at::"):   # torch's own kernels: the cache flush between steps
            continue
        lines.append(f"| {short} | {r['Calls']} | {avg:.3f} | {float(r['MinNs']) / 1e6:.3f} | "
                     f"{float(r['MaxNs']) / 1e6:.3f} | {float(r['Percentage']):.2f} |")
    v = line["variants"][line["config"]["variant"]]
    lines += ["", f"bench.py (HIP events around the attention call, same run): {v['attn_ms']:.3f} ms per launch, "
              f"{v['tflops_attn']:.1f} TFLOP/s over {line['config']['flop_per_step']:.4g} FLOP; "
              f"step {v['ms_per_step']:.3f} ms."]
    if attn_avg:
        lines.append(f"rocprofv3 attention kernel average: {attn_avg:.3f} ms "
                     f"({line['config']['flop_per_step'] / (attn_avg * 1e-3) / 1e12:.1f} TFLOP/s).")
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_producer_trace(rows, line, out_md: str, command_note: str) -> None:
    """Kernel table of a `bench.py --producer` run: the producer's kernels against the HBM roofline
    of reading Q and K once and writing the mask, and the path on the produced mask."""
    lines = [f"# kernel trace: pooled-score top-k mask producer, {line['workload']}", "",
             f"Command: `{command_note}`", "",
             "| kernel | calls | average ms | min ms | max ms | share % |", "|---|---|---|---|---|---|"]
    prod_ms, launches = 0.0, 0
    calls = line.get("producer_calls") or 1
    for r in rows:
        short = r["Name"].replace("(anonymous namespace)::", "").replace("void ", "").split("(")[0]
        avg = float(r["AverageNs"]) / 1e6
        if "producer_kernel" in r["Name"] or "producer_init_kernel" in r["Name"]:  # two launches per call
            prod_ms += float(r["TotalDurationNs"]) / 1e6 / calls
            launches += int(r["Calls"])
        if short.startswith("at::") or "elementwise" in short or "reduce_kernel" in short:
            continue
        lines.append(f"| {short} | {r['Calls']} | {avg:.3f} | {float(r['MinNs']) / 1e6:.3f} | "
                     f"{float(r['MaxNs']) / 1e6:.3f} | {float(r['Percentage']):.2f} |")
    rf = line["producer_roofline"]
    lines += ["", f"keep {line['keep']} blocks per row + the diagonal (density {100 * line['density']:.2f}%).",
              f"bench.py (HIP events around wa_produce_block_mask, same run): {line['producer_ms']:.3f} ms; "
              f"{rf['achieved']:.0f} GB/s of {rf['algorithmic_bytes'] / 1e9:.2f} GB algorithmic bytes "
              f"(Q and K read once, mask written) = {100 * rf['frac']:.1f}% of 8 TB/s.",
              f"rocprofv3: the producer's {launches // calls} launches per call take {prod_ms:.3f} ms "
              f"per call ({calls} calls).", "",
              "Path on the produced mask (step = permutation if built + compaction + attention):", ""]
    for v, r in line["path"].items():
        extra = f", {r['identity_heads']} heads kept the identity order" if "identity_heads" in r else ""
        lines.append(f"* {v}: step {r['step_ms']:.2f} ms, attention {r['attn_ms']:.2f} ms, "
                     f"{r['tflops_step']:.1f} TFLOP/s{extra}")
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def cpu_baseline(wl, q, k, v, mask, total_flop, budget_s: float):
    """The oracle, as it stands, timed on a bounded sample of the workload on the host cores."""
    from oracle import attention as A
    from oracle import permutation as P
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        pools = threadpool_info()
        cores = max([p.get("num_threads", 1) for p in pools] or [1])
        libs = [f"{p.get('internal_api')} {p.get('version')} ({p.get('threading_layer', '?')} threads)"
                for p in pools if p.get("user_api") == "blas"]
        blas = "; ".join(libs) or blas
    except Exception:
        cores = os.cpu_count() or 1
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next(ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name"))
    except (OSError, StopIteration):
        pass
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
        "cpu_model": cpu_model,
        "host_threads": os.cpu_count(),
        "blas": blas,
        "kind": "oracle",
        "sample": (f"fp64 oracle attention on {blocks} random query blocks ({flop_done / 1e9:.1f} GFLOP, "
                   f"{t_attn:.1f} s) plus the permutation oracle on 1 of {wl.batch * wl.heads} heads "
                   f"({t_perm_head:.1f} s); step time extrapolated by FLOPs and head count "
                   f"(est. {est_step:.0f} s per step)"),
    }


# Row orders and queue layouts compared by the benchmark. n_xcd is the kernel's queue count and the
# permutation's segment count: 1 = one queue in slot order for the whole chip, waves of W = resident
# tasks per CU x CUs rows (Alg. 2 with the paper's W); 8 = one queue per XCD (segment x of every head
# runs on XCD x), waves of W / 8 rows per segment.
VARIANTS = {
    "reordered": dict(perm="two-stage", skip="never", n_xcd=1, wave_mult=8),
    "natural": dict(perm=None, n_xcd=1),
    "auto": dict(perm="two-stage", skip="auto", n_xcd=1, wave_mult=8),
    "s1-only": dict(perm="stage1", skip="never", n_xcd=1, wave_mult=8),
    "s2-only": dict(perm="s2-only", n_xcd=1, wave_mult=8),
    "random": dict(perm="random", n_xcd=1),
    "reordered-xcd": dict(perm="two-stage", skip="never", n_xcd=8),
    "natural-xcd": dict(perm=None, n_xcd=8),
    "natural-interleaved": dict(perm=None, n_xcd=1, head_order="interleaved"),
    "reordered-interleaved": dict(perm="two-stage", skip="never", n_xcd=1, wave_mult=8, head_order="interleaved"),
    "auto-vnatural": dict(perm="two-stage", skip="auto", n_xcd=1, wave_mult=8, v_layout="natural"),
}
VARIANT_HELP = {
    "reordered": "two-stage order (Stage 1 polar sort + Stage 2 bucket sort), chip-wide waves, one queue, "
                 "skip never",
    "natural": "identity order, one queue (plain slot order)",
    "auto": "as reordered, with the adaptive skip rule deciding per head",
    "s1-only": "Stage-1 order only (no bucket sort), one queue",
    "s2-only": "identity order with the Stage-2 bucket sort over chip-wide waves only (built on the host)",
    "random": "a seeded random order, one queue (built on the host)",
    "reordered-xcd": "two-stage order, work-balanced XCD segments, one queue per XCD, skip never",
    "natural-xcd": "identity order, equal row-count XCD segments, one queue per XCD",
    "natural-interleaved": "identity order, one queue, the heads' slots dealt round-robin (head-parallel)",
    "reordered-interleaved": "as reordered, the heads' slots dealt round-robin (head-parallel)",
    "auto-vnatural": "as auto, V passed in its natural [B][H][N][d] layout (transposed inside every call)",
}
# Every other variant passes V as V^T ([B][H][d][M_B*block], written once by transpose_v before the
# timed steps, the layout a value projection can emit directly) and runs the heads in order.


FLAG_NAMES = ((1, "fits_cache"), (2, "little_work"), (4, "local"), (8, "unstructured"), (16, "degenerate"))


def gemm_reference(attn_tflops: float, n: int = 16384, reps: int = 5) -> dict:
    """Context for the roofline fraction: the rate of a large dense bf16 GEMM from the vendor library
    (torch.matmul -> hipBLASLt) on the same GPU and clock conditions. Not part of the path."""
    import torch
    a = torch.randn((n, n), device="cuda", dtype=torch.bfloat16)
    b = torch.randn((n, n), device="cuda", dtype=torch.bfloat16)
    for _ in range(2):
        c = a @ b
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        c = a @ b
    e1.record()
    torch.cuda.synchronize()
    tflops = 2.0 * n ** 3 / (e0.elapsed_time(e1) / reps * 1e-3) / 1e12
    del a, b, c
    torch.cuda.empty_cache()
    log(f"library bf16 GEMM {n}^3: {tflops:.1f} TFLOP/s")
    return {"op": f"torch.matmul bf16 {n}x{n}x{n}", "tflops": tflops, "frac_of_peak": tflops / MFMA_BF16_PEAK_TFLOPS,
            "attention_vs_gemm": attn_tflops / tflops}


def _median(xs):
    return float(np.median(np.asarray(xs, dtype=np.float64)))


def run_skip_sweep(args) -> int:
    """Kernel-level latency with and without reordering (overhead included) over sequence length and
    density, each repetition starting from a flushed L2 and last-level cache, and the decision the
    adaptive skip rule takes at each point. One JSON line per point on stdout."""
    import torch
    import paper_2609_34814_amd as W
    from workloads import skip_sweep_workloads

    points = skip_sweep_workloads()
    if args.sweep_points:
        keep = [s.strip() for s in args.sweep_points.split(",") if s.strip()]
        points = [p for p in points if any(s in p.name for s in keep)]
    # 1 GiB, larger than the L2s and the last-level cache together, written then read before each
    # repetition (the read evicts the written lines, so no repetition pays for write-backs)
    flush = torch.zeros(1 << 28, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    for wl in points:
        t0 = time.perf_counter()
        mask = make_mask(wl, threads=16)
        b_, h_, mb, n, d, blk = wl.batch, wl.heads, wl.mb, wl.seq_len, wl.head_dim, wl.block
        nnz = int(mask.sum(dtype=np.int64))
        distinct = mask.any(axis=2).sum(axis=-1)
        kv_mib = float(distinct.mean()) * 2 * blk * d * 2 / 2 ** 20
        md = torch.from_numpy(mask).cuda()
        del mask
        gen = torch.Generator(device="cuda")
        gen.manual_seed(wl.seed)
        q, k, v = (torch.randn((b_, h_, n, d), generator=gen, device="cuda", dtype=torch.bfloat16) for _ in range(3))
        vt = W.transpose_v(v, block=blk)
        del v
        shape = W.shape_of(b_, h_, n, d, blk)
        perm_ws = torch.empty(W.perm_workspace_size(shape), dtype=torch.uint8, device="cuda")
        attn_ws = torch.empty(W.attn_vt_workspace_size(shape), dtype=torch.uint8, device="cuda")
        perm = torch.empty((b_, h_, mb), dtype=torch.int32, device="cuda")
        seg = torch.empty((b_, h_, 2), dtype=torch.int32, device="cuda")
        flags = torch.empty((b_, h_), dtype=torch.uint8, device="cuda")
        row_ptr = torch.empty((b_, h_, mb + 1), dtype=torch.int32, device="cuda")
        col_idx = torch.empty((b_ * h_ * mb * mb,), dtype=torch.int32, device="cuda")
        o = torch.empty_like(q)
        wave = W.wave_size(d, blk) * 8
        log(f"{wl.name}: N={n} M_B={mb} nnz={nnz} K/V per head {kv_mib:.1f} MiB "
            f"(inputs {time.perf_counter() - t0:.1f} s)")

        def step(variant, ev):
            ev[0].record(stream)
            p = sg = None
            if variant != "natural":
                W.build_permutation(md, seq_len=n, block=blk, head_dim=d, wave=wave, n_xcd=1,
                                    skip="never" if variant == "reordered" else "auto", workspace=perm_ws,
                                    out=perm, flags_out=flags, seg_out=seg)
                p, sg = perm, seg
            ev[1].record(stream)
            rp, ci = W.compact_mask(md, seq_len=n, block=blk, head_dim=d, row_ptr=row_ptr, col_idx=col_idx)
            ev[2].record(stream)
            W.sparse_attn_vt(q, k, vt, rp, ci, p, sg, block=blk, n_xcd=1, out=o, workspace=attn_ws)
            ev[3].record(stream)

        rec = {"point": wl.name, "frames": wl.grid[0], "seq_len": n, "mb": mb, "heads": h_,
               "kind": "mixed" if "mixed" in wl.name else "spatial",
               "rho": float(wl.name.rsplit("rho", 1)[1]), "density": nnz / (b_ * h_ * mb * mb), "nnz": nnz,
               "kv_mib_per_head": kv_mib, "reps": args.sweep_reps}
        for variant in ("natural", "reordered", "auto"):
            times = {"step": [], "perm": [], "compact": [], "attn": []}
            for r in range(1 + args.sweep_reps):
                flush.fill_(1.0)
                flush.sum()
                ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
                step(variant, ev)
                torch.cuda.synchronize()
                if r == 0:
                    continue  # warm-up
                times["step"].append(ev[0].elapsed_time(ev[3]))
                times["perm"].append(ev[0].elapsed_time(ev[1]))
                times["compact"].append(ev[1].elapsed_time(ev[2]))
                times["attn"].append(ev[2].elapsed_time(ev[3]))
            rec[variant] = {key: _median(val) for key, val in times.items()}
            if variant != "natural":
                f = flags.cpu().numpy().reshape(-1)
                rec[variant]["identity_heads"] = int(np.count_nonzero(f & 64))
                if variant == "reordered":
                    rec["cases"] = {name: int(np.count_nonzero(f & bit)) for bit, name in FLAG_NAMES}
        rec["gain_step"] = rec["natural"]["step"] / rec["reordered"]["step"]
        rec["gain_attn"] = rec["natural"]["attn"] / rec["reordered"]["attn"]
        rec["auto_vs_best"] = rec["auto"]["step"] / min(rec["natural"]["step"], rec["reordered"]["step"])
        log(f"  natural {rec['natural']['step']:.2f} ms, reordered {rec['reordered']['step']:.2f} ms "
            f"(perm {rec['reordered']['perm']:.2f}), auto {rec['auto']['step']:.2f} ms with "
            f"{rec['auto']['identity_heads']}/{h_} heads skipped; gain step {rec['gain_step']:.3f} "
            f"attention {rec['gain_attn']:.3f}")
        print(json.dumps(rec), flush=True)
        del md, q, k, vt, perm_ws, attn_ws, perm, seg, flags, row_ptr, col_idx, o
        torch.cuda.empty_cache()
    return 0


def run_producer(args) -> int:
    """The pooled-score top-k mask producer on the 363,600-token shape with positional Q/K: its time
    and HBM roofline, then the path (natural / reordered / auto) on the mask it produced."""
    import torch
    import paper_2609_34814_amd as W
    from workloads.gen import PRODUCER_CONFIGS

    wl = PRODUCER_CONFIGS["produced-long-720p-401f"]
    t0 = time.perf_counter()
    q, k, v = make_qkv(wl, threads=16)
    log(f"generated {wl.name} in {time.perf_counter() - t0:.1f} s")

    def dev(bits):
        return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()

    qd, kd, vd = dev(q), dev(k), dev(v)
    del q, k, v
    b_, h_, mb, n, d, blk = wl.batch, wl.heads, wl.mb, wl.seq_len, wl.head_dim, wl.block
    keep = round(args.producer_density * mb)
    shape = W.shape_of(b_, h_, n, d, blk)
    pws = torch.empty(W.mask_producer_workspace_size(shape), dtype=torch.uint8, device="cuda")
    md = torch.empty((b_, h_, mb, mb), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")   # as in the main benchmark
    times = []
    for r in range(args.warmup + args.steps):
        flush.fill_(1.0)
        flush.sum()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        W.produce_block_mask(qd, kd, block=blk, keep=keep, diagonal=True, out=md, workspace=pws)
        e1.record(stream)
        torch.cuda.synchronize()
        if r >= args.warmup:
            times.append(e0.elapsed_time(e1))
    prod_ms = _median(times)
    hbm_bytes = 2.0 * b_ * h_ * n * d * 2 + float(b_ * h_ * mb * mb)
    nnz = int(md.sum(dtype=torch.int64).item())
    log(f"producer: {prod_ms:.3f} ms, keep {keep} + diagonal, nnz {nnz} ({nnz / (b_ * h_ * mb * mb):.4f})")
    roof = {"bound": "hbm", "achieved": hbm_bytes / (prod_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": hbm_bytes / (prod_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": hbm_bytes}
    if args.producer_only:
        print(json.dumps({"mode": "producer", "workload": wl.name, "keep": keep, "diagonal": True,
                          "density": nnz / (b_ * h_ * mb * mb), "producer_ms": prod_ms,
                          "producer_calls": args.warmup + args.steps, "producer_roofline": roof, "path": {}}),
              flush=True)
        return 0

    perm_ws = torch.empty(W.perm_workspace_size(shape), dtype=torch.uint8, device="cuda")
    attn_ws = torch.empty(W.attn_vt_workspace_size(shape), dtype=torch.uint8, device="cuda")
    perm = torch.empty((b_, h_, mb), dtype=torch.int32, device="cuda")
    seg = torch.empty((b_, h_, 2), dtype=torch.int32, device="cuda")
    flags = torch.empty((b_, h_), dtype=torch.uint8, device="cuda")
    row_ptr = torch.empty((b_, h_, mb + 1), dtype=torch.int32, device="cuda")
    col_idx = torch.empty((b_ * h_ * mb * mb,), dtype=torch.int32, device="cuda")
    o = torch.empty_like(qd)
    vtd = W.transpose_v(vd, block=blk)
    del vd
    wave = W.wave_size(d, blk) * 8
    flop = 4.0 * blk * blk * d * nnz
    res = {}
    for variant in ("natural", "reordered", "auto"):
        st = []
        for r in range(args.warmup + args.steps):
            flush.fill_(1.0)
            flush.sum()
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            ev[0].record(stream)
            p = sg = None
            if variant != "natural":
                W.build_permutation(md, seq_len=n, block=blk, head_dim=d, wave=wave, n_xcd=1,
                                    skip="never" if variant == "reordered" else "auto", workspace=perm_ws,
                                    out=perm, flags_out=flags, seg_out=seg)
                p, sg = perm, seg
            rp, ci = W.compact_mask(md, seq_len=n, block=blk, head_dim=d, row_ptr=row_ptr, col_idx=col_idx)
            ev[1].record(stream)
            W.sparse_attn_vt(qd, kd, vtd, rp, ci, p, sg, block=blk, n_xcd=1, out=o, workspace=attn_ws)
            ev[2].record(stream)
            torch.cuda.synchronize()
            if r >= args.warmup:
                st.append((ev[0].elapsed_time(ev[2]), ev[1].elapsed_time(ev[2])))
        step_ms, attn_ms = (_median([x[i] for x in st]) for i in range(2))
        res[variant] = {"step_ms": step_ms, "attn_ms": attn_ms, "tflops_step": flop / (step_ms * 1e-3) / 1e12}
        if variant != "natural":
            res[variant]["identity_heads"] = int(((flags & 64) != 0).sum().item())
        log(f"{variant}: step {step_ms:.2f} ms, attention {attn_ms:.2f} ms")
    print(json.dumps({
        "mode": "producer", "workload": wl.name, "keep": keep, "diagonal": True, "density": nnz / (b_ * h_ * mb * mb),
        "producer_ms": prod_ms, "producer_calls": args.warmup + args.steps, "producer_roofline": roof,
        "path": res}), flush=True)
    return 0


def summarize_sweep(jsonl: str, out_md: str, command_note: str) -> None:
    recs = []
    with open(jsonl) as f:
        for ln in f:
            if ln.startswith("{"):
                recs.append(json.loads(ln))
    lines = ["# Adaptive skip sweep: kernel-level latency with and without reordering", "",
             "Each figure is the median over the repetitions of one step (permutation, when built, + mask",
             "compaction + attention call); every repetition starts after a 1 GiB read that evicts the L2s",
             "and the last-level cache. `gain` = natural / reordered (> 1: reordering pays).",
             "`skip cases` counts heads per case of the rule under the built-in profile (one head can",
             "hit several); `auto` runs with the rule deciding per head.", "",
             f"Command: `{command_note}`", "",
             "| point | tokens | density | K/V per head MiB | natural ms | reordered ms (perm) | gain step | "
             "gain attention | auto ms (heads skipped) | auto / best | skip cases |",
             "|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in recs:
        cases = ", ".join(f"{k} {v}" for k, v in r.get("cases", {}).items() if v)
        lines.append(f"| {r['point']} | {r['seq_len']} | {r['density'] * 100:.1f}% | {r['kv_mib_per_head']:.1f} | "
                     f"{r['natural']['step']:.2f} | {r['reordered']['step']:.2f} ({r['reordered']['perm']:.2f}) | "
                     f"{r['gain_step']:.3f} | {r['gain_attn']:.3f} | {r['auto']['step']:.2f} "
                     f"({r['auto']['identity_heads']}/{r['heads']}) | {r['auto_vs_best']:.3f} | {cases or '-'} |")
    # calibration of the skip rule's cost model (case 2): the permutation's time per head, amortised
    # over the heads that run concurrently, as a linear function of M_B (both forms multiply the whole
    # bit mask on the matrix cores, so the head's kept blocks do not enter), fitted separately for the
    # two forms that build it (one workgroup per head up to 1024 blocks, many workgroups per head
    # above); and the attention time saved per kept block by the reordered order
    lines += ["", "Overhead model fitted to the permutation times above (least squares, per head = step share / "
              "heads), one line per form that builds the permutation:"]
    for form, sel, cols in (("one workgroup per head (M_B <= 1024)", lambda r: r["mb"] <= 1024, 2),
                            ("sliced, many workgroups per head (M_B > 1024)", lambda r: r["mb"] > 1024, 2)):
        rs = [r for r in recs if sel(r)]
        if len(rs) < cols:
            continue
        xs = np.array([[1.0, r["mb"], r["nnz"] / r["heads"]][:cols] for r in rs])
        ys = np.array([r["reordered"]["perm"] * 1e6 / r["heads"] for r in rs])
        coef = np.linalg.lstsq(xs, ys, rcond=None)[0]
        rel = np.abs(xs @ coef - ys) / ys
        terms = f"fixed = {coef[0]:.0f} ns, per row = {coef[1]:.2f} ns" + (
            f", per kept block = {coef[2]:.4f} ns" if cols == 3 else "")
        lines.append(f"* {form}, {len(rs)} points: {terms} (largest relative residual {100 * rel.max():.1f}%).")
    lines += ["", "Attention time saved per kept block by the reordered order, ns (natural - reordered attention "
              "call over the kept blocks):", ""]
    lines.append(" | ".join(f"{r['point']}: {(r['natural']['attn'] - r['reordered']['attn']) * 1e6 / r['nnz']:+.3f}"
                            for r in recs))
    lines += ["", "Below about 50K tokens the whole step takes a few ms and the attention call runs faster after any "
              "permutation kernel, also when the order stays the identity (the auto column), so the savings "
              "there are not an effect of the order."]
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="long-720p-401f", choices=sorted(ALL_CONFIGS))
    ap.add_argument("--variants", default="auto,reordered,natural",
                    help="comma list of: " + "; ".join(f"{k}: {v}" for k, v in VARIANT_HELP.items()))
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-order-stats", action="store_true",
                    help="skip the host-side statistics of each executed order (per-XCD compulsory K/V bytes, "
                         "adjacent-row overlap, Eq. 1 objective)")
    ap.add_argument("--no-gemm-reference", action="store_true",
                    help="skip timing the vendor library's dense bf16 GEMM (context for the roofline fraction)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of this many MiB (3 times), to calibrate the HBM counters")
    ap.add_argument("--summarize-pmc", metavar="DIR", help="summarize rocprofv3 counter passes found in DIR "
                    "into profiles/attn_traffic.json and a markdown table (no GPU needed)")
    ap.add_argument("--pmc-command", default="", help="command line recorded in the counter summary")
    ap.add_argument("--pmc-bench-json", default="", help="bench line of the unprofiled run summarized with --summarize-pmc")
    ap.add_argument("--summarize-trace", nargs=2, metavar=("STATS_CSV", "BENCH_JSON"),
                    help="summarize a rocprofv3 --kernel-trace --stats run of bench.py into profiles/ (no GPU needed)")
    ap.add_argument("--trace-command", default="", help="command line recorded in the trace summary")
    ap.add_argument("--skip-sweep", action="store_true",
                    help="time natural / reordered / auto over the sequence-length and density sweep (JSON lines)")
    ap.add_argument("--sweep-points", default="", help="comma list of substrings selecting sweep points")
    ap.add_argument("--sweep-reps", type=int, default=5)
    ap.add_argument("--summarize-sweep", metavar="JSONL", help="write profiles/skip_sweep.md from a sweep's output")
    ap.add_argument("--producer", action="store_true",
                    help="time the pooled-score top-k mask producer and the path on its mask (JSON line)")
    ap.add_argument("--producer-density", type=float, default=0.05, help="kept blocks per row / M_B")
    ap.add_argument("--producer-only", action="store_true",
                    help="with --producer: time the producer alone, not the path on its mask")
    ap.add_argument("--sweep-command", default="", help="command line recorded in the sweep summary")
    args = ap.parse_args()

    if args.summarize_sweep:
        summarize_sweep(args.summarize_sweep, os.path.join(ROOT, "profiles", "skip_sweep.md"), args.sweep_command)
        return 0

    if args.summarize_trace:
        stats_csv, bench_json = args.summarize_trace
        with open(bench_json) as f:
            cfg = json.loads([ln for ln in f.read().splitlines() if ln.startswith("{")][-1]).get("config")
        if cfg is None:
            md = os.path.join(ROOT, "profiles", "mask_producer_produced-long-720p-401f_kernel_trace.md")
        else:
            md = os.path.join(ROOT, "profiles", f"attn_fwd_{cfg['workload']}_{cfg['variant']}_kernel_trace.md")
        summarize_trace(stats_csv, bench_json, md, args.trace_command)
        return 0
    if args.summarize_pmc:
        md = os.path.join(ROOT, "profiles", f"attn_fwd_{args.config}_counters.md")
        summarize_pmc(args.summarize_pmc, args.config, [x.strip() for x in args.variants.split(",") if x.strip()],
                      args.warmup, args.steps, args.pmc_bench_json, TRAFFIC_FILE, md, args.pmc_command)
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the path is a single-GPU kernel pipeline; across GPUs the "
              "heads would shard with no exchange, each GPU running this path on its share", file=sys.stderr)
        return 2

    import torch
    import paper_2609_34814_amd as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.skip_sweep:
        return run_skip_sweep(args)
    if args.producer:
        return run_producer(args)
    if args.copy_calibration:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 3}))
        return 0
    wl = ALL_CONFIGS[args.config]
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
    # compulsory bytes of one attention call: Q read and O written once, every distinct K/V block of a
    # head read once (the ragged last block at its true size), and the KV index lists
    blk_tokens = np.full(wl.mb, wl.block, dtype=np.int64)
    blk_tokens[-1] = wl.seq_len - (wl.mb - 1) * wl.block
    used = mask.any(axis=2)                              # [B][H][N_B]
    kv_bytes = int((used * blk_tokens).sum()) * wl.head_dim * 2 * 2
    qo_bytes = 2 * wl.batch * wl.heads * wl.seq_len * wl.head_dim * 2
    list_bytes = 4 * nnz
    algo_bytes = kv_bytes + qo_bytes + list_bytes
    b_, h_, mb = wl.batch, wl.heads, wl.mb
    shape = W.shape_of(b_, h_, wl.seq_len, wl.head_dim, wl.block)
    perm_ws = torch.empty(W.perm_workspace_size(shape), dtype=torch.uint8, device="cuda")
    perm = torch.empty((b_, h_, mb), dtype=torch.int32, device="cuda")
    row_ptr = torch.empty((b_, h_, mb + 1), dtype=torch.int32, device="cuda")
    col_idx = torch.empty((b_ * h_ * mb * mb,), dtype=torch.int32, device="cuda")
    o = torch.empty_like(qd)
    flags = torch.empty((b_, h_), dtype=torch.uint8, device="cuda")
    status = torch.zeros((1,), dtype=torch.int32, device="cuda")
    # V^T, as a value projection can emit it: written once here, an input of every timed step
    vtd = W.transpose_v(vd, block=wl.block)
    need_vnat = any(VARIANTS[x.strip()].get("v_layout") == "natural" for x in args.variants.split(",") if x.strip())
    attn_ws = torch.empty(W.attn_workspace_size(shape) if need_vnat else W.attn_vt_workspace_size(shape),
                          dtype=torch.uint8, device="cuda")
    wave = W.wave_size(wl.head_dim, wl.block)
    stream = torch.cuda.current_stream()
    # 1 GiB written, then read, before every timed step: more than the eight L2s and the shared
    # last-level cache hold, and the read evicts the written lines, so no step starts with cached
    # K/V or pays for another call's write-backs
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    log(f"uploaded; nnz={nnz} density={nnz / (b_ * h_ * mb * mb):.4f} wave_per_xcd={wave}")

    rng = np.random.default_rng(12345)
    row_nnz = mask.reshape(b_ * h_, mb, mb).sum(axis=2, dtype=np.int64)

    def host_perm(kind, n_seg, wave_rows):
        """Ablation orders built once on the host (not part of the timed step)."""
        out = np.empty((b_ * h_, mb), dtype=np.int32)
        for hh in range(b_ * h_):
            if kind == "random":
                out[hh] = rng.permutation(mb)
            else:  # s2-only: identity order, buckets of `wave_rows` rows per segment sorted by descending n_i
                base, extra = divmod(mb, n_seg)
                starts = [x * base + min(x, extra) for x in range(n_seg + 1)]
                order = []
                for x in range(n_seg):
                    for s0 in range(starts[x], starts[x + 1], wave_rows):
                        rows = np.arange(s0, min(s0 + wave_rows, starts[x + 1]))
                        order.extend(rows[np.argsort(-row_nnz[hh, rows], kind="stable")])
                out[hh] = order
        return torch.from_numpy(out).cuda().reshape(b_, h_, mb)

    def make_step(variant):
        spec = VARIANTS[variant]
        n_xcd = spec["n_xcd"]
        head_order = spec.get("head_order", "in-order")
        v_natural = spec.get("v_layout") == "natural"
        fixed = (host_perm(spec["perm"], n_xcd, wave * spec.get("wave_mult", 1))
                 if spec["perm"] in ("random", "s2-only") else None)
        s1 = torch.empty((b_, h_, mb), dtype=torch.int32, device="cuda") if spec["perm"] == "stage1" else None
        seg_q = torch.empty((b_, h_, n_xcd + 1), dtype=torch.int32, device="cuda")
        used_perm = {}

        def step(ev=None):
            p, sg = fixed, None
            if ev is not None:
                ev[2].record(stream)
            if spec["perm"] in ("two-stage", "stage1"):
                W.build_permutation(md, seq_len=wl.seq_len, block=wl.block, head_dim=wl.head_dim,
                                    wave=wave * spec.get("wave_mult", 1), n_xcd=n_xcd, skip=spec["skip"],
                                    workspace=perm_ws, out=perm, flags_out=flags, seg_out=seg_q,
                                    stage1_out=s1)
                p = s1 if s1 is not None else perm
                sg = seg_q
            if ev is not None:
                ev[3].record(stream)
            rp, ci = W.compact_mask(md, seq_len=wl.seq_len, block=wl.block, head_dim=wl.head_dim,
                                    row_ptr=row_ptr, col_idx=col_idx)
            if ev is not None:
                ev[0].record(stream)
            if v_natural:
                W.sparse_attn_csr(qd, kd, vd, rp, ci, p, sg, block=wl.block, n_xcd=n_xcd, out=o, workspace=attn_ws,
                                  status=status)
            else:
                W.sparse_attn_vt(qd, kd, vtd, rp, ci, p, sg, block=wl.block, n_xcd=n_xcd, head_order=head_order,
                                 out=o, workspace=attn_ws, status=status)
            if ev is not None:
                ev[1].record(stream)
            used_perm["perm"], used_perm["seg"] = p, sg
        step.used = used_perm
        return step

    def order_stats(variant, used_perm):
        """Host-side statistics of the order a variant executed (rows in slot order, per head):
        * per-XCD compulsory K/V bytes: every distinct block the rows of one XCD reference, fetched once
          per XCD; with one queue per XCD (n_xcd = 8) the rows of segment x run on XCD x, with one queue
          the slots go round-robin over the 8 XCDs (slot t on XCD t mod 8, the order in which the first
          workgroups start). Over the global compulsory bytes: the duplication across the private L2s;
        * adjacent-row overlap J = sum |M_s & M_s+1| / sum |M_s | M_s+1| over consecutive slots;
        * the Eq. 1 objective: over consecutive waves of W = resident workgroups of the chip rows, the
          summed squared distance of every ordered pair of rows of a wave."""
        spec = VARIANTS[variant]
        p, sg = used_perm.get("perm"), used_perm.get("seg")
        ph = p.cpu().numpy().reshape(b_ * h_, mb) if p is not None else None
        sgh = sg.cpu().numpy().reshape(b_ * h_, -1) if sg is not None else None
        total = 0
        adj_and = adj_or = 0
        eq1 = 0
        w_chip = wave * 8
        mk = mask.reshape(b_ * h_, mb, mb)
        for hh in range(b_ * h_):
            order = ph[hh] if ph is not None else np.arange(mb)
            rows_h = mk[hh][order].astype(bool)
            adj_and += int((rows_h[1:] & rows_h[:-1]).sum())
            adj_or += int((rows_h[1:] | rows_h[:-1]).sum())
            for s0 in range(0, mb, w_chip):
                wv = rows_h[s0:s0 + w_chip]
                col = wv.sum(axis=0, dtype=np.int64)
                eq1 += 2 * wv.shape[0] * int(col.sum()) - 2 * int((col * col).sum())
            for x in range(8):
                if spec["n_xcd"] == 8:
                    if sgh is not None:
                        rows = order[sgh[hh, x]:sgh[hh, x + 1]]
                    else:
                        base, extra = divmod(mb, 8)
                        a0 = x * base + min(x, extra)
                        rows = order[a0:a0 + base + (1 if x < extra else 0)]
                else:
                    rows = order[x::8]
                if rows.size:
                    total += int((mk[hh, rows].any(axis=0) * blk_tokens).sum())
        return {"kv_compulsory_xcd_bytes": total * wl.head_dim * 2 * 2,
                "adj_jaccard": adj_and / adj_or if adj_or else 0.0, "eq1_objective": eq1, "eq1_wave": w_chip}

    results = {}
    xcd_bytes = {}
    for variant in [s.strip() for s in args.variants.split(",") if s.strip()]:
        step = make_step(variant)
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        # per step: [0] attention start, [1] attention end, [2] step start, [3] permutation end
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for i in range(args.steps):
            flush.fill_(1.0)
            flush.sum()
            step(evs[i])
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        steps_ms = [e[2].elapsed_time(e[1]) for e in evs]
        attn = [e[0].elapsed_time(e[1]) for e in evs]
        ms_step = _median(steps_ms)
        attn_ms = _median(attn)
        perm_ms = _median([e[2].elapsed_time(e[3]) for e in evs])
        compact_ms = _median([e[3].elapsed_time(e[0]) for e in evs])
        st = int(status.item())
        if st != 0:
            raise RuntimeError(f"{variant}: the attention call reported status {st}")
        results[variant] = dict(ms_per_step=ms_step, wall_ms_per_step=wall * 1e3 / args.steps, attn_ms=attn_ms,
                                attn_ms_min=float(min(attn)), attn_ms_max=float(max(attn)),
                                perm_ms=perm_ms, compact_ms=compact_ms,
                                tflops_step=flop / (ms_step * 1e-3) / 1e12,
                                tflops_attn=flop / (attn_ms * 1e-3) / 1e12)
        if VARIANTS[variant]["perm"] in ("two-stage", "stage1"):
            f = flags.cpu().numpy().reshape(-1)
            results[variant]["identity_heads"] = int(np.count_nonzero(f & 64))
        if not args.no_order_stats:
            xcd_bytes[variant] = order_stats(variant, step.used)
        log(f"{variant}: step {ms_step:.2f} ms, attention call {attn_ms:.2f} ms "
            f"({results[variant]['tflops_attn']:.1f} TFLOP/s)")

    head = next((v for v in ("auto", "reordered") if v in results), next(iter(results)))
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
    # LDS, the kernel's on-chip operand path. Per kept block each of the block/32 wavefronts reads the
    # whole K tile and V^T tile from LDS (its MFMA operands) and the global->LDS copies write both tiles
    # once: (block/32 + 1) x 2 tiles of block x d bf16. gfx950 serves 128-bit LDS reads at 256 B/clk/CU
    # (225 measured with two wavefronts per SIMD, this kernel's occupancy), so at the 2.4 GHz peak clock
    # 256 x 256 x 2.4e9 B/s. The MFMA work of a kept block takes 4 block^2 d / (2500e12 / 256 / 2.4e9
    # FLOP/clk/CU) cycles; LDS would cap MFMA use only if a block's LDS cycles exceeded those.
    lds_bytes_block = (wl.block // 32 + 1) * 2 * wl.block * wl.head_dim * 2
    lds_b_per_clk = 256.0
    lds_peak = 256 * lds_b_per_clk * 2.4e9
    lds_achieved = lds_bytes_block * nnz / (r["attn_ms"] * 1e-3)
    mfma_cycles = 4.0 * wl.block * wl.block * wl.head_dim / (MFMA_BF16_PEAK_TFLOPS * 1e12 / 256 / 2.4e9)
    lds_cycles = lds_bytes_block / lds_b_per_clk
    lds_roof = {"bytes_per_kept_block": lds_bytes_block, "achieved_TBps": lds_achieved / 1e12,
                "peak_TBps": lds_peak / 1e12, "frac": lds_achieved / lds_peak,
                "lds_cycles_per_mfma_cycle": lds_cycles / mfma_cycles,
                "mfma_cap": min(1.0, mfma_cycles / lds_cycles), "binding": lds_cycles > mfma_cycles,
                "kind": "derived from the kernel's tile traffic, not a counter"}
    # Where the bf16 fraction goes: the clock the chip held under the kernel (power-limited) times the
    # share of those cycles the MFMA pipes were busy, both from the committed counter summary.
    cnt = load_counters(wl.name, head)
    clock_split = None
    if cnt and cnt.get("clock_ghz") and cnt.get("mfma_busy") is not None:
        clock_split = {"clock_ghz": cnt["clock_ghz"], "clock_share_of_2.4GHz": cnt["clock_ghz"] / 2.4,
                       "mfma_busy": cnt["mfma_busy"],
                       "frac_at_that_clock": roof["frac"] * 2.4 / cnt["clock_ghz"],
                       "source": cnt["source"]}
    out = {
        "metric": "sparse-attn effective TFLOP/s (skip rule + reordering + attention, overhead included)",
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
                   "flop_per_step": flop, "variant": head, "wave_per_xcd": wave, "v_input": "transposed",
                   "timing": "median over steps, each after a 1 GiB write + read cache flush"},
        "roofline": roof,
        "lds_roofline": lds_roof,
        "clock_split": clock_split,
        "algorithmic_bytes": {"kv_compulsory": kv_bytes, "q_and_o": qo_bytes, "kv_lists": list_bytes,
                              "total": algo_bytes, "flop_per_byte": flop / algo_bytes},
        "variants": results,
    }
    if xcd_bytes:
        out["algorithmic_bytes"]["kv_compulsory_per_xcd"] = {
            v: {"bytes": st["kv_compulsory_xcd_bytes"], "vs_global": st["kv_compulsory_xcd_bytes"] / kv_bytes}
            for v, st in xcd_bytes.items()}
        nat = xcd_bytes.get("natural")
        out["order_stats"] = {
            v: {"adj_jaccard": st["adj_jaccard"], "eq1_objective": st["eq1_objective"], "eq1_wave": st["eq1_wave"],
                "eq1_vs_natural": st["eq1_objective"] / nat["eq1_objective"] if nat and nat["eq1_objective"] else None}
            for v, st in xcd_bytes.items()}
    if "natural" in results:
        out["speedup_vs_natural"] = {
            v: {"step": results["natural"]["ms_per_step"] / rv["ms_per_step"],
                "attention_kernel": results["natural"]["attn_ms"] / rv["attn_ms"]}
            for v, rv in results.items() if v != "natural"}
    counters = {v: c for v in results if (c := load_counters(wl.name, v)) is not None}
    if counters:
        out["counters"] = counters
    if not args.no_gemm_reference:
        out["library_gemm_reference"] = gemm_reference(r["tflops_attn"])
    if not args.no_cpu_baseline:
        log("timing the oracle on the host")
        out["cpu_baseline"] = cpu_baseline(wl, q, k, v, mask, flop, args.cpu_budget)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
