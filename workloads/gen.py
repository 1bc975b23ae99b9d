"""Seeded synthetic inputs for the block-sparse attention path.

This module only draws inputs: bf16 Q/K/V tensors and binary block masks. It
contains none of the method's arithmetic and is shared by the CPU oracle, the
GPU tests and the benchmark.

Shapes follow the paper's long-video setting (Sec. VI-A): tokens are the raster
order (frame, y, x) of a video latent grid, blocks are runs of consecutive
tokens (Sec. II-B), 128-token blocks for the large models and 64-token blocks
for the small backend configuration. Real Q/K/V captured from video DiTs are
not available; N(0,1) tensors and masks with local spatio-temporal structure
plus scattered "global" blocks and heavy-tailed row counts stand in for them
(Sec. III-C describes dispersed K/V accesses and uneven per-row block counts;
Sec. VI-F shows diagonal-dominated masks; Table I uses a random-mask floor).

Random streams: every array is drawn from its own NumPy ``SeedSequence``
``[seed, stream, flat_head]`` so any head can be regenerated alone.
Stream ids: 0 Q, 1 K, 2 V, 3 mask row counts / Bernoulli draws, 4 global
columns, 5 tie-break hashes, 6 positional features.

Workloads whose masks are to be produced from Q and K (the pooled-score mask
producer) add a positional component to Q and K: per head, random Fourier
features of the token's (frame, y, x) position, so that the expected product of
two tokens' features is a Gaussian kernel of their distance. "spatial" heads
decay with distance in time and space, "temporal" heads ignore the frame index,
so that tokens at the same in-frame position match across all frames.
"""
from __future__ import annotations

import math
import statistics
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace
from typing import Optional, Sequence

import numpy as np

STREAM_Q, STREAM_K, STREAM_V, STREAM_COUNT, STREAM_GLOBAL, STREAM_TIE, STREAM_POS = 0, 1, 2, 3, 4, 5, 6


# --------------------------------------------------------------------------------------
# bf16 N(0,1) codes
# --------------------------------------------------------------------------------------
def _f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp64 -> fp32 (round to nearest even) -> bf16 bits (round to nearest even)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def _normal_table() -> np.ndarray:
    """bf16 bits of the standard normal quantile at (k + 1/2) / 65536, k = 0..65535."""
    nd = statistics.NormalDist()
    q = np.array([nd.inv_cdf((k + 0.5) / 65536.0) for k in range(65536)], dtype=np.float64)
    return _f64_to_bf16_bits(q)


_TABLE: Optional[np.ndarray] = None


def normal_table() -> np.ndarray:
    global _TABLE
    if _TABLE is None:
        _TABLE = _normal_table()
    return _TABLE


def bf16_normal(seed: int, stream: int, flat_head: int, count: int) -> np.ndarray:
    """``count`` bf16 bit patterns distributed as N(0,1) (inverse CDF of 16-bit uniform codes)."""
    ss = np.random.SeedSequence([seed, stream, flat_head])
    codes = np.random.Generator(np.random.Philox(ss)).integers(0, 65536, size=count, dtype=np.uint16)
    return np.take(normal_table(), codes)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------------------
# workload description
# --------------------------------------------------------------------------------------
@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    heads: int
    head_dim: int
    block: int
    grid: tuple  # (frames, height, width) in latent tokens; seq_len = product
    seed: int
    # mask recipe, one entry per head group: list of (first_head, last_head_exclusive, rule dict)
    mask_rules: tuple = field(default_factory=tuple)
    seq_len_override: Optional[int] = None
    # positional component of Q and K, one entry per head group: (first, last_exclusive, rule dict)
    qk_rules: tuple = field(default_factory=tuple)

    @property
    def seq_len(self) -> int:
        if self.seq_len_override is not None:
            return self.seq_len_override
        f, h, w = self.grid
        return f * h * w

    @property
    def mb(self) -> int:
        return -(-self.seq_len // self.block)

    @property
    def frame_tokens(self) -> int:
        return self.grid[1] * self.grid[2]

    def shape(self):
        return (self.batch, self.heads, self.seq_len, self.head_dim, self.block)


def _rules(*groups):
    return tuple((a, b, tuple(sorted(r.items()))) for a, b, r in groups)


# The five configurations of the path (name, shapes and mask recipe).
CONFIGS = {
    "tiny": Workload("tiny", 1, 2, 64, 64, (4, 32, 32), 1001,
                     _rules((0, 2, dict(kind="radius", rt=1, rs=2, g=4)))),
    "wan1.3b-480p-81f": Workload("wan1.3b-480p-81f", 1, 12, 128, 128, (21, 30, 52), 1002,
                                 _rules((0, 12, dict(kind="radius", rt=2, rs=3, g=8)))),
    "wan14b-720p-81f": Workload("wan14b-720p-81f", 1, 40, 128, 128, (21, 45, 80), 1003,
                                _rules((0, 40, dict(kind="count", rho_lo=0.05, rho_hi=0.25, sigma=0.8, g=8)))),
    "long-720p-401f": Workload("long-720p-401f", 1, 40, 128, 128, (101, 45, 80), 1004,
                               _rules((0, 40, dict(kind="count", rho_lo=0.05, rho_hi=0.05, sigma=0.8, g=8)))),
    "skip-d64": Workload("skip-d64", 1, 32, 64, 128, (31, 32, 48), 1005,
                         _rules((0, 16, dict(kind="bernoulli", p=0.20)),
                                (16, 32, dict(kind="count_fixed", frac=0.15, g=0)))),
}
CONFIG_ORDER = ["tiny", "wan1.3b-480p-81f", "wan14b-720p-81f", "long-720p-401f", "skip-d64"]

# An additional workload with the shapes of the 401-frame one: half of the heads are "spatial"
# (the count rule above), half are "temporal", keeping the blocks at (about) the same in-frame
# position in every frame plus scattered globals. Temporal heads are where raster order puts rows
# that share no K/V block next to each other (Sec. III-C, root cause 1).
EXTRA_CONFIGS = {
    "long-720p-401f-mixed": Workload("long-720p-401f-mixed", 1, 40, 128, 128, (101, 45, 80), 1006,
                                     _rules((0, 20, dict(kind="count", rho_lo=0.05, rho_hi=0.05, sigma=0.8, g=8)),
                                            (20, 40, dict(kind="radius", rt=101, rs=0.5, g=8)))),
}
# Workloads for the pooled-score mask producer: Q and K carry the positional component above
# (heads 0..H/2-1 spatial, the rest temporal); their masks are produced from Q and K, so
# mask_rules is empty. The large one has the shapes of the 401-frame workload.
_SPATIAL_QK = dict(amp=3.0, lt=2.0, ly=6.0, lx=40.0)
_TEMPORAL_QK = dict(amp=3.0, lt=math.inf, ly=4.0, lx=30.0)
PRODUCER_CONFIGS = {
    "produced-tiny": Workload("produced-tiny", 1, 2, 64, 64, (4, 32, 32), 1101,
                              qk_rules=_rules((0, 1, _SPATIAL_QK), (1, 2, _TEMPORAL_QK))),
    "produced-ragged": Workload("produced-ragged", 2, 2, 128, 128, (5, 30, 52), 1102,
                                qk_rules=_rules((0, 1, _SPATIAL_QK), (1, 2, _TEMPORAL_QK))),
    "produced-long-720p-401f": Workload("produced-long-720p-401f", 1, 40, 128, 128, (101, 45, 80), 1103,
                                        qk_rules=_rules((0, 20, _SPATIAL_QK), (20, 40, _TEMPORAL_QK))),
}
ALL_CONFIGS = {**CONFIGS, **EXTRA_CONFIGS}


def sweep_workload(frames: int, rho: float, kind: str, seed: int) -> Workload:
    """One point of the skip-rule sweep: the 720p latent grid (45 x 80 tokens a frame) over ``frames``
    frames, 40 heads, d = 128, 128-token blocks. ``kind`` "spatial": every head takes the count rule
    at density ``rho``; "mixed": heads 20-39 take the temporal rule of the mixed workload instead."""
    spatial = dict(kind="count", rho_lo=rho, rho_hi=rho, sigma=0.8, g=8)
    if kind == "spatial":
        groups = ((0, 40, spatial),)
    elif kind == "mixed":
        groups = ((0, 20, spatial), (20, 40, dict(kind="radius", rt=frames, rs=0.5, g=8)))
    else:
        raise ValueError(kind)
    return Workload(f"sweep-{frames}f-{kind}-rho{rho:g}", 1, 40, 128, 128, (frames, 45, 80), seed, _rules(*groups))


def skip_sweep_workloads():
    """The sweep of the adaptive skip (Sec. VI-F): sequence length from 25,200 to 522,000 tokens
    (7 to 145 latent frames; 145 frames are 4,079 blocks, just under the 4,096-block limit) at 5%
    density, spatial and mixed heads; then density 1.7% to 25% at 363,600 tokens."""
    out = []
    for frames in (7, 14, 27, 55, 101, 145):
        for kind in ("spatial", "mixed"):
            out.append(sweep_workload(frames, 0.05, kind, 3000 + len(out)))
    for rho in (0.017, 0.067, 0.145, 0.25):
        out.append(sweep_workload(101, rho, "spatial", 3000 + len(out)))
    return out


def custom(name: str, *, batch=1, heads=2, head_dim=64, block=64, grid=(2, 16, 16), seed=7,
           rule=None, seq_len=None) -> Workload:
    """A small workload for tests; ``rule`` is one mask-rule dict applied to every head."""
    if rule is None:
        rule = dict(kind="radius", rt=1, rs=1, g=2)
    return Workload(name, batch, heads, head_dim, block, tuple(grid), seed,
                    _rules((0, heads, rule)), seq_len_override=seq_len)


# --------------------------------------------------------------------------------------
# tensors
# --------------------------------------------------------------------------------------
def qk_rule_for_head(wl: Workload, h: int) -> Optional[dict]:
    for a, b, r in wl.qk_rules:
        if a <= h < b:
            return dict(r)
    return None


def positional_features(wl: Workload, flat_head: int, rule: dict) -> np.ndarray:
    """float64 [N][d]: sqrt(2/d) cos(w_c . p_t + phi_c) with p_t = (frame, y, x) of token t,
    w_c ~ N(0, diag(1/lt^2, 1/ly^2, 1/lx^2)) (lt = inf: no time dependence), phi_c ~ U[0, 2 pi)."""
    n, d = wl.seq_len, wl.head_dim
    f_, hh, ww = wl.grid
    rng = _rng(wl, STREAM_POS, flat_head)
    g = rng.standard_normal((3, d))
    inv_l = np.array([0.0 if math.isinf(rule["lt"]) else 1.0 / rule["lt"], 1.0 / rule["ly"], 1.0 / rule["lx"]])
    w = g * inv_l[:, None]
    phi = rng.uniform(0.0, 2.0 * math.pi, size=d)
    t = np.arange(n, dtype=np.int64)
    pos = np.stack([t // (hh * ww), (t // ww) % hh, t % ww], axis=1).astype(np.float64)
    # the phase written out element by element (a BLAS product here gave wrong values when the
    # generator ran in several threads at once, so the inputs were not reproducible)
    arg = pos[:, 0:1] * w[0] + pos[:, 1:2] * w[1] + pos[:, 2:3] * w[2] + phi
    return math.sqrt(2.0 / d) * np.cos(arg)


def make_tensor(wl: Workload, stream: int, heads: Optional[Sequence[int]] = None,
                threads: int = 8) -> np.ndarray:
    """bf16 bit patterns, shape [B][H][N][d] (or [len(heads)] flat heads if ``heads`` given)."""
    n, d = wl.seq_len, wl.head_dim
    flat = list(range(wl.batch * wl.heads)) if heads is None else list(heads)
    out = np.empty((len(flat), n, d), dtype=np.uint16)

    def one(k):
        bits = bf16_normal(wl.seed, stream, flat[k], n * d).reshape(n, d)
        rule = qk_rule_for_head(wl, flat[k] % wl.heads) if stream in (STREAM_Q, STREAM_K) else None
        if rule is not None:
            x = bf16_bits_to_f32(bits).astype(np.float64) + rule["amp"] * positional_features(wl, flat[k], rule)
            bits = _f64_to_bf16_bits(x)
        out[k] = bits

    if len(flat) > 1 and threads > 1:
        with ThreadPoolExecutor(min(threads, len(flat))) as ex:
            list(ex.map(one, range(len(flat))))
    else:
        for k in range(len(flat)):
            one(k)
    if heads is None:
        return out.reshape(wl.batch, wl.heads, n, d)
    return out


def make_qkv(wl: Workload, threads: int = 8):
    return tuple(make_tensor(wl, s, threads=threads) for s in (STREAM_Q, STREAM_K, STREAM_V))


# --------------------------------------------------------------------------------------
# masks
# --------------------------------------------------------------------------------------
def block_centres(wl: Workload):
    """Frame index t_j and in-frame raster position p_j of each block's centre token."""
    n, blk, hw = wl.seq_len, wl.block, wl.frame_tokens
    start = np.arange(wl.mb, dtype=np.int64) * blk
    end = np.minimum(start + blk, n)
    c = (start + end - 1) // 2
    return c // hw, c % hw


def _rng(wl: Workload, stream: int, flat_head: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([wl.seed, stream, flat_head])))


def _add_globals(keep: np.ndarray, g: int, rng: np.random.Generator) -> None:
    """Add ``g`` distinct random columns per row, drawn among the columns not yet kept."""
    if g <= 0:
        return
    m, n = keep.shape
    keys = rng.integers(0, np.iinfo(np.int64).max, size=(m, n), dtype=np.int64)
    keys[keep] = np.iinfo(np.int64).max
    gg = min(g, n)
    pick = np.argpartition(keys, gg - 1, axis=1)[:, :gg]
    rows = np.repeat(np.arange(m), gg)
    sel = pick.reshape(-1)
    ok = keys[rows, sel] != np.iinfo(np.int64).max
    keep[rows[ok], sel[ok]] = True


def _radius_head(wl, t, p, rule, fh):
    keep = (np.abs(t[:, None] - t[None, :]) <= rule["rt"]) & \
           (np.abs(p[:, None] - p[None, :]) <= rule["rs"] * wl.block)
    _add_globals(keep, rule["g"], _rng(wl, STREAM_GLOBAL, fh))
    return keep


def _count_keep(wl, t, p, n_rows, g, fh):
    """Keep the ``n_i - g`` nearest blocks (block distance D, seeded tie-break) plus ``g`` globals."""
    m = wl.mb
    dt = np.abs(t[:, None] - t[None, :])
    dp = -(-np.abs(p[:, None] - p[None, :]) // wl.block)
    dist = np.maximum(dt, dp).astype(np.int64)
    tie = _rng(wl, STREAM_TIE, fh).integers(0, 1 << 32, size=(m, m), dtype=np.int64)
    key = (dist << 32) | tie
    srt = np.sort(key, axis=1)
    near = np.clip(n_rows - g, 1, m)
    thr = srt[np.arange(m), near - 1]
    keep = key <= thr[:, None]
    _add_globals(keep, g, _rng(wl, STREAM_GLOBAL, fh))
    return keep


def _count_head(wl, t, p, rule, fh):
    m, g = wl.mb, rule["g"]
    rng = _rng(wl, STREAM_COUNT, fh)
    rho = rng.uniform(rule["rho_lo"], rule["rho_hi"]) if rule["rho_hi"] > rule["rho_lo"] else rule["rho_lo"]
    lengths = rng.lognormal(0.0, rule["sigma"], size=m)
    n_rows = np.rint(rho * m * lengths / lengths.mean()).astype(np.int64)
    n_rows = np.clip(n_rows, g + 1, m)
    return _count_keep(wl, t, p, n_rows, g, fh)


def _count_fixed_head(wl, t, p, rule, fh):
    m, g = wl.mb, rule["g"]
    n_rows = np.full(m, int(np.rint(rule["frac"] * m)), dtype=np.int64)
    n_rows = np.clip(n_rows, g + 1, m)
    return _count_keep(wl, t, p, n_rows, g, fh)


def _bernoulli_head(wl, t, p, rule, fh):
    m = wl.mb
    keep = _rng(wl, STREAM_COUNT, fh).random((m, m)) < rule["p"]
    empty = ~keep.any(axis=1)
    keep[np.nonzero(empty)[0], np.nonzero(empty)[0]] = True
    return keep


def _ones_head(wl, t, p, rule, fh):
    return np.ones((wl.mb, wl.mb), dtype=bool)


def _diag_head(wl, t, p, rule, fh):
    return np.eye(wl.mb, dtype=bool)


def _empty_rows_head(wl, t, p, rule, fh):
    """Bernoulli(p) mask where a seeded fraction of rows is left empty (edge case)."""
    m = wl.mb
    rng = _rng(wl, STREAM_COUNT, fh)
    keep = rng.random((m, m)) < rule.get("p", 0.3)
    drop = rng.random(m) < rule.get("empty", 0.25)
    keep[drop] = False
    return keep


_RULES = {
    "radius": _radius_head,
    "count": _count_head,
    "count_fixed": _count_fixed_head,
    "bernoulli": _bernoulli_head,
    "ones": _ones_head,
    "diag": _diag_head,
    "empty_rows": _empty_rows_head,
}


def rule_for_head(wl: Workload, h: int) -> dict:
    for a, b, r in wl.mask_rules:
        if a <= h < b:
            return dict(r)
    raise ValueError(f"no mask rule covers head {h} of {wl.name}")


def make_mask_head(wl: Workload, b: int, h: int) -> np.ndarray:
    t, p = block_centres(wl)
    rule = rule_for_head(wl, h)
    keep = _RULES[rule["kind"]](wl, t, p, rule, b * wl.heads + h)
    return keep.astype(np.uint8)


def make_mask(wl: Workload, threads: int = 8) -> np.ndarray:
    """Block mask, uint8 [B][H][M_B][N_B], 1 = the query block attends to the KV block."""
    m = wl.mb
    out = np.empty((wl.batch, wl.heads, m, m), dtype=np.uint8)
    jobs = [(b, h) for b in range(wl.batch) for h in range(wl.heads)]

    def one(bh):
        b, h = bh
        out[b, h] = make_mask_head(wl, b, h)

    if threads > 1 and len(jobs) > 1:
        with ThreadPoolExecutor(min(threads, len(jobs))) as ex:
            list(ex.map(one, jobs))
    else:
        for j in jobs:
            one(j)
    return out


def with_seed(wl: Workload, seed: int) -> Workload:
    return replace(wl, seed=seed)
