"""Reference query-row permutation: an integer-exact reading of Alg. 1 and Alg. 2.

TEST INFRASTRUCTURE ONLY. The GPU permutation must reproduce this bit for bit.

What the paper fixes (Sec. IV-B .. IV-E):
  * Stage 1 (Sec. IV-C, Alg. 1, Eq. 2-4): embed each mask row i by the top-2 left
    singular vectors (u1[i], u2[i]) of the column-centred mask
    M~ = (I - 11^T/m) M, obtained by matrix-free centred subspace iteration
    (MFCSI): starting from a random orthonormal m x 2 block X, repeat T times
    Y = M^T X - c (1^T X)/m,  Z = M Y - 1 (c^T Y)/m,  X = Q of qr(Z),
    with c = M^T 1; then (Rayleigh-Ritz) B = X^T Z, (L, R) = eig(B), X = X R.
    Rows are sorted by the polar angle atan2(u2[i], u1[i]) (Eq. 4).
  * Stage 2 (Sec. IV-D, Alg. 2): cut the Stage-1 order into consecutive buckets
    of at most W rows (one execution wave each) and sort every bucket by
    descending row count n_i = sum_j M[i, j].

What the paper leaves open, and the reading taken here (each one is needed so
that two independent implementations agree exactly):
  R1 precision: X, Y, Z are fixed-point integers. X carries 2^30 per unit. The
     products M^T X and M Y and every sum are exact int64; the centring terms
     are applied exactly by scaling with m: Ym = m*M^T X - c*(1^T X) equals
     m * M~^T X with no rounding, Zm = m*M Ys - 1*(c^T Ys) equals m * M~ Ys.
     Ym is shifted right (floor) to 30 significant bits before the second
     product; scalar factors do not matter to a subspace iteration.
  R2 random start: Z0[i, k] = (splitmix64(seed + 2*(flat_head*m + i) + k) >> 40) - 2^23,
     then X = orth(Z0).
  R3 QR: Cholesky-QR of the 2 x 2 Gram matrix (R with non-negative diagonal),
     the Gram entries summed exactly over inputs shifted to 24 bits, then fp64
     with one IEEE rounding per operation (no fused multiply-add). The second
     column is dropped (set to 0) when its residual u = G22 - r12^2 is not above
     G22 * 2^-30 (numerically rank one).
  R4 Rayleigh-Ritz is always applied (Alg. 1 calls it optional) so that the basis
     is canonical: the symmetric 2 x 2 eigenproblem is solved by one Jacobi
     rotation (Golub & Van Loan, sym.schur2) and the column with the larger
     eigenvalue becomes u1.
  R5 sign: each column is negated if its entry of largest magnitude (smallest
     row index on ties) is negative. The angular order is only invariant to
     rotations and reflections cyclically, so a fixed sign and basis are needed.
  R6 angle sort: atan2 on (-pi, pi] is replaced by an exact comparator on the
     integer points (half-plane class, then the sign of the 2-D cross product);
     equal angles (and the origin, angle 0) keep ascending row index.
  R7 degenerate heads (the centred mask has no direction at all, e.g. all rows
     equal): Stage 1 returns the identity order.
  R8 waves: the Stage-1 order is first split into n_xcd contiguous segments, one
     per group of compute units that shares a private L2 (an XCD), balanced by
     work: with w_i = n_i + 1 (one block-time of fixed cost per row) and W_p the
     sum of w over the first p positions of the order, position p belongs to
     segment min(n_xcd - 1, floor(n_xcd * W_p / W_m)). Each segment is cut into
     buckets of W rows from its start (the last bucket may be shorter); Stage 2
     sorts each bucket by descending n_i, stably (ties keep Stage-1 order).
     n_xcd = 1 is Alg. 2 as printed.
  R9 T = 10 iterations by default (the paper uses 5-15).

Bounds: all int64 intermediates stay below 2^61 for m, n <= 4096.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional

import numpy as np

from .splitmix import splitmix64

X_BITS = 30          # fixed-point scale of X and U: 2^30 per unit
GRAM_BITS = 24       # inputs to Gram sums are shifted to this many bits
Y_BITS = 30          # Ym is shifted to this many bits before the second product
RR_X_SHIFT = 6       # X >> 6 (24 bits) in the Rayleigh-Ritz sums
MAX_BLOCKS = 4096    # bound under which every int64 intermediate is exact


def _bl(x: int) -> int:
    return abs(int(x)).bit_length()


def _max_abs(a: np.ndarray) -> int:
    return int(np.abs(a).max()) if a.size else 0


def _exact_int_matmul(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Exact integer product of a 0/1 matrix and an int64 matrix.

    Every partial sum is an integer below 2^53 (asserted), so an fp64 product
    is exact whatever order the library sums in.
    """
    bound = a.shape[1] * max(_max_abs(b), 1)
    assert bound < (1 << 53), "integer product would not be exact in fp64"
    return (a.astype(np.float64) @ b.astype(np.float64)).astype(np.int64)


# ---------------------------------------------------------------------------------------
# R2: random start
# ---------------------------------------------------------------------------------------
def random_start(m: int, seed: int, flat_head: int) -> np.ndarray:
    z = np.empty((m, 2), dtype=np.int64)
    for i in range(m):
        for k in range(2):
            ctr = (seed + 2 * (flat_head * m + i) + k) & ((1 << 64) - 1)
            z[i, k] = (splitmix64(ctr) >> 40) - (1 << 23)
    return z


# ---------------------------------------------------------------------------------------
# R3: orthonormalisation (QR of an m x 2 block)
# ---------------------------------------------------------------------------------------
def orth(z: np.ndarray):
    """Q factor of z (m x 2 int64) in 2^30 fixed point. Returns (X, degenerate)."""
    s = max(0, _bl(_max_abs(z)) - GRAM_BITS)
    zs = z >> s
    z0, z1 = zs[:, 0], zs[:, 1]
    g11 = int(np.dot(z0, z0))
    g12 = int(np.dot(z0, z1))
    g22 = int(np.dot(z1, z1))
    assert max(g11, g22, abs(g12)) < (1 << 62)
    x = np.zeros_like(z)
    if g11 == 0:
        return x, True
    G11, G12, G22 = float(g11), float(g12), float(g22)
    r11 = math.sqrt(G11)
    r12 = G12 / r11
    u = G22 - r12 * r12
    q0 = z0.astype(np.float64) / r11
    x[:, 0] = np.rint(q0 * float(1 << X_BITS)).astype(np.int64)
    if u > G22 * 2.0 ** -30:
        r22 = math.sqrt(u)
        q1 = (z1.astype(np.float64) - r12 * q0) / r22
        x[:, 1] = np.rint(q1 * float(1 << X_BITS)).astype(np.int64)
    assert _max_abs(x) < (1 << 31)
    return x, False


# ---------------------------------------------------------------------------------------
# R1: the centred products  m*M~^T X  and  m*M~ Ys
# ---------------------------------------------------------------------------------------
def centred_apply(mask: np.ndarray, col_counts: np.ndarray, x: np.ndarray):
    """Returns (Zm, sy): Zm = m * M~ (Ym >> sy) with Ym = m * M~^T X, both exact."""
    m = mask.shape[0]
    c = col_counts.astype(np.int64)
    ya = _exact_int_matmul(mask.T, x)                      # M^T X
    sx = x.sum(axis=0)                                      # 1^T X
    ym = m * ya - c[:, None] * sx[None, :]                  # m * M~^T X
    assert _max_abs(ym) < (1 << 61)
    sy = max(0, _bl(_max_abs(ym)) - Y_BITS)
    ys = ym >> sy
    za = _exact_int_matmul(mask, ys)                        # M Ys
    syy = c @ ys                                            # c^T Ys
    zm = m * za - syy[None, :]                              # m * M~ Ys
    assert _max_abs(zm) < (1 << 61)
    return zm, sy


# ---------------------------------------------------------------------------------------
# R4: Rayleigh-Ritz with one Jacobi rotation
# ---------------------------------------------------------------------------------------
@dataclass
class RitzResult:
    u: np.ndarray        # m x 2 int64, 2^30 fixed point, column 0 = larger eigenvalue
    trace: int           # b00 + b11 (exact integer)
    scale_exp: int       # trace * 2^scale_exp / m^2 = trace of X^T M~ M~^T X
    lam: tuple           # fp64 eigenvalue estimates in the same scaled units (diagnostic)


def rayleigh_ritz(mask, col_counts, x) -> RitzResult:
    zm, sy = centred_apply(mask, col_counts, x)
    s_r = max(0, _bl(_max_abs(zm)) - GRAM_BITS)
    xs = x >> RR_X_SHIFT
    zs = zm >> s_r
    b00 = int(np.dot(xs[:, 0], zs[:, 0]))
    b01 = int(np.dot(xs[:, 0], zs[:, 1]))
    b10 = int(np.dot(xs[:, 1], zs[:, 0]))
    b11 = int(np.dot(xs[:, 1], zs[:, 1]))
    a = float(b00)
    c = float(b11)
    b = float((b01 + b10) >> 1)
    if b == 0.0:
        t, cs, sn = 0.0, 1.0, 0.0
    else:
        tau = (c - a) / (2.0 * b)
        sgn = 1.0 if tau >= 0.0 else -1.0
        t = sgn / (abs(tau) + math.sqrt(1.0 + tau * tau))
        cs = 1.0 / math.sqrt(1.0 + t * t)
        sn = t * cs
    lam0 = a - t * b
    lam1 = c + t * b
    x0 = x[:, 0].astype(np.float64)
    x1 = x[:, 1].astype(np.float64)
    u0 = np.rint(cs * x0 - sn * x1).astype(np.int64)
    u1 = np.rint(sn * x0 + cs * x1).astype(np.int64)
    if lam1 > lam0:
        u0, u1 = u1, u0
        lam0, lam1 = lam1, lam0
    # X has 2^30 per unit and is read as X >> 6; Zm carries m^2 * 2^-sy * 2^30 * 2^-s_r.
    scale_exp = sy + s_r + RR_X_SHIFT - 2 * X_BITS
    return RitzResult(np.stack([u0, u1], axis=1), b00 + b11, scale_exp, (lam0, lam1))


# ---------------------------------------------------------------------------------------
# R5: canonical sign
# ---------------------------------------------------------------------------------------
def canonical_sign(u: np.ndarray) -> np.ndarray:
    u = u.copy()
    for k in range(2):
        col = u[:, k]
        if col.size == 0:
            continue
        i_star = int(np.argmax(np.abs(col)))   # first index of the maximum
        if col[i_star] < 0:
            u[:, k] = -col
    return u


# ---------------------------------------------------------------------------------------
# R6: exact polar-angle order
# ---------------------------------------------------------------------------------------
def angle_class(x: int, y: int) -> int:
    """0: angle in (-pi, 0); 1: angle 0 (incl. origin); 2: (0, pi); 3: angle pi."""
    if y < 0:
        return 0
    if y == 0:
        return 1 if x >= 0 else 3
    return 2


def angle_precedes(p, q) -> bool:
    """True if point p = (x, y, idx) comes before q in ascending atan2 order (ties by index)."""
    cp, cq = angle_class(p[0], p[1]), angle_class(q[0], q[1])
    if cp != cq:
        return cp < cq
    if cp in (0, 2):
        cross = p[0] * q[1] - p[1] * q[0]
        if cross != 0:
            return cross > 0
    return p[2] < q[2]


def angle_order(u: np.ndarray) -> np.ndarray:
    """Row indices sorted by ascending polar angle of (u[:,0], u[:,1]) (Eq. 4), exact."""
    import functools

    pts = [(int(u[i, 0]), int(u[i, 1]), i) for i in range(u.shape[0])]

    def cmp(p, q):
        if p[2] == q[2]:
            return 0
        return -1 if angle_precedes(p, q) else 1

    pts.sort(key=functools.cmp_to_key(cmp))
    return np.array([p[2] for p in pts], dtype=np.int32)


# ---------------------------------------------------------------------------------------
# Stage 1 driver
# ---------------------------------------------------------------------------------------
@dataclass
class Stage1Result:
    order: np.ndarray          # Stage-1 row order (int32 [m])
    embedding: np.ndarray      # canonical (u1, u2) in 2^30 fixed point, int64 [m][2]
    degenerate: bool
    trace: int                 # Rayleigh-Ritz trace (exact integer), 0 if degenerate
    scale_exp: int


def mfcsi_embedding(mask: np.ndarray, seed: int, flat_head: int, iters: int = 10):
    """Alg. 1 under readings R1-R5. Returns (U, degenerate, RitzResult or None)."""
    mask = (np.asarray(mask) != 0).astype(np.uint8)
    m, n = mask.shape
    assert m <= MAX_BLOCKS and n <= MAX_BLOCKS
    c = mask.sum(axis=0).astype(np.int64)
    x, degen = orth(random_start(m, seed, flat_head))
    for _ in range(iters):
        if degen:
            break
        zm, _ = centred_apply(mask, c, x)
        x, degen = orth(zm)
    if degen:
        return np.zeros((m, 2), dtype=np.int64), True, None
    rr = rayleigh_ritz(mask, c, x)
    return canonical_sign(rr.u), False, rr


def stage1(mask: np.ndarray, seed: int, flat_head: int, iters: int = 10) -> Stage1Result:
    m = mask.shape[0]
    u, degen, rr = mfcsi_embedding(mask, seed, flat_head, iters)
    if degen:
        return Stage1Result(np.arange(m, dtype=np.int32), u, True, 0, 0)
    return Stage1Result(angle_order(u), u, False, rr.trace, rr.scale_exp)


# ---------------------------------------------------------------------------------------
# R8: XCD segments, wave buckets and Stage 2
# ---------------------------------------------------------------------------------------
def segment_bounds(m: int, n_xcd: int):
    """[start, end) of n_xcd contiguous segments of m slots with equal row counts
    (the first m mod n_xcd get one more row): the slot layout of an unscheduled launch."""
    base, extra = divmod(m, n_xcd)
    bounds, s = [], 0
    for x in range(n_xcd):
        ln = base + (1 if x < extra else 0)
        bounds.append((s, s + ln))
        s += ln
    return bounds


def work_segments(order: np.ndarray, row_nnz: np.ndarray, n_xcd: int):
    """seg_start[0..n_xcd]: work-balanced contiguous segments of the order (reading R8)."""
    m = order.size
    w = [int(row_nnz[int(r)]) + 1 for r in order]
    total = sum(w)
    seg_of = []
    prefix = 0
    for p in range(m):
        seg_of.append(min(n_xcd - 1, (n_xcd * prefix) // total))
        prefix += w[p]
    starts = []
    for x in range(n_xcd):
        starts.append(next((p for p in range(m) if seg_of[p] >= x), m))
    return starts + [m]


def stage2(order: np.ndarray, row_nnz: np.ndarray, n_xcd: int, wave: int, seg_start=None) -> np.ndarray:
    """Descending-n_i stable sort inside every wave bucket of every segment (Alg. 2)."""
    m = order.size
    perm = np.empty(m, dtype=np.int32)
    if seg_start is None:
        seg_start = work_segments(order, row_nnz, n_xcd)
    for s0, s1 in zip(seg_start[:-1], seg_start[1:]):
        for b0 in range(s0, s1, wave):
            b1 = min(b0 + wave, s1)
            bucket = [int(r) for r in order[b0:b1]]
            bucket_sorted = sorted(bucket, key=lambda r: -int(row_nnz[r]))  # Python sort is stable
            perm[b0:b1] = bucket_sorted
    return perm


def two_stage_permutation(mask: np.ndarray, *, seed: int, flat_head: int, wave: int,
                          n_xcd: int = 8, iters: int = 10):
    """perm[s] = original row executed at slot s (Alg. 2 with readings R1-R9)."""
    s1 = stage1(mask, seed, flat_head, iters)
    nnz = (np.asarray(mask) != 0).sum(axis=1)
    return stage2(s1.order, nnz, n_xcd, wave), s1


def two_stage_schedule(mask: np.ndarray, *, seed: int, flat_head: int, wave: int, n_xcd: int = 8, iters: int = 10):
    """(perm, seg_start, Stage-1 result): the permutation and its work-balanced XCD segments."""
    s1 = stage1(mask, seed, flat_head, iters)
    nnz = (np.asarray(mask) != 0).sum(axis=1)
    seg = work_segments(s1.order, nnz, n_xcd)
    return stage2(s1.order, nnz, n_xcd, wave, seg), seg, s1


def identity_permutation(m: int) -> np.ndarray:
    return np.arange(m, dtype=np.int32)
