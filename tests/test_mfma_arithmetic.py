"""Host checks of the integer identities the matrix-core permutation kernels rely on.

The kernels multiply the 0/1 mask by the balanced base-256 digits of X (and of Ys) with int8
MFMAs and recombine the int32 products exactly in int64; the mask's bits become the MFMA's bytes
through one 24-bit multiply per nibble. These tests check the identities on the CPU, with the
same integer steps written in numpy.
"""
import numpy as np


def balanced_digits(v: np.ndarray) -> np.ndarray:
    """Four digits d_b in [-128, 127] with v = sum_b d_b 256^b: d_0 is the low byte read as a signed
    byte, then v <- (v - d_0) / 256 exactly, and so on."""
    v = v.astype(np.int64)
    out = []
    for _ in range(4):
        d = ((v & 0xFF) ^ 0x80) - 0x80        # the low byte as a signed byte
        out.append(d)
        assert np.all((v - d) % 256 == 0)
        v = (v - d) >> 8
    return np.stack(out, axis=-1)


def test_balanced_digits_reconstruct_every_value_in_range():
    # |v| <= 2^31 - 2^25: the lower digits add at most 128 (1 + 256 + 65536) to the last one; X and Ys
    # never exceed 2^30 + 1
    rng = np.random.default_rng(0)
    lim = (1 << 31) - (1 << 25)
    edge = np.arange(lim - 100000, lim + 1)
    v = np.concatenate([rng.integers(-lim, lim + 1, 200000), edge, -edge,
                        np.array([0, 1, -1, 127, 128, -128, -129, 255, 256, 1 << 30, -(1 << 30), (1 << 30) + 1])])
    d = balanced_digits(v)
    assert d.min() >= -128 and d.max() <= 127
    back = d[..., 0] + 256 * d[..., 1] + 65536 * d[..., 2] + 16777216 * d[..., 3]
    assert np.array_equal(back, v)
    # further out the last digit can leave [-128, 127]: 2^31 - 128 (1 + 256 + 65536) has lower digits
    # -128, -128, -128 and would need a last digit of 128
    over = np.array([(1 << 31) - 128 * (1 + 256 + 65536)])
    d = balanced_digits(over)
    assert d[0, 0] + 256 * d[0, 1] + 65536 * d[0, 2] + 16777216 * d[0, 3] != over[0]


def test_digit_products_are_exact_in_int32():
    # a column sum over at most 4096 rows of 0/1 x int8 stays far inside int32, and the int64
    # recombination of the four digit products equals the direct product
    rng = np.random.default_rng(1)
    m = 4096
    mask = (rng.random((m, 64)) < 0.3).astype(np.int64)
    x = rng.integers(-(1 << 30), 1 << 30, m)
    d = balanced_digits(x)
    parts = mask.T @ d                                     # [64 columns][4 digits]
    assert np.abs(parts).max() <= m * 128 < (1 << 31)
    combined = parts[:, 0] + 256 * parts[:, 1] + 65536 * parts[:, 2] + 16777216 * parts[:, 3]
    assert np.array_equal(combined, mask.T @ x)


def test_nibble_spread_expands_bits_to_bytes():
    b = np.arange(1 << 16, dtype=np.uint64)
    words = [(((b >> np.uint64(4 * k)) & np.uint64(0xF)) * np.uint64(0x204081)) & np.uint64(0x01010101)
             for k in range(4)]
    for t in range(16):
        byte = (words[t // 4] >> np.uint64(8 * (t % 4))) & np.uint64(0xFF)
        assert np.array_equal(byte, (b >> np.uint64(t)) & np.uint64(1)), t


def test_bit_block_swap_transposes_a_64x64_tile():
    # the recursive block swap of the mask transpose, one lane per row: at distance s a lane trades
    # its columns with bit s set for the partner's columns with bit s clear
    rng = np.random.default_rng(2)
    rows = [int(x) for x in rng.integers(0, 1 << 62, 64)]
    low = {32: 0x00000000FFFFFFFF, 16: 0x0000FFFF0000FFFF, 8: 0x00FF00FF00FF00FF, 4: 0x0F0F0F0F0F0F0F0F,
           2: 0x3333333333333333, 1: 0x5555555555555555}
    full = (1 << 64) - 1
    v = list(rows)
    for s in (32, 16, 8, 4, 2, 1):
        lo = low[s]
        t = [v[lane ^ s] for lane in range(64)]
        v = [((v[i] & ~lo & full) | ((t[i] >> s) & lo)) if i & s else ((v[i] & lo) | (((t[i] & lo) << s) & full))
             for i in range(64)]
    for r in range(64):
        for c in range(64):
            assert (v[c] >> r) & 1 == (rows[r] >> c) & 1
