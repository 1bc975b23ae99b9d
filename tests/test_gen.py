"""The seeded input generator: determinism, distributions and mask recipes."""
import numpy as np
import pytest

from workloads import CONFIGS, custom, make_mask, make_mask_head, make_tensor, bf16_bits_to_f32, block_centres
from workloads import gen as G


def test_normal_table_is_symmetric_monotone_standard():
    t = bf16_bits_to_f32(G.normal_table()).astype(np.float64)
    assert np.all(np.diff(t) >= 0)
    assert np.array_equal(t, -t[::-1])
    assert abs(t.mean()) < 1e-12
    assert abs(t.var() - 1.0) < 2e-3


def test_tensor_determinism_and_head_independence():
    wl = custom("t", heads=3, head_dim=64, block=64, grid=(1, 8, 16))
    a = make_tensor(wl, 0)
    b = make_tensor(wl, 0)
    assert np.array_equal(a, b)
    one = make_tensor(wl, 0, heads=[2])
    assert np.array_equal(one[0], a[0, 2])
    assert not np.array_equal(make_tensor(wl, 1), a)
    x = bf16_bits_to_f32(a).astype(np.float64)
    assert abs(x.mean()) < 0.02 and abs(x.std() - 1) < 0.02


def test_positional_tensors_same_in_threads():
    """Q with a positional component, generated one head at a time and by four threads at once, is the
    same bit for bit. (The generator once took the phase from a BLAS product, which returned wrong
    values now and then when several threads called it at once at the 363,600-token size.)"""
    wl = G.Workload("pos", 1, 4, 128, 128, (12, 45, 80), 1103,
                    qk_rules=G._rules((0, 2, G._SPATIAL_QK), (2, 4, G._TEMPORAL_QK)))
    a = make_tensor(wl, G.STREAM_Q, threads=1)
    b = make_tensor(wl, G.STREAM_Q, threads=4)
    assert np.array_equal(a, b)


def test_block_centres_ragged_last_block():
    wl = CONFIGS["wan1.3b-480p-81f"]
    t, p = block_centres(wl)
    assert wl.mb == 256 and wl.seq_len - 255 * 128 == 120
    c_last = (255 * 128 + wl.seq_len - 1) // 2
    assert t[-1] == c_last // (30 * 52) and p[-1] == c_last % (30 * 52)


@pytest.mark.parametrize("name,lo,hi", [("tiny", 0.24, 0.245), ("wan1.3b-480p-81f", 0.13, 0.133)])
def test_radius_rule_density(name, lo, hi):
    wl = CONFIGS[name]
    m = make_mask(wl)
    assert lo < m.mean() < hi
    # the radius neighbourhood always includes the diagonal
    assert np.all(np.diagonal(m, axis1=2, axis2=3) == 1)


def test_count_rule_rows():
    wl = CONFIGS["wan14b-720p-81f"]
    for h in (0, 7):
        m = make_mask_head(wl, 0, h)
        n = m.sum(1)
        assert n.min() >= 9
        assert np.all(np.diagonal(m) == 1)
    dens = [make_mask_head(wl, 0, h).mean() for h in range(40)]
    assert 0.04 < min(dens) and max(dens) < 0.27


def test_skip_config_halves():
    wl = CONFIGS["skip-d64"]
    r = make_mask_head(wl, 0, 3)
    assert abs(r.mean() - 0.20) < 0.01
    s = make_mask_head(wl, 0, 20)
    assert np.all(s.sum(1) == 56)


def test_mask_determinism_per_head():
    wl = CONFIGS["wan14b-720p-81f"]
    full = make_mask(wl)
    assert np.array_equal(full[0, 5], make_mask_head(wl, 0, 5))
