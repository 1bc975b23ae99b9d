"""Writes tests/golden/perm_small.txt from the oracle alone (inputs from the seeded generator).

Run:  python -m tests.golden.make_golden
The stored permutations guard the oracle against unnoticed changes; they are not
the paper's values (the paper prints none).
"""
import os

import numpy as np

from oracle import reorder as R
from oracle import skip as S
from workloads import CONFIGS, custom, make_mask


def golden_cases():
    return [
        ("tiny_h0_never_w16", ("tiny", 0, 16, 8, S.SKIP_NEVER)),
        ("tiny_h1_never_w64_x1", ("tiny", 1, 64, 1, S.SKIP_NEVER)),
        ("wan13b_h5_never_w64", ("wan1.3b-480p-81f", 5, 64, 8, S.SKIP_NEVER)),
        ("rand_h0_auto_w8", ("rand-small", 0, 8, 8, S.SKIP_AUTO)),
    ]


def _mask(name):
    if name == "rand-small":
        wl = custom("rand-small", heads=1, head_dim=64, block=64, grid=(3, 8, 16),
                    rule=dict(kind="bernoulli", p=0.25), seed=5)
    else:
        wl = CONFIGS[name]
    return wl, make_mask(wl)


# The skip rule's constants are fixed here so that the stored flags do not move when the
# built-in profile is recalibrated.
PROFILE = S.SkipProfile(cache_bytes=4.0 * 1024 * 1024, gain_ns_per_block=1.0, ovh_ns_fixed=2000.0,
                        ovh_ns_per_row=2.0, ovh_ns_per_nnz=0.05, j_max=0.75, eta_min=0.05)


def compute_case(name, head, wave, n_xcd, mode):
    wl, mask = _mask(name)
    perm, flags, _ = R.build_permutation(mask[:, head:head + 1], block=wl.block, head_dim=wl.head_dim,
                                         wave=wave, n_xcd=n_xcd, iters=10, seed=head * 0 + 0,
                                         skip_mode=mode, profile=PROFILE)
    return [int(v) for v in perm[0, 0]] + [int(flags[0, 0])]


def main():
    path = os.path.join(os.path.dirname(__file__), "perm_small.txt")
    with open(path, "w") as f:
        f.write("# key perm... flags  (written by tests/golden/make_golden.py from oracle/ only)\n")
        for key, args in golden_cases():
            f.write(key + " " + " ".join(str(v) for v in compute_case(*args)) + "\n")


if __name__ == "__main__":
    main()
