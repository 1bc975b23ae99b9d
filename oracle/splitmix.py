"""SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014), used as a counter-based generator: ``splitmix64(x)``
is the first output of a SplitMix64 generator whose state is x, i.e. the state
is advanced by the golden-ratio increment and passed through the published
64-bit finaliser. Test infrastructure only.
"""
MASK64 = (1 << 64) - 1
GOLDEN_GAMMA = 0x9E3779B97F4A7C15


def splitmix64(x: int) -> int:
    z = (x + GOLDEN_GAMMA) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def splitmix64_stream(seed: int, count: int):
    """The first ``count`` outputs of a SplitMix64 generator seeded with ``seed``."""
    out = []
    state = seed & MASK64
    for _ in range(count):
        out.append(splitmix64(state))
        state = (state + GOLDEN_GAMMA) & MASK64
    return out
