"""CPU oracle for the block-sparse attention path with cache-aware query-row reordering.

TEST INFRASTRUCTURE ONLY. Nothing in the product path (the HIP library and its
Python binding) may import, call, link or execute anything in this package.
Only the test suite, the smoke check and the benchmark's CPU-baseline leg use it.

The oracle is deliberately plain and slow: NumPy and Python integers, fp64 for
floating point (float32 where a step is defined by float32 roundings), no
blocking or fusion beyond what the paper's definitions state.
It shares no code with the GPU path.

Modules
  attention    fp64 masked softmax attention over a block mask (Sec. II-B, II-C)
  compaction   per-row KV-block index lists (the mask-selected inner loop, Sec. II-C)
  splitmix     SplitMix64, the counter-based generator that seeds the subspace iteration
  permutation  integer-exact reading of Alg. 1 (MFCSI) and Alg. 2 (two-stage reordering)
  skip         mask statistics and the adaptive reordering skip (Sec. IV-E)
  objective    the intra-wave distance objective of Eq. 1 (diagnostic)
  mask_producer  pooled-score top-k block mask from Q and K (a content-dependent producer of the
               mask the path consumes, Sec. II-B; float32 where the method rounds, fixed order)
"""
