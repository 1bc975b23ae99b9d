"""Seeded synthetic workloads (inputs only; no arithmetic of the method)."""
from .gen import (ALL_CONFIGS, CONFIGS, CONFIG_ORDER, EXTRA_CONFIGS, Workload, custom, make_mask, make_mask_head, make_qkv,
                  make_tensor, bf16_bits_to_f32, block_centres, with_seed, skip_sweep_workloads, sweep_workload,
                  STREAM_Q, STREAM_K, STREAM_V)

__all__ = ["ALL_CONFIGS", "CONFIGS", "CONFIG_ORDER", "EXTRA_CONFIGS", "Workload", "custom", "make_mask", "make_mask_head", "make_qkv",
           "make_tensor", "bf16_bits_to_f32", "block_centres", "with_seed", "skip_sweep_workloads", "sweep_workload", "STREAM_Q", "STREAM_K", "STREAM_V"]
