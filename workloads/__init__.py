"""Seeded synthetic MoE inputs shared by the oracle tests and the GPU path."""
from .generate import (CONFIGS, CONFIG_TITLES, SWEEP_SKEW, SWEEP_T, Workload,
                       config, custom, explicit, f32_to_bf16_bits,
                       layer_inputs, make_workload, sweep_workload, sweep_workloads,
                       target_counts, zipf_targets)
