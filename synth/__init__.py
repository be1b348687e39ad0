"""Seeded synthetic workloads shared by the oracle side and the GPU side.

Holds random draws and data layout only, never the method's arithmetic.
"""
from .workloads import (CONFIGS, SEED_BASE, LoopWorkload, StepInputs, add_near_ties,  # noqa: F401
                        bf16_bits_to_f32, config_seed, f32_to_bf16_bits, make_config,
                        make_loop_workload, make_step, uniform_offsets)
