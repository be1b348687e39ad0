"""Seeded synthetic workloads shared by the oracle side and the GPU side.

Holds random draws and data layout only, never the method's arithmetic.
"""
from .workloads import (LOOP, NEARTIE, SEED_BASE, SMALL, V60K, V90K, WORKLOADS,  # noqa: F401
                        LoopWorkload, StepInputs, add_near_ties, bf16_bits_to_f32, f32_to_bf16_bits,
                        make_eos_workload, make_loop_workload, make_step, make_workload, uniform_offsets,
                        workload_index, workload_seed, EosWorkload)
