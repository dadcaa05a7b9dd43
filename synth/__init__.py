"""Seeded synthetic inputs for the true-tail update (shared by the oracle tests,
the GPU parity tests and the benchmark).

This package holds workload construction only: shapes, random draws and the
record (removal-range) sampling. It contains none of the method's arithmetic
(no RoPE, no attention, no recurrence, no compaction), so that the CPU oracle
and the HIP path can both consume its outputs without sharing code.
"""
from .workloads import (  # noqa: F401
    AttnShape,
    DeltaShape,
    Config,
    CONFIGS,
    T_SWEEP,
    t_sweep_config,
    sub_rng,
    to_bf16_bits,
    bf16_bits_to_f32,
    gen_attn_cache,
    gen_attn_tail,
    gen_delta_state,
    gen_delta_inputs,
    gen_conv_inputs,
    draw_records,
    subtract_ranges,
    append_interval,
    initial_intervals,
    Scenario,
    Round,
    CharacterPlan,
    make_scenario,
    Revision,
    PaperTrace,
    make_paper_trace,
)
