"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

Holds no attention arithmetic; see ``workloads.generate``.
"""
from .generate import (  # noqa: F401
    group_starts, grouped_case, stage_units, batch_from_tables,
    GENERATOR_PROMPT, FIXER_PROMPT, FIRST_ATTEMPT,
    BLOCK_SIZE, BF16_QNAN, CONFIG_NAMES, CONFIG_DESCRIPTIONS, LogicalCase, Workload,
    build_config, duplicate_shared_blocks, f32_to_bf16_bits, logical_case, logical_tokens,
    normal_bf16, page_case, permute_blocks, touched_slots,
)
