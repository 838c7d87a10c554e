"""Seeded synthetic workloads for the KV tier-migration path: inputs, and an
exact check of a tier state against the content-addressed KV values."""
from .configs import (CHURN, CONFIGS, LLAMA3_70B, LLAMA3_70B_TP2, LLAMA3_70B_TP4, LLAMA3_70B_TP8, LLAMA3_8B,  # noqa: F401
                      MLA, TINY, WINDOW_K, KVConfig)
from .synth import (BANK, FREE_OWNER, NO_PAGE, TIER_CPU, TIER_GPU, TIER_WAIT, Geometry,  # noqa: F401
                    Instance, budget_bytes, churn_steps, eviction_blocks, draw_windows, fill_pool_np, fill_pool_torch,
                    make_bank, make_instance, page_owners, program_content_torch, program_host_content, random_instance, run_content,
                    rotation_windows, run_offset, run_tag, runs_torch)
from .check import check_tier_bytes  # noqa: F401
