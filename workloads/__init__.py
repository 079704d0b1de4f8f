"""Seeded synthetic inputs (shapes and statistics of the paper's workloads)."""
from .synthetic import (WORKLOADS, Workload, scaled, head_crs, effective_crs,  # noqa: F401
                        precompressed_lengths, decision_logits, decode_inputs_np,
                        prompt_np, decode_inputs_torch, prompt_torch, prompt_full_torch,
                        precompressed_torch, sample_units, seed_for, pool_pages,
                        train_inputs_torch, TRAIN_C, TRAIN_TAU, TRAIN_WINDOW)
