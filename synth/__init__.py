"""Seeded synthetic inputs shared by the oracle and the GPU path.

This package holds only workload descriptions (topologies, shapes, the
threshold table and schedule constants that are *inputs* to the method) and
seeded random generators.  It contains none of the method's arithmetic: no
similarity, no selector, no network layer, no sampler update.
"""
from .configs import (UNET_TINY, UNET_SD15, UNET_SDXL, SCHEDULE_SD, THRESHOLDS_PAPER,
                      THRESHOLDS_TINY, WORKLOADS, unet_config)
from .weights import param_specs, make_weights, param_count, bf16_round
from .data import (make_cache, make_cache_device, cluster_centres_device, make_queries_at_sims,
                   make_cluster_queries, cluster_queries_from, make_contexts, make_pooled, make_k_values,
                   cache_rows_f32, cluster_centres, make_latents, to_bf16_bits, from_bf16_bits,
                   make_prompt_stream)

__all__ = [
    "UNET_TINY", "UNET_SD15", "UNET_SDXL", "SCHEDULE_SD", "THRESHOLDS_PAPER", "THRESHOLDS_TINY",
    "WORKLOADS", "unet_config", "param_specs", "make_weights", "param_count", "bf16_round",
    "make_cache", "make_queries_at_sims", "make_cluster_queries", "make_contexts", "make_latents",
    "to_bf16_bits", "from_bf16_bits", "make_k_values", "cache_rows_f32", "cluster_centres",
    "make_cache_device", "cluster_centres_device", "cluster_queries_from", "make_pooled",
    "make_prompt_stream",
]
