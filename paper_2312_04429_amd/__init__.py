"""MI355X-native cache-hit generation path of approximate caching for diffusion serving.

Entry points (same names as the C ABI in include/nv.h):
  nv_cache_lookup   exact cosine top-1 over the cached prompt embeddings + cache selector
  nv_gather_states  fetch the matched entry's intermediate latent at the chosen K
  nv_gather_pool    the same from a maintained state pool, with hole handling
  NvLCBFU           host LCBFU maintainer (evictions, row compaction plans)
  NvIVF             IVF approximate index (build and search on the device)
  nv_ocsvm_train    train the match predictor (linear one-class SVM, host)
  nv_match_gate     score queries with it and turn predicted misses into "no match"
  nv_cache_lookup_gated  the lookup with the predictor in front: only predicted
                    matches are searched (Alg. 1)
  NvUNet            device-resident latent-diffusion UNet; .nv_denoise runs the
                    remaining N - K guided DDIM steps, .nv_unet_eps one evaluation

Importing the package loads libnv.so and fails if it has not been built.
"""
from .api import (NvIVF, NvLCBFU, NvUNet, nv_cache_insert, nv_cache_move_rows, nv_gather_pool,
                  nv_match_gate, nv_ocsvm_train, nv_table_update, nv_cache_lookup, nv_cache_lookup_gated, nv_cache_lookup_gated_workspace,
                  nv_cache_lookup_static, nv_cache_lookup_workspace, nv_gather_states,
                  nv_op_attention, nv_op_conv3x3, nv_op_linear, nv_probe_peaks, nv_trace_disable,
                  nv_trace_enable, nv_trace_read, nv_trace_records, nv_unet_param_count,
                  nv_unet_param_info, workspace)

from ._native import NV_FAM_ATTN as FAM_ATTN, NV_FAM_CONV as FAM_CONV
from ._native import NV_FAM_LINEAR as FAM_LINEAR, NV_FAM_SCAN as FAM_SCAN

__all__ = ["FAM_ATTN", "FAM_CONV", "FAM_LINEAR", "FAM_SCAN", "NvIVF", "NvLCBFU", "NvUNet",
           "nv_cache_move_rows", "nv_gather_pool", "nv_match_gate", "nv_ocsvm_train",
           "nv_table_update", "nv_cache_insert", "nv_cache_lookup", "nv_cache_lookup_gated", "nv_cache_lookup_gated_workspace", "nv_cache_lookup_static", "nv_cache_lookup_workspace", "nv_gather_states",
           "nv_op_attention", "nv_op_conv3x3", "nv_op_linear", "nv_probe_peaks", "nv_trace_disable", "nv_trace_enable",
           "nv_trace_read", "nv_trace_records", "nv_unet_param_count", "nv_unet_param_info", "workspace"]
