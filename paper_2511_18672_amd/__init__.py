"""Selective partial-denoising step of Sphinx (arXiv 2511.18672) on AMD MI355X.

The compute path is ``libsphinx.so`` (hand-written HIP for gfx950 behind the C
ABI of include/sphinx.h).  This package is its thin Python binding plus the
step driver; it has no CPU fallback and raises if the library is missing.
"""
from .binding import (ATTN_FACTORISED, ATTN_JOINT, GRID_PER_FRAME, GRID_SHARED, sphinx_plan_step_grid, BF16, F32, KLogic, make_klogic, sphinx_adaptive_start, KERNEL_CLASSES, NCHW, PEAK_BLOCKS, PEAK_CONSTANT, PEAK_RANDOM, TOKENS, EXPORTED, SphinxError, gather, lib,
                      make_requests, model_desc, plan_step, refine_step, scatter_blend, select_mask, sphinx_gather,
                      sphinx_gather_ctx, sphinx_kv_cache_bytes, sphinx_mask_frontend,
                      sphinx_mask_frontend_workspace_bytes, sphinx_model_blob_bytes, sphinx_model_param,
                      sphinx_peak_mfma, sphinx_plan_cache, sphinx_plan_step, sphinx_refine_step,
                      sphinx_refine_step_cached, sphinx_refine_workspace_bytes, sphinx_scatter_blend,
                      sphinx_scatter_masked, sphinx_select_mask, sphinx_select_mask_static, sphinx_select_workspace_bytes, sphinx_varlen_attention,
                      sphinx_status_string, sphinx_timing_enable, sphinx_timing_read)
from .refiner import Refiner, from_workload, pack_weights

__all__ = ["ATTN_FACTORISED", "ATTN_JOINT", "GRID_PER_FRAME", "GRID_SHARED", "sphinx_plan_step_grid", "BF16", "F32", "KLogic", "make_klogic", "sphinx_adaptive_start", "KERNEL_CLASSES", "NCHW", "PEAK_BLOCKS", "PEAK_CONSTANT", "PEAK_RANDOM", "TOKENS", "EXPORTED", "SphinxError", "Refiner",
           "from_workload", "pack_weights", "lib", "make_requests", "model_desc", "sphinx_gather",
           "sphinx_gather_ctx", "sphinx_kv_cache_bytes", "sphinx_mask_frontend",
           "sphinx_mask_frontend_workspace_bytes", "sphinx_model_blob_bytes", "sphinx_model_param",
           "sphinx_peak_mfma", "sphinx_plan_cache", "sphinx_plan_step", "sphinx_refine_step",
           "sphinx_refine_step_cached", "sphinx_refine_workspace_bytes", "sphinx_scatter_blend",
           "sphinx_scatter_masked", "sphinx_select_mask", "sphinx_select_mask_static", "sphinx_select_workspace_bytes", "sphinx_varlen_attention", "sphinx_status_string",
           "sphinx_timing_enable", "sphinx_timing_read", "select_mask", "gather", "refine_step", "scatter_blend",
           "plan_step"]
