"""PatchKV context-loading path on MI355X (gfx950): HIP kernels behind a C ABI.

The library (``lib/libpatchkv.so``) is loaded on first use by :mod:`.binding`;
there is no CPU fallback.
"""
from .binding import (BF16, F32, F64, IDX_PER_HEAD, IDX_SHARED, KV_MXINT4, KV_MXINT8, KV_PLAIN, RIDGE_ABSOLUTE,
                      RIDGE_ADAPTIVE, RIDGE_TRACE_MEAN, SOLVE_EXACT_F32, SOLVE_FAST_BF16, PatchKVError, accumulate_normal_eq,
                      attend_cache, attend_chunk, attend_compressed, attend_compressed_noalloc,
                      attend_full, compute_block_targets, compute_layer_patch, compute_targets,
                      layer_workspace_bytes, lib, low_rank_patch, mlp_features, propagate_student,
                      solve_patch, solve_patch_dual)

__all__ = ["BF16", "F32", "F64", "IDX_PER_HEAD", "IDX_SHARED", "KV_MXINT4", "KV_MXINT8", "KV_PLAIN", "RIDGE_ABSOLUTE",
           "RIDGE_ADAPTIVE", "RIDGE_TRACE_MEAN", "SOLVE_EXACT_F32", "SOLVE_FAST_BF16", "PatchKVError", "accumulate_normal_eq",
           "attend_cache", "attend_chunk", "attend_compressed", "attend_compressed_noalloc",
           "attend_full", "compute_block_targets", "compute_layer_patch", "compute_targets",
           "layer_workspace_bytes", "lib", "low_rank_patch", "mlp_features", "propagate_student",
           "solve_patch", "solve_patch_dual"]
