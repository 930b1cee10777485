"""Seeded synthetic workloads for the PatchKV context-loading path.

This package only *draws inputs*: random normals, key scales, eviction index
sets and synthesized compressed caches. It contains none of the arithmetic of
the patch construction itself (attention, targets, statistics, ridge solve);
both the fp64 oracle and the GPU path read the bytes it produces.
"""
from .configs import CONFIGS, Config, get_config
from .generate import (ChunkInputs, LayerInputs, MlpWeights, QuantCache, make_cache_bias,
                       make_chunk_inputs, make_layer_inputs, make_custom_inputs, make_mlp_weights,
                       make_quant_cache, make_cache_extras, pack_int4, unpack_int4, quantize_mx,
                       bf16_round_bits, bf16_bits_to_f32)

__all__ = ["CONFIGS", "Config", "get_config", "LayerInputs", "make_layer_inputs",
           "make_custom_inputs", "bf16_round_bits", "bf16_bits_to_f32", "ChunkInputs",
           "make_chunk_inputs", "MlpWeights", "make_mlp_weights", "QuantCache", "make_cache_bias",
           "make_quant_cache", "make_cache_extras", "pack_int4", "unpack_int4", "quantize_mx"]
