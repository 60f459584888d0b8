"""Seeded synthetic inputs shared by the oracle and the HIP path.

This module only *generates inputs*: model weights, camera frames, text ids,
extra embedding rows, workload shapes and thresholds.  It holds none of the
method's arithmetic (no patch similarity, no model math, no margin).  Both the
CPU oracle and the GPU path receive exactly the tensors produced here.

Random numbers come from a counter-based hash: every element is a pure
function of (seed, tensor id, element index), so any tensor (or any slice of
one) can be regenerated on any device without generating the rest.  The hash
is the 32-bit "lowbias32" integer mixer published by C. Wellons (hash
prospector, 2018): x ^= x>>16; x *= 0x7feb352d; x ^= x>>15; x *= 0x846ca68b;
x ^= x>>16, all mod 2^32.  It is evaluated in int64 torch arithmetic with the
32x32-bit products split into 16-bit halves so nothing overflows; integer
arithmetic makes CPU and GPU results identical.

Weights are uniform on [-a, a) with a = 2^s: a 24-bit hash value k maps to
(k - 2^23) * 2^(s-23) in one IEEE fp32 multiply (exact for integer s), then
rounds to bf16 with round-to-nearest-even (torch's fp32->bf16 cast); the
bits are the same on every device.
"""
from .hashgen import lowbias32, hash_u32, uniform_f32, uniform_bf16, uniform_u8
from .configs import (VLAConfig, config_c1, config_mid, config_c4_tiny, config_c2, config_c3, config_c4, config_c5,
                      config_c1v, config_c2v, ALL_CONFIGS)
from .workload import (
    TensorId, layer_weights, global_weights, model_weights, vit_weights,
    random_frame, changed_patch_order, perturb_patches, text_ids, extra_rows,
    step_inputs, c3_episode_frames, reuse_schedule,
)

__all__ = [
    "lowbias32", "hash_u32", "uniform_f32", "uniform_bf16", "uniform_u8",
    "VLAConfig", "config_c1", "config_mid", "config_c4_tiny", "config_c2", "config_c3", "config_c4", "config_c5",
    "config_c1v", "config_c2v", "ALL_CONFIGS",
    "TensorId", "layer_weights", "global_weights", "model_weights", "vit_weights",
    "random_frame", "changed_patch_order", "perturb_patches", "text_ids", "extra_rows",
    "step_inputs", "c3_episode_frames", "reuse_schedule",
]
