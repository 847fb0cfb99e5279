"""Seeded synthetic workloads for the single-stage forward.

This package is shared by the CPU oracle (``oracle/``) and the HIP path
(``paper_2512_21835_amd``).  It holds shapes, seeds and random-number generation
only -- none of the decoder-layer arithmetic -- so that both sides consume the
same bits without sharing any code of the method itself.

The paper serves LLaMA2-13B / Qwen3-32B / LLaMA3.3-70B checkpoints on a
fixed-length text dataset (Section IV-A, "Models").  Neither is available, so
every workload here is a seeded synthetic stand-in with the layer shapes of a
LLaMA-3-8B or LLaMA-3.3-70B decoder stage: weights bf16(N(0, 0.02)), RMSNorm
gains bf16(1 + N(0, 0.02)), hidden states N(0, 1) fp32.
"""
from .inputs import (  # noqa: F401
    StageShape, Workload, TINY, LLAMA8B_STAGE, LLAMA70B_STAGE, WORKLOADS,
    TENSOR_IDS, seed_of, normal_bf16, normal_f32, layer_weights, layer_weight_shapes,
    prefill_inputs, decode_input, bf16_to_f32, draws, lib_path, build_lib,
)
