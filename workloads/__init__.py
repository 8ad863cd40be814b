"""Seeded synthetic inputs for the boosted-decode hot path.

This package is shared by the CPU oracle and by the GPU path. It only draws
random numbers and lays out inputs (vocabulary case classes, per-stream phrase
lists, joint-logit tensors); it holds none of the boosting arithmetic.
"""

from .synth import (  # noqa: F401
    CONFIGS,
    Config,
    bf16_bits_to_f32,
    class_map,
    class_members,
    config_by_name,
    logit_chunks,
    logits,
    model_ids,
    phrase_csr,
    phrases,
    plants,
)
