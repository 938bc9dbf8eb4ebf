"""Seeded synthetic inputs for the Whisper-Flash draft-and-verify step.

This module holds shapes, the weight manifest order and seeded random
generators only.  It contains none of the method's arithmetic: both the
CPU oracle (``oracle/``) and the HIP path (``paper_2609_32869_amd``) take
their inputs from here, and neither imports the other.

Workload shapes follow the paper's setup: the target is Whisper large-v3
(Section 4), the drafter has two blocks and fills K=8 mask positions
(Section 3.2, Eq. 2), history taps come from target blocks 1, 8, 15, 22, 29
(Appendix A.2), the acoustic memory is one 30 s window of 1500 encoder
frames, and text positions stop at Whisper's 448-token context.
"""
from .configs import (ModelConfig, TINY, LARGE_V3, MICRO, VOCAB64, PURPOSE, config_by_name,
                      EncoderConfig, LARGE_V3_ENC, MICRO_ENC)
from .manifest import target_manifest, drafter_manifest, full_manifest, param_count, encoder_manifest
from .gen import (make_weights, make_memory, make_prefix, make_prefix_lengths,
                  plant_drafts, bf16_round_bits, bits_to_f32, WeightSet, make_encoder_weights, make_audio)

__all__ = [
    "ModelConfig", "TINY", "LARGE_V3", "MICRO", "VOCAB64", "PURPOSE", "config_by_name",
    "target_manifest", "drafter_manifest", "full_manifest", "param_count",
    "make_weights", "make_memory", "make_prefix", "make_prefix_lengths", "plant_drafts",
    "bf16_round_bits", "bits_to_f32", "WeightSet",
    "EncoderConfig", "LARGE_V3_ENC", "MICRO_ENC", "encoder_manifest", "make_encoder_weights", "make_audio",
]
