"""Seeded synthetic step inputs shared by the oracle side and the HIP side.

Holds no arithmetic of the decoding step itself."""
from .generator import (VERSION, CONFIGS, StepConfig, StepCase, make_step, custom_config,
                        f32_to_bf16_bits, bf16_bits_to_f32, to_storage, widen_f64,
                        router_scores, suffix_segment, lbs_window)

__all__ = ["VERSION", "CONFIGS", "StepConfig", "StepCase", "make_step", "custom_config",
           "f32_to_bf16_bits", "bf16_bits_to_f32", "to_storage", "widen_f64", "router_scores",
           "suffix_segment", "lbs_window"]
