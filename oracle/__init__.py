"""fp64 CPU oracle of the Early-Bird denoising step.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the package smoke check
and the benchmark's CPU-baseline leg, never by the HIP product path."""
from .eb_oracle import (block_attention, lmhead_logits, confidence_stats, lmhead_confidence,
                        unmask_select, decode_step, lps_features, unmask_select_lps,
                        unmask_select_topm, lbs_select)
from . import margins

__all__ = ["block_attention", "lmhead_logits", "confidence_stats", "lmhead_confidence",
           "unmask_select", "decode_step", "lps_features", "unmask_select_lps",
           "unmask_select_topm", "lbs_select", "margins"]
