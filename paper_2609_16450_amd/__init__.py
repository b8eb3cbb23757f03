"""MI355X (gfx950) implementation of one Early-Bird denoising step.

The computation lives in libeb.so (hand-written HIP kernels behind the C ABI of
include/eb.h); this package only builds it and binds it with ctypes."""
from .binding import (EB_BF16, EB_F32, EB_NOALLOC_SCRATCH_BYTES, EbError, Ragged, StepBuffers,
                      eb_block_attn, eb_block_attn_dual, eb_block_attn_workspace, eb_decode_step,
                      eb_decode_step_attn_in_lmhead, eb_decode_step_noalloc,
                      eb_decode_step_workspace, eb_last_error, eb_lbs_select,
                      eb_lmhead_confidence, eb_lmhead_features, eb_lmhead_features_workspace,
                      eb_lmhead_workspace, eb_lps_features, eb_probe_mfma_bf16, eb_status_string,
                      eb_unmask_select, eb_unmask_select_lps, eb_unmask_select_topm, eb_version,
                      lib_path, load)

__all__ = ["EB_BF16", "EB_F32", "EB_NOALLOC_SCRATCH_BYTES", "EbError", "Ragged", "StepBuffers",
           "eb_block_attn", "eb_block_attn_dual", "eb_block_attn_workspace", "eb_decode_step",
           "eb_decode_step_attn_in_lmhead", "eb_decode_step_noalloc", "eb_decode_step_workspace",
           "eb_last_error", "eb_lbs_select", "eb_lmhead_confidence", "eb_lmhead_features",
           "eb_lmhead_features_workspace", "eb_lmhead_workspace", "eb_lps_features",
           "eb_probe_mfma_bf16", "eb_status_string", "eb_unmask_select", "eb_unmask_select_lps",
           "eb_unmask_select_topm", "eb_version", "lib_path", "load"]
