// Host-side launch interface between the C ABI (eb_api.hip) and the kernel files.
// Callers have validated every argument; these functions only choose tiles and launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace eb {

// ---- LM head + confidence -------------------------------------------------------------
// Number of vocabulary slices whose per-row partials are written to the workspace.
int lmhead_num_slices(bool bf16, int n_rows, int vocab);
// With top2 the workspace also holds each partial's second-largest logit.
size_t lmhead_ws_bytes(bool bf16, int n_rows, int vocab, bool top2);
// Partials [n_rows, n_slices] go to ws; the combine writes the per-row outputs (top2_gap only
// when the partials were formed with top2).
hipError_t lmhead_partials(bool bf16, int n_rows, int hidden, int vocab, const void* h,
                           const void* w, void* ws, bool top2, hipStream_t s);
hipError_t lmhead_combine(bool bf16, int n_rows, int vocab, const void* ws, float* conf,
                          float* entropy, int32_t* argmax, float* max_logit, float* top2_gap,
                          hipStream_t s);

// ---- block attention ------------------------------------------------------------------
struct AttnArgs {
  int batch, total_block, max_block, total_prefix, max_prefix;
  const int32_t* cu_block;
  const int32_t* cu_prefix;
  int hq, hkv, head_dim;
  float scale;
  const void *q, *k_blk, *v_blk, *k_pre, *v_pre;
  void* out;
  // optional cached suffix segment (dual cache); cu_suffix == nullptr: none
  int max_suffix = 0;
  const int32_t* cu_suffix = nullptr;
  const void* k_suf = nullptr;
  const void* v_suf = nullptr;
};
// Workspace for key-split partials (0 when the launch needs no split).  Without allow_split
// one workgroup covers all keys of its query tile and no workspace is used.  max_keys is the
// largest number of keys of a sequence (prefix + block + suffix).
size_t block_attn_ws_bytes(bool bf16, bool allow_split, int batch, int total_block,
                           int max_block, int max_keys, int hq, int hkv, int head_dim);
// With defer_merge a key-split launch leaves its partials in ws for step_finish to merge.
hipError_t block_attn(bool bf16, bool allow_split, const AttnArgs& a, void* ws, hipStream_t s,
                      bool defer_merge = false);

// LM-head partials and the block attention of `a` in one launch: the attention's workgroups are
// queued behind the LM head's vocabulary slices (key-split partials in attn_ws, merged by
// step_finish).  Possible when lmhead_hosts_attn(...) holds; the attention then computes
// exactly what block_attn computes for the same arguments.
bool lmhead_hosts_attn(bool bf16, int n_rows, int vocab, const AttnArgs& a);
hipError_t lmhead_partials_attn(int n_rows, int hidden, int vocab, const void* h, const void* w,
                                void* ws, const AttnArgs& a, void* attn_ws, hipStream_t s);

// ---- measurement aid -------------------------------------------------------------------
// Register-only bf16 32x32x16 MFMA loop over `groups` workgroups of 256 threads; each thread
// writes one float of out[groups * 256].  mfma_probe_flops gives the launch's flop count.
double mfma_probe_flops(int groups, int iters);
hipError_t mfma_probe(float* out, int groups, int iters, hipStream_t s);

// ---- unmask ---------------------------------------------------------------------------
hipError_t unmask_select(int batch, int max_block, const int32_t* cu_block, const float* conf,
                         const int32_t* argmax, const float* tau, uint8_t* masked,
                         int32_t* tokens, uint8_t* unmask, int32_t* n_commit, uint8_t* resolved,
                         hipStream_t s);
hipError_t unmask_select_lps(int batch, const int32_t* cu_block, const float* conf,
                             const int32_t* argmax, const float* tau, const float* p_psi,
                             float tau_psi, uint8_t* masked, int32_t* tokens, uint8_t* unmask,
                             int32_t* n_commit, uint8_t* resolved, hipStream_t s);
hipError_t unmask_select_topm(int batch, const int32_t* cu_block, const float* conf,
                              const int32_t* argmax, const float* tau, int m, uint8_t* masked,
                              int32_t* tokens, uint8_t* unmask, int32_t* n_commit,
                              uint8_t* resolved, hipStream_t s);
hipError_t lps_features(int batch, const int32_t* cu_block, int vocab, const float* conf,
                        const float* entropy, const float* gap, const uint8_t* masked,
                        const int32_t* seq_pos, float* feat, float* pos, float* mask_ratio,
                        hipStream_t s);

// ---- fused step epilogue ---------------------------------------------------------------
// One launch after block_attn(..., defer_merge = true) and lmhead_partials: merges the attention
// key splits, combines each row's LM-head partials into conf / entropy / argmax / max_logit,
// and applies the threshold unmask per block.  Usable when one workgroup can reduce a block's
// partials (max_block * n_slices <= kFinishMaxPartials).
constexpr long kFinishMaxPartials = 1L << 16;
bool step_finish_fusable(int max_block, int n_slices);
hipError_t step_finish(bool bf16, const AttnArgs& a, void* attn_ws, int n_rows, int vocab,
                       const void* lm_ws, float* conf, float* entropy, int32_t* argmax,
                       float* max_logit, const float* tau, uint8_t* masked, int32_t* tokens,
                       uint8_t* unmask, int32_t* n_commit, uint8_t* resolved, hipStream_t s);

// ---- LBS post-pass ----------------------------------------------------------------------
hipError_t lbs_select(int n_seq, int window, const uint8_t* masked, const float* p_phi,
                      const int32_t* x_hat, int eos, int l_min, int l_b, int g_max,
                      uint8_t* block, int32_t* size, int32_t* first, hipStream_t s);

}  // namespace eb
