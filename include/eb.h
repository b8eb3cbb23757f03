/*
 * eb.h - C ABI of the Early-Bird denoising-step library (libeb.so), MI355X / gfx950.
 *
 * One denoising step of a masked diffusion LM over ragged, variable-length active blocks
 * (Early-Bird Decoding, Sec. 5 and Alg. 5):
 *   1. bidirectional attention of each block's queries over the sequence's cached prefix
 *      keys/values plus the block's own keys/values        -> eb_block_attn
 *   2. LM-head logits z = W h for every block position, reduced on chip to the top-1
 *      confidence kappa = max_v p(v), the top-1 token x_hat and the entropy of
 *      p = softmax(z); the logits never reach device memory  -> eb_lmhead_confidence
 *   3. threshold commit kappa >= tau with the anti-stall fallback inside each block
 *                                                          -> eb_unmask_select
 *   4. all of the above on one stream                      -> eb_decode_step
 *
 * Conventions shared by every entry point
 *   - Every pointer argument is a DEVICE pointer owned by the caller unless stated
 *     otherwise; descriptor structs themselves live in host memory and are read during the
 *     call only.  The library allocates no device memory and keeps no state besides a
 *     per-thread last-error string.
 *   - Every call enqueues work on `stream` (a hipStream_t; NULL = default stream) and
 *     returns without synchronising.  Outputs are valid once the stream reaches them.
 *   - Arguments are checked on the host before anything is launched: a bad argument
 *     returns EB_ERR_INVALID (or EB_ERR_WORKSPACE for a short workspace) and launches
 *     nothing.  A valid but unimplemented combination returns EB_ERR_UNSUPPORTED.
 *     A launch failure returns EB_ERR_HIP.  eb_last_error() describes the last failure
 *     of the calling thread.
 *   - Device-array contents are the caller's contract and are not checked: cu arrays are
 *     non-decreasing, start at 0 and end at the totals given on the host, maxima are
 *     true maxima, tau lies in (0, 1], inputs are finite.  For debugging, the environment
 *     variable EB_DEBUG_CHECKS (any value but "0") makes every entry point that takes cu
 *     arrays or tau copy them to the host after the work already on its stream (which
 *     synchronises that stream) and return EB_ERR_INVALID, launching nothing, when they break
 *     this contract.  Such calls cannot be captured in a graph.  For testing, the environment
 *     variable EB_ATTN_STAGED (any value but "0") makes the bf16 attention at head dimension
 *     128 use the kernel it otherwise keeps for K/V segments too long for 32-bit offsets;
 *     results agree with the default kernel to the attention tolerance, not bit for bit.
 *   - Rows are packed: the block rows of sequence b are rows cu_block[b] .. cu_block[b+1]-1,
 *     in ascending sequence position (a non-contiguous block is gathered in order), its
 *     cached prefix rows are cu_prefix[b] .. cu_prefix[b+1]-1.  Empty blocks are legal.
 *   - bf16 tensors are raw bfloat16 bit patterns (uint16) and must be 16-byte aligned.
 *   - Results are deterministic: the same inputs give bit-identical outputs run to run.
 */
#ifndef EB_H_
#define EB_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* eb_stream_t; /* identical to hipStream_t */
typedef struct ihipEvent_t* eb_event_t;   /* identical to hipEvent_t */

typedef enum { EB_F32 = 0, EB_BF16 = 1 } eb_dtype;

typedef enum {
  EB_OK = 0,
  EB_ERR_INVALID = 1,     /* bad argument; nothing launched */
  EB_ERR_UNSUPPORTED = 2, /* valid but not implemented (e.g. head_dim not 64/128) */
  EB_ERR_WORKSPACE = 3,   /* ws_bytes below the matching *_workspace() query */
  EB_ERR_HIP = 4          /* HIP runtime / launch failure */
} eb_status;

/* Ragged batch.  Host integers size the launch grids; device arrays hold exclusive prefix
 * sums of the per-sequence block and prefix lengths. */
typedef struct {
  int32_t batch;            /* number of sequences B >= 1 */
  int32_t total_block;      /* T = cu_block[B] (block rows over all sequences) */
  int32_t max_block;        /* max_b (cu_block[b+1] - cu_block[b]) */
  int32_t total_prefix;     /* S = cu_prefix[B] (cached prefix rows) */
  int32_t max_prefix;       /* max_b (cu_prefix[b+1] - cu_prefix[b]) */
  const int32_t* cu_block;  /* device [B+1] */
  const int32_t* cu_prefix; /* device [B+1]; unused (may be NULL) by eb_unmask_select */
} eb_ragged;

/* ---------------------------------------------------------------------------------------
 * Block attention with a prefix KV cache (Sec. 3 / App. B: the mask predictor is a
 * bidirectional Transformer, so a block query sees every key of its sequence; Sec. 6.3:
 * keys/values of the committed context left of the block come from a prefix cache).
 *
 *   out[i, h, :] = sum_j softmax_j(scale * q[i, h, :] . k_j) v_j
 *
 * over the keys j of i's sequence b: its prefix rows (k_pre, v_pre) and its block rows
 * (k_blk, v_blk).  No causal mask, no masking by [MASK] state.  Query head h reads key/value
 * head h / (hq / hkv) (grouped-query attention with contiguous groups).  K arrives after any
 * positional encoding.
 *
 *   q      [T, hq, head_dim]    k_blk, v_blk [T, hkv, head_dim]
 *   k_pre, v_pre [S, hkv, head_dim]             out [T, hq, head_dim]   (all of dtype dt)
 *
 * Requires hq % hkv == 0, head_dim in {64, 128}, scale > 0 and finite; scale = 0 selects
 * 1/sqrt(head_dim) (rounded to fp32, the same bits eb_decode_step uses for attn_scale <= 0).
 * Arithmetic: bf16 inputs, fp32 scores / softmax / accumulation, the probabilities rounded to
 * bf16 for the product with V (at head_dim 128 the softmax denominator sums those same rounded
 * values), output rounded to bf16 (round to nearest even); EB_F32 computes in fp32 throughout.
 * ------------------------------------------------------------------------------------- */
size_t eb_block_attn_workspace(eb_dtype dt, const eb_ragged* r, int hq, int hkv, int head_dim);
eb_status eb_block_attn(eb_dtype dt, const eb_ragged* r, int hq, int hkv, int head_dim,
                        float scale, const void* q, const void* k_blk, const void* v_blk,
                        const void* k_pre, const void* v_pre, void* out, void* ws,
                        size_t ws_bytes, eb_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * Block attention with a dual cache (Sec. 6.3, Tab. 6): as eb_block_attn, with each
 * sequence's keys extended by its cached suffix rows, the context right of the block,
 *
 *   keys of sequence b = prefix rows cu_prefix[b] .. cu_prefix[b+1]-1 of k_pre / v_pre
 *                      + block rows  cu_block[b]  .. cu_block[b+1]-1  of k_blk / v_blk
 *                      + suffix rows cu_suffix[b] .. cu_suffix[b+1]-1 of k_suf / v_suf
 *
 * (the keys form a set: the order of the segments does not change the result).
 *   k_suf, v_suf [total_suffix, hkv, head_dim] of dtype dt; cu_suffix device [batch+1] int32,
 *   non-decreasing from 0 to total_suffix; max_suffix its largest difference.
 * ws: at least eb_block_attn_dual_workspace(...) bytes.
 * ------------------------------------------------------------------------------------- */
typedef struct {
  int32_t total_suffix, max_suffix;
  const int32_t* cu_suffix; /* device [batch+1] */
} eb_suffix;

size_t eb_block_attn_dual_workspace(eb_dtype dt, const eb_ragged* r, const eb_suffix* sfx, int hq,
                                    int hkv, int head_dim);
eb_status eb_block_attn_dual(eb_dtype dt, const eb_ragged* r, const eb_suffix* sfx, int hq,
                             int hkv, int head_dim, float scale, const void* q, const void* k_blk,
                             const void* v_blk, const void* k_pre, const void* v_pre,
                             const void* k_suf, const void* v_suf, void* out, void* ws,
                             size_t ws_bytes, eb_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * Fused LM head and confidence statistics (Alg. 5: softmax of the backbone logits, top-1
 * confidence and token; Eq. app-confidence; Sec. 5.1: entropy, normalised by ln|V| for the
 * block selector).  For each row i of h:
 *
 *   z = W h_i (fp32 accumulation),  p = softmax(z)
 *   conf[i]         = max_v p(v)                      (kappa)
 *   argmax[i]       = lowest v with z_v = max z       (x_hat; ties to the lowest id)
 *   entropy_nats[i] = -sum_v p(v) ln p(v)             (raw nats; divide by ln(vocab) for H~)
 *   max_logit[i]    = max_v z_v                       (optional; pass NULL to skip)
 *
 *   h [n_rows, hidden]   w [vocab, hidden] (nn.Linear layout)   outputs [n_rows]
 *
 * Requires n_rows >= 0, vocab >= 1, hidden >= 1; EB_BF16 also needs hidden % 64 == 0.
 * ws: at least eb_lmhead_workspace(...) bytes of device memory, contents ignored; it holds
 * per-(row, vocabulary slice) partial reductions merged in a fixed order.
 * ------------------------------------------------------------------------------------- */
size_t eb_lmhead_workspace(eb_dtype dt, int n_rows, int hidden, int vocab);
eb_status eb_lmhead_confidence(eb_dtype dt, int n_rows, int hidden, int vocab, const void* h,
                               const void* w, float* conf, float* entropy_nats,
                               int32_t* argmax, float* max_logit, void* ws, size_t ws_bytes,
                               eb_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * Threshold unmask inside each variable-length block (Eq. prelim-update, threshold branch;
 * Alg. 5 accept rule without the router term, anti-stall fallback and commit).
 * For each sequence b, over its block rows i:
 *
 *   A_b = { i : masked[i] && conf[i] >= tau[b] }
 *   if A_b is empty and some row is masked:
 *       A_b = { the lowest i among masked rows with maximal conf[i] }
 *   for i in A_b: tokens[i] = argmax[i]; masked[i] = 0
 *   unmask[i]   = (i in A_b)            for every block row
 *   n_commit[b] = |A_b|
 *   resolved[b] = no masked row left in block b (1 for an empty block)
 *
 *   conf [T] f32, argmax [T] i32, tau [B] f32        (inputs)
 *   masked [T] u8 (1 = [MASK]), tokens [T] i32         (updated in place)
 *   unmask [T] u8, n_commit [B] i32, resolved [B] u8   (outputs)
 *
 * Only r->batch, r->total_block, r->max_block and r->cu_block are used.
 * ------------------------------------------------------------------------------------- */
eb_status eb_unmask_select(const eb_ragged* r, const float* conf, const int32_t* argmax,
                           const float* tau, uint8_t* masked, int32_t* tokens, uint8_t* unmask,
                           int32_t* n_commit, uint8_t* resolved, eb_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * LM head with the LPS gap feature (Sec. 5.2, Alg. 5): everything eb_lmhead_confidence
 * computes, plus the gap between the two largest probabilities of each row
 *
 *   top2_gap[i] = p_(1) - p_(2)    (p sorted in decreasing order, counted with multiplicity:
 *                                   0 when the largest logit is shared; p_(2) = 0 if vocab = 1)
 *
 * computed as (1 - exp(z_(2) - z_(1))) / sum_v exp(z_v - z_(1)) from the two largest logits,
 * which the kernels track next to the row maximum.  Same requirements as eb_lmhead_confidence;
 * top2_gap [n_rows] f32 is required.  ws: at least eb_lmhead_features_workspace(...) bytes.
 * ------------------------------------------------------------------------------------- */
size_t eb_lmhead_features_workspace(eb_dtype dt, int n_rows, int hidden, int vocab);
eb_status eb_lmhead_features(eb_dtype dt, int n_rows, int hidden, int vocab, const void* h,
                             const void* w, float* conf, float* entropy_nats, int32_t* argmax,
                             float* max_logit, float* top2_gap, void* ws, size_t ws_bytes,
                             eb_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * LPS router inputs of every block row (Sec. 5.2; Alg. 5, feature tuple and intra-block
 * position).  For row i of block b (rows cu_block[b] .. cu_block[b+1]-1, len_b rows):
 *
 *   rho_b      = (masked rows of block b) / len_b     (block-wise mask ratio before commit)
 *   feat[i]    = (conf[i], entropy_nats[i] / ln(vocab), top2_gap[i], rho_b)   [T, 4] f32
 *   pos[i]     = (p_i - p_first) / len_b              [T] f32, the normalised intra-block
 *                position (i - b) / |B| of Sec. 5.2 and Alg. 5, with b the block's left
 *                boundary and |B| its size, where
 *                  seq_pos != NULL:  p_i = seq_pos[i], the sequence position of row i (a
 *                                    block chosen by eb_lbs_select may have gaps, and then
 *                                    pos exceeds 1 towards its right end);
 *                  seq_pos == NULL:  p_i = i, the packed row, so pos is the row's rank within
 *                                    its block over len_b, in [0, 1) (equal to the above for
 *                                    a contiguous block);
 *                p_first is p_i of the block's first row.  Computed in fp32 (the integer
 *                difference, exact below 2^24, divided by len_b with one rounding).
 *   mask_ratio[b] = rho_b                             [B] f32, optional (NULL to skip)
 *
 *   seq_pos [T] i32, optional; ascending within each block (the caller's contract).
 *
 * The router itself is not part of this library: its commit probability p_psi comes back
 * through eb_unmask_select_lps.  Requires vocab >= 2 and feat 16-byte aligned; only r->batch,
 * r->total_block and r->cu_block are used.
 * ------------------------------------------------------------------------------------- */
eb_status eb_lps_features(const eb_ragged* r, int vocab, const float* conf,
                          const float* entropy_nats, const float* top2_gap,
                          const uint8_t* masked, const int32_t* seq_pos, float* feat, float* pos,
                          float* mask_ratio, eb_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * Union accept rule of Alg. 5 (Sec. 5.2, LPS router inference): as eb_unmask_select, with
 *
 *   A_b = { i : masked[i] && (conf[i] >= tau[b] || p_psi[i] > tau_psi) }
 *
 * and the same anti-stall fallback and commit.  p_psi [T] f32 is the caller's router commit
 * probability per block row (rows that are not masked are ignored).
 * ------------------------------------------------------------------------------------- */
eb_status eb_unmask_select_lps(const eb_ragged* r, const float* conf, const int32_t* argmax,
                               const float* tau, const float* p_psi, float tau_psi,
                               uint8_t* masked, int32_t* tokens, uint8_t* unmask,
                               int32_t* n_commit, uint8_t* resolved, eb_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * Budgeted block update (Eq. prelim-update with a per-step budget m): as eb_unmask_select,
 * with
 *
 *   A_b = { i : masked[i] && conf[i] >= tau[b] }  united with
 *         Top-m_b = the m masked rows of block b with the largest conf (equal conf: the lower
 *                   row first; every masked row if fewer than m)
 *
 * m = 0 gives the threshold rule with its anti-stall fallback; a tau above 1 disables the
 * threshold.  Requires m >= 0.
 * ------------------------------------------------------------------------------------- */
eb_status eb_unmask_select_topm(const eb_ragged* r, const float* conf, const int32_t* argmax,
                                const float* tau, int32_t m, uint8_t* masked, int32_t* tokens,
                                uint8_t* unmask, int32_t* n_commit, uint8_t* resolved,
                                eb_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * LBS active-block selection post-pass (Sec. 5.1; Alg. 5, block selection) for each of n_seq
 * sequences over a generation window of `window` positions.
 *
 * Contract.  For every sequence s the call picks a set B_s of its masked positions (the next
 * active block) and writes it as a 0/1 mask.  A sequence with at most l_min masked positions
 * takes all of them.  Otherwise B_s is grown from the left over the masked positions that the
 * LBS router includes (p_phi > 0.5, strictly) and whose predicted token is not eos_id, and
 * growth stops before the first such position that lies more than g_max positions after the
 * last one taken, so nothing beyond a wide gap joins.  When that leaves fewer than l_min
 * positions, B_s becomes the l_b lowest masked positions instead.  Distances are differences of
 * positions: g_max = 1 admits contiguous runs only.
 *
 *   masked [n_seq, window] u8, p_phi [n_seq, window] f32 (the LBS router's probability; the
 *   router itself is not part of this library), x_hat [n_seq, window] i32   (inputs)
 *   block [n_seq, window] u8 (1 = in B_s), size [n_seq] i32 = |B_s|,
 *   first [n_seq] i32 = smallest position of B_s, or -1 when B_s is empty    (outputs)
 *
 * Requires l_min, l_b >= 0 and g_max >= 1.  Integer-exact.
 * ------------------------------------------------------------------------------------- */
eb_status eb_lbs_select(int32_t n_seq, int32_t window, const uint8_t* masked,
                        const float* p_phi, const int32_t* x_hat, int32_t eos_id, int32_t l_min,
                        int32_t l_b, int32_t g_max, uint8_t* block, int32_t* size,
                        int32_t* first, eb_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * One whole denoising step (Alg. 5, one loop iteration): eb_block_attn, then
 * eb_lmhead_confidence over the T block rows of h, then eb_unmask_select, enqueued on `stream`
 * with no host synchronisation.  Every output equals, bit for bit, what those three calls
 * produce; the step merely launches fewer kernels: the attention's key-split merge, the
 * merge of the LM-head partials and the unmask run as one epilogue launch (unless a block's
 * rows times the LM head's vocabulary slices exceed 65536, when they run separately), and in
 * small bf16 steps (at most 64 block rows, at most 256 query rows per sequence and K/V head,
 * head_dim 64 or 128, an LM head streamed by 16-wave workgroups) the attention's workgroups are
 * queued behind the LM head's in the same launch, which starts them as the LM head's
 * workgroups finish.  The attention does not depend on the LM head or the reverse, so this
 * changes no result.  The workspace holds the attention's key-split partials followed by the
 * LM-head partials.
 * Field meanings, layouts and requirements are those of the three calls above; the LM-head
 * rows are the block rows (n_rows = ragged.total_block).
 *
 * Optional tracing: when `trace` is non-NULL, each non-NULL event in it is recorded on the
 * step's stream at the named point (events created by the caller, e.g. with
 * hipEventCreate); this times the kernels of one step without a host synchronisation.
 * ------------------------------------------------------------------------------------- */
typedef struct {
  eb_event_t attn_begin, attn_end;     /* around the attention kernel (its split merge, if
                                          any, runs in the epilogue); recorded back to back
                                          when the attention shares the LM-head launch */
  eb_event_t lmhead_begin, lmhead_end; /* around the fused LM-head kernel (without its merge),
                                          including the attention when it shares the launch */
  eb_event_t select_begin, select_end; /* around the epilogue: split merges and unmask */
} eb_step_trace;

typedef struct {
  eb_dtype dtype;
  eb_ragged ragged;
  /* attention */
  int32_t hq, hkv, head_dim;
  float attn_scale; /* <= 0 selects 1/sqrt(head_dim) */
  const void* q;
  const void* k_blk;
  const void* v_blk;
  const void* k_pre;
  const void* v_pre;
  void* attn_out;
  /* LM head + statistics */
  int32_t hidden, vocab;
  const void* h;
  const void* w;
  float* conf;
  float* entropy_nats;
  int32_t* argmax;
  float* max_logit; /* nullable */
  /* unmask */
  const float* tau;
  uint8_t* masked;
  int32_t* tokens;
  uint8_t* unmask;
  int32_t* n_commit;
  uint8_t* resolved;
  /* tracing */
  const eb_step_trace* trace; /* nullable */
} eb_step_desc;

size_t eb_decode_step_workspace(const eb_step_desc* d);
eb_status eb_decode_step(const eb_step_desc* d, void* ws, size_t ws_bytes, eb_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * eb_decode_step without a caller workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid allocation).
 *
 * Same descriptor, same work and bit-identical outputs as eb_decode_step; the workspace is a
 * device array inside the library of EB_NOALLOC_SCRATCH_BYTES (128 MiB), one per device,
 * present from the moment the library is loaded on that device until the process ends.  The
 * call allocates and frees nothing.  On its first call for a device it looks up that device's
 * copy of the array (the device of `stream`, or the current device for a NULL stream).
 *
 * Limit: a step needing more than EB_NOALLOC_SCRATCH_BYTES of workspace
 * (eb_decode_step_workspace) returns EB_ERR_WORKSPACE and launches nothing.  The array's
 * contents are left over from the previous call and are not needed to be zero.
 * Every call on a device shares that device's array: calls that may overlap in time on one
 * device (different streams without ordering between them, or different threads) race on it
 * and must be serialised by the caller.
 * ------------------------------------------------------------------------------------- */
#define EB_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
eb_status eb_decode_step_noalloc(const eb_step_desc* d, eb_stream_t stream);

/* 1 when eb_decode_step with this descriptor runs the attention's workgroups inside the LM-head
 * launch (the small-step case above), else 0 (also for a NULL descriptor).  Reads only the
 * descriptor's host fields (dtype, ragged sizes, heads, head_dim, vocab); launches nothing.  For
 * profilers that attribute the shared launch's time and bytes. */
int32_t eb_decode_step_attn_in_lmhead(const eb_step_desc* d);

/* ---------------------------------------------------------------------------------------
 * Measurement aid (not part of the denoising step).
 *
 * A register-only loop of dense bf16 32x32x16 MFMAs: `groups` workgroups of 256 threads, each
 * wave running 8 independent accumulator chains for `iters` iterations, with no memory traffic
 * except one float per thread written to out[groups * 256] at the end (a caller-owned device
 * buffer of at least groups * 256 floats; its values mean nothing).  Timing the launch gives the
 * matrix-core rate the chip sustains at the clock it holds under MFMA load, beside the dense
 * bf16 peak that the step's matrix-bound kernels are rated against.
 * eb_probe_mfma_bf16_flops returns the launch's flop count (2 * 32 * 32 * 16 per MFMA), or 0.0
 * for arguments the probe rejects.  groups in [1, 65536], iters in [1, 2^20], else
 * EB_ERR_INVALID and nothing is launched.
 * ------------------------------------------------------------------------------------- */
eb_status eb_probe_mfma_bf16(float* out, int32_t groups, int32_t iters, eb_stream_t stream);
double eb_probe_mfma_bf16_flops(int32_t groups, int32_t iters);

/* ---------------------------------------------------------------------------------------
 * Diagnostics.
 * ------------------------------------------------------------------------------------- */
const char* eb_status_string(eb_status s); /* static string */
const char* eb_last_error(void);           /* per-thread; "" if none; valid until next call */
const char* eb_version(void);              /* static string */

#ifdef __cplusplus
}
#endif

#endif /* EB_H_ */
