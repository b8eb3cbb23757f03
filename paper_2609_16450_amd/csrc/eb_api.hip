// C ABI of libeb.so: argument checks, workspace sizing, error reporting, step composition.
// The declarations and the contract of every entry point are in include/eb.h.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <string>
#include <vector>

#include "../../include/eb.h"
#include "eb_internal.hpp"

namespace {

thread_local std::string g_last_error;

eb_status fail(eb_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
eb_status fail(eb_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

eb_status ok() {
  g_last_error.clear();
  return EB_OK;
}

eb_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(EB_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr size_t kWsAlign = 256;
constexpr int kProbeMaxGroups = 65536;
constexpr int kProbeMaxIters = 1 << 20;
size_t round_up(size_t n) { return (n + kWsAlign - 1) / kWsAlign * kWsAlign; }

eb_status check_ragged(const eb_ragged* r, bool need_prefix) {
  if (!r) return fail(EB_ERR_INVALID, "ragged descriptor is NULL");
  if (r->batch < 1) return fail(EB_ERR_INVALID, "batch must be >= 1 (got %d)", r->batch);
  if (r->total_block < 0 || r->max_block < 0 || r->max_block > r->total_block)
    return fail(EB_ERR_INVALID, "bad block totals (total_block %d, max_block %d)",
                r->total_block, r->max_block);
  if (r->total_block > 0 && r->max_block == 0)
    return fail(EB_ERR_INVALID, "max_block is 0 but total_block is %d", r->total_block);
  if (!r->cu_block) return fail(EB_ERR_INVALID, "cu_block is NULL");
  if (need_prefix) {
    if (r->total_prefix < 0 || r->max_prefix < 0 || r->max_prefix > r->total_prefix)
      return fail(EB_ERR_INVALID, "bad prefix totals (total_prefix %d, max_prefix %d)",
                  r->total_prefix, r->max_prefix);
    if (!r->cu_prefix) return fail(EB_ERR_INVALID, "cu_prefix is NULL");
  }
  return EB_OK;
}

// The attention scale: 0 selects 1 / sqrt(head_dim), computed here in fp32 for every entry point
// (so that eb_block_attn and eb_decode_step use the same bits).
float attn_scale_or_default(float scale, int head_dim) {
  return scale == 0.f && head_dim > 0 ? 1.0f / sqrtf(static_cast<float>(head_dim)) : scale;
}

eb_status check_attn(eb_dtype dt, const eb_ragged* r, int hq, int hkv, int head_dim, float scale,
                     const void* q, const void* k_blk, const void* v_blk, const void* k_pre,
                     const void* v_pre, const void* out) {
  if (dt != EB_F32 && dt != EB_BF16) return fail(EB_ERR_INVALID, "unknown dtype %d", (int)dt);
  eb_status st = check_ragged(r, true);
  if (st != EB_OK) return st;
  if (hq < 1 || hkv < 1 || hq % hkv)
    return fail(EB_ERR_INVALID, "need hq, hkv >= 1 and hq %% hkv == 0 (hq %d, hkv %d)", hq, hkv);
  if (head_dim < 1) return fail(EB_ERR_INVALID, "head_dim must be >= 1 (got %d)", head_dim);
  if (!(scale > 0.f) || !isfinite(scale))
    return fail(EB_ERR_INVALID, "scale must be finite and > 0");
  if (head_dim != 64 && head_dim != 128)
    return fail(EB_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", head_dim);
  if (r->total_block > 0 && (!q || !k_blk || !v_blk || !out))
    return fail(EB_ERR_INVALID, "NULL q / k_blk / v_blk / out");
  if (r->total_prefix > 0 && (!k_pre || !v_pre))
    return fail(EB_ERR_INVALID, "NULL k_pre / v_pre with total_prefix > 0");
  if (dt == EB_BF16) {
    const void* ps[] = {q, k_blk, v_blk, k_pre, v_pre, out};
    for (const void* p : ps)
      if (p && !aligned16(p)) return fail(EB_ERR_INVALID, "bf16 tensors must be 16-byte aligned");
  }
  return EB_OK;
}

eb_status check_lmhead(eb_dtype dt, int n_rows, int hidden, int vocab, const void* h,
                       const void* w, const void* conf, const void* entropy,
                       const void* argmax) {
  if (dt != EB_F32 && dt != EB_BF16) return fail(EB_ERR_INVALID, "unknown dtype %d", (int)dt);
  if (n_rows < 0 || hidden < 1 || vocab < 1)
    return fail(EB_ERR_INVALID, "need n_rows >= 0, hidden >= 1, vocab >= 1 (got %d, %d, %d)",
                n_rows, hidden, vocab);
  if (dt == EB_BF16 && hidden % 64)
    return fail(EB_ERR_UNSUPPORTED, "bf16 LM head needs hidden %% 64 == 0 (got %d)", hidden);
  if (n_rows > 0 && (!h || !w || !conf || !entropy || !argmax))
    return fail(EB_ERR_INVALID, "NULL h / w / conf / entropy / argmax");
  if (dt == EB_BF16 && n_rows > 0 && (!aligned16(h) || !aligned16(w)))
    return fail(EB_ERR_INVALID, "bf16 tensors must be 16-byte aligned");
  return EB_OK;
}

eb_status check_unmask(const eb_ragged* r, const void* conf, const void* argmax, const void* tau,
                       const void* masked, const void* tokens, const void* unmask,
                       const void* n_commit, const void* resolved) {
  eb_status st = check_ragged(r, false);
  if (st != EB_OK) return st;
  if (!tau || !n_commit || !resolved) return fail(EB_ERR_INVALID, "NULL tau / n_commit / resolved");
  if (r->total_block > 0 && (!conf || !argmax || !masked || !tokens || !unmask))
    return fail(EB_ERR_INVALID, "NULL conf / argmax / masked / tokens / unmask");
  return EB_OK;
}

// ---- optional checks of the device-array contract --------------------------------------
// With the environment variable EB_DEBUG_CHECKS set (to anything but "0"), an entry point copies
// its offset arrays (and tau) to the host after the work already on `stream`, and returns
// EB_ERR_INVALID, launching nothing, when they break the contract stated in eb.h.  The copy
// synchronises the stream, so these checks are for debugging, not for captured or timed code.
bool debug_checks() {
  const char* v = getenv("EB_DEBUG_CHECKS");
  return v && *v && strcmp(v, "0") != 0;
}

template <class T>
eb_status fetch(std::vector<T>& h, const T* d, int n, hipStream_t s) {
  h.resize(n);
  hipError_t e = hipMemcpyAsync(h.data(), d, sizeof(T) * n, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  return e == hipSuccess ? EB_OK : fail(EB_ERR_HIP, "debug check copy: %s", hipGetErrorString(e));
}

// cu [batch + 1]: starts at 0, non-decreasing, ends at `total`, largest step `max`.
eb_status check_cu(const char* name, const int32_t* cu, int batch, int total, int max,
                   hipStream_t s) {
  std::vector<int32_t> h;
  eb_status st = fetch(h, cu, batch + 1, s);
  if (st != EB_OK) return st;
  if (h[0] != 0) return fail(EB_ERR_INVALID, "%s[0] = %d, expected 0", name, h[0]);
  int mx = 0;
  for (int b = 0; b < batch; ++b) {
    if (h[b + 1] < h[b])
      return fail(EB_ERR_INVALID, "%s decreases at %d (%d -> %d)", name, b, h[b], h[b + 1]);
    mx = h[b + 1] - h[b] > mx ? h[b + 1] - h[b] : mx;
  }
  if (h[batch] != total)
    return fail(EB_ERR_INVALID, "%s[%d] = %d but the host total is %d", name, batch, h[batch],
                total);
  if (mx != max)
    return fail(EB_ERR_INVALID, "largest %s step is %d but the host maximum is %d", name, mx, max);
  return EB_OK;
}

eb_status check_tau(const float* tau, int batch, hipStream_t s) {
  std::vector<float> h;
  eb_status st = fetch(h, tau, batch, s);
  if (st != EB_OK) return st;
  for (int b = 0; b < batch; ++b)
    if (!(h[b] > 0.f && h[b] <= 1.f))
      return fail(EB_ERR_INVALID, "tau[%d] = %g is not in (0, 1]", b, (double)h[b]);
  return EB_OK;
}

// The ragged descriptor's arrays (cu_prefix too when need_prefix) and, when given, tau.
eb_status check_device(const eb_ragged* r, bool need_prefix, const float* tau, hipStream_t s) {
  if (!debug_checks()) return EB_OK;
  eb_status st = check_cu("cu_block", r->cu_block, r->batch, r->total_block, r->max_block, s);
  if (st == EB_OK && need_prefix)
    st = check_cu("cu_prefix", r->cu_prefix, r->batch, r->total_prefix, r->max_prefix, s);
  if (st == EB_OK && tau) st = check_tau(tau, r->batch, s);
  return st;
}

// ---------------------------------------------------------------------------------------
// Device scratch of eb_decode_step_noalloc.  The array exists once per device the library's
// code object is loaded on and lives until the process ends.  Host code never uses its name
// as an address (on the host it is only a stand-in for the symbol): the device address of each
// device's copy comes from hipGetSymbolAddress, taken once per device with that device current,
// and only that address is passed to kernels.
// ---------------------------------------------------------------------------------------
constexpr size_t kNoAllocScratchBytes = EB_NOALLOC_SCRATCH_BYTES;
static_assert(kNoAllocScratchBytes % 256 == 0, "scratch size is a multiple of the alignment");

}  // namespace

static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

namespace {

std::mutex g_scratch_mu;
std::vector<void*> g_scratch_addr;  // indexed by device ordinal; nullptr until looked up

// Device address of `scratch` on device `dev` (looked up on the first call for that device).
eb_status scratch_address(int dev, void** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (dev < 0) return fail(EB_ERR_INVALID, "bad device ordinal %d", dev);
  if (static_cast<size_t>(dev) >= g_scratch_addr.size()) g_scratch_addr.resize(dev + 1, nullptr);
  if (!g_scratch_addr[dev]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    void* p = nullptr;
    if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    const hipError_t e2 = (cur >= 0 && cur != dev) ? hipSetDevice(cur) : hipSuccess;
    if (e != hipSuccess) return hip_status(e, "scratch symbol lookup");
    if (e2 != hipSuccess) return hip_status(e2, "restoring the current device");
    if (!p) return fail(EB_ERR_HIP, "scratch symbol lookup returned NULL");
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return EB_OK;
}

}  // namespace

extern "C" {

const char* eb_status_string(eb_status s) {
  switch (s) {
    case EB_OK: return "EB_OK";
    case EB_ERR_INVALID: return "EB_ERR_INVALID";
    case EB_ERR_UNSUPPORTED: return "EB_ERR_UNSUPPORTED";
    case EB_ERR_WORKSPACE: return "EB_ERR_WORKSPACE";
    case EB_ERR_HIP: return "EB_ERR_HIP";
  }
  return "EB_ERR_UNKNOWN";
}

const char* eb_last_error(void) { return g_last_error.c_str(); }

const char* eb_version(void) { return "libeb 0.1 (gfx950)"; }

double eb_probe_mfma_bf16_flops(int32_t groups, int32_t iters) {
  if (groups < 1 || groups > kProbeMaxGroups || iters < 1 || iters > kProbeMaxIters) return 0.0;
  return eb::mfma_probe_flops(groups, iters);
}

eb_status eb_probe_mfma_bf16(float* out, int32_t groups, int32_t iters, eb_stream_t stream) {
  if (!out) return fail(EB_ERR_INVALID, "out is NULL");
  if (groups < 1 || groups > kProbeMaxGroups)
    return fail(EB_ERR_INVALID, "groups must be in [1, %d] (got %d)", kProbeMaxGroups, groups);
  if (iters < 1 || iters > kProbeMaxIters)
    return fail(EB_ERR_INVALID, "iters must be in [1, %d] (got %d)", kProbeMaxIters, iters);
  return hip_status(eb::mfma_probe(out, groups, iters, stream), "mfma probe launch");
}

size_t eb_block_attn_workspace(eb_dtype dt, const eb_ragged* r, int hq, int hkv, int head_dim) {
  if (!r || r->batch < 1 || hq < 1 || hkv < 1 || hq % hkv || r->total_block <= 0) return 0;
  return round_up(eb::block_attn_ws_bytes(dt == EB_BF16, true, r->batch, r->total_block,
                                          r->max_block, r->max_prefix + r->max_block, hq, hkv,
                                          head_dim));
}

eb_status eb_block_attn(eb_dtype dt, const eb_ragged* r, int hq, int hkv, int head_dim,
                        float scale, const void* q, const void* k_blk, const void* v_blk,
                        const void* k_pre, const void* v_pre, void* out, void* ws,
                        size_t ws_bytes, eb_stream_t stream) {
  scale = attn_scale_or_default(scale, head_dim);
  eb_status st = check_attn(dt, r, hq, hkv, head_dim, scale, q, k_blk, v_blk, k_pre, v_pre, out);
  if (st != EB_OK) return st;
  const size_t need = eb_block_attn_workspace(dt, r, hq, hkv, head_dim);
  if (ws_bytes < need || (need && !ws))
    return fail(EB_ERR_WORKSPACE, "attention workspace %zu bytes < required %zu", ws_bytes, need);
  st = check_device(r, true, nullptr, stream);
  if (st != EB_OK) return st;
  eb::AttnArgs a{r->batch, r->total_block, r->max_block, r->total_prefix, r->max_prefix,
                 r->cu_block, r->cu_prefix, hq, hkv, head_dim, scale, q, k_blk, v_blk,
                 k_pre, v_pre, out};
  return hip_status(eb::block_attn(dt == EB_BF16, true, a, ws, stream), "eb_block_attn launch");
}

size_t eb_block_attn_dual_workspace(eb_dtype dt, const eb_ragged* r, const eb_suffix* sfx, int hq,
                                    int hkv, int head_dim) {
  if (!r || !sfx || r->batch < 1 || hq < 1 || hkv < 1 || hq % hkv || r->total_block <= 0 ||
      sfx->max_suffix < 0)
    return 0;
  return round_up(eb::block_attn_ws_bytes(dt == EB_BF16, true, r->batch, r->total_block,
                                          r->max_block,
                                          r->max_prefix + r->max_block + sfx->max_suffix, hq,
                                          hkv, head_dim));
}

eb_status eb_block_attn_dual(eb_dtype dt, const eb_ragged* r, const eb_suffix* sfx, int hq,
                             int hkv, int head_dim, float scale, const void* q, const void* k_blk,
                             const void* v_blk, const void* k_pre, const void* v_pre,
                             const void* k_suf, const void* v_suf, void* out, void* ws,
                             size_t ws_bytes, eb_stream_t stream) {
  scale = attn_scale_or_default(scale, head_dim);
  eb_status st = check_attn(dt, r, hq, hkv, head_dim, scale, q, k_blk, v_blk, k_pre, v_pre, out);
  if (st != EB_OK) return st;
  if (!sfx) return fail(EB_ERR_INVALID, "suffix descriptor is NULL");
  if (sfx->total_suffix < 0 || sfx->max_suffix < 0 || !sfx->cu_suffix)
    return fail(EB_ERR_INVALID, "need total_suffix, max_suffix >= 0 and cu_suffix");
  if (sfx->total_suffix > 0 && (!k_suf || !v_suf))
    return fail(EB_ERR_INVALID, "NULL k_suf / v_suf with total_suffix > 0");
  if (dt == EB_BF16 && ((k_suf && !aligned16(k_suf)) || (v_suf && !aligned16(v_suf))))
    return fail(EB_ERR_INVALID, "bf16 tensors must be 16-byte aligned");
  const size_t need = eb_block_attn_dual_workspace(dt, r, sfx, hq, hkv, head_dim);
  if (ws_bytes < need || (need && !ws))
    return fail(EB_ERR_WORKSPACE, "attention workspace %zu bytes < required %zu", ws_bytes, need);
  st = check_device(r, true, nullptr, stream);
  if (st == EB_OK && debug_checks())
    st = check_cu("cu_suffix", sfx->cu_suffix, r->batch, sfx->total_suffix, sfx->max_suffix,
                  stream);
  if (st != EB_OK) return st;
  eb::AttnArgs a{r->batch, r->total_block, r->max_block, r->total_prefix, r->max_prefix,
                 r->cu_block, r->cu_prefix, hq, hkv, head_dim, scale, q, k_blk, v_blk,
                 k_pre, v_pre, out, sfx->max_suffix, sfx->cu_suffix, k_suf, v_suf};
  return hip_status(eb::block_attn(dt == EB_BF16, true, a, ws, stream),
                    "eb_block_attn_dual launch");
}

size_t eb_lmhead_workspace(eb_dtype dt, int n_rows, int hidden, int vocab) {
  (void)hidden;
  if (n_rows <= 0 || vocab <= 0) return 0;
  return round_up(eb::lmhead_ws_bytes(dt == EB_BF16, n_rows, vocab, false));
}

size_t eb_lmhead_features_workspace(eb_dtype dt, int n_rows, int hidden, int vocab) {
  (void)hidden;
  if (n_rows <= 0 || vocab <= 0) return 0;
  return round_up(eb::lmhead_ws_bytes(dt == EB_BF16, n_rows, vocab, true));
}

namespace {
eb_status lmhead_run(eb_dtype dt, int n_rows, int hidden, int vocab, const void* h,
                     const void* w, float* conf, float* entropy_nats, int32_t* argmax,
                     float* max_logit, float* top2_gap, void* ws, size_t ws_bytes,
                     eb_stream_t stream) {
  eb_status st = check_lmhead(dt, n_rows, hidden, vocab, h, w, conf, entropy_nats, argmax);
  if (st != EB_OK) return st;
  const bool top2 = top2_gap != nullptr;
  const size_t need = top2 ? eb_lmhead_features_workspace(dt, n_rows, hidden, vocab)
                           : eb_lmhead_workspace(dt, n_rows, hidden, vocab);
  if (ws_bytes < need || (need && !ws))
    return fail(EB_ERR_WORKSPACE, "LM-head workspace %zu bytes < required %zu", ws_bytes, need);
  if (n_rows == 0) return ok();
  const bool bf16 = dt == EB_BF16;
  hipError_t e = eb::lmhead_partials(bf16, n_rows, hidden, vocab, h, w, ws, top2, stream);
  if (e != hipSuccess) return hip_status(e, "LM-head partial launch");
  e = eb::lmhead_combine(bf16, n_rows, vocab, ws, conf, entropy_nats, argmax, max_logit,
                         top2_gap, stream);
  return hip_status(e, "LM-head combine launch");
}
}  // namespace

eb_status eb_lmhead_confidence(eb_dtype dt, int n_rows, int hidden, int vocab, const void* h,
                               const void* w, float* conf, float* entropy_nats,
                               int32_t* argmax, float* max_logit, void* ws, size_t ws_bytes,
                               eb_stream_t stream) {
  return lmhead_run(dt, n_rows, hidden, vocab, h, w, conf, entropy_nats, argmax, max_logit,
                    nullptr, ws, ws_bytes, stream);
}

eb_status eb_lmhead_features(eb_dtype dt, int n_rows, int hidden, int vocab, const void* h,
                             const void* w, float* conf, float* entropy_nats, int32_t* argmax,
                             float* max_logit, float* top2_gap, void* ws, size_t ws_bytes,
                             eb_stream_t stream) {
  if (n_rows > 0 && !top2_gap) return fail(EB_ERR_INVALID, "NULL top2_gap");
  return lmhead_run(dt, n_rows, hidden, vocab, h, w, conf, entropy_nats, argmax, max_logit,
                    top2_gap, ws, ws_bytes, stream);
}

eb_status eb_lps_features(const eb_ragged* r, int vocab, const float* conf,
                          const float* entropy_nats, const float* top2_gap,
                          const uint8_t* masked, const int32_t* seq_pos, float* feat, float* pos,
                          float* mask_ratio, eb_stream_t stream) {
  eb_status st = check_ragged(r, false);
  if (st != EB_OK) return st;
  if (vocab < 2) return fail(EB_ERR_INVALID, "vocab must be >= 2 (got %d)", vocab);
  if (r->total_block > 0 && (!conf || !entropy_nats || !top2_gap || !masked || !feat || !pos))
    return fail(EB_ERR_INVALID, "NULL conf / entropy / top2_gap / masked / feat / pos");
  if (r->total_block > 0 && !aligned16(feat))
    return fail(EB_ERR_INVALID, "feat must be 16-byte aligned");
  st = check_device(r, false, nullptr, stream);
  if (st != EB_OK) return st;
  return hip_status(eb::lps_features(r->batch, r->cu_block, vocab, conf, entropy_nats, top2_gap,
                                     masked, seq_pos, feat, pos, mask_ratio, stream),
                    "eb_lps_features launch");
}

eb_status eb_unmask_select_lps(const eb_ragged* r, const float* conf, const int32_t* argmax,
                               const float* tau, const float* p_psi, float tau_psi,
                               uint8_t* masked, int32_t* tokens, uint8_t* unmask,
                               int32_t* n_commit, uint8_t* resolved, eb_stream_t stream) {
  eb_status st = check_unmask(r, conf, argmax, tau, masked, tokens, unmask, n_commit, resolved);
  if (st != EB_OK) return st;
  if (r->total_block > 0 && !p_psi) return fail(EB_ERR_INVALID, "NULL p_psi");
  st = check_device(r, false, tau, stream);
  if (st != EB_OK) return st;
  return hip_status(eb::unmask_select_lps(r->batch, r->cu_block, conf, argmax, tau, p_psi,
                                          tau_psi, masked, tokens, unmask, n_commit, resolved,
                                          stream),
                    "eb_unmask_select_lps launch");
}

eb_status eb_unmask_select_topm(const eb_ragged* r, const float* conf, const int32_t* argmax,
                                const float* tau, int32_t m, uint8_t* masked, int32_t* tokens,
                                uint8_t* unmask, int32_t* n_commit, uint8_t* resolved,
                                eb_stream_t stream) {
  eb_status st = check_unmask(r, conf, argmax, tau, masked, tokens, unmask, n_commit, resolved);
  if (st != EB_OK) return st;
  if (m < 0) return fail(EB_ERR_INVALID, "m must be >= 0 (got %d)", m);
  st = check_device(r, false, tau, stream);
  if (st != EB_OK) return st;
  return hip_status(eb::unmask_select_topm(r->batch, r->cu_block, conf, argmax, tau, m, masked,
                                           tokens, unmask, n_commit, resolved, stream),
                    "eb_unmask_select_topm launch");
}

eb_status eb_unmask_select(const eb_ragged* r, const float* conf, const int32_t* argmax,
                           const float* tau, uint8_t* masked, int32_t* tokens, uint8_t* unmask,
                           int32_t* n_commit, uint8_t* resolved, eb_stream_t stream) {
  eb_status st = check_unmask(r, conf, argmax, tau, masked, tokens, unmask, n_commit, resolved);
  if (st != EB_OK) return st;
  st = check_device(r, false, tau, stream);
  if (st != EB_OK) return st;
  return hip_status(eb::unmask_select(r->batch, r->max_block, r->cu_block, conf, argmax, tau,
                                      masked, tokens, unmask, n_commit, resolved, stream),
                    "eb_unmask_select launch");
}

eb_status eb_lbs_select(int32_t n_seq, int32_t window, const uint8_t* masked,
                        const float* p_phi, const int32_t* x_hat, int32_t eos_id, int32_t l_min,
                        int32_t l_b, int32_t g_max, uint8_t* block, int32_t* size,
                        int32_t* first, eb_stream_t stream) {
  if (n_seq < 0 || window < 0)
    return fail(EB_ERR_INVALID, "need n_seq, window >= 0 (got %d, %d)", n_seq, window);
  if (l_min < 0 || l_b < 0 || g_max < 1)
    return fail(EB_ERR_INVALID, "need l_min, l_b >= 0 and g_max >= 1 (got %d, %d, %d)", l_min,
                l_b, g_max);
  if (n_seq == 0) return ok();
  if (!size || !first) return fail(EB_ERR_INVALID, "NULL size / first");
  if (window > 0 && (!masked || !p_phi || !x_hat || !block))
    return fail(EB_ERR_INVALID, "NULL masked / p_phi / x_hat / block");
  return hip_status(eb::lbs_select(n_seq, window, masked, p_phi, x_hat, eos_id, l_min, l_b, g_max,
                                   block, size, first, stream),
                    "eb_lbs_select launch");
}

int32_t eb_decode_step_attn_in_lmhead(const eb_step_desc* d) {
  if (!d || d->hkv < 1 || d->hq < 1) return 0;
  const eb_ragged* r = &d->ragged;
  const bool bf16 = d->dtype == EB_BF16;
  const int T = r->total_block;
  eb::AttnArgs a{r->batch, T, r->max_block, r->total_prefix, r->max_prefix, r->cu_block,
                 r->cu_prefix, d->hq, d->hkv, d->head_dim, 1.0f, d->q, d->k_blk, d->v_blk,
                 d->k_pre, d->v_pre, d->attn_out};
  const int n_slices = T > 0 && d->vocab > 0 ? eb::lmhead_num_slices(bf16, T, d->vocab) : 0;
  return eb::step_finish_fusable(r->max_block, n_slices) &&
                 eb::lmhead_hosts_attn(bf16, T, d->vocab, a)
             ? 1
             : 0;
}

size_t eb_decode_step_workspace(const eb_step_desc* d) {
  if (!d) return 0;
  return eb_block_attn_workspace(d->dtype, &d->ragged, d->hq, d->hkv, d->head_dim) +
         eb_lmhead_workspace(d->dtype, d->ragged.total_block, d->hidden, d->vocab);
}

eb_status eb_decode_step(const eb_step_desc* d, void* ws, size_t ws_bytes, eb_stream_t stream) {
  if (!d) return fail(EB_ERR_INVALID, "step descriptor is NULL");
  const float scale = attn_scale_or_default(d->attn_scale > 0.f ? d->attn_scale : 0.f, d->head_dim);
  eb_status st = check_attn(d->dtype, &d->ragged, d->hq, d->hkv, d->head_dim, scale, d->q,
                            d->k_blk, d->v_blk, d->k_pre, d->v_pre, d->attn_out);
  if (st != EB_OK) return st;
  const int T = d->ragged.total_block;
  st = check_lmhead(d->dtype, T, d->hidden, d->vocab, d->h, d->w, d->conf, d->entropy_nats,
                    d->argmax);
  if (st != EB_OK) return st;
  st = check_unmask(&d->ragged, d->conf, d->argmax, d->tau, d->masked, d->tokens, d->unmask,
                    d->n_commit, d->resolved);
  if (st != EB_OK) return st;
  const size_t need = eb_decode_step_workspace(d);
  if (ws_bytes < need || (need && !ws))
    return fail(EB_ERR_WORKSPACE, "step workspace %zu bytes < required %zu", ws_bytes, need);
  st = check_device(&d->ragged, true, d->tau, stream);
  if (st != EB_OK) return st;

  const bool bf16 = d->dtype == EB_BF16;
  const eb_ragged* r = &d->ragged;
  const eb_step_trace* tr = d->trace;
  auto mark = [&](eb_event_t ev) -> hipError_t {
    return ev ? hipEventRecord(reinterpret_cast<hipEvent_t>(ev), stream) : hipSuccess;
  };
  eb::AttnArgs a{r->batch, r->total_block, r->max_block, r->total_prefix, r->max_prefix,
                 r->cu_block, r->cu_prefix, d->hq, d->hkv, d->head_dim, scale, d->q, d->k_blk,
                 d->v_blk, d->k_pre, d->v_pre, d->attn_out};
  const size_t attn_ws = eb_block_attn_workspace(d->dtype, r, d->hq, d->hkv, d->head_dim);
  char* lm_ws = static_cast<char*>(ws) + attn_ws;
  // One epilogue launch (attention split merge + row statistics + unmask) when one workgroup
  // can reduce a block's LM-head partials; otherwise the three kernels run one after another.
  const int n_slices = T > 0 ? eb::lmhead_num_slices(bf16, T, d->vocab) : 0;
  const bool fuse = eb::step_finish_fusable(r->max_block, n_slices);

  // Small steps: the attention's workgroups ride in the LM-head launch, behind its slices (its
  // split merge then happens in the epilogue, which is why this needs `fuse`).
  const bool hosted = eb_decode_step_attn_in_lmhead(d) != 0;

  hipError_t e = tr ? mark(tr->attn_begin) : hipSuccess;
  if (e == hipSuccess && !hosted) e = eb::block_attn(bf16, true, a, ws, stream, fuse);
  if (e == hipSuccess && tr) e = mark(tr->attn_end);
  if (e != hipSuccess) return hip_status(e, "step attention launch");

  if (tr) e = mark(tr->lmhead_begin);
  if (e == hipSuccess && hosted)
    e = eb::lmhead_partials_attn(T, d->hidden, d->vocab, d->h, d->w, lm_ws, a, ws, stream);
  else if (e == hipSuccess && T > 0)
    e = eb::lmhead_partials(bf16, T, d->hidden, d->vocab, d->h, d->w, lm_ws, false, stream);
  if (e == hipSuccess && tr) e = mark(tr->lmhead_end);
  if (e != hipSuccess) return hip_status(e, "step LM-head launch");
  if (tr) e = mark(tr->select_begin);
  if (fuse) {
    if (e == hipSuccess)
      e = eb::step_finish(bf16, a, ws, T, d->vocab, lm_ws, d->conf, d->entropy_nats, d->argmax,
                          d->max_logit, d->tau, d->masked, d->tokens, d->unmask, d->n_commit,
                          d->resolved, stream);
  } else {
    if (e == hipSuccess && T > 0)
      e = eb::lmhead_combine(bf16, T, d->vocab, lm_ws, d->conf, d->entropy_nats, d->argmax,
                             d->max_logit, nullptr, stream);
    if (e == hipSuccess)
      e = eb::unmask_select(r->batch, r->max_block, r->cu_block, d->conf, d->argmax, d->tau,
                            d->masked, d->tokens, d->unmask, d->n_commit, d->resolved, stream);
  }
  if (e == hipSuccess && tr) e = mark(tr->select_end);
  return hip_status(e, "step select launch");
}

eb_status eb_decode_step_noalloc(const eb_step_desc* d, eb_stream_t stream) {
  if (!d) return fail(EB_ERR_INVALID, "step descriptor is NULL");
  const size_t need = eb_decode_step_workspace(d);
  if (need > kNoAllocScratchBytes)
    return fail(EB_ERR_WORKSPACE,
                "step needs %zu bytes of scratch; eb_decode_step_noalloc holds %zu (use "
                "eb_decode_step with a caller workspace)",
                need, kNoAllocScratchBytes);
  int dev = -1;
  hipError_t e = stream ? hipStreamGetDevice(reinterpret_cast<hipStream_t>(stream), &dev)
                        : hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "device of the stream");
  void* ws = nullptr;
  const eb_status st = scratch_address(dev, &ws);
  if (st != EB_OK) return st;
  return eb_decode_step(d, ws, kNoAllocScratchBytes, stream);
}

}  // extern "C"
