// Segmented unmask with the anti-stall fallback, one workgroup per block, and the LPS feature
// rows of each block.
//
// For block b: masked rows passing the accept rule are committed; if none passes and a row is
// still masked, the masked row of largest conf (lowest row on ties) is committed.  A commit
// writes the top-1 token and clears the mask flag.
#include "eb_common.hpp"
#include "eb_internal.hpp"

namespace eb {
namespace {

constexpr int kThreads = 256;

struct Best {
  float c;
  int32_t i;
};

// Larger conf wins; equal conf -> lower row.  Symmetric, so both butterfly lanes agree.
__device__ __forceinline__ Best best_of(Best a, Best b) {
  if (a.c > b.c) return a;
  if (b.c > a.c) return b;
  return a.i <= b.i ? a : b;
}

// Accept rules of one block step:
//   kThreshold: conf >= tau_b (Eq. prelim-update, threshold branch);
//   kUnion:     conf >= tau_b or p_psi > tau_psi (Alg. 5, union accept rule);
//   kTopM:      conf >= tau_b or the row is among the m most confident masked rows of the block
//               (Eq. prelim-update with a budget; equal conf: lower row first).
// Masked rows only.  When no masked row passes, the masked row of largest conf (lowest row on
// ties) is committed (Alg. 5, anti-stall fallback).
enum Rule { kThreshold = 0, kUnion = 1, kTopM = 2 };

struct RuleArgs {
  const float* p_psi;
  float tau_psi;
  int m;
};

constexpr int kRankTile = 2048;  // rows of a block staged in LDS per pass of the rank count

// Number of masked rows of [beg, end) that rank above row i (larger conf, or equal conf and a
// lower row), computed over LDS tiles of the block; every thread of the workgroup must call it
// the same number of times.  Rows i < 0 return 0.
__device__ __forceinline__ void rank_rows(int beg, int end, const float* __restrict__ conf,
                                          const uint8_t* __restrict__ masked, int i0,
                                          int (&rank)[4], int n_own) {
  __shared__ float s_conf[kRankTile];
  __shared__ uint8_t s_mask[kRankTile];
  float ci[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    rank[k] = 0;
    const int i = i0 + k * kThreads;
    ci[k] = (k < n_own && i < end) ? conf[i] : 0.f;
  }
  for (int t0 = beg; t0 < end; t0 += kRankTile) {
    const int tn = min(kRankTile, end - t0);
    __syncthreads();
    for (int j = threadIdx.x; j < tn; j += kThreads) {
      s_conf[j] = conf[t0 + j];
      s_mask[j] = masked[t0 + j];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int i = i0 + k * kThreads;
      if (k >= n_own || i >= end) continue;
      int r = 0;
      for (int j = 0; j < tn; ++j) {
        const float cj = s_conf[j];
        r += (s_mask[j] && (cj > ci[k] || (cj == ci[k] && t0 + j < i))) ? 1 : 0;
      }
      rank[k] += r;
    }
  }
}

// Step of block b by one workgroup of kThreads threads under rule R.
template <Rule R>
__device__ __forceinline__ void unmask_block(
    int b, const int32_t* __restrict__ cu_block, const float* __restrict__ conf,
    const int32_t* __restrict__ argmax, const float* __restrict__ tau, RuleArgs ra,
    uint8_t* __restrict__ masked,
    int32_t* __restrict__ tokens, uint8_t* __restrict__ unmask, int32_t* __restrict__ n_commit,
    uint8_t* __restrict__ resolved) {
  __shared__ int s_pass[kThreads / 64], s_masked[kThreads / 64];
  __shared__ Best s_best[kThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int beg = cu_block[b], end = cu_block[b + 1];
  const float tb = tau[b];

  // masked-row count first (the top-m rule needs it to skip the rank count)
  int n_masked = 0;
  Best best{-INFINITY, kNoIndex};
  for (int i = beg + tid; i < end; i += kThreads) {
    if (masked[i]) {
      const float c = conf[i];
      ++n_masked;
      if (c > best.c) best = Best{c, i};  // rows ascend per thread: strict > keeps the lowest
    }
  }
  for (int mask = 32; mask >= 1; mask >>= 1) {
    n_masked += __shfl_xor(n_masked, mask);
    Best o{__shfl_xor(best.c, mask), __shfl_xor(best.i, mask)};
    best = best_of(best, o);
  }
  if (lane == 0) {
    s_masked[wave] = n_masked;
    s_best[wave] = best;
  }
  __syncthreads();
  n_masked = 0;
  best = Best{-INFINITY, kNoIndex};
  for (int k = 0; k < kThreads / 64; ++k) {
    n_masked += s_masked[k];
    best = best_of(best, s_best[k]);
  }

  // Rows this thread owns: beg + tid + k * kThreads.  The top-m rule ranks them when needed
  // (blocks of up to 4 * kThreads rows go through the LDS rank count; longer blocks in rounds).
  auto passes = [&](int i, int rank) -> bool {
    if (!masked[i]) return false;
    const float c = conf[i];
    if (c >= tb) return true;
    if constexpr (R == kUnion) return ra.p_psi[i] > ra.tau_psi;
    if constexpr (R == kTopM) return rank < ra.m;
    return false;
  };
  const bool rank_all = (R == kTopM) && ra.m > 0 && ra.m < n_masked;
  const bool all_topm = (R == kTopM) && ra.m >= n_masked;
  // pass 1: count passing rows
  int n_pass = 0;
  for (int r0 = beg; r0 < end; r0 += 4 * kThreads) {
    int rank[4] = {0, 0, 0, 0};
    if (rank_all) rank_rows(beg, end, conf, masked, r0 + tid, rank, 4);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int i = r0 + tid + k * kThreads;
      if (i < end && (passes(i, all_topm ? 0 : (rank_all ? rank[k] : 1 << 30))))
        ++n_pass;
    }
  }
  for (int mask = 32; mask >= 1; mask >>= 1) n_pass += __shfl_xor(n_pass, mask);
  __syncthreads();
  if (lane == 0) s_pass[wave] = n_pass;
  __syncthreads();
  n_pass = 0;
  for (int k = 0; k < kThreads / 64; ++k) n_pass += s_pass[k];

  // pass 2: decide every row (ranks recomputed from the unchanged mask flags) into `unmask`,
  // then commit the decided rows once the whole block is decided
  const bool use_rule = n_pass > 0;
  for (int r0 = beg; r0 < end; r0 += 4 * kThreads) {
    int rank[4] = {0, 0, 0, 0};
    if (rank_all && use_rule) rank_rows(beg, end, conf, masked, r0 + tid, rank, 4);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int i = r0 + tid + k * kThreads;
      if (i >= end) continue;
      const bool take = use_rule ? passes(i, all_topm ? 0 : (rank_all ? rank[k] : 1 << 30))
                                 : (masked[i] && i == best.i);
      unmask[i] = take ? 1 : 0;
    }
  }
  __syncthreads();  // every decision is made before any mask flag changes
  for (int i = beg + tid; i < end; i += kThreads) {
    if (unmask[i]) {
      tokens[i] = argmax[i];
      masked[i] = 0;
    }
  }
  if (tid == 0) {
    const int commits = use_rule ? n_pass : (n_masked > 0 ? 1 : 0);
    n_commit[b] = commits;
    resolved[b] = (n_masked - commits == 0) ? 1 : 0;
  }
}

template <Rule R>
__global__ __launch_bounds__(kThreads) void unmask_kernel(
    const int32_t* __restrict__ cu_block, const float* __restrict__ conf,
    const int32_t* __restrict__ argmax, const float* __restrict__ tau, RuleArgs ra,
    uint8_t* __restrict__ masked, int32_t* __restrict__ tokens, uint8_t* __restrict__ unmask,
    int32_t* __restrict__ n_commit, uint8_t* __restrict__ resolved) {
  unmask_block<R>(blockIdx.x, cu_block, conf, argmax, tau, ra, masked, tokens, unmask, n_commit,
                  resolved);
}

// LPS router inputs (Sec. 5.2, Alg. 5), one workgroup per block: the block's mask ratio rho
// before this step's commit, then per row feat = (kappa, H * inv_ln_v, Delta, rho) and
// pos = (i - b0) / len.
__global__ __launch_bounds__(kThreads) void lps_features_kernel(
    const int32_t* __restrict__ cu_block, float inv_ln_v, const float* __restrict__ conf,
    const float* __restrict__ entropy, const float* __restrict__ gap,
    const uint8_t* __restrict__ masked, float* __restrict__ feat, float* __restrict__ pos,
    float* __restrict__ mask_ratio) {
  __shared__ int s_cnt[kThreads / 64];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int beg = cu_block[b], end = cu_block[b + 1], len = end - beg;
  int cnt = 0;
  for (int i = beg + tid; i < end; i += kThreads) cnt += masked[i] ? 1 : 0;
  for (int mask = 32; mask >= 1; mask >>= 1) cnt += __shfl_xor(cnt, mask);
  if (lane == 0) s_cnt[wave] = cnt;
  __syncthreads();
  cnt = 0;
  for (int k = 0; k < kThreads / 64; ++k) cnt += s_cnt[k];
  const float rho = len > 0 ? static_cast<float>(cnt) / static_cast<float>(len) : 0.f;
  if (tid == 0 && mask_ratio) mask_ratio[b] = rho;
  for (int i = beg + tid; i < end; i += kThreads) {
    *reinterpret_cast<f32x4*>(feat + 4 * static_cast<size_t>(i)) =
        f32x4{conf[i], entropy[i] * inv_ln_v, gap[i], rho};
    pos[i] = static_cast<float>(i - beg) / static_cast<float>(len);
  }
}

}  // namespace

hipError_t unmask_select(int batch, int max_block, const int32_t* cu_block, const float* conf,
                         const int32_t* argmax, const float* tau, uint8_t* masked,
                         int32_t* tokens, uint8_t* unmask, int32_t* n_commit, uint8_t* resolved,
                         hipStream_t s) {
  (void)max_block;
  const RuleArgs ra{nullptr, 0.f, 0};
  hipLaunchKernelGGL(unmask_kernel<kThreshold>, dim3(batch), dim3(kThreads), 0, s, cu_block,
                     conf, argmax, tau, ra, masked, tokens, unmask, n_commit, resolved);
  return hipGetLastError();
}

hipError_t unmask_select_lps(int batch, const int32_t* cu_block, const float* conf,
                             const int32_t* argmax, const float* tau, const float* p_psi,
                             float tau_psi, uint8_t* masked, int32_t* tokens, uint8_t* unmask,
                             int32_t* n_commit, uint8_t* resolved, hipStream_t s) {
  const RuleArgs ra{p_psi, tau_psi, 0};
  hipLaunchKernelGGL(unmask_kernel<kUnion>, dim3(batch), dim3(kThreads), 0, s, cu_block, conf,
                     argmax, tau, ra, masked, tokens, unmask, n_commit, resolved);
  return hipGetLastError();
}

hipError_t unmask_select_topm(int batch, const int32_t* cu_block, const float* conf,
                              const int32_t* argmax, const float* tau, int m, uint8_t* masked,
                              int32_t* tokens, uint8_t* unmask, int32_t* n_commit,
                              uint8_t* resolved, hipStream_t s) {
  const RuleArgs ra{nullptr, 0.f, m};
  hipLaunchKernelGGL(unmask_kernel<kTopM>, dim3(batch), dim3(kThreads), 0, s, cu_block, conf,
                     argmax, tau, ra, masked, tokens, unmask, n_commit, resolved);
  return hipGetLastError();
}

hipError_t lps_features(int batch, const int32_t* cu_block, int vocab, const float* conf,
                        const float* entropy, const float* gap, const uint8_t* masked,
                        float* feat, float* pos, float* mask_ratio, hipStream_t s) {
  const float inv_ln_v = static_cast<float>(1.0 / log(static_cast<double>(vocab)));
  hipLaunchKernelGGL(lps_features_kernel, dim3(batch), dim3(kThreads), 0, s, cu_block, inv_ln_v,
                     conf, entropy, gap, masked, feat, pos, mask_ratio);
  return hipGetLastError();
}

}  // namespace eb
