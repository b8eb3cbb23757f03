// One block step of the unmask rules, shared by the unmask kernels and the fused step epilogue.
//
// For block b: masked rows passing the accept rule are committed; if none passes and a row is
// still masked, the masked row of largest conf (lowest row on ties) is committed.  A commit
// writes the top-1 token and clears the mask flag.
#pragma once

#include "eb_common.hpp"

namespace eb {
namespace {

constexpr int kUnmaskThreads = 256;  // threads of a workgroup running unmask_block

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
    const int i = i0 + k * kUnmaskThreads;
    ci[k] = (k < n_own && i < end) ? conf[i] : 0.f;
  }
  for (int t0 = beg; t0 < end; t0 += kRankTile) {
    const int tn = min(kRankTile, end - t0);
    __syncthreads();
    for (int j = threadIdx.x; j < tn; j += kUnmaskThreads) {
      s_conf[j] = conf[t0 + j];
      s_mask[j] = masked[t0 + j];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int i = i0 + k * kUnmaskThreads;
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

// Block step of a block of at most 64 rows by one wavefront (the commit, fallback and tie-break
// of unmask_block): lane l holds row `row` (valid when `mine`), its mask flag m, its conf c, its
// top-1 token x, and whether it passes the accept rule.
__device__ __forceinline__ void unmask_wave(int b, int row, bool mine, bool m, float c, int32_t x,
                                            bool pass, uint8_t* __restrict__ masked,
                                            int32_t* __restrict__ tokens,
                                            uint8_t* __restrict__ unmask,
                                            int32_t* __restrict__ n_commit,
                                            uint8_t* __restrict__ resolved, int lane) {
  const bool mk = mine && m;
  int n_masked = mk ? 1 : 0;
  int n_pass = (mk && pass) ? 1 : 0;
  Best best = mk ? Best{c, row} : Best{-INFINITY, kNoIndex};
  for (int mask = 32; mask >= 1; mask >>= 1) {
    n_masked += __shfl_xor(n_masked, mask);
    n_pass += __shfl_xor(n_pass, mask);
    Best o{__shfl_xor(best.c, mask), __shfl_xor(best.i, mask)};
    best = best_of(best, o);
  }
  const bool use_rule = n_pass > 0;
  if (mine) {
    const bool take = mk && (use_rule ? pass : row == best.i);
    unmask[row] = take ? 1 : 0;
    if (take) {
      tokens[row] = x;
      masked[row] = 0;
    }
  }
  if (lane == 0) {
    const int commits = use_rule ? n_pass : (n_masked > 0 ? 1 : 0);
    n_commit[b] = commits;
    resolved[b] = (n_masked - commits == 0) ? 1 : 0;
  }
}

// Step of block b by one workgroup of kThreads threads under rule R (the top-m rank count runs
// on kUnmaskThreads threads).
template <Rule R, int kThreads = kUnmaskThreads>
__device__ __forceinline__ void unmask_block(
    int b, const int32_t* __restrict__ cu_block, const float* __restrict__ conf,
    const int32_t* __restrict__ argmax, const float* __restrict__ tau, RuleArgs ra,
    uint8_t* __restrict__ masked,
    int32_t* __restrict__ tokens, uint8_t* __restrict__ unmask, int32_t* __restrict__ n_commit,
    uint8_t* __restrict__ resolved) {
  static_assert(R != kTopM || kThreads == kUnmaskThreads, "rank_rows assumes kUnmaskThreads");
  __shared__ int s_pass[kThreads / 64], s_masked[kThreads / 64];
  __shared__ Best s_best[kThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int beg = cu_block[b], end = cu_block[b + 1];
  const float tb = tau[b];

  if constexpr (R != kTopM) {
    if (end - beg <= 64) {  // one wavefront: no reduction across waves, no barrier
      if (wave == 0) {
        const int i = beg + lane;
        const bool mine = i < end;
        const bool m = mine && masked[i];
        const float c = mine ? conf[i] : 0.f;
        const int32_t x = mine ? argmax[i] : 0;
        bool pass = c >= tb;
        if constexpr (R == kUnion) pass = pass || (mine && ra.p_psi[i] > ra.tau_psi);
        unmask_wave(b, i, mine, m, c, x, pass, masked, tokens, unmask, n_commit, resolved, lane);
      }
      return;
    }
    // One pass counts the masked rows, finds the best masked row and counts the rows passing
    // the rule.  Each thread then decides and commits its own rows: the rule reads no other
    // row's mask flag, so a row is committed as soon as it is decided.
    int n_masked = 0, n_pass = 0;
    Best best{-INFINITY, kNoIndex};
    for (int i = beg + tid; i < end; i += kThreads) {
      if (masked[i]) {
        const float c = conf[i];
        ++n_masked;
        if (c > best.c) best = Best{c, i};  // rows ascend per thread: strict > keeps the lowest
        bool ok = c >= tb;
        if constexpr (R == kUnion) ok = ok || ra.p_psi[i] > ra.tau_psi;
        n_pass += ok ? 1 : 0;
      }
    }
    for (int mask = 32; mask >= 1; mask >>= 1) {
      n_masked += __shfl_xor(n_masked, mask);
      n_pass += __shfl_xor(n_pass, mask);
      Best o{__shfl_xor(best.c, mask), __shfl_xor(best.i, mask)};
      best = best_of(best, o);
    }
    if (lane == 0) {
      s_masked[wave] = n_masked;
      s_pass[wave] = n_pass;
      s_best[wave] = best;
    }
    __syncthreads();
    n_masked = 0;
    n_pass = 0;
    best = Best{-INFINITY, kNoIndex};
    for (int k = 0; k < kThreads / 64; ++k) {
      n_masked += s_masked[k];
      n_pass += s_pass[k];
      best = best_of(best, s_best[k]);
    }
    const bool use_rule = n_pass > 0;
    for (int i = beg + tid; i < end; i += kThreads) {
      bool take = false;
      if (masked[i]) {
        if (use_rule) {
          take = conf[i] >= tb;
          if constexpr (R == kUnion) take = take || ra.p_psi[i] > ra.tau_psi;
        } else {
          take = i == best.i;
        }
      }
      unmask[i] = take ? 1 : 0;
      if (take) {
        tokens[i] = argmax[i];
        masked[i] = 0;
      }
    }
    if (tid == 0) {
      const int commits = use_rule ? n_pass : (n_masked > 0 ? 1 : 0);
      n_commit[b] = commits;
      resolved[b] = (n_masked - commits == 0) ? 1 : 0;
    }
    return;
  }

  // Top-m: the masked-row count first (it decides whether the rank count is needed)
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

}  // namespace
}  // namespace eb
