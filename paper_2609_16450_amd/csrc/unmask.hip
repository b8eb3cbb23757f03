// Segmented threshold unmask with the anti-stall fallback, one workgroup per block.
//
// For block b: rows passing (masked && conf >= tau_b) are committed; if none passes and a row
// is still masked, the masked row of largest conf (lowest row on ties) is committed.  A commit
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

// Unmask of block b by one workgroup of kThreads threads.
__device__ __forceinline__ void unmask_block(
    int b, const int32_t* __restrict__ cu_block, const float* __restrict__ conf,
    const int32_t* __restrict__ argmax, const float* __restrict__ tau,
    uint8_t* __restrict__ masked,
    int32_t* __restrict__ tokens, uint8_t* __restrict__ unmask, int32_t* __restrict__ n_commit,
    uint8_t* __restrict__ resolved) {
  __shared__ int s_pass[kThreads / 64], s_masked[kThreads / 64];
  __shared__ Best s_best[kThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int beg = cu_block[b], end = cu_block[b + 1];
  const float tb = tau[b];

  int n_pass = 0, n_masked = 0;
  Best best{-INFINITY, kNoIndex};
  for (int i = beg + tid; i < end; i += kThreads) {
    if (masked[i]) {
      const float c = conf[i];
      ++n_masked;
      n_pass += (c >= tb) ? 1 : 0;
      if (c > best.c) best = Best{c, i};  // rows ascend per thread: strict > keeps the lowest
    }
  }
  for (int mask = 32; mask >= 1; mask >>= 1) {
    n_pass += __shfl_xor(n_pass, mask);
    n_masked += __shfl_xor(n_masked, mask);
    Best o{__shfl_xor(best.c, mask), __shfl_xor(best.i, mask)};
    best = best_of(best, o);
  }
  if (lane == 0) {
    s_pass[wave] = n_pass;
    s_masked[wave] = n_masked;
    s_best[wave] = best;
  }
  __syncthreads();
  n_pass = 0;
  n_masked = 0;
  best = Best{-INFINITY, kNoIndex};
  for (int k = 0; k < kThreads / 64; ++k) {
    n_pass += s_pass[k];
    n_masked += s_masked[k];
    best = best_of(best, s_best[k]);
  }

  const bool use_threshold = n_pass > 0;
  for (int i = beg + tid; i < end; i += kThreads) {
    bool take = false;
    if (masked[i]) take = use_threshold ? (conf[i] >= tb) : (i == best.i);
    unmask[i] = take ? 1 : 0;
    if (take) {
      tokens[i] = argmax[i];
      masked[i] = 0;
    }
  }
  if (tid == 0) {
    const int commits = use_threshold ? n_pass : (n_masked > 0 ? 1 : 0);
    n_commit[b] = commits;
    resolved[b] = (n_masked - commits == 0) ? 1 : 0;
  }
}

__global__ __launch_bounds__(kThreads) void unmask_kernel(
    const int32_t* __restrict__ cu_block, const float* __restrict__ conf,
    const int32_t* __restrict__ argmax, const float* __restrict__ tau,
    uint8_t* __restrict__ masked, int32_t* __restrict__ tokens, uint8_t* __restrict__ unmask,
    int32_t* __restrict__ n_commit, uint8_t* __restrict__ resolved) {
  unmask_block(blockIdx.x, cu_block, conf, argmax, tau, masked, tokens, unmask, n_commit,
               resolved);
}

}  // namespace

hipError_t unmask_select(int batch, int max_block, const int32_t* cu_block, const float* conf,
                         const int32_t* argmax, const float* tau, uint8_t* masked,
                         int32_t* tokens, uint8_t* unmask, int32_t* n_commit, uint8_t* resolved,
                         hipStream_t s) {
  (void)max_block;
  hipLaunchKernelGGL(unmask_kernel, dim3(batch), dim3(kThreads), 0, s, cu_block, conf, argmax,
                     tau, masked, tokens, unmask, n_commit, resolved);
  return hipGetLastError();
}

}  // namespace eb
