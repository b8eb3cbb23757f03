// Fused epilogue of one decoding step (Alg. 5, one loop iteration, after the attention and the
// LM-head partials, which in small steps come from one launch): a single launch that
//   * merges the attention key-split partials of every (block row, query head) pair, and
//   * per block: merges each row's LM-head partials into conf, entropy, argmax and top logit
//     (Alg. 5, confidence of the softmax), then applies the threshold unmask with the
//     anti-stall fallback (Eq. prelim-update, Alg. 5).
// The two roles touch disjoint data, so they share one grid: workgroups [0, n_merge) merge
// attention pairs, the next `batch` workgroups each finish one block.  Each block's rows are
// reduced by the block's own workgroup, whose unmask step then reads them back after a barrier
// (a block of at most 64 rows: from LDS, by one wavefront), so no cross-workgroup ordering is
// needed.  The arithmetic is that of the separate kernels
// (same partial merge order, same row statistics, same block step), so the outputs are
// bit-identical to attention merge + combine + unmask launched one after another.
#include "attn_common.hpp"
#include "eb_common.hpp"
#include "eb_internal.hpp"
#include "unmask_block.hpp"

namespace eb {
namespace {

constexpr int kFinishThreads = 1024;  // 16 waves: the rows of a block spread over all four SIMDs

// D: attention head dimension of the merge role (unused when n_merge == 0).
template <int D>
__global__ __launch_bounds__(kFinishThreads) void step_finish_kernel(
    AttnParams ap, int total_block, int batch, int n_merge, const Partial* __restrict__ part,
    int n_slices, float* __restrict__ conf, float* __restrict__ entropy,
    int32_t* __restrict__ argmax, float* __restrict__ max_logit, const float* __restrict__ tau,
    uint8_t* __restrict__ masked, int32_t* __restrict__ tokens, uint8_t* __restrict__ unmask,
    int32_t* __restrict__ n_commit, uint8_t* __restrict__ resolved) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (static_cast<int>(blockIdx.x) < n_merge) {
    const int rh = blockIdx.x * (kFinishThreads / 64) + wave;
    if (rh < total_block * ap.hq) attn_merge_pair<D>(ap, rh, batch, lane);
    return;  // whole workgroup: the merge role has no barrier
  }
  const int b = blockIdx.x - n_merge;
  const int beg = ap.cu_block[b], end = ap.cu_block[b + 1];
  // A block of at most 64 rows also leaves its rows' conf and argmax in LDS, and wave 0 then runs
  // the block step alone (one barrier, no reduction across waves; its lanes read their rows' mask
  // flags up front).  Larger blocks run the workgroup-wide step.
  const bool small = end - beg <= 64;
  __shared__ float s_conf[64];
  __shared__ int32_t s_arg[64];
  const int own_row = beg + lane;
  const bool own_ok = small && wave == 0 && own_row < end;
  const uint8_t m_own = own_ok ? masked[own_row] : uint8_t{0};
  // Wave w reduces rows beg + w, beg + w + 16, ...; kRowBatch rows at a time with their loads in
  // flight together and their merges interleaved.  Each row is merged exactly as wave_merge does
  // it (lane-strided in index order, loads grouped by 4, an empty partial in place of a missing
  // one, then wave_finish).
  constexpr int kWaves = kFinishThreads / 64, kRowBatch = 2, kLoads = 4;
  for (int r0 = beg + wave; r0 < end; r0 += kWaves * kRowBatch) {
    Partial acc[kRowBatch];
#pragma unroll
    for (int i = 0; i < kRowBatch; ++i) acc[i] = partial_empty();
    for (int base = 0; base < n_slices; base += 64 * kLoads) {  // uniform trip count
      Partial q[kRowBatch][kLoads];
#pragma unroll
      for (int i = 0; i < kRowBatch; ++i) {
        const Partial* pr = part + static_cast<size_t>(min(r0 + kWaves * i, end - 1)) * n_slices;
#pragma unroll
        for (int j = 0; j < kLoads; ++j) q[i][j] = pr[min(base + 64 * j + lane, n_slices - 1)];
      }
#pragma unroll
      for (int j = 0; j < kLoads; ++j) {
        const bool ok = base + 64 * j + lane < n_slices;
#pragma unroll
        for (int i = 0; i < kRowBatch; ++i)
          acc[i] = partial_merge(acc[i], ok ? q[i][j] : partial_empty());
      }
    }
#pragma unroll
    for (int i = 0; i < kRowBatch; ++i) {
      const Partial p = wave_finish(acc[i]);
      const int row = r0 + kWaves * i;
      if (lane == 0 && row < end) {
        write_row_stats(p, row, conf, entropy, argmax, max_logit);
        if (small) {
          s_conf[row - beg] = 1.0f / p.s;  // the value write_row_stats stores
          s_arg[row - beg] = p.idx;
        }
      }
    }
  }
  __syncthreads();  // the block's conf / argmax rows are written before the block step reads them
  if (small) {
    if (wave == 0) {
      const float c = own_ok ? s_conf[lane] : 0.f;
      unmask_wave(b, own_row, own_ok, m_own != 0, c, own_ok ? s_arg[lane] : 0, c >= tau[b],
                  masked, tokens, unmask, n_commit, resolved, lane);
    }
    return;
  }
  unmask_block<kThreshold, kFinishThreads>(b, ap.cu_block, conf, argmax, tau,
                                           RuleArgs{nullptr, 0.f, 0}, masked, tokens, unmask,
                                           n_commit, resolved);
}

}  // namespace

bool step_finish_fusable(int max_block, int n_slices) {
  // one workgroup reduces a whole block's partials
  return static_cast<long>(max_block) * n_slices <= kFinishMaxPartials;
}

hipError_t step_finish(bool bf16, const AttnArgs& a, void* attn_ws, int n_rows, int vocab,
                       const void* lm_ws, float* conf, float* entropy, int32_t* argmax,
                       float* max_logit, const float* tau, uint8_t* masked, int32_t* tokens,
                       uint8_t* unmask, int32_t* n_commit, uint8_t* resolved, hipStream_t s) {
  SplitPlan sp{1, 0};
  if (bf16 && a.total_block > 0 && a.max_block > 0)
    sp = split_plan(a.batch, a.max_block, attn_max_keys(a), a.hq, a.hkv);
  const AttnParams ap = attn_params(a, sp, attn_ws);
  const long pairs = static_cast<long>(a.total_block) * a.hq;
  const int n_merge =
      sp.nsplit > 1 ? static_cast<int>((pairs + kFinishThreads / 64 - 1) / (kFinishThreads / 64))
                    : 0;
  const int n_slices = n_rows > 0 ? lmhead_num_slices(bf16, n_rows, vocab) : 0;
  const Partial* part = static_cast<const Partial*>(lm_ws);
  const dim3 grid(static_cast<unsigned>(n_merge + a.batch));
  if (a.head_dim == 64)
    hipLaunchKernelGGL(step_finish_kernel<64>, grid, dim3(kFinishThreads), 0, s, ap,
                       a.total_block, a.batch, n_merge, part, n_slices, conf, entropy, argmax,
                       max_logit, tau, masked, tokens, unmask, n_commit, resolved);
  else
    hipLaunchKernelGGL(step_finish_kernel<128>, grid, dim3(kFinishThreads), 0, s, ap,
                       a.total_block, a.batch, n_merge, part, n_slices, conf, entropy, argmax,
                       max_logit, tau, masked, tokens, unmask, n_commit, resolved);
  return hipGetLastError();
}

}  // namespace eb
