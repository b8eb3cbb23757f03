// Segmented unmask with the anti-stall fallback (the block step is in unmask_block.hpp), one
// workgroup per block, and the LPS feature rows of each block.
#include "eb_common.hpp"
#include "eb_internal.hpp"
#include "unmask_block.hpp"

namespace eb {
namespace {

constexpr int kThreads = kUnmaskThreads;

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
// before this step's commit, then per row feat = (kappa, H * inv_ln_v, Delta, rho) and the
// intra-block position pos = (p_i - p_first) / len, where p is the row's sequence position
// (seq_pos) or, without seq_pos, its packed row index.
__global__ __launch_bounds__(kThreads) void lps_features_kernel(
    const int32_t* __restrict__ cu_block, float inv_ln_v, const float* __restrict__ conf,
    const float* __restrict__ entropy, const float* __restrict__ gap,
    const uint8_t* __restrict__ masked, const int32_t* __restrict__ seq_pos,
    float* __restrict__ feat, float* __restrict__ pos, float* __restrict__ mask_ratio) {
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
  const int first = (seq_pos && len > 0) ? seq_pos[beg] : beg;
  for (int i = beg + tid; i < end; i += kThreads) {
    *reinterpret_cast<f32x4*>(feat + 4 * static_cast<size_t>(i)) =
        f32x4{conf[i], entropy[i] * inv_ln_v, gap[i], rho};
    const int p = seq_pos ? seq_pos[i] : i;
    pos[i] = static_cast<float>(p - first) / static_cast<float>(len);
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
                        const int32_t* seq_pos, float* feat, float* pos, float* mask_ratio,
                        hipStream_t s) {
  const float inv_ln_v = static_cast<float>(1.0 / log(static_cast<double>(vocab)));
  hipLaunchKernelGGL(lps_features_kernel, dim3(batch), dim3(kThreads), 0, s, cu_block, inv_ln_v,
                     conf, entropy, gap, masked, seq_pos, feat, pos, mask_ratio);
  return hipGetLastError();
}

}  // namespace eb
