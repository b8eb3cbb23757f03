// LBS block-selection post-pass (Sec. 5.1, Alg. 5), one workgroup per sequence.
//
// With M the masked positions of the generation window: |M| <= L_min selects M (size
// fallback); otherwise the candidates are the masked positions with router probability
// p_phi > 0.5 whose predicted token is not EOS; the first candidate farther than g_max
// positions from the previous candidate is dropped with every later one (max-gap filter); if
// fewer than L_min positions remain, the first L_B masked positions are selected instead
// (min-tokens fallback).  Integer work only: scans over the window in chunks of the workgroup
// size, carried across chunks.
#include "eb_common.hpp"
#include "eb_internal.hpp"

namespace eb {
namespace {

constexpr int kLbsThreads = 256;
constexpr int kLbsWaves = kLbsThreads / 64;

// Workgroup-wide reductions and scans (every thread calls; every thread gets the result).
struct WgScratch {
  int v[kLbsWaves];
};

__device__ __forceinline__ int wg_sum(int x, WgScratch& s) {
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) s.v[threadIdx.x >> 6] = x;
  __syncthreads();
  int t = 0;
#pragma unroll
  for (int k = 0; k < kLbsWaves; ++k) t += s.v[k];
  return t;
}

__device__ __forceinline__ int wg_min(int x, WgScratch& s) {
  for (int m = 32; m >= 1; m >>= 1) x = min(x, __shfl_xor(x, m));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) s.v[threadIdx.x >> 6] = x;
  __syncthreads();
  int t = s.v[0];
#pragma unroll
  for (int k = 1; k < kLbsWaves; ++k) t = min(t, s.v[k]);
  return t;
}

// Exclusive scan in thread order with operator op (sum or max) and identity id; `total`
// receives the reduction over the whole workgroup.
template <bool kMax>
__device__ __forceinline__ int wg_exclusive_scan(int x, int id, WgScratch& s, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = x;
  for (int off = 1; off < 64; off <<= 1) {
    const int t = __shfl_up(inc, off);
    if (lane >= off) inc = kMax ? max(inc, t) : inc + t;
  }
  int exc = __shfl_up(inc, 1);
  if (lane == 0) exc = id;
  __syncthreads();
  if (lane == 63) s.v[wave] = inc;
  __syncthreads();
  int before = id;
  total = id;
#pragma unroll
  for (int k = 0; k < kLbsWaves; ++k) {
    if (k < wave) before = kMax ? max(before, s.v[k]) : before + s.v[k];
    total = kMax ? max(total, s.v[k]) : total + s.v[k];
  }
  return kMax ? max(before, exc) : before + exc;
}

__global__ __launch_bounds__(kLbsThreads) void lbs_select_kernel(
    int L, const uint8_t* __restrict__ masked, const float* __restrict__ p_phi,
    const int32_t* __restrict__ x_hat, int eos, int l_min, int l_b, int g_max,
    uint8_t* __restrict__ block, int32_t* __restrict__ size, int32_t* __restrict__ first) {
  __shared__ WgScratch s;
  const int tid = threadIdx.x;
  const size_t base = static_cast<size_t>(blockIdx.x) * L;
  const uint8_t* mk = masked + base;
  const float* pp = p_phi + base;
  const int32_t* xh = x_hat + base;
  uint8_t* out = block + base;
  auto cand = [&](int i) -> bool { return mk[i] && pp[i] > 0.5f && xh[i] != eos; };

  int cnt = 0, fm = L;
  for (int i = tid; i < L; i += kLbsThreads) {
    if (mk[i]) {
      ++cnt;
      fm = min(fm, i);
    }
  }
  const int n_masked = wg_sum(cnt, s);
  const int first_masked = wg_min(fm, s);

  if (n_masked <= l_min) {  // size fallback: the block is every masked position
    for (int i = tid; i < L; i += kLbsThreads) out[i] = mk[i];
    if (tid == 0) {
      size[blockIdx.x] = n_masked;
      first[blockIdx.x] = n_masked ? first_masked : -1;
    }
    return;
  }

  // max-gap cut: the first candidate whose previous candidate is more than g_max away
  int cut = L, carry = -1;
  for (int c0 = 0; c0 < L; c0 += kLbsThreads) {
    const int i = c0 + tid;
    const bool c = i < L && cand(i);
    int chunk_last;
    const int prev = max(carry, wg_exclusive_scan<true>(c ? i : -1, -1, s, chunk_last));
    const bool bad = c && prev >= 0 && i - prev > g_max;
    const int b = wg_min(bad ? i : L, s);
    if (b < L) {
      cut = b;
      break;  // uniform: every thread sees the same b
    }
    carry = max(carry, chunk_last);
  }
  int kc = 0, fk = L;
  for (int i = tid; i < cut; i += kLbsThreads) {
    if (cand(i)) {
      ++kc;
      fk = min(fk, i);
    }
  }
  const int kept = wg_sum(kc, s);
  const int first_kept = wg_min(fk, s);

  if (kept >= l_min) {
    for (int i = tid; i < L; i += kLbsThreads) out[i] = (i < cut && cand(i)) ? 1 : 0;
    if (tid == 0) {
      size[blockIdx.x] = kept;
      first[blockIdx.x] = kept ? first_kept : -1;
    }
    return;
  }
  // min-tokens fallback: the first l_b masked positions
  int rank_carry = 0;
  for (int c0 = 0; c0 < L; c0 += kLbsThreads) {
    const int i = c0 + tid;
    const int m = (i < L && mk[i]) ? 1 : 0;
    int chunk_total;
    const int rank = rank_carry + wg_exclusive_scan<false>(m, 0, s, chunk_total);
    if (i < L) out[i] = (m && rank < l_b) ? 1 : 0;
    rank_carry += chunk_total;
  }
  if (tid == 0) {
    const int n = min(l_b, n_masked);
    size[blockIdx.x] = n;
    first[blockIdx.x] = n ? first_masked : -1;
  }
}

}  // namespace

hipError_t lbs_select(int n_seq, int window, const uint8_t* masked, const float* p_phi,
                      const int32_t* x_hat, int eos, int l_min, int l_b, int g_max,
                      uint8_t* block, int32_t* size, int32_t* first, hipStream_t s) {
  hipLaunchKernelGGL(lbs_select_kernel, dim3(n_seq), dim3(kLbsThreads), 0, s, window, masked,
                     p_phi, x_hat, eos, l_min, l_b, g_max, block, size, first);
  return hipGetLastError();
}

}  // namespace eb
