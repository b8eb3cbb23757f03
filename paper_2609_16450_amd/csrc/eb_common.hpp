// Device-side helpers shared by the gfx950 kernels: bf16 vectors, MFMA wrappers, and the
// (max, sum, entropy-moment, argmax) partial used to reduce softmax statistics over a
// vocabulary that never leaves the chip.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace eb {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegBig = -3.402823466e38f;  // empty-partial max (finite, so 0 * (m - M) = 0)
constexpr int32_t kNoIndex = 0x7fffffff;

// 32x32 output tile, K = 16 per instruction, bf16 inputs, fp32 accumulate.
// Lane l holds A[l % 32][8 * (l / 32) + 0..7] and B[8 * (l / 32) + 0..7][l % 32];
// accumulator register r of lane l is C[8 * (r / 4) + 4 * (l / 32) + r % 4][l % 32].
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// 16x16 output tile, K = 32 per instruction, bf16 inputs, fp32 accumulate.
// Lane l holds A[l % 16][8 * (l / 16) + 0..7] and B[8 * (l / 16) + 0..7][l % 16];
// accumulator register r of lane l is C[4 * (l / 16) + r][l % 16].
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Two floats to two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32; lo in bits 0-15.
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// acc + lo + hi of the two bf16 values packed in w (one dot instruction against (1, 1)).  Takes
// the word as a scalar: the front end lowers a bit cast of a vector-element expression
// (__builtin_bit_cast(T, v[i])) to element 0 whatever i is.
__device__ __forceinline__ float sum2_bf16(uint32_t w, float acc) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w),
                                         __builtin_bit_cast(bf16x2, 0x3f803f80u), acc, false);
}

// Buffer loads straight into LDS.  A raw buffer resource over memory starting at `base` (2 GiB
// range, word 3 as gfx9 raw dword loads need); 16 bytes per lane from byte offset voff + soff
// into LDS at l + 16 * lane (the LDS address is wave-uniform).  The builtins sit in device
// functions of their own: inside a kernel body the host compilation would drop the kernel.
// (Loads into LDS issued as global loads count on the LDS-read counter as well, and the
// compiler then waits for every outstanding LDS read before each use of one; buffer loads do
// not.)
typedef __attribute__((address_space(3))) void lds_void_t;
constexpr int kBufferWord3 = 0x00020000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, 0x7fffffff, kBufferWord3);
}
__device__ __forceinline__ void buffer_load_to_lds(__amdgpu_buffer_rsrc_t rs, void* l,
                                                   uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)(l), 16, voff, soff, 0, 0);
}

// Wait until at most N vector-memory instructions of this wave are outstanding and all of its
// LDS reads have returned, then barrier.
template <int N>
__device__ __forceinline__ void wait_vm_lds_and_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0x0 << 8));
  asm volatile("s_barrier" ::: "memory");
}

// bf16 <-> f32
__device__ __forceinline__ float bf16_bits_to_f32(uint16_t u) {
  return __uint_as_float(static_cast<uint32_t>(u) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16_bits_rne(float f) {
  uint32_t b = __float_as_uint(f);
  b += 0x7fffu + ((b >> 16) & 1u);
  return static_cast<uint16_t>(b >> 16);
}

// Partial softmax statistics of a set of logits, in base-2 units:
//   m = max z,  s = sum 2^((z - m) log2 e),  t = sum 2^((z - m) log2 e) * (z - m) log2 e,
//   idx = lowest index attaining m.
// Then kappa = 1 / s and H = ln s - ln2 * t / s.
struct alignas(16) Partial {
  float m, s, t;
  int32_t idx;
};


__device__ __forceinline__ Partial partial_empty() { return Partial{kNegBig, 0.f, 0.f, kNoIndex}; }

// Merge two partials.  The result does not depend on argument order for m and idx; s and t
// are combined in the order given (callers fix that order for determinism).
__device__ __forceinline__ Partial partial_merge(const Partial& a, const Partial& b) {
  const float M = fmaxf(a.m, b.m);
  // <= 0; clamped so that an empty side (s = 0, m = kNegBig) contributes 0 * finite = 0
  const float da = fmaxf((a.m - M) * kLog2e, -1.0e30f);
  const float db = fmaxf((b.m - M) * kLog2e, -1.0e30f);
  const float fa = fast_exp2(da);
  const float fb = fast_exp2(db);
  Partial r;
  r.m = M;
  r.s = a.s * fa + b.s * fb;
  r.t = fa * (a.t + a.s * da) + fb * (b.t + b.s * db);
  r.idx = (a.m > b.m) ? a.idx : (b.m > a.m) ? b.idx : min(a.idx, b.idx);
  return r;
}

__device__ __forceinline__ Partial partial_shfl_xor(const Partial& p, int mask) {
  Partial q;
  q.m = __shfl_xor(p.m, mask);
  q.s = __shfl_xor(p.s, mask);
  q.t = __shfl_xor(p.t, mask);
  q.idx = __shfl_xor(p.idx, mask);
  return q;
}

// Butterfly step: lanes lane and lane ^ mask both end with merge(lower lane, higher lane),
// evaluated by the same expression, hence bit-identical on both lanes.
__device__ __forceinline__ Partial partial_xor_merge(const Partial& p, int mask, int lane) {
  const Partial q = partial_shfl_xor(p, mask);
  return (lane & mask) ? partial_merge(q, p) : partial_merge(p, q);
}

// Reduction of one partial per lane to the wavefront's partial, returned on every lane: the
// maximum M and the lowest index attaining it by max / min butterflies, then each lane's partial
// rescaled to M (s 2^d and 2^d (t + s d) with d = (m - M) log2 e, the partial_merge formulas)
// and s, t summed by a butterfly.  Each lane's sums use the same additions in the same order
// (a + b on one lane, b + a on its partner), so every lane ends with identical bits.
__device__ __forceinline__ Partial wave_finish(const Partial& acc) {
  float M = acc.m;
  for (int mask = 32; mask >= 1; mask >>= 1) M = fmaxf(M, __shfl_xor(M, mask));
  int32_t idx = acc.m == M ? acc.idx : kNoIndex;
  for (int mask = 32; mask >= 1; mask >>= 1) idx = min(idx, __shfl_xor(idx, mask));
  const float d = fmaxf((acc.m - M) * kLog2e, -1.0e30f);  // empty lane: 2^d = 0
  const float f = fast_exp2(d);
  float s = acc.s * f;
  float t = f * (acc.t + acc.s * d);
  for (int mask = 32; mask >= 1; mask >>= 1) {
    s += __shfl_xor(s, mask);
    t += __shfl_xor(t, mask);
  }
  return Partial{M, s, t, idx};
}

// Merge of n partials p[0..n) by one wavefront in a fixed order: lane l merges p[l], p[l+64],
// ... in index order, then wave_finish; every lane ends with the same result.  Loads are issued
// kBatch at a time, unconditionally (clamped index), so that their latencies overlap; a lane
// past the end merges an empty partial, which leaves its partial unchanged exactly (m and idx
// kept, s + 0 * 0, t + 0), so the code has no branch.
template <int kBatch = 4>
__device__ __forceinline__ Partial wave_merge(const Partial* __restrict__ p, int n, int lane) {
  Partial acc = partial_empty();
  for (int base = 0; base < n; base += 64 * kBatch) {  // uniform trip count
    Partial q[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) q[j] = p[min(base + 64 * j + lane, n - 1)];
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
      acc = partial_merge(acc, base + 64 * j + lane < n ? q[j] : partial_empty());
  }
  return wave_finish(acc);
}

// Per-row outputs from a row's merged partial p: conf = 1 / s (the top-1 probability),
// entropy in nats = ln s - ln 2 * t / s, argmax, and the top logit (max_logit optional).
__device__ __forceinline__ void write_row_stats(const Partial& p, int row, float* conf,
                                                float* entropy, int32_t* argmax,
                                                float* max_logit) {
  conf[row] = 1.0f / p.s;
  entropy[row] = logf(p.s) - kLn2 * p.t / p.s;
  argmax[row] = p.idx;
  if (max_logit) max_logit[row] = p.m;
}

}  // namespace eb
