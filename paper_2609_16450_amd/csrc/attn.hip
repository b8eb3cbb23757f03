// Block attention with a prefix KV cache for gfx950.
//
// Every query row of a sequence's active block attends, without a causal mask, to the
// sequence's cached prefix keys followed by the block's own keys.  Grouped-query attention:
// query head h reads key/value head h / G with G = hq / hkv, so one workgroup serves the
// G query heads of one key/value head and its K/V tiles are read once for all of them.
//
// bf16 path: scores are computed transposed, S^T = K Q^T, so each lane owns one query row
// (an MFMA column) and reduces its softmax statistics in registers; the probabilities then
// feed P V directly as the B operand of O^T = V^T P^T, with V staged transposed in LDS.
// Small steps (attn_small_ok) take the 16-row role of attn_small.hpp instead, here as a kernel
// of its own; the decode step runs the same role inside the LM-head launch.
#include "attn_common.hpp"
#include "attn_small.hpp"
#include "eb_common.hpp"
#include "eb_internal.hpp"

namespace eb {
namespace {

constexpr int kThreads = 256;   // 4 waves
constexpr int kRowsPerWg = kAttnRowsPerWg;
constexpr int kKeys = kAttnKeys;


// Two workgroups per compute unit (<= 256 VGPRs per lane, no spills at D = 128), so one
// wave's softmax arithmetic overlaps another wave's MFMAs on the same SIMD (batch 64 at
// D = 128: 1.85 ms with one workgroup per compute unit, 1.07 ms with two).
template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_bf16_kernel(AttnParams p) {
  constexpr int kKRow = D + 8;       // K tile pitch (bf16)
  constexpr int kVRow = kKeys + 4;   // V^T tile pitch (bf16)
  constexpr int kDSteps = D / 16;    // MFMA k-steps over the head dimension
  constexpr int kDBlocks = D / 32;   // 32-row blocks of O^T
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kKeys * kKRow];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * kVRow];

  const int b = blockIdx.z / p.nsplit;
  const int sp = blockIdx.z % p.nsplit;
  const int g = blockIdx.y;
  const int G = p.group;
  const int bbeg = p.cu_block[b];
  const int len = p.cu_block[b + 1] - bbeg;
  const int pbeg = p.cu_prefix[b];
  const int plen = p.cu_prefix[b + 1] - pbeg;
  const int n_rows = len * G;
  const int row0 = blockIdx.x * kRowsPerWg;
  if (row0 >= n_rows) return;  // whole workgroup: this tile lies past the block
  const int sbeg = p.cu_suffix ? p.cu_suffix[b] : 0;
  const int slen = p.cu_suffix ? p.cu_suffix[b + 1] - sbeg : 0;
  const int n_keys = plen + len + slen;
  const int kbeg = sp * p.kps;
  if (kbeg >= n_keys) return;  // whole workgroup: this key range lies past the sequence
  const int kend = min(n_keys, kbeg + p.kps);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;

  // This lane's query row.
  const int myrow = row0 + wave * 32 + l32;
  const bool row_ok = myrow < n_rows;
  const int rr = row_ok ? myrow : 0;
  const int pos = rr / G, hh = rr % G;
  const size_t q_off = (static_cast<size_t>(bbeg + pos) * p.hq + g * G + hh) * D;

  // Q^T fragments (B operand): step s, half hf holds d = 16 s + 8 hf .. +7.
  bf16x8 qf[kDSteps];
#pragma unroll
  for (int s = 0; s < kDSteps; ++s)
    qf[s] = *reinterpret_cast<const bf16x8*>(p.q + q_off + 16 * s + 8 * half);

  f32x16 o[kDBlocks];
#pragma unroll
  for (int db = 0; db < kDBlocks; ++db) o[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  // Loader assignments.  K: 16-byte chunks, chunk c = key c / (D/8), columns 8 (c % (D/8)).
  constexpr int kKChunks = kKeys * (D / 8);
  constexpr int kKPer = kKChunks / kThreads;
  // V: thread handles keys 2 kp, 2 kp + 1 (kp = tid % 32) and d range [dg * D/8, +D/8).
  const int kp = tid & 31, dg = tid >> 5;
  constexpr int kVd = D / 8;

  // key j of the sequence: prefix rows, then block rows, then suffix rows (an unordered set)
  auto key_src = [&](int j, const uint16_t* pre, const uint16_t* blk,
                     const uint16_t* suf) -> const uint16_t* {
    if (j < plen) return pre + (static_cast<size_t>(pbeg + j) * p.hkv + g) * D;
    if (j < plen + len) return blk + (static_cast<size_t>(bbeg + j - plen) * p.hkv + g) * D;
    return suf + (static_cast<size_t>(sbeg + j - plen - len) * p.hkv + g) * D;
  };

  // Loads are unconditional with clamped key indices (a conditional load would be waited for
  // on the spot); keys past the end are replaced by zeros when stored to LDS.
  u32x4 kreg[kKPer];
  u32x4 vreg[2][kVd / 8];
  const int key_stride = p.hkv * D;  // elements between consecutive keys of one K/V head
  auto gload = [&](int kv0) {
    if (kv0 + kKeys <= plen) {
      // the whole stage lies in the prefix: one base pointer per tensor, no per-key segment choice
      const size_t base = (static_cast<size_t>(pbeg + kv0) * p.hkv + g) * D;
      const uint16_t* kb = p.k_pre + base;
      const uint16_t* vb = p.v_pre + base;
#pragma unroll
      for (int i = 0; i < kKPer; ++i) {
        const int c = tid + i * kThreads;
        const int key = c / (D / 8), col = (c % (D / 8)) * 8;
        kreg[i] = *reinterpret_cast<const u32x4*>(kb + key * key_stride + col);
      }
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int c = 0; c < kVd / 8; ++c)
          vreg[e][c] = *reinterpret_cast<const u32x4*>(vb + (2 * kp + e) * key_stride +
                                                       dg * kVd + 8 * c);
      return;
    }
#pragma unroll
    for (int i = 0; i < kKPer; ++i) {
      const int c = tid + i * kThreads;
      const int key = c / (D / 8), col = (c % (D / 8)) * 8;
      const int j = min(kv0 + key, kend - 1);
      kreg[i] = *reinterpret_cast<const u32x4*>(key_src(j, p.k_pre, p.k_blk, p.k_suf) + col);
    }
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int j = min(kv0 + 2 * kp + e, kend - 1);
#pragma unroll
      for (int c = 0; c < kVd / 8; ++c)
        vreg[e][c] = *reinterpret_cast<const u32x4*>(key_src(j, p.v_pre, p.v_blk, p.v_suf) +
                                                     dg * kVd + 8 * c);
    }
  };
  // Keys past the end were loaded from a clamped (valid) row: finite values whose scores are
  // masked to -inf below, so their probabilities are exactly 0 and they add nothing to O.
  auto sstore = [&]() {
#pragma unroll
    for (int i = 0; i < kKPer; ++i) {
      const int c = tid + i * kThreads;
      const int key = c / (D / 8), col = (c % (D / 8)) * 8;
      *reinterpret_cast<u32x4*>(Ks + key * kKRow + col) = kreg[i];
    }
    // V^T: the 16-bit values of keys 2 kp and 2 kp + 1 at one d form one 32-bit word
#pragma unroll
    for (int c = 0; c < kVd / 8; ++c)
#pragma unroll
      for (int w4 = 0; w4 < 4; ++w4) {
        const int d = dg * kVd + 8 * c + 2 * w4;
        const uint32_t k0 = vreg[0][c][w4], k1 = vreg[1][c][w4];
        *reinterpret_cast<uint32_t*>(Vt + d * kVRow + 2 * kp) =
            __builtin_amdgcn_perm(k1, k0, 0x05040100u);  // low halves: value at d
        *reinterpret_cast<uint32_t*>(Vt + (d + 1) * kVRow + 2 * kp) =
            __builtin_amdgcn_perm(k1, k0, 0x07060302u);  // high halves: value at d + 1
      }
  };

  const int n_stages = (kend - kbeg + kKeys - 1) / kKeys;
  gload(kbeg);
  for (int st = 0; st < n_stages; ++st) {
    const int kv0 = kbeg + st * kKeys;
    __syncthreads();  // previous stage's LDS reads are done
    sstore();
    __syncthreads();
    if (st + 1 < n_stages) gload(kv0 + kKeys);

    // S^T for two 32-key blocks: acc[kb][r] = S[query l32][key kb*32 + 8(r/4) + 4 half + r%4]
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sacc[kb] = f32x16{};
#pragma unroll
      for (int s = 0; s < kDSteps; ++s) {
        const bf16x8 kf =
            *reinterpret_cast<const bf16x8*>(Ks + (kb * 32 + l32) * kKRow + 16 * s + 8 * half);
        sacc[kb] = mfma32(kf, qf[s], sacc[kb]);
      }
    }
    // raw scores; keys past the end (last stage only) masked to -inf
    if (kv0 + kKeys > kend) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kv0 + kb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          if (key >= kend) sacc[kb][r] = -INFINITY;
        }
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, sacc[kb][r]);
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    // scale > 0, so max(scale * s) = scale * max(s); e = 2^(scale s - m) with one FMA
    const float m_new = fmaxf(m_run, mloc * p.scale_log2);
    const float alpha = fast_exp2(m_run - m_new);
    m_run = m_new;
    float lsum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = fast_exp2(fmaf(sacc[kb][r], p.scale_log2, -m_new));
        sacc[kb][r] = e;
        lsum += e;
      }
    l_run = l_run * alpha + lsum;
    if (__any(alpha != 1.0f)) {  // some row's running max moved (alpha = 1 leaves O as it is)
#pragma unroll
      for (int db = 0; db < kDBlocks; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
    }

    // O^T += V^T P^T.  MFMA u of key block kb covers keys kb*32 + 16u + {4 half + 0..3,
    // 8 + 4 half + 0..3}, which are exactly accumulator registers 8u .. 8u+7 of sacc[kb].
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        u32x4 pb;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          pb[e] = pack2_bf16(sacc[kb][8 * u + 2 * e], sacc[kb][8 * u + 2 * e + 1]);
        const bf16x8 pf = __builtin_bit_cast(bf16x8, pb);
        const int kbase = kb * 32 + 16 * u + 4 * half;
#pragma unroll
        for (int db = 0; db < kDBlocks; ++db) {
          const uint16_t* vr = Vt + (db * 32 + l32) * kVRow;
          const u32x2 lo = *reinterpret_cast<const u32x2*>(vr + kbase);
          const u32x2 hi = *reinterpret_cast<const u32x2*>(vr + kbase + 8);
          const u32x4 va{lo[0], lo[1], hi[0], hi[1]};
          o[db] = mfma32(__builtin_bit_cast(bf16x8, va), pf, o[db]);
        }
      }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!row_ok) return;
  if (p.nsplit > 1) {
    const size_t idx = (static_cast<size_t>(bbeg + pos) * p.hq + g * G + hh) * p.nsplit + sp;
    float* dst = p.o_part + idx * D;
#pragma unroll
    for (int db = 0; db < kDBlocks; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = db * 32 + 8 * q4 + 4 * half;
        *reinterpret_cast<f32x4*>(dst + d) =
            f32x4{o[db][4 * q4 + 0], o[db][4 * q4 + 1], o[db][4 * q4 + 2], o[db][4 * q4 + 3]};
      }
    if (half == 0) {
      p.m_part[idx] = m_run;
      p.l_part[idx] = l_tot;
    }
    return;
  }
  const float inv = 1.0f / l_tot;
  uint16_t* dst = p.out + q_off;
#pragma unroll
  for (int db = 0; db < kDBlocks; ++db)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int d = db * 32 + 8 * q4 + 4 * half;
      const u32x2 v{pack2_bf16(o[db][4 * q4 + 0] * inv, o[db][4 * q4 + 1] * inv),
                    pack2_bf16(o[db][4 * q4 + 2] * inv, o[db][4 * q4 + 3] * inv)};
      *reinterpret_cast<u32x2*>(dst + d) = v;
    }
}

// Small steps on their own: the 16-query-row role of attn_small.hpp with kSmallAloneThreads
// threads, one workgroup per (unit, group of row tiles).
#ifndef EB_SMALL_ALONE_THREADS
#define EB_SMALL_ALONE_THREADS 256
#endif
constexpr int kSmallAloneThreads = EB_SMALL_ALONE_THREADS;
template <int D>
__global__ __launch_bounds__(kSmallAloneThreads) void attn_small_kernel(AttnParams p) {
  attn_small_role<D, kSmallAloneThreads>(p, static_cast<int>(blockIdx.x),
                                          static_cast<int>(blockIdx.y));
}

// Combine the key-split partials of each (block row, query head), one wavefront per pair.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnParams p, int total_block, int batch) {
  const int rh = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (rh >= total_block * p.hq) return;  // uniform per wavefront
  attn_merge_pair<D>(p, rh, batch, threadIdx.x & 63);
}

// fp32 path (small shapes): one wavefront per (block row, query head); lanes split the head
// dimension; keys are visited one by one with an online softmax.
struct AttnParamsF32 {
  const int32_t* cu_block;
  const int32_t* cu_prefix;
  int hq, hkv, group, head_dim;
  float scale;
  const float* q;
  const float* k_blk;
  const float* v_blk;
  const float* k_pre;
  const float* v_pre;
  float* out;
  const int32_t* cu_suffix;  // nullptr: no suffix segment
  const float* k_suf;
  const float* v_suf;
};

__global__ __launch_bounds__(64) void attn_f32_kernel(AttnParamsF32 p) {
  const int b = blockIdx.z, h = blockIdx.y, i = blockIdx.x;
  const int bbeg = p.cu_block[b];
  const int len = p.cu_block[b + 1] - bbeg;
  if (i >= len) return;
  const int pbeg = p.cu_prefix[b];
  const int plen = p.cu_prefix[b + 1] - pbeg;
  const int D = p.head_dim;
  const int g = h / p.group;
  const int lane = threadIdx.x;
  const float* qr = p.q + (static_cast<size_t>(bbeg + i) * p.hq + h) * D;
  const float q0 = lane < D ? qr[lane] : 0.f;
  const float q1 = lane + 64 < D ? qr[lane + 64] : 0.f;
  const int sbeg = p.cu_suffix ? p.cu_suffix[b] : 0;
  const int slen = p.cu_suffix ? p.cu_suffix[b + 1] - sbeg : 0;
  float m = -INFINITY, l = 0.f, a0 = 0.f, a1 = 0.f;
  for (int j = 0; j < plen + len + slen; ++j) {
    size_t off;
    const float *kb, *vb;
    if (j < plen) {
      off = static_cast<size_t>(pbeg + j);
      kb = p.k_pre;
      vb = p.v_pre;
    } else if (j < plen + len) {
      off = static_cast<size_t>(bbeg + j - plen);
      kb = p.k_blk;
      vb = p.v_blk;
    } else {
      off = static_cast<size_t>(sbeg + j - plen - len);
      kb = p.k_suf;
      vb = p.v_suf;
    }
    const float* kr = kb + (off * p.hkv + g) * D;
    const float* vr = vb + (off * p.hkv + g) * D;
    float dot = (lane < D ? q0 * kr[lane] : 0.f) + (lane + 64 < D ? q1 * kr[lane + 64] : 0.f);
    for (int mask = 32; mask >= 1; mask >>= 1) dot += __shfl_xor(dot, mask);
    const float sc = dot * p.scale;
    const float mn = fmaxf(m, sc);
    const float alpha = expf(m - mn);
    const float e = expf(sc - mn);
    l = l * alpha + e;
    a0 = a0 * alpha + e * (lane < D ? vr[lane] : 0.f);
    a1 = a1 * alpha + e * (lane + 64 < D ? vr[lane + 64] : 0.f);
    m = mn;
  }
  float* dst = p.out + (static_cast<size_t>(bbeg + i) * p.hq + h) * D;
  if (lane < D) dst[lane] = a0 / l;
  if (lane + 64 < D) dst[lane + 64] = a1 / l;
}

}  // namespace

size_t block_attn_ws_bytes(bool bf16, bool allow_split, int batch, int total_block, int max_block,
                           int max_keys, int hq, int hkv, int head_dim) {
  if (!bf16 || !allow_split || total_block == 0 || max_block == 0) return 0;
  const SplitPlan sp = split_plan(batch, max_block, max_keys, hq, hkv);
  if (sp.nsplit == 1) return 0;
  return static_cast<size_t>(total_block) * hq * sp.nsplit * (head_dim + 2) * sizeof(float);
}

hipError_t block_attn(bool bf16, bool allow_split, const AttnArgs& a, void* ws, hipStream_t s,
                      bool defer_merge) {
  if (a.total_block == 0 || a.max_block == 0) return hipSuccess;
  const int group = a.hq / a.hkv;
  const int max_keys = attn_max_keys(a);
  if (!bf16) {
    AttnParamsF32 p{a.cu_block, a.cu_prefix, a.hq, a.hkv, group, a.head_dim, a.scale,
                    static_cast<const float*>(a.q), static_cast<const float*>(a.k_blk),
                    static_cast<const float*>(a.v_blk), static_cast<const float*>(a.k_pre),
                    static_cast<const float*>(a.v_pre), static_cast<float*>(a.out), a.cu_suffix,
                    static_cast<const float*>(a.k_suf), static_cast<const float*>(a.v_suf)};
    hipLaunchKernelGGL(attn_f32_kernel, dim3(a.max_block, a.hq, a.batch), dim3(64), 0, s, p);
    return hipGetLastError();
  }
  const SplitPlan sp = allow_split ? split_plan(a.batch, a.max_block, max_keys, a.hq, a.hkv)
                                   : SplitPlan{1, (max_keys + kKeys - 1) / kKeys * kKeys};
  const AttnParams p = attn_params(a, sp, ws);
  if (allow_split && attn_small_ok(bf16, a)) {
    const long tiles = (static_cast<long>(a.max_block) * group + kSmallTile - 1) / kSmallTile;
    const int waves = kSmallAloneThreads / 64;
    const dim3 grid(static_cast<unsigned>(attn_small_units(a, sp)),
                    static_cast<unsigned>((tiles + waves - 1) / waves));
    if (a.head_dim == 128)
      hipLaunchKernelGGL(attn_small_kernel<128>, grid, dim3(kSmallAloneThreads), 0, s, p);
    else
      hipLaunchKernelGGL(attn_small_kernel<64>, grid, dim3(kSmallAloneThreads), 0, s, p);
  } else {
    const long rows = static_cast<long>(a.max_block) * group;
    dim3 grid(static_cast<unsigned>((rows + kRowsPerWg - 1) / kRowsPerWg), a.hkv,
              static_cast<unsigned>(a.batch) * sp.nsplit);
    if (a.head_dim == 128)
      hipLaunchKernelGGL(attn_bf16_kernel<128>, grid, dim3(kThreads), 0, s, p);
    else
      hipLaunchKernelGGL(attn_bf16_kernel<64>, grid, dim3(kThreads), 0, s, p);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || sp.nsplit == 1 || defer_merge) return e;
  const long pairs = static_cast<long>(a.total_block) * a.hq;
  dim3 mgrid(static_cast<unsigned>((pairs + 3) / 4));
  if (a.head_dim == 128)
    hipLaunchKernelGGL(attn_merge_kernel<128>, mgrid, dim3(256), 0, s, p, a.total_block, a.batch);
  else
    hipLaunchKernelGGL(attn_merge_kernel<64>, mgrid, dim3(256), 0, s, p, a.total_block, a.batch);
  return hipGetLastError();
}

}  // namespace eb
