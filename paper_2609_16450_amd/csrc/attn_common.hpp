// Block-attention pieces shared by the attention kernels and the fused step epilogue: the bf16
// kernel parameters, the key-split plan, and the merge of one (block row, query head)'s splits.
#pragma once

#include "eb_common.hpp"
#include "eb_internal.hpp"

namespace eb {
namespace {

constexpr int kAttnRowsPerWg = 128;  // query rows (position, head-in-group) per workgroup
constexpr int kAttnKeys = 64;        // keys per LDS stage
constexpr int kAttnTargetWgs = 512;  // the key split aims at this many workgroups

struct AttnParams {
  const int32_t* cu_block;
  const int32_t* cu_prefix;
  int hq, hkv, group;
  float scale_log2;  // scale * log2(e)
  const uint16_t* q;
  const uint16_t* k_blk;
  const uint16_t* v_blk;
  const uint16_t* k_pre;
  const uint16_t* v_pre;
  uint16_t* out;
  // optional cached suffix segment (dual cache): rows cu_suffix[b] .. cu_suffix[b+1]-1 of
  // k_suf / v_suf are further keys of sequence b; cu_suffix == nullptr: none
  const int32_t* cu_suffix;
  const uint16_t* k_suf;
  const uint16_t* v_suf;
  // key split: keys of a sequence are cut into ranges of kps keys, one workgroup per range;
  // with nsplit > 1 the workgroups write unnormalised partials that attn_merge_kernel (or the
  // fused step epilogue) combines
  int nsplit, kps;
  float* o_part;  // [T * hq * nsplit, D]
  float* m_part;  // [T * hq * nsplit]  running max (log2 units)
  float* l_part;  // [T * hq * nsplit]  sum of 2^(s - m)
};

struct SplitPlan {
  int nsplit, kps;
};

// Key-split plan: enough workgroups to fill the chip, in whole 64-key stages.  max_keys is the
// largest number of keys of a sequence (prefix + block + suffix).
inline SplitPlan split_plan(int batch, int max_block, int max_keys, int hq, int hkv) {
  const int group = hq / hkv;
  const long row_tiles =
      (static_cast<long>(max_block) * group + kAttnRowsPerWg - 1) / kAttnRowsPerWg;
  const long base = row_tiles * hkv * batch;
  const int stages = (max_keys + kAttnKeys - 1) / kAttnKeys;
  int nsplit = static_cast<int>((kAttnTargetWgs + base - 1) / base);
  nsplit = max(1, min(nsplit, stages));
  const int stages_per = (stages + nsplit - 1) / nsplit;
  const int kps = stages_per * kAttnKeys;
  nsplit = (stages * kAttnKeys + kps - 1) / kps;
  return SplitPlan{nsplit, kps};
}

inline int attn_max_keys(const AttnArgs& a) {
  return a.max_prefix + a.max_block + (a.cu_suffix ? a.max_suffix : 0);
}

// Parameters of a bf16 launch under plan sp; with a split the partials live in ws as
// o [T * hq * nsplit, D], then m and l [T * hq * nsplit] each.
inline AttnParams attn_params(const AttnArgs& a, const SplitPlan& sp, void* ws) {
  const size_t n_part = static_cast<size_t>(a.total_block) * a.hq * sp.nsplit;
  float* o_part = sp.nsplit > 1 ? static_cast<float*>(ws) : nullptr;
  float* m_part = sp.nsplit > 1 ? o_part + n_part * a.head_dim : nullptr;
  float* l_part = sp.nsplit > 1 ? m_part + n_part : nullptr;
  return AttnParams{a.cu_block, a.cu_prefix, a.hq, a.hkv, a.hq / a.hkv, a.scale * kLog2e,
                    static_cast<const uint16_t*>(a.q), static_cast<const uint16_t*>(a.k_blk),
                    static_cast<const uint16_t*>(a.v_blk), static_cast<const uint16_t*>(a.k_pre),
                    static_cast<const uint16_t*>(a.v_pre), static_cast<uint16_t*>(a.out),
                    a.cu_suffix, static_cast<const uint16_t*>(a.k_suf),
                    static_cast<const uint16_t*>(a.v_suf), sp.nsplit, sp.kps, o_part, m_part,
                    l_part};
}

// Combine the key-split partials of pair rh = row * hq + head (one wavefront, lane = lane id):
// splits merged in index order (max, rescale, sum), output rounded to bf16.
template <int D>
__device__ __forceinline__ void attn_merge_pair(const AttnParams& p, int rh, int batch, int lane) {
  const int row = rh / p.hq;
  // sequence of this row: largest b with cu_block[b] <= row (blocks are non-empty here)
  int lo = 0, hi = batch - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.cu_block[mid] <= row) lo = mid; else hi = mid - 1;
  }
  const int b = lo;
  const int n_keys = (p.cu_prefix[b + 1] - p.cu_prefix[b]) + (p.cu_block[b + 1] - p.cu_block[b]) +
                     (p.cu_suffix ? p.cu_suffix[b + 1] - p.cu_suffix[b] : 0);
  const int nvalid = min(p.nsplit, (n_keys + p.kps - 1) / p.kps);
  const size_t base = static_cast<size_t>(rh) * p.nsplit;
  // kGroup splits at a time, loaded together (clamped index, masked use), combined in index order
  constexpr int kGroup = 16;
  constexpr int kPer = D / 64;  // values per lane
  float M = -INFINITY;
  for (int k0 = 0; k0 < nvalid; k0 += kGroup) {
    float mk[kGroup];
#pragma unroll
    for (int j = 0; j < kGroup; ++j) mk[j] = p.m_part[base + min(k0 + j, nvalid - 1)];
#pragma unroll
    for (int j = 0; j < kGroup; ++j)
      if (k0 + j < nvalid) M = fmaxf(M, mk[j]);
  }
  float acc[kPer] = {};
  float L = 0.f;
  for (int k0 = 0; k0 < nvalid; k0 += kGroup) {
    float mk[kGroup], lk[kGroup], ok[kGroup][kPer];
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
      const size_t k = base + min(k0 + j, nvalid - 1);
      mk[j] = p.m_part[k];
      lk[j] = p.l_part[k];
#pragma unroll
      for (int e = 0; e < kPer; ++e) ok[j][e] = p.o_part[k * D + lane * kPer + e];
    }
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
      if (k0 + j >= nvalid) continue;
      const float f = fast_exp2(mk[j] - M);
      L += f * lk[j];
#pragma unroll
      for (int e = 0; e < kPer; ++e) acc[e] += f * ok[j][e];
    }
  }
  const float inv = 1.0f / L;
  uint16_t* dst = p.out + static_cast<size_t>(rh) * D + lane * kPer;
#pragma unroll
  for (int e = 0; e < kPer; ++e) dst[e] = f32_to_bf16_bits_rne(acc[e] * inv);
}

}  // namespace
}  // namespace eb
