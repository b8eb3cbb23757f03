// Block attention for small steps (at most 64 block rows in all), written as the role of a
// workgroup of up to 1024 threads that stays within 128 VGPRs per lane at that size.  The role
// runs as a kernel of its own (attn_small_kernel, 256-thread workgroups) and, with 1024 threads,
// as extra workgroups of the streaming LM-head launch, queued behind its vocabulary slices: the
// dispatcher starts them on the compute units that the slices free at the end, so the attention
// fills the LM head's tail instead of taking a launch of its own.
//
// One workgroup per (sequence b, K/V head g, key range) and group of 16-row query tiles: the
// query rows of (b, g) are the (position, head-in-group) pairs, 16 per wave (at most 256 rows,
// one 1024-thread workgroup for all of them); the workgroup stages each 64-key stage of K and V
// in LDS, and the waves that own query rows compute.  Scores are formed transposed,
// S^T = K Q^T, with 16x16x32 MFMAs, so lane l owns query l % 16 and holds keys 4 (l / 16) + r of
// each 16-key tile; exactly those keys are the k-slots of the B operand of O^T = V^T P^T once
// the contraction index is permuted, and the matching V^T operand comes from two transposed LDS
// reads (ds_read_b64_tr_b16) of row-major V.  Same key split, partial layout and online-softmax
// convention as the 128-row kernel.
#pragma once

#include "attn_common.hpp"
#include "eb_common.hpp"

namespace eb {
namespace {

constexpr int kSmallThreads = 1024;                 // 16 waves (inside the LM-head launch)
constexpr int kSmallTile = 16;                      // query rows per wave
constexpr int kSmallMaxRows = 16 * kSmallTile;      // query rows of one (sequence, K/V head)
constexpr int kSmallMaxTotal = 64;                  // block rows of the whole step

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// Eligible shapes: bf16, D in {64, 128}, at most kSmallMaxTotal block rows and at most
// kSmallMaxRows query rows per (sequence, K/V head).
inline bool attn_small_ok(bool bf16, const AttnArgs& a) {
  return bf16 && (a.head_dim == 64 || a.head_dim == 128) && a.total_block > 0 &&
         a.max_block > 0 && a.total_block <= kSmallMaxTotal &&
         static_cast<long>(a.max_block) * (a.hq / a.hkv) <= kSmallMaxRows;
}

// Workgroups of the role under plan sp: one per (sequence, K/V head, key range).
inline int attn_small_units(const AttnArgs& a, const SplitPlan& sp) {
  return a.batch * a.hkv * sp.nsplit;
}

// Attention role of unit `unit` (= (b hkv + g) nsplit + split) for the query-row tiles
// tile_group * kThreads/64 .. +kThreads/64 - 1 of its (sequence, K/V head), one per wave; every
// thread of the workgroup calls it, and every thread returns from it.  A row's arithmetic does
// not depend on kThreads, so every workgroup size gives the same bits.
template <int D, int kThreads>
__device__ __forceinline__ void attn_small_role(const AttnParams& p, int unit, int tile_group) {
  constexpr int kKeys = kAttnKeys;    // keys per stage
  constexpr int kKPitch = D + 8;      // K row pitch (bf16)
  constexpr int kVPitch = D + 16;     // V row pitch (bf16): rows 8 banks apart, so the 8 rows
                                      // x 32 B that 32 lanes of a transposed read touch fall on
                                      // distinct banks
  constexpr int kDSteps = D / 32;     // MFMA k-steps of S^T over the head dimension
  constexpr int kDTiles = D / 16;     // 16-row tiles of O^T
  constexpr int kChunks = kKeys * D / 8;  // 16-byte pieces of one K (or V) stage
  constexpr int kPer = kChunks >= kThreads ? kChunks / kThreads : 1;  // pieces per thread
  static_assert(kChunks % kThreads == 0 || kThreads % kChunks == 0, "pieces split evenly");
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kKeys * kKPitch];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[kKeys * kVPitch];

  const int sp = unit % p.nsplit;
  const int bg = unit / p.nsplit;
  const int g = bg % p.hkv, b = bg / p.hkv;
  const int G = p.group;
  const int bbeg = p.cu_block[b];
  const int len = p.cu_block[b + 1] - bbeg;
  const int pbeg = p.cu_prefix[b];
  const int plen = p.cu_prefix[b + 1] - pbeg;
  const int sbeg = p.cu_suffix ? p.cu_suffix[b] : 0;
  const int slen = p.cu_suffix ? p.cu_suffix[b + 1] - sbeg : 0;
  const int n_keys = plen + len + slen;
  const int n_rows = len * G;
  const int kbeg = sp * p.kps;
  const int row0 = tile_group * (kThreads / 64) * kSmallTile;
  if (row0 >= n_rows || kbeg >= n_keys) return;  // whole workgroup: nothing to do here
  const int kend = min(n_keys, kbeg + p.kps);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = lane >> 4, l16 = lane & 15;
  const bool active = row0 + wave * kSmallTile < n_rows;  // wave-uniform: the wave owns rows
  const int myrow = row0 + wave * kSmallTile + l16;
  const bool row_ok = myrow < n_rows;
  const int rr = row_ok ? myrow : n_rows - 1;
  const int pos = rr / G, hh = rr % G;
  const size_t q_off = (static_cast<size_t>(bbeg + pos) * p.hq + g * G + hh) * D;

  // Q^T fragments (B operand of S^T): step s holds d = 32 s + 8 grp .. +7 of query l16.
  bf16x8 qf[kDSteps];
#pragma unroll
  for (int s = 0; s < kDSteps; ++s)
    qf[s] = *reinterpret_cast<const bf16x8*>(p.q + q_off + 32 * s + 8 * grp);

  f32x4 o[kDTiles];
#pragma unroll
  for (int t = 0; t < kDTiles; ++t) o[t] = f32x4{};
  float m_run = -INFINITY, l_run = 0.f;

  // key j of the sequence: prefix rows, then block rows, then suffix rows (an unordered set)
  auto key_src = [&](int j, const uint16_t* pre, const uint16_t* blk,
                     const uint16_t* suf) -> const uint16_t* {
    if (j < plen) return pre + (static_cast<size_t>(pbeg + j) * p.hkv + g) * D;
    if (j < plen + len) return blk + (static_cast<size_t>(bbeg + j - plen) * p.hkv + g) * D;
    return suf + (static_cast<size_t>(sbeg + j - plen - len) * p.hkv + g) * D;
  };
  // Thread tid moves pieces tid + i kThreads (i < kPer) of K and of V: piece c is key c / (D/8),
  // columns 8 (c % (D/8)).  Keys past the end are loaded from a clamped, valid row; their scores
  // are set to -inf.
  const bool loader = tid < kChunks;  // wave-uniform (kChunks is a multiple of 64)
  u32x4 kreg[kPer], vreg[kPer];
  auto gload = [&](int kv0) {
    if (!loader) return;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = tid + i * kThreads;
      const int j = min(kv0 + c / (D / 8), kend - 1), col = (c % (D / 8)) * 8;
      kreg[i] = *reinterpret_cast<const u32x4*>(key_src(j, p.k_pre, p.k_blk, p.k_suf) + col);
      vreg[i] = *reinterpret_cast<const u32x4*>(key_src(j, p.v_pre, p.v_blk, p.v_suf) + col);
    }
  };
  auto sstore = [&]() {
    if (!loader) return;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = tid + i * kThreads;
      const int key = c / (D / 8), col = (c % (D / 8)) * 8;
      *reinterpret_cast<u32x4*>(Ks + key * kKPitch + col) = kreg[i];
      *reinterpret_cast<u32x4*>(Vs + key * kVPitch + col) = vreg[i];
    }
  };
  // V^T fragment for keys kbase + 4 grp + 0..3 at d = d0 + l16: lanes 4j .. 4j+3 of a 16-lane
  // group address row kbase + 4 grp + j, columns d0 + 4 (l16 % 4) .. +3; the transposed read
  // hands lane i of the group element i % 4 of the piece addressed by lane 4 j + i / 4.
  auto vt_read = [&](int kbase, int d0) -> v4i16 {
    const uint16_t* a = Vs + (kbase + 4 * grp + (l16 >> 2)) * kVPitch + d0 + 4 * (l16 & 3);
    // address-space cast (generic -> LDS) needs a C-style cast
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(const_cast<uint16_t*>(a)));
  };

  const int n_stages = (kend - kbeg + kKeys - 1) / kKeys;
  gload(kbeg);
  for (int st = 0; st < n_stages; ++st) {
    const int kv0 = kbeg + st * kKeys;
    __syncthreads();  // previous stage's LDS reads are done
    sstore();
    __syncthreads();
    if (st + 1 < n_stages) gload(kv0 + kKeys);
    if (!active) continue;

    // S^T tile t: sacc[t][r] = S[query l16][key 16 t + 4 grp + r]
    f32x4 sacc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      sacc[t] = f32x4{};
#pragma unroll
      for (int s = 0; s < kDSteps; ++s) {
        const bf16x8 kf =
            *reinterpret_cast<const bf16x8*>(Ks + (16 * t + l16) * kKPitch + 32 * s + 8 * grp);
        sacc[t] = mfma16(kf, qf[s], sacc[t]);
      }
    }
    if (kv0 + kKeys > kend) {  // last, partial stage: keys past the end get -inf
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (kv0 + 16 * t + 4 * grp + r >= kend) sacc[t][r] = -INFINITY;
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) mloc = fmaxf(mloc, sacc[t][r]);
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    // scale > 0, so max(scale * s) = scale * max(s); e = 2^(scale s - m) with one FMA
    const float m_new = fmaxf(m_run, mloc * p.scale_log2);
    const float alpha = fast_exp2(m_run - m_new);
    m_run = m_new;
    float lsum = 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float e = fast_exp2(fmaf(sacc[t][r], p.scale_log2, -m_new));
        sacc[t][r] = e;
        lsum += e;
      }
    l_run = l_run * alpha + lsum;
    if (__any(alpha != 1.0f)) {  // some row's running max moved
#pragma unroll
      for (int t = 0; t < kDTiles; ++t) o[t] *= alpha;
    }

    // O^T += V^T P^T over 32-key steps u: k-slot 8 grp + j stands for key
    // 32 u + 16 (j / 4) + 4 grp + j % 4, which is where sacc[2u + j/4][j % 4] already sits.
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const u32x4 pb{pack2_bf16(sacc[2 * u][0], sacc[2 * u][1]),
                     pack2_bf16(sacc[2 * u][2], sacc[2 * u][3]),
                     pack2_bf16(sacc[2 * u + 1][0], sacc[2 * u + 1][1]),
                     pack2_bf16(sacc[2 * u + 1][2], sacc[2 * u + 1][3])};
      const bf16x8 pf = __builtin_bit_cast(bf16x8, pb);
#pragma unroll
      for (int t = 0; t < kDTiles; ++t) {
        const v4i16 lo = vt_read(32 * u, 16 * t);
        const v4i16 hi = vt_read(32 * u + 16, 16 * t);
        const v8i16 vv = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        o[t] = mfma16(__builtin_bit_cast(bf16x8, vv), pf, o[t]);
      }
    }
  }
  if (!active) return;

  // the four lane groups of a query hold disjoint keys: sum their l (same bits on every lane)
  float l_tot = l_run + __shfl_xor(l_run, 16);
  l_tot = l_tot + __shfl_xor(l_tot, 32);
  if (!row_ok) return;
  if (p.nsplit > 1) {
    const size_t idx = (static_cast<size_t>(bbeg + pos) * p.hq + g * G + hh) * p.nsplit + sp;
    float* dst = p.o_part + idx * D;
#pragma unroll
    for (int t = 0; t < kDTiles; ++t)
      *reinterpret_cast<f32x4*>(dst + 16 * t + 4 * grp) = o[t];
    if (grp == 0) {
      p.m_part[idx] = m_run;
      p.l_part[idx] = l_tot;
    }
    return;
  }
  const float inv = 1.0f / l_tot;
  uint16_t* dst = p.out + q_off;
#pragma unroll
  for (int t = 0; t < kDTiles; ++t) {
    const u32x2 v{pack2_bf16(o[t][0] * inv, o[t][1] * inv),
                  pack2_bf16(o[t][2] * inv, o[t][3] * inv)};
    *reinterpret_cast<u32x2*>(dst + 16 * t + 4 * grp) = v;
  }
}

}  // namespace
}  // namespace eb
