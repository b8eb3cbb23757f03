// Fused LM head + softmax statistics for gfx950.
//
// z = W h is formed tile by tile with bf16 MFMA (fp32 accumulation) and folded straight into
// per-(row, vocabulary tile) partials (max, sum of exponentials, entropy moment, argmax); the
// logits never leave registers.  A second kernel merges the partials of each row in a fixed
// order and emits kappa = 1/s, H = ln s - t/s, the argmax and the max logit.
//
// Orientation: the MFMA "row" dimension is the vocabulary and the "column" dimension is the
// block position, so every lane owns one position and reduces the logits it holds in
// registers before a single cross-half exchange.
#include "attn_small.hpp"
#include "eb_common.hpp"
#include "eb_internal.hpp"

namespace eb {
namespace {

// ---------------------------------------------------------------------------------------
// Streaming kernel for few block positions (n_rows <= 32 * NT).
//
// With a handful of positions the product is a bandwidth-bound pass over W.  One workgroup per
// compute unit owns a contiguous slice of vocabulary rows.  Each of its 16 waves (8 for slices
// above 768 rows) streams its share of the slice from HBM straight into MFMA A-operand
// registers, keeping kDepth k-steps of loads in flight; h, the B operand shared by all waves,
// goes through a double-buffered LDS chunk.  Every W byte is read once, by one lane, with no
// LDS round trip.  (Loading h per wave straight into registers instead, with no LDS and no
// barrier, measured 237 us against 203 us at 32 positions: the per-wave h traffic from L2 costs
// more than the shared chunks.)
// ---------------------------------------------------------------------------------------
#ifndef EB_STREAM_GROUPS
#define EB_STREAM_GROUPS 256
#endif
constexpr int kStreamGroups = EB_STREAM_GROUPS;  // workgroups (256: one per compute unit)

// The streaming kernel uses 16x16x32 MFMA tiles (mfma16).  A lane of the A operand holds 8
// consecutive k-values of row l % 16 and the four lanes of a row cover 64 contiguous bytes, so
// each load instruction reads 16 rows x 64 B of W (a 32x32x16 layout reads half that run per row
// and measured 4.65 TB/s at best against 5.4).

// Second-largest logit (with multiplicity) of the union of two sets whose largest values are
// m_a, m_b and second-largest m2_a, m2_b.  Exact and order-free, so every merge order gives
// the same bits.  kNegBig stands for "none".
__device__ __forceinline__ float top2_merge(float m_a, float m2_a, float m_b, float m2_b) {
  return fmaxf(fminf(m_a, m_b), fmaxf(m2_a, m2_b));
}

// top2_merge of a lane's (m, m2) with the lane `mask` away.
__device__ __forceinline__ float top2_shfl_merge(float m, float m2, int mask) {
  return top2_merge(m, m2, __shfl_xor(m, mask), __shfl_xor(m2, mask));
}

// kTop2: also track the second-largest logit of each (row, slice) into part2.
// kWaves waves per workgroup, TM 16-row tiles per wave, NT 16-position tiles.
// kAttnD != 0: workgroups n_slices and up run the small block attention (head dimension kAttnD)
// on unit blockIdx.x - n_slices of ap; the dispatcher starts them as the slices finish.
template <int kWaves, int TM, int NT, int kDepth, bool kTop2, int kAttnD>
__global__ __launch_bounds__(kWaves * 64) void lmhead_stream16_kernel(
    const uint16_t* __restrict__ h, const uint16_t* __restrict__ w, int n_rows, int hidden,
    int vocab, int rows_per_wg, Partial* __restrict__ part, float* __restrict__ part2,
    int n_slices, AttnParams ap) {
  static_assert(kAttnD == 0 || kWaves * 64 == kSmallThreads, "attention role shape");
  if constexpr (kAttnD != 0) {
    if (static_cast<int>(blockIdx.x) >= n_slices) {  // whole workgroup
      attn_small_role<kAttnD, kSmallThreads>(ap, static_cast<int>(blockIdx.x) - n_slices, 0);
      return;
    }
  }
  constexpr int KC = 1024 / NT;        // h columns per LDS chunk
  constexpr int kPitch = KC + 8;       // LDS row pitch (bf16)
  constexpr int kSpc = KC / 32;        // k-steps per chunk
  constexpr int kHRows = NT * 16;
  constexpr int kHChunks16 = kHRows * KC / 8;
  constexpr int kThreads = kWaves * 64;
  constexpr int kHPer = kHChunks16 / kThreads;
  static_assert(kHChunks16 % kThreads == 0, "h chunk splits evenly");
  static_assert(kSpc % kDepth == 0, "chunk boundary falls on a group boundary");
  __shared__ __attribute__((aligned(16))) uint16_t hs[2][kHRows * kPitch];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = lane >> 4, l16 = lane & 15;
  const int wg = blockIdx.x;
  const int vb = wg * rows_per_wg;
  const int ve = min(vocab, vb + rows_per_wg);
  const int rw = (rows_per_wg + kWaves - 1) / kWaves;
  const int wb = vb + wave * rw;
  const int we = min(ve, wb + rw);

  // Unconditional loads with clamped addresses, as in the 32x32 kernel.
  const int wlast = max(min(we, vocab) - 1, 0);
  const uint16_t* wp[TM];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int row = min(wb + tm * 16 + l16, wlast);
    wp[tm] = w + static_cast<size_t>(row) * hidden + 8 * grp;
  }
  const int nsteps = hidden / 32;
  const int nsteps_p = (nsteps + kDepth - 1) / kDepth * kDepth;
  const int nchunks = (hidden + KC - 1) / KC;

  u32x4 buf[kDepth][TM];
  auto issue = [&](int j, int step) {
    const int st = min(step, nsteps - 1);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) buf[j][tm] = *reinterpret_cast<const u32x4*>(wp[tm] + 32 * st);
  };
  u32x4 hreg[kHPer];
  auto load_h = [&](int c) {
#pragma unroll
    for (int i = 0; i < kHPer; ++i) {
      const int idx = tid + i * kThreads;
      const int row = min(idx / (KC / 8), n_rows - 1);
      const int col = min(c * KC + (idx % (KC / 8)) * 8, hidden - 8);
      hreg[i] = *reinterpret_cast<const u32x4*>(h + static_cast<size_t>(row) * hidden + col);
    }
  };
  auto store_h = [&](int b, int c) {
#pragma unroll
    for (int i = 0; i < kHPer; ++i) {
      const int idx = tid + i * kThreads;
      const int row = idx / (KC / 8), col = (idx % (KC / 8)) * 8;
      const bool ok = c * KC + col < hidden;
      *reinterpret_cast<u32x4*>(&hs[b][row * kPitch + col]) = ok ? hreg[i] : u32x4{0u, 0u, 0u, 0u};
    }
  };

  f32x4 acc[TM][NT];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < NT; ++b) acc[a][b] = f32x4{};

#pragma unroll
  for (int j = 0; j < kDepth; ++j) issue(j, j);
  load_h(0);
  store_h(0, 0);
  __syncthreads();
  if (nchunks > 1) load_h(1);

  auto consume = [&](int g, int j) {
    const uint16_t* hb = hs[(g / kSpc) & 1] + (g % kSpc) * 32 + 8 * grp + 32 * j;
    bf16x8 b[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      b[nt] = *reinterpret_cast<const bf16x8*>(hb + (nt * 16 + l16) * kPitch);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const bf16x8 a = __builtin_bit_cast(bf16x8, buf[j][tm]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[tm][nt] = mfma16(a, b[nt], acc[tm][nt]);
    }
  };
  auto chunk_boundary = [&](int g) {
    if (g > 0 && g % kSpc == 0) {
      const int c = g / kSpc;
      store_h(c & 1, c);
      __syncthreads();
      if (c + 1 < nchunks) load_h(c + 1);
    }
  };

  for (int g = 0; g < nsteps_p - kDepth; g += kDepth) {
    chunk_boundary(g);
#pragma unroll
    for (int j = 0; j < kDepth; ++j) {
      consume(g, j);
      issue(j, g + kDepth + j);
    }
  }
  chunk_boundary(nsteps_p - kDepth);
#pragma unroll
  for (int j = 0; j < kDepth; ++j) consume(nsteps_p - kDepth, j);

  __syncthreads();
  Partial* red = reinterpret_cast<Partial*>(&hs[0][0]);  // [kWaves][kHRows]
  float* red2 = reinterpret_cast<float*>(red + kWaves * kHRows);
  static_assert(kWaves * kHRows * (sizeof(Partial) + 4) <= sizeof(hs), "reduction fits");
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float m = kNegBig, m2 = kNegBig;
    int32_t idx = kNoIndex;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int v = wb + tm * 16 + 4 * grp + r;
        const float z = acc[tm][nt][r];
        if (kTop2 && v < we) m2 = __builtin_amdgcn_fmed3f(m, m2, z);
        if (v < we && z > m) {
          m = z;
          idx = v;
        }
      }
    float s = 0.f, t = 0.f;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int v = wb + tm * 16 + 4 * grp + r;
        if (v < we) {
          const float y = (acc[tm][nt][r] - m) * kLog2e;
          const float e = fast_exp2(y);
          s += e;
          t = fmaf(e, y, t);
        }
      }
    Partial p{m, s, t, idx};
    if (kTop2) m2 = top2_shfl_merge(p.m, m2, 16);
    p = partial_xor_merge(p, 16, lane);
    if (kTop2) m2 = top2_shfl_merge(p.m, m2, 32);
    p = partial_xor_merge(p, 32, lane);
    if (lane < 16) {
      red[wave * kHRows + nt * 16 + l16] = p;
      if (kTop2) red2[wave * kHRows + nt * 16 + l16] = m2;
    }
  }
  __syncthreads();
  if (tid < kHRows && tid < n_rows) {
    Partial p = red[tid];
    float m2 = kTop2 ? red2[tid] : kNegBig;
#pragma unroll
    for (int k = 1; k < kWaves; ++k) {
      const Partial q = red[k * kHRows + tid];
      if (kTop2) m2 = top2_merge(p.m, m2, q.m, red2[k * kHRows + tid]);
      p = partial_merge(p, q);
    }
    part[static_cast<size_t>(tid) * n_slices + wg] = p;
    if (kTop2) part2[static_cast<size_t>(tid) * n_slices + wg] = m2;
  }
}

// k-steps of W loads in flight per wave with 16 waves (measured on MI355X; the macro exists so
// that other settings can be built and timed).
#ifndef EB_STREAM_DEPTH
#define EB_STREAM_DEPTH 8
#endif
constexpr int kStreamShape = 16;  // rows (and positions) per MFMA tile
constexpr int kStreamDepth = EB_STREAM_DEPTH;
// 16 waves per workgroup while each wave's share of the slice fits in kStreamMaxTm16 row tiles
// (at 1024 threads a lane has 128 VGPRs; four tiles with two or more position tiles spill), else
// 8 waves, which leaves 256 VGPRs per lane for up to 8 row tiles (16 waves with depth 8 measured
// 186 us against 195 us for 8 waves with depth 2 at 32 positions of a 126464 x 4096 head).
constexpr int kStreamMaxTm16 = 3;
constexpr int kStreamMaxTm8 = 8;

struct StreamPlan {
  int groups, rows_per_wg, waves, tm;  // tm: MFMA row tiles per wave
};

StreamPlan stream_plan(int vocab) {
  const int groups = min(kStreamGroups, (vocab + 31) / 32);
  const int rows = (vocab + groups - 1) / groups;
  auto tiles = [&](int waves) {
    const int rw = (rows + waves - 1) / waves;
    return (rw + kStreamShape - 1) / kStreamShape;
  };
  if (tiles(16) <= kStreamMaxTm16) return StreamPlan{groups, rows, 16, tiles(16)};
  return StreamPlan{groups, rows, 8, tiles(8)};
}

constexpr int kStreamMaxRows = 64;  // n_rows handled by the streaming kernel

bool use_stream(int n_rows, int vocab) {
  if (n_rows > kStreamMaxRows) return false;
  const StreamPlan pl = stream_plan(vocab);
  if (pl.waves == 16) return true;
  if (n_rows > 2 * kStreamShape) return pl.tm <= 6;  // register budget with four position tiles
  return pl.tm <= kStreamMaxTm8;
}

// Block attention queued behind the slices of a streaming launch (attn_d 0: none).
struct HostedAttn {
  AttnParams p;
  int units, attn_d;
};

template <int kWaves, int TM, int NT, bool kTop2, int kAttnD = 0>
hipError_t launch_stream_tm(int n_rows, int hidden, int vocab, const StreamPlan& pl,
                            const void* h, const void* w, Partial* part, float* part2,
                            hipStream_t s, const HostedAttn& ha) {
  // 16 waves: up to 16 W registers in flight per lane (16 bytes each; 8 with four position
  // tiles), at most kStreamDepth k-steps.  8 waves: two k-steps (more measured no faster).
  constexpr int kBudget = kWaves == 8 ? 2 * TM : (NT >= 4 ? 8 : 16);
  constexpr int D0 = kBudget / TM >= 1 ? kBudget / TM : 1;
  constexpr int D = (kWaves == 16 && D0 > kStreamDepth) ? kStreamDepth : D0;
  // a power of two that divides the per-chunk step count
  constexpr int Dp = D >= 8 ? 8 : (D >= 4 ? 4 : (D >= 2 ? 2 : 1));
  const int extra = kAttnD != 0 ? ha.units : 0;
  hipLaunchKernelGGL((lmhead_stream16_kernel<kWaves, TM, NT, Dp, kTop2, kAttnD>),
                     dim3(pl.groups + extra), dim3(kWaves * 64), 0, s,
                     static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(w), n_rows,
                     hidden, vocab, pl.rows_per_wg, part, part2, pl.groups, ha.p);
  return hipGetLastError();
}

// 16 waves, TM row tiles: the variant for the hosted attention's head dimension.
template <int TM, int NT, bool kTop2>
hipError_t launch_stream16(int n_rows, int hidden, int vocab, const StreamPlan& pl,
                           const void* h, const void* w, Partial* part, float* part2,
                           hipStream_t s, const HostedAttn& ha) {
  if constexpr (!kTop2) {
    if (ha.attn_d == 128)
      return launch_stream_tm<16, TM, NT, false, 128>(n_rows, hidden, vocab, pl, h, w, part,
                                                      part2, s, ha);
    if (ha.attn_d == 64)
      return launch_stream_tm<16, TM, NT, false, 64>(n_rows, hidden, vocab, pl, h, w, part,
                                                     part2, s, ha);
  }
  if (ha.attn_d != 0) return hipErrorInvalidValue;  // excluded by lmhead_hosts_attn
  return launch_stream_tm<16, TM, NT, kTop2>(n_rows, hidden, vocab, pl, h, w, part, part2, s,
                                             ha);
}

// NT: 16-position tiles covering n_rows.
template <int NT, bool kTop2>
hipError_t launch_stream(int n_rows, int hidden, int vocab, const void* h, const void* w,
                         Partial* part, float* part2, hipStream_t s, const HostedAttn& ha) {
  const StreamPlan pl = stream_plan(vocab);
  if (pl.waves == 16) {
    switch (pl.tm) {
      case 1:
        return launch_stream16<1, NT, kTop2>(n_rows, hidden, vocab, pl, h, w, part, part2, s, ha);
      case 2:
        return launch_stream16<2, NT, kTop2>(n_rows, hidden, vocab, pl, h, w, part, part2, s, ha);
      case 3:
        return launch_stream16<3, NT, kTop2>(n_rows, hidden, vocab, pl, h, w, part, part2, s, ha);
      default: return hipErrorInvalidValue;  // excluded by stream_plan
    }
  }
  if (ha.attn_d != 0) return hipErrorInvalidValue;  // excluded by lmhead_hosts_attn
  // More than 48 tiles of rows per workgroup: the 8-wave shape has 7 or 8 tiles per wave.
  switch (pl.tm) {
    case 7:
      if constexpr (NT < 4)
        return launch_stream_tm<8, 7, NT, kTop2>(n_rows, hidden, vocab, pl, h, w, part, part2, s,
                                                 ha);
      return hipErrorInvalidValue;
    case 8:
      if constexpr (NT < 4)
        return launch_stream_tm<8, 8, NT, kTop2>(n_rows, hidden, vocab, pl, h, w, part, part2, s,
                                                 ha);
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;  // excluded by use_stream
  }
}

template <bool kTop2>
hipError_t launch_stream_rows(int n_rows, int hidden, int vocab, const void* h, const void* w,
                              Partial* part, float* part2, hipStream_t s,
                              const HostedAttn& ha = HostedAttn{}) {
  if (n_rows <= 16)
    return launch_stream<1, kTop2>(n_rows, hidden, vocab, h, w, part, part2, s, ha);
  if (n_rows <= 32)
    return launch_stream<2, kTop2>(n_rows, hidden, vocab, h, w, part, part2, s, ha);
  if (n_rows <= 64)
    return launch_stream<4, kTop2>(n_rows, hidden, vocab, h, w, part, part2, s, ha);
  return hipErrorInvalidValue;  // excluded by use_stream
}

// ---------------------------------------------------------------------------------------
// Large-batch kernel: 256 (vocabulary) x 256 (positions) tiles.
//
// Both operands are streamed HBM -> LDS by direct loads (global_load_lds_dwordx4: lane l of a
// wave writes its 16 bytes to LDS base + 16 l) into a ring of RING stages of BK = 32 hidden
// columns, RING - 1 stages in flight; no staging registers and no LDS store instructions.  LDS
// rows are 64 bytes without padding; the 16-byte chunk c of row r is kept in slot
// c ^ ((r / 4) % 4), which makes the 32-row MFMA operand reads free of bank conflicts.
// Four waves form a 2 x 2 grid of 128 x 128 sub-tiles of 32x32x16 MFMA blocks.
//
// Launch order is XCD-aware: vocabulary tiles are grouped in bands of kBand, band b goes to XCD
// b % 8 (workgroups are dealt to the 8 XCDs round-robin by id), and each XCD sweeps its band row
// tile by row tile, so the workgroups an XCD runs at once share a few W and h tiles in its L2
// and each W tile is fetched from HBM about once.
// ---------------------------------------------------------------------------------------
constexpr int kXcds = 8;
constexpr int kBand = 4;
constexpr int kTileBM = 256;
constexpr int kTileBK = 32;

struct TileMap {
  int n_vtiles, n_rtiles, n_bands, grid;
};

TileMap tile_map(int n_rows, int vocab, int bn) {
  TileMap m;
  m.n_vtiles = (vocab + kTileBM - 1) / kTileBM;
  m.n_rtiles = (n_rows + bn - 1) / bn;
  m.n_bands = (m.n_vtiles + kBand - 1) / kBand;
  const int bands_per_xcd = (m.n_bands + kXcds - 1) / kXcds;
  m.grid = kXcds * bands_per_xcd * kBand * m.n_rtiles;
  return m;
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void global_void_t;

__device__ __forceinline__ void load_to_lds(const void* g, void* l) {
  // address-space casts (generic -> global / LDS) need C-style casts
  __builtin_amdgcn_global_load_lds((global_void_t*)(const_cast<void*>(g)), (lds_void_t*)(l), 16, 0,
                                   0);
}

// Partial statistics of one lane's column over TM 32-row MFMA blocks.  Element (tm, r) of the
// lane is vocabulary row vbase + o with o = 32 tm + 8 (r / 4) + (r % 4).  Four independent chains
// (by r % 4) carry the max, the sums and the first argmax, so the reduction is not bound by the
// latency of one long dependency chain; each chain walks its rows in decreasing order, so its
// last z == max hit is its lowest row, and the chains are combined at the end.  The argmax is
// tracked as the offset o, a constant of the unrolled code, and kFull (every row inside the
// vocabulary) drops the per-row bounds test: neither a row index nor a mask is then kept per
// element.  With kTop2 the max pass also tracks each chain's second-largest logit; m2 returns
// the lane's second-largest (kNegBig if none).
template <int TM, int TN, bool kTop2, bool kFull>
__device__ __forceinline__ Partial column_partial(const f32x16 (&acc)[TM][TN], int tn, int vbase,
                                                  int vocab, float* m2) {
  float mc[4] = {kNegBig, kNegBig, kNegBig, kNegBig};
  float mc2[4] = {kNegBig, kNegBig, kNegBig, kNegBig};
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int o = tm * 32 + 8 * (r >> 2) + (r & 3);
      if (kFull || vbase + o < vocab) {
        const float z = acc[tm][tn][r];
        // with mc >= mc2, the new second-largest is the median of (mc, mc2, z): one v_med3
        if (kTop2) mc2[r & 3] = __builtin_amdgcn_fmed3f(mc[r & 3], mc2[r & 3], z);
        mc[r & 3] = fmaxf(mc[r & 3], z);
      }
    }
  const float m = fmaxf(fmaxf(mc[0], mc[1]), fmaxf(mc[2], mc[3]));
  if (kTop2)
    *m2 = top2_merge(fmaxf(mc[0], mc[1]), top2_merge(mc[0], mc2[0], mc[1], mc2[1]),
                     fmaxf(mc[2], mc[3]), top2_merge(mc[2], mc2[2], mc[3], mc2[3]));
  float sc[4] = {0.f, 0.f, 0.f, 0.f}, tc[4] = {0.f, 0.f, 0.f, 0.f};
  int32_t oc[4] = {kNoIndex, kNoIndex, kNoIndex, kNoIndex};
#pragma unroll
  for (int tm = TM - 1; tm >= 0; --tm)
#pragma unroll
    for (int r = 15; r >= 0; --r) {
      const int o = tm * 32 + 8 * (r >> 2) + (r & 3);
      const float z = acc[tm][tn][r];
      if (kFull) {
        const float y = (z - m) * kLog2e;
        const float e = fast_exp2(y);
        sc[r & 3] += e;
        tc[r & 3] = fmaf(e, y, tc[r & 3]);
        oc[r & 3] = z == m ? o : oc[r & 3];
      } else {
        const bool ok = vbase + o < vocab;
        // rows past the vocabulary contribute e = 0 and y = 0 (a lane with no valid row keeps
        // m = kNegBig, where z - m would overflow and 0 * inf would poison t)
        const float y = ok ? (z - m) * kLog2e : 0.f;
        const float e = ok ? fast_exp2(y) : 0.f;
        sc[r & 3] += e;
        tc[r & 3] = fmaf(e, y, tc[r & 3]);
        oc[r & 3] = (ok && z == m) ? o : oc[r & 3];
      }
    }
  const int32_t ob = min(min(oc[0], oc[1]), min(oc[2], oc[3]));
  return Partial{m, (sc[0] + sc[1]) + (sc[2] + sc[3]), (tc[0] + tc[1]) + (tc[2] + tc[3]),
                 ob == kNoIndex ? kNoIndex : vbase + ob};
}

// column_partial with the bounds test only where the tile reaches past the vocabulary.
template <int TM, int TN, bool kTop2>
__device__ __forceinline__ Partial column_partial(const f32x16 (&acc)[TM][TN], int tn, int vbase,
                                                  int vocab, bool full, float* m2) {
  return full ? column_partial<TM, TN, kTop2, true>(acc, tn, vbase, vocab, m2)
              : column_partial<TM, TN, kTop2, false>(acc, tn, vbase, vocab, m2);
}

// Wait until at most N vector-memory instructions of this wave are outstanding and all of its
// LDS reads have returned, then barrier.
template <int N>
__device__ __forceinline__ void wait_vm_lds_and_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0x0 << 8));
  asm volatile("s_barrier" ::: "memory");
}

// 256 x 256 tiles computed by 4 waves as a 2 x 2 grid of 128 x 128 sub-tiles (4 x 4 blocks of
// 32x32x16 MFMAs, 256 accumulator registers per lane).  Per 32-column k step a wave reads
// 16 KB of operand fragments from LDS (the 8-wave 128 x 64 split reads 12 KB per wave, 96 KB
// per tile against 64 KB here).  The fragments of the two 16-column halves of a k step are
// double-buffered in registers: the reads of one half are issued before the MFMAs of the
// other, so LDS latency hides under 16 MFMAs.  The DMA ring keeps RING stages occupied: right
// after the barrier that ends the reads of stage kt, stage kt + RING is issued into its slot.
template <int RING, bool kTop2>
__global__ __launch_bounds__(256, 1) void lmhead_tile4_kernel(
    const uint16_t* __restrict__ h, const uint16_t* __restrict__ w, int n_rows, int hidden,
    int vocab, int n_vtiles, int n_rtiles, int n_bands, Partial* __restrict__ part,
    float* __restrict__ part2) {
  constexpr int BM = kTileBM, BN = 256, BK = kTileBK;
  constexpr int WM = 2, WN = 2, kWaves = WM * WN;
  constexpr int kWaveM = BM / WM, kWaveN = BN / WN;
  constexpr int TM = kWaveM / 32, TN = kWaveN / 32;
  constexpr int kRowB = BK * 2;                   // 64 bytes per LDS row
  constexpr int kStageBytes = (BM + BN) * kRowB;  // 32 KB
  constexpr int kInst = (BM + BN) / 16;           // 1 KB wave instructions per stage
  constexpr int kInstPerWave = kInst / kWaves;    // 8
  static_assert(RING >= 2 && RING <= 4, "ring of 2 to 4 stages");
  static_assert((RING - 1) * kInstPerWave < 64, "vmcnt range");
  __shared__ __attribute__((aligned(16))) uint8_t smem[RING * kStageBytes];
  static_assert(WM * BN * sizeof(Partial) <= RING * kStageBytes, "reduction fits in the ring");

  const int id = blockIdx.x;
  const int xcd = id % kXcds, k = id / kXcds;
  const int per_band = kBand * n_rtiles;
  const int band = xcd + kXcds * (k / per_band);
  if (band >= n_bands) return;
  const int tt = k % per_band;
  const int nv = min(kBand, n_vtiles - band * kBand);
  if (tt >= nv * n_rtiles) return;
  const int vt = band * kBand + tt % nv;
  const int rt = tt / nv;
  const int v0 = vt * BM, r0 = rt * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int half = lane >> 5, l32 = lane & 31;

  // Load instruction i of this wave covers tile rows 16 q .. 16 q + 15, q = wave * 8 + i (rows
  // below BM are W, the rest h); lane L fetches row 16 q + L / 4, global chunk
  // (L % 4) ^ swizzle(row) into LDS slot L % 4 of the row.  Rows past the end are clamped.
  const uint16_t* src[kInstPerWave];
#pragma unroll
  for (int i = 0; i < kInstPerWave; ++i) {
    const int q = wave * kInstPerWave + i;
    const int row = 16 * q + (lane >> 2);
    const int chunk = (lane & 3) ^ ((row >> 2) & 3);
    src[i] = row < BM
                 ? w + static_cast<size_t>(min(v0 + row, vocab - 1)) * hidden + chunk * 8
                 : h + static_cast<size_t>(min(r0 + row - BM, n_rows - 1)) * hidden + chunk * 8;
  }
  // Stage `stage` of the k loop into ring slot `slot`.
  auto issue = [&](int stage, int slot) {
    uint8_t* base = smem + slot * kStageBytes;
#pragma unroll
    for (int i = 0; i < kInstPerWave; ++i)
      load_to_lds(src[i] + stage * BK, base + (wave * kInstPerWave + i) * 1024);
  };
  // Fragments of half s (k columns 16 s .. 16 s + 15 of the stage, chunk 2 half + s per lane).
  auto read = [&](int kt, int s, bf16x8 (&a)[TM], bf16x8 (&b)[TN]) {
    const uint8_t* st = smem + (kt % RING) * kStageBytes;
    const int c = 2 * half + s;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int r = wm * kWaveM + tm * 32 + l32;
      a[tm] = *reinterpret_cast<const bf16x8*>(st + r * kRowB + 16 * (c ^ ((r >> 2) & 3)));
    }
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int r = BM + wn * kWaveN + tn * 32 + l32;
      b[tn] = *reinterpret_cast<const bf16x8*>(st + r * kRowB + 16 * (c ^ ((r >> 2) & 3)));
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b) acc[a][b] = f32x16{};
  auto mma = [&](const bf16x8 (&a)[TM], const bf16x8 (&b)[TN]) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = mfma32(a[tm], b[tn], acc[tm][tn]);
  };
  // Every iteration issues exactly one stage (past the end: the last stage again, into the slot
  // just freed, never read), so the number of younger stages in flight at each barrier is
  // always RING - 2 and every wait is the same; straight-line code lets the fragment reads of
  // one half stay in flight under the MFMAs of the other.
  const int nk = hidden / BK;  // >= 1
#pragma unroll
  for (int j = 0; j < RING; ++j) issue(min(j, nk - 1), j);
  wait_vm_lds_and_barrier<(RING - 1) * kInstPerWave>();
  bf16x8 xa[TM], xb[TN], ya[TM], yb[TN];
  read(0, 0, xa, xb);
  for (int kt = 0; kt + 1 < nk; ++kt) {
    read(kt, 1, ya, yb);
    mma(xa, xb);
    // one fragment read after each of the first 8 MFMAs
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    __builtin_amdgcn_sched_barrier(0);
    wait_vm_lds_and_barrier<(RING - 2) * kInstPerWave>();  // stage kt + 1 has landed
    issue(min(kt + RING, nk - 1), kt % RING);               // slot of stage kt, fully read
    read(kt + 1, 0, xa, xb);
    mma(ya, yb);
    // one DMA load after each of the first 8 MFMAs, one fragment read after each of the rest
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x010, 1, 0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  read(nk - 1, 1, ya, yb);
  mma(xa, xb);
  mma(ya, yb);
  wait_vm_lds_and_barrier<0>();  // no DMA in flight; every wave is done reading the ring

  Partial* red = reinterpret_cast<Partial*>(smem);  // [WM][BN]
  float* red2 = reinterpret_cast<float*>(red + WM * BN);
  static_assert(WM * BN * (sizeof(Partial) + 4) <= sizeof(smem), "reduction fits in LDS");
  const bool full = v0 + BM <= vocab;
  const int vbase = v0 + wm * kWaveM + 4 * half;
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
    float m2 = kNegBig;
    Partial p = column_partial<TM, TN, kTop2>(acc, tn, vbase, vocab, full, &m2);
    if (kTop2) m2 = top2_shfl_merge(p.m, m2, 32);
    p = partial_xor_merge(p, 32, lane);
    if (lane < 32) {
      red[wm * BN + wn * kWaveN + tn * 32 + l32] = p;
      if (kTop2) red2[wm * BN + wn * kWaveN + tn * 32 + l32] = m2;
    }
  }
  __syncthreads();
  for (int c = tid; c < BN; c += kWaves * 64) {
    Partial p = red[c];
    float m2 = kTop2 ? red2[c] : kNegBig;
#pragma unroll
    for (int q = 1; q < WM; ++q) {
      const Partial o = red[q * BN + c];
      if (kTop2) m2 = top2_merge(p.m, m2, o.m, red2[q * BN + c]);
      p = partial_merge(p, o);
    }
    const int row = r0 + c;
    if (row < n_rows) {
      part[static_cast<size_t>(row) * n_vtiles + vt] = p;
      if (kTop2) part2[static_cast<size_t>(row) * n_vtiles + vt] = m2;
    }
  }
}

// Tile kernel of the large-batch path: lmhead_tile4_kernel, 256 x 256 tiles, 4 waves of
// 128 x 128, ring of 4 (128 KB LDS, one workgroup per compute unit); batch 64: 9.6 ms.
// Measured and dropped: 8 waves of 128 x 64 (10.55 ms), 256 x 128 tiles with a ring of 3 at two
// workgroups per compute unit (11.8 ms), stages reaching LDS through registers (9.65 ms),
// 64-column stages with one barrier per 64 MFMAs (10.1 ms), DMA loads spread over both halves of
// a step (no change); with every operand L2-resident the kernel runs at the same speed, so it is
// bound by the issue/LDS schedule of one wave per SIMD, not by memory.
constexpr int kTileBN = 256;

template <bool kTop2>
hipError_t launch_tile(int n_rows, int hidden, int vocab, const void* h, const void* w,
                       Partial* part, float* part2, hipStream_t s) {
  const TileMap m = tile_map(n_rows, vocab, kTileBN);
  hipLaunchKernelGGL((lmhead_tile4_kernel<4, kTop2>), dim3(m.grid), dim3(256), 0, s,
                     static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(w), n_rows,
                     hidden, vocab, m.n_vtiles, m.n_rtiles, m.n_bands, part, part2);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// fp32 kernel (small shapes): one thread per vocabulary entry, plain fp32 FMA dot products.
// ---------------------------------------------------------------------------------------
constexpr int kF32SliceRows = 256;

template <bool kTop2>
__global__ __launch_bounds__(256) void lmhead_f32_kernel(const float* __restrict__ h,
                                                         const float* __restrict__ w,
                                                         int n_rows, int hidden, int vocab,
                                                         int n_slices,
                                                         Partial* __restrict__ part,
                                                         float* __restrict__ part2) {
  __shared__ Partial red[4];
  __shared__ float red2[4];
  const int slice = blockIdx.x;
  const int row = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int v = slice * kF32SliceRows + threadIdx.x;
  Partial p = partial_empty();
  float m2 = kNegBig;
  if (v < vocab) {
    const float* wr = w + static_cast<size_t>(v) * hidden;
    const float* hr = h + static_cast<size_t>(row) * hidden;
    float z = 0.f;
    for (int k = 0; k < hidden; ++k) z = fmaf(wr[k], hr[k], z);
    p = Partial{z, 1.f, 0.f, v};
  }
  for (int mask = 32; mask >= 1; mask >>= 1) {
    if (kTop2) m2 = top2_shfl_merge(p.m, m2, mask);
    p = partial_xor_merge(p, mask, lane);
  }
  if (lane == 0) {
    red[wave] = p;
    red2[wave] = m2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    Partial q = red[0];
    float q2 = red2[0];
    for (int k = 1; k < 4; ++k) {
      if (kTop2) q2 = top2_merge(q.m, q2, red[k].m, red2[k]);
      q = partial_merge(q, red[k]);
    }
    part[static_cast<size_t>(row) * n_slices + slice] = q;
    if (kTop2) part2[static_cast<size_t>(row) * n_slices + slice] = q2;
  }
}

// ---------------------------------------------------------------------------------------
// combine: one wavefront per row, fixed merge order (lane-strided, then butterfly)
// ---------------------------------------------------------------------------------------
template <bool kTop2>
__global__ __launch_bounds__(256) void lmhead_combine_kernel(const Partial* __restrict__ part,
                                                             const float* __restrict__ part2,
                                                             int n_rows, int n_slices,
                                                             float* __restrict__ conf,
                                                             float* __restrict__ entropy,
                                                             int32_t* __restrict__ argmax,
                                                             float* __restrict__ max_logit,
                                                             float* __restrict__ top2_gap) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;  // uniform per wavefront
  const Partial* pr = part + static_cast<size_t>(row) * n_slices;
  const Partial p = wave_merge(pr, n_slices, lane);
  float m2 = kNegBig;
  if (kTop2) {
    // (max, second max) over the slices: lane-strided, then a butterfly; exact in any order
    float m = kNegBig;
    const float* p2 = part2 + static_cast<size_t>(row) * n_slices;
    for (int j = lane; j < n_slices; j += 64) {
      const float mj = pr[j].m;
      m2 = top2_merge(m, m2, mj, p2[j]);
      m = fmaxf(m, mj);
    }
    for (int mask = 32; mask >= 1; mask >>= 1) {
      m2 = top2_shfl_merge(m, m2, mask);
      m = fmaxf(m, __shfl_xor(m, mask));
    }
  }
  if (lane == 0) {
    write_row_stats(p, row, conf, entropy, argmax, max_logit);
    // p_(1) - p_(2) = (1 - e^(z2 - m)) / s; 0 when the maximum is shared (z2 = m)
    if (kTop2) top2_gap[row] = (1.0f - fast_exp2((m2 - p.m) * kLog2e)) * (1.0f / p.s);
  }
}

}  // namespace

int lmhead_num_slices(bool bf16, int n_rows, int vocab) {
  if (bf16 && use_stream(n_rows, vocab)) return stream_plan(vocab).groups;
  if (bf16) return tile_map(n_rows, vocab, kTileBN).n_vtiles;
  return (vocab + kF32SliceRows - 1) / kF32SliceRows;
}

// Workspace: partials [n_rows, n_slices] (16 B each), then with top2 the second-largest logits
// [n_rows, n_slices] (4 B each) from the next 256-byte boundary.
static size_t lmhead_part_bytes(bool bf16, int n_rows, int vocab) {
  const size_t b = static_cast<size_t>(n_rows) * lmhead_num_slices(bf16, n_rows, vocab) *
                   sizeof(Partial);
  return (b + 255) / 256 * 256;
}

size_t lmhead_ws_bytes(bool bf16, int n_rows, int vocab, bool top2) {
  size_t b = lmhead_part_bytes(bf16, n_rows, vocab);
  if (top2) b += static_cast<size_t>(n_rows) * lmhead_num_slices(bf16, n_rows, vocab) * 4;
  return b;
}

hipError_t lmhead_partials(bool bf16, int n_rows, int hidden, int vocab, const void* h,
                           const void* w, void* ws, bool top2, hipStream_t s) {
  if (n_rows == 0) return hipSuccess;
  Partial* part = static_cast<Partial*>(ws);
  float* part2 = top2 ? reinterpret_cast<float*>(static_cast<char*>(ws) +
                                                 lmhead_part_bytes(bf16, n_rows, vocab))
                      : nullptr;
  if (!bf16) {
    const int n_slices = lmhead_num_slices(false, n_rows, vocab);
    dim3 grid(n_slices, n_rows);
    const float* hp = static_cast<const float*>(h);
    const float* wp = static_cast<const float*>(w);
    if (top2)
      hipLaunchKernelGGL(lmhead_f32_kernel<true>, grid, dim3(256), 0, s, hp, wp, n_rows, hidden,
                         vocab, n_slices, part, part2);
    else
      hipLaunchKernelGGL(lmhead_f32_kernel<false>, grid, dim3(256), 0, s, hp, wp, n_rows, hidden,
                         vocab, n_slices, part, part2);
    return hipGetLastError();
  }
  if (use_stream(n_rows, vocab))
    return top2 ? launch_stream_rows<true>(n_rows, hidden, vocab, h, w, part, part2, s)
                : launch_stream_rows<false>(n_rows, hidden, vocab, h, w, part, part2, s);
  return top2 ? launch_tile<true>(n_rows, hidden, vocab, h, w, part, part2, s)
              : launch_tile<false>(n_rows, hidden, vocab, h, w, part, part2, s);
}

bool lmhead_hosts_attn(bool bf16, int n_rows, int vocab, const AttnArgs& a) {
  return bf16 && n_rows > 0 && use_stream(n_rows, vocab) && stream_plan(vocab).waves == 16 &&
         attn_small_ok(bf16, a);
}

hipError_t lmhead_partials_attn(int n_rows, int hidden, int vocab, const void* h, const void* w,
                                void* ws, const AttnArgs& a, void* attn_ws, hipStream_t s) {
  const SplitPlan sp = split_plan(a.batch, a.max_block, attn_max_keys(a), a.hq, a.hkv);
  const HostedAttn ha{attn_params(a, sp, attn_ws), attn_small_units(a, sp), a.head_dim};
  return launch_stream_rows<false>(n_rows, hidden, vocab, h, w, static_cast<Partial*>(ws),
                                   nullptr, s, ha);
}

hipError_t lmhead_combine(bool bf16, int n_rows, int vocab, const void* ws, float* conf,
                          float* entropy, int32_t* argmax, float* max_logit, float* top2_gap,
                          hipStream_t s) {
  if (n_rows == 0) return hipSuccess;
  const int n_slices = lmhead_num_slices(bf16, n_rows, vocab);
  const Partial* part = static_cast<const Partial*>(ws);
  const dim3 grid((n_rows + 3) / 4);
  if (top2_gap) {
    const float* part2 = reinterpret_cast<const float*>(static_cast<const char*>(ws) +
                                                        lmhead_part_bytes(bf16, n_rows, vocab));
    hipLaunchKernelGGL(lmhead_combine_kernel<true>, grid, dim3(256), 0, s, part, part2, n_rows,
                       n_slices, conf, entropy, argmax, max_logit, top2_gap);
  } else {
    hipLaunchKernelGGL(lmhead_combine_kernel<false>, grid, dim3(256), 0, s, part, nullptr,
                       n_rows, n_slices, conf, entropy, argmax, max_logit, nullptr);
  }
  return hipGetLastError();
}

}  // namespace eb
