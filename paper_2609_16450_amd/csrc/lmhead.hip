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
// Both operands go HBM/L2 -> LDS by buffer loads straight into LDS (lane l of a wave writes its
// 16 bytes to LDS base + 16 l) into a ring of RING stages of BK = 32 hidden columns, RING - 1
// stages in flight; no staging registers and no LDS store instructions.  LDS rows are 64 bytes
// without padding; the 16-byte chunk c of row r is kept in slot c ^ ((r / 4) % 4), which makes
// the 16-row MFMA operand reads (rows in the order rho of lmhead_tile_kernel) free of bank
// conflicts.  Four waves form a 2 x 2 grid of 128 x 128 sub-tiles of 16x16x32 MFMA blocks.
//
// Tile order is XCD-aware: the launch sequence takes vocabulary tiles in bands of kBand, each
// band swept position tile by position tile, and is cut into one contiguous segment per XCD
// (lmhead_tile_kernel), so the workgroups an XCD runs at once work on neighbouring tiles that
// share a few W and h tiles in its L2.
// ---------------------------------------------------------------------------------------
constexpr int kXcds = 8;
constexpr int kBand = 4;
constexpr int kTileBM = 256;     // vocabulary rows per tile
constexpr int kTileBN = 256;     // block positions per tile
constexpr int kTileBK = 32;      // hidden columns per ring stage
constexpr int kTileRing = 4;     // ring stages
constexpr int kTileGroups = 256; // persistent workgroups (one per compute unit)

int tile_vtiles(int vocab) { return (vocab + kTileBM - 1) / kTileBM; }

// 16x16x32 MFMA with its accumulator tied to the same AGPRs as input and output.  Written as asm:
// with the builtin, the compiler picks the untied form for this size and moves the accumulators
// through other registers around every MFMA of a 64-accumulator loop (hundreds of copies per
// step, seen in the ISA).
__device__ __forceinline__ void mfma16_tied(f32x4& c, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}

// The compiler does not see that the asm above is an MFMA, so it inserts none of the wait states
// between an MFMA and other instructions touching its accumulators.  Every accumulator passes
// through an empty asm that "writes" it, which no access of it can cross, and s_nops supply the
// wait states: acc_fence_in after the accumulators are written and before the first MFMA reads
// them, acc_fence_out after the last MFMA and before anything reads its results.
template <int TM, int TN>
__device__ __forceinline__ void acc_fence_in(f32x4 (&acc)[TM][TN]) {
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b) asm volatile("" : "+a"(acc[a][b]));
  asm volatile("s_nop 7");
}
template <int TM, int TN>
__device__ __forceinline__ void acc_fence_out(f32x4 (&acc)[TM][TN]) {
  asm volatile("s_nop 7\n s_nop 7\n s_nop 7\n s_nop 7");
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b) asm volatile("" : "+a"(acc[a][b]));
}

// Reductions over the four lanes l % 16 + 16 q (q < 4) of a column, in registers: the gfx950
// swaps v_permlane16_swap / v_permlane32_swap hand every lane the values of the lower and upper
// lane of its pair (l & ~16 and l | 16, then l & ~32 and l | 32), which are combined as
// lower op upper, so both lanes of a pair evaluate the same expression and end with the same
// bits.
__device__ __forceinline__ void lane_pair16(float x, float& lo, float& hi) {
  const auto r =
      __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
}
__device__ __forceinline__ void lane_pair32(float x, float& lo, float& hi) {
  const auto r =
      __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
}
__device__ __forceinline__ float pair_max(float m) {
  float lo, hi;
  lane_pair16(m, lo, hi);
  m = fmaxf(lo, hi);
  lane_pair32(m, lo, hi);
  return fmaxf(lo, hi);
}
__device__ __forceinline__ void pair_sum_min(float& s, float& t, int32_t& idx) {
  float lo, hi, lo2, hi2, lo3, hi3;
  lane_pair16(s, lo, hi);
  lane_pair16(t, lo2, hi2);
  lane_pair16(__int_as_float(idx), lo3, hi3);
  s = lo + hi;
  t = lo2 + hi2;
  idx = min(__float_as_int(lo3), __float_as_int(hi3));
  lane_pair32(s, lo, hi);
  lane_pair32(t, lo2, hi2);
  lane_pair32(__int_as_float(idx), lo3, hi3);
  s = lo + hi;
  t = lo2 + hi2;
  idx = min(__float_as_int(lo3), __float_as_int(hi3));
}

// Statistics of one column of a wave's 16x16x32 accumulator tile: lane l holds, for column block
// tn, vocabulary rows vbase + 16 tm + 4 r (tm < TM, r < 4; vbase includes the lane's l / 16) of
// one column, and the four lanes l % 16 + 16 q together hold the column's 16 TM rows (the rows
// of a 16-row block reach the MFMA in the order the fragment reads use, see
// lmhead_tile_kernel).  A max pass in four chains (by r), the column maximum M over the four
// lanes (pair_max), one exponential pass against M, then the four lanes' sums added pairwise in
// registers (pair_sum_min): identical bits on all four lanes.  Each chain walks its rows in
// decreasing order, so its last z == M is its lowest row; the argmax is kept as the block index
// tm, a constant of the unrolled code.  kFull (every row inside the vocabulary) drops the
// per-row bounds test.  With kTop2, m2 returns the column's second-largest logit (kNegBig if
// none).
template <int TM, int TN, bool kTop2, bool kFull>
__device__ __forceinline__ Partial column_stats16(const f32x4 (&acc)[TM][TN], int tn, int vbase,
                                                  int vocab, float* m2) {
  float mc[4] = {kNegBig, kNegBig, kNegBig, kNegBig};
  float mc2[4] = {kNegBig, kNegBig, kNegBig, kNegBig};
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if (kFull || vbase + tm * 16 + 4 * r < vocab) {
        const float z = acc[tm][tn][r];
        // with mc >= mc2, the new second-largest is the median of (mc, mc2, z): one v_med3
        if (kTop2) mc2[r] = __builtin_amdgcn_fmed3f(mc[r], mc2[r], z);
        mc[r] = fmaxf(mc[r], z);
      }
    }
  const float m = fmaxf(fmaxf(mc[0], mc[1]), fmaxf(mc[2], mc[3]));
  if (kTop2) {
    float x = top2_merge(fmaxf(mc[0], mc[1]), top2_merge(mc[0], mc2[0], mc[1], mc2[1]),
                         fmaxf(mc[2], mc[3]), top2_merge(mc[2], mc2[2], mc[3], mc2[3]));
    x = top2_shfl_merge(m, x, 16);
    *m2 = top2_shfl_merge(fmaxf(m, __shfl_xor(m, 16)), x, 32);
  }
  float M = pair_max(m);
  constexpr int kNoK = TM;  // "not seen"
  float sc[4] = {0.f, 0.f, 0.f, 0.f}, tc[4] = {0.f, 0.f, 0.f, 0.f};
  int32_t kc[4] = {kNoK, kNoK, kNoK, kNoK};
#pragma unroll
  for (int tm = TM - 1; tm >= 0; --tm)
#pragma unroll
    for (int r = 3; r >= 0; --r) {
      const float z = acc[tm][tn][r];
      if (kFull) {
        const float y = (z - M) * kLog2e;
        const float e = fast_exp2(y);
        sc[r] += e;
        tc[r] = fmaf(e, y, tc[r]);
        kc[r] = z == M ? tm : kc[r];
      } else {
        // rows past the vocabulary contribute e = 0 and y = 0 (with no valid row in the
        // column, M = kNegBig, where z - M would overflow and 0 * inf would poison t)
        const bool ok = vbase + tm * 16 + 4 * r < vocab;
        const float y = ok ? (z - M) * kLog2e : 0.f;
        const float e = ok ? fast_exp2(y) : 0.f;
        sc[r] += e;
        tc[r] = fmaf(e, y, tc[r]);
        kc[r] = (ok && z == M) ? tm : kc[r];
      }
    }
  int32_t ob = kNoIndex;
#pragma unroll
  for (int c = 0; c < 4; ++c) ob = min(ob, kc[c] == kNoK ? kNoIndex : 16 * kc[c] + 4 * c);
  int32_t idx = ob == kNoIndex ? kNoIndex : vbase + ob;
  float s = (sc[0] + sc[1]) + (sc[2] + sc[3]), t = (tc[0] + tc[1]) + (tc[2] + tc[3]);
  pair_sum_min(s, t, idx);
  return Partial{M, s, t, idx};
}

// column_stats16 with the bounds test only where the tile reaches past the vocabulary.
template <int TM, int TN, bool kTop2>
__device__ __forceinline__ Partial column_stats16(const f32x4 (&acc)[TM][TN], int tn, int vbase,
                                                  int vocab, bool full, float* m2) {
  return full ? column_stats16<TM, TN, kTop2, true>(acc, tn, vbase, vocab, m2)
              : column_stats16<TM, TN, kTop2, false>(acc, tn, vbase, vocab, m2);
}

// Tile (vt, rt) of position s of the launch sequence: bands of kBand vocabulary tiles (the last
// band may be narrower), each band swept position tile by position tile (vocabulary tiles of the
// band innermost).  Every s in [0, n_vtiles * n_rtiles) is a tile.
__device__ __forceinline__ void band_tile(int s, int n_vtiles, int n_rtiles, int& vt, int& rt) {
  const int per_band = kBand * n_rtiles;
  const int band = s / per_band;
  const int tt = s - band * per_band;
  const int nv = min(kBand, n_vtiles - band * kBand);
  vt = band * kBand + tt % nv;
  rt = tt / nv;
}

// Persistent form of the large-batch kernel: kTileGroups workgroups, one per compute unit, each
// computing a sequence of 256 x 256 tiles (vocabulary rows x block positions).  The launch
// sequence is cut into 8 contiguous segments, one per XCD (workgroup g runs on XCD g % 8 and
// takes every 32nd tile of its XCD's segment), so each XCD gets the same number of tiles and
// its 32 resident workgroups share a few W and h tiles in its L2.  With fewer tiles than
// workgroups, workgroup g computes tile g.
//
// Per tile: 4 waves form a 2 x 2 grid of 128 x 128 sub-tiles, each 8 x 8 blocks of 16x16x32 bf16
// MFMAs (256 accumulator registers per lane).  A 32-column ring stage is one MFMA k step: per
// stage a wave reads 16 fragments (16 KB) from LDS and issues 64 MFMAs.  Step kt: one barrier
// (stage kt + 1 has landed, and every wave's reads of stage kt are done), then the 64 MFMAs of
// stage kt from one register set while the fragments of stage kt + 1 go into the other and
// stage kt + RING is loaded into the slot of stage kt; groups of six MFMAs carry one load into
// LDS and two fragment reads, so both are spread over the step.  The ring slot of a stage is its
// index in the workgroup's whole sequence modulo RING, so the last steps of a tile issue the
// next tile's first stages and read its stage 0: its operands arrive while this tile finishes
// and runs its epilogue.  Measured against 32x32x16 blocks (the same tiles and ring): 16x16x32
// MFMAs sustain a higher clock under the chip's power limit.
template <int BM, int RING, bool kTop2>
__global__ __launch_bounds__(256, 1) void lmhead_tile_kernel(
    const uint16_t* __restrict__ h, const uint16_t* __restrict__ w, int n_rows, int hidden,
    int vocab, int n_vtiles, int n_rtiles, Partial* __restrict__ part,
    float* __restrict__ part2) {
  constexpr int BN = kTileBN, BK = kTileBK;
  constexpr int WM = 2, WN = 2, kWaves = WM * WN;
  constexpr int kWaveM = BM / WM, kWaveN = BN / WN;
  constexpr int TM = kWaveM / 16, TN = kWaveN / 16;
  constexpr int kRowB = BK * 2;                   // 64 bytes per LDS row
  constexpr int kStageBytes = (BM + BN) * kRowB;  // 32 KB
  constexpr int kInst = (BM + BN) / 16;           // 1 KB wave instructions per stage
  constexpr int kInstPerWave = kInst / kWaves;    // 8
  constexpr int kRedBytes = WM * BN * (sizeof(Partial) + 4);
  constexpr int kReads = TM + TN, kMfmas = TM * TN;
  static_assert(RING == 4, "ring of 4 stages (steps go in pairs, and RING - 1 stages in flight)");
  static_assert(BK == 32, "one 16x16x32 k step per stage");
  static_assert(kInst % kWaves == 0, "stage loads split evenly over the waves");
  static_assert(6 * kInstPerWave <= kMfmas && kReads == 2 * kInstPerWave, "interleave pattern");
  static_assert(RING * kStageBytes + kRedBytes <= 160 * 1024, "ring and reduction fit in LDS");
  static_assert((RING - 1) * kInstPerWave < 64, "vmcnt range");
  __shared__ __attribute__((aligned(16))) uint8_t smem[RING * kStageBytes + kRedBytes];

  // this workgroup's tiles: s0, s0 + step, ... below s_end
  const int n_tiles = n_vtiles * n_rtiles;
  const int g = blockIdx.x, groups = gridDim.x;
  int s0 = g, step = groups, s_end = n_tiles;
  if (groups == kTileGroups) {
    const int x = g % kXcds;
    s_end = static_cast<int>(static_cast<long long>(n_tiles) * (x + 1) / kXcds);
    s0 = static_cast<int>(static_cast<long long>(n_tiles) * x / kXcds) + g / kXcds;
    step = kTileGroups / kXcds;
  }
  if (s0 >= s_end) return;  // whole workgroup

  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index is the same on every lane: taken as a scalar, so the LDS destinations of the
  // loads (M0) are scalar arithmetic
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % WM, wn = wave / WM;
  const int q4 = lane >> 4, l16 = lane & 15;
  const int nk = hidden / BK;     // even (hidden is a multiple of 64), >= 2
  const bool chain = nk >= RING;  // the tail of a tile issues the next tile's first stages

  // Load instruction i of this wave covers tile rows 16 q .. 16 q + 15, q = wave * 8 + i (rows
  // below BM are W, the rest h, so a wave loads from one operand only); lane L fetches row
  // 16 q + L / 4, global chunk (L % 4) ^ swizzle(row) into LDS slot L % 4 of the row.  Rows past
  // the end are clamped.  The loads are buffer loads into LDS: a resource per tile (its first
  // row of the operand) in scalar registers, a byte offset per load instruction in a vector
  // register, and the stage's column offset as the scalar offset.  (Global loads into LDS would
  // count on the LDS-read counter as well, and the compiler then waits for every outstanding
  // fragment read before each use of one.)
  static_assert((BM / 16) % kInstPerWave == 0, "a wave loads from one operand");
  const bool w_wave = wave * kInstPerWave * 16 < BM;
  struct Src {
    __amdgpu_buffer_rsrc_t rs;
    uint32_t off[kInstPerWave];
  };
  auto set_src = [&](Src& d, int vt_, int rt_) {
    const uint16_t* base =
        w_wave ? w + static_cast<size_t>(vt_) * BM * hidden
               : h + static_cast<size_t>(rt_) * BN * hidden;
    const int last = w_wave ? vocab - 1 - vt_ * BM : n_rows - 1 - rt_ * BN;  // >= 0
    d.rs = make_rsrc(base);
#pragma unroll
    for (int i = 0; i < kInstPerWave; ++i) {
      const int q = wave * kInstPerWave + i;
      const int row = 16 * q + (lane >> 2);
      const int chunk = (lane & 3) ^ ((row >> 2) & 3);
      const int r = min(w_wave ? row : row - BM, last);
      d.off[i] = static_cast<uint32_t>(r * hidden * 2 + chunk * 16);
    }
  };
  // A source chosen by value, field by field (a conditional reference to one of two sources
  // makes the compiler take their addresses and keep them in scratch memory).
  auto pick = [&](bool c, const Src& x, const Src& y) {
    Src r;
    r.rs = c ? x.rs : y.rs;
#pragma unroll
    for (int i = 0; i < kInstPerWave; ++i) r.off[i] = c ? x.off[i] : y.off[i];
    return r;
  };
  // Stage `stage` of the tile described by d, into ring slot `slot`.
  auto issue = [&](const Src& d, int stage, int slot) {
    uint8_t* base = smem + slot * kStageBytes;
#pragma unroll
    for (int i = 0; i < kInstPerWave; ++i)
      buffer_load_to_lds(d.rs, base + (wave * kInstPerWave + i) * 1024, d.off[i], stage * BK * 2);
  };
  // Fragment f of a stage (f < TM: W block f of this wave, else h block f - TM): lane l reads
  // row rho(l % 16) = 4 (l % 4) + (l % 16) / 4 of the 16-row block, 16-byte chunk l / 16
  // (k = 8 (l / 16) .. + 7).  Rows in their natural order (lane l, row l % 16) make every read a
  // 2-way LDS bank conflict (rocprofv3 SQ_LDS_BANK_CONFLICT: 4 extra cycles per read, none with
  // rho).  The MFMA then sees the block's rows permuted by rho, on both operands: accumulator
  // register r of lane l holds vocabulary row 16 tm + rho(4 (l / 16) + r) = 16 tm + 4 r + l / 16
  // of the wave's W rows, for position tn * 16 + rho(l % 16) of its h rows.
  const int rho = 4 * (l16 & 3) + (l16 >> 2);
  auto frag = [&](const uint8_t* st, int f) {
    const int r = f < TM ? wm * kWaveM + f * 16 + rho : BM + wn * kWaveN + (f - TM) * 16 + rho;
    return *reinterpret_cast<const bf16x8*>(st + r * kRowB + 16 * (q4 ^ ((r >> 2) & 3)));
  };
  auto read = [&](int slot, bf16x8 (&a)[TM], bf16x8 (&b)[TN]) {
    const uint8_t* st = smem + slot * kStageBytes;
#pragma unroll
    for (int f = 0; f < TM; ++f) a[f] = frag(st, f);
#pragma unroll
    for (int f = 0; f < TN; ++f) b[f] = frag(st, TM + f);
  };

  f32x4 acc[TM][TN];
  Partial* red = reinterpret_cast<Partial*>(smem + RING * kStageBytes);  // [WM][BN]
  float* red2 = reinterpret_cast<float*>(red + WM * BN);

  int s = s0, vt, rt;
  band_tile(s, n_vtiles, n_rtiles, vt, rt);
  Src src, nsrc;
  set_src(src, vt, rt);
  int slot0 = 0;  // ring slot of the current tile's stage 0
#pragma unroll
  for (int j = 0; j < RING; ++j) issue(src, min(j, nk - 1), j);
  bf16x8 xa[TM], xb[TN], ya[TM], yb[TN];
  wait_vm_lds_and_barrier<(RING - 1) * kInstPerWave>();  // stage 0 has landed
  read(0, xa, xb);
  for (;;) {
    const int ns = s + step;
    const bool next = ns < s_end;
    int nvt = 0, nrt = 0;
    if (next) {
      band_tile(ns, n_vtiles, n_rtiles, nvt, nrt);
      set_src(nsrc, nvt, nrt);
    }
    const bool pre = next && chain;
    auto slot = [&](int kt) { return static_cast<int>(static_cast<unsigned>(slot0 + kt) % RING); };

    // Step kt: the barrier, stage `stage` of p into the slot of stage kt, the fragments of
    // stage kt + 1 into (na, nb) and the MFMAs of stage kt from (ca, cb).  Every step issues
    // exactly one stage, so RING - 2 younger stages are in flight at each barrier.
    auto body = [&](int kt, const Src& p, int stage, const bf16x8 (&ca)[TM],
                    const bf16x8 (&cb)[TN], bf16x8 (&na)[TM], bf16x8 (&nb)[TN]) {
      wait_vm_lds_and_barrier<(RING - 2) * kInstPerWave>();
      uint8_t* lbase = smem + slot(kt) * kStageBytes;
      const uint8_t* rbase = smem + slot(kt + 1) * kStageBytes;
#pragma unroll
      for (int i = 0; i < kMfmas; ++i) {
        mfma16_tied(acc[i / TN][i % TN], ca[i / TN], cb[i % TN]);
        if (i < 6 * kInstPerWave) {
          const int grp = i / 6, r = i % 6;
          if (r == 1)
            buffer_load_to_lds(p.rs, lbase + (wave * kInstPerWave + grp) * 1024, p.off[grp],
                               stage * BK * 2);
          if (r == 3 || r == 5) {
            const int f = 2 * grp + (r == 5);
            if (f < TM)
              na[f] = frag(rbase, f);
            else
              nb[f - TM] = frag(rbase, f);
          }
        }
      }
    };
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b) acc[a][b] = f32x4{};
    acc_fence_in(acc);  // the zeros are in place before the first MFMA reads them
    // Steps go in pairs, alternating the two register sets (nk and RING are even, so a pair
    // never straddles the end of this tile's stages).  Once this tile has no stage kt + RING,
    // a step issues the next tile's first stages (or, without a next tile or with fewer than
    // RING stages per tile, this tile's last stage again into the slot just freed, never read).
    const Src tsrc = pick(pre, nsrc, src);
    int kt = 0;
    for (; kt + RING < nk; kt += 2) {
      body(kt, src, kt + RING, xa, xb, ya, yb);
      body(kt + 1, src, kt + 1 + RING, ya, yb, xa, xb);
    }
    for (; kt < nk; kt += 2) {
      body(kt, tsrc, pre ? kt + RING - nk : nk - 1, xa, xb, ya, yb);
      body(kt + 1, tsrc, pre ? kt + 1 + RING - nk : nk - 1, ya, yb, xa, xb);
    }
    if (!pre) wait_vm_lds_and_barrier<0>();  // no DMA in flight
    acc_fence_out(acc);  // every MFMA has written its accumulator before the epilogue reads it

    const bool full = vt * BM + BM <= vocab;
    const int vbase = vt * BM + wm * kWaveM + q4;
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      float m2 = kNegBig;
      const Partial p = column_stats16<TM, TN, kTop2>(acc, tn, vbase, vocab, full, &m2);
      if (lane < 16) {
        red[wm * BN + wn * kWaveN + tn * 16 + rho] = p;
        if (kTop2) red2[wm * BN + wn * kWaveN + tn * 16 + rho] = m2;
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
      const int row = rt * BN + c;
      if (row < n_rows) {
        part[static_cast<size_t>(row) * n_vtiles + vt] = p;
        if (kTop2) part2[static_cast<size_t>(row) * n_vtiles + vt] = m2;
      }
    }
    if (!next) break;
    s = ns;
    vt = nvt;
    rt = nrt;
    src = nsrc;
    if (pre) {
      slot0 = (slot0 + nk) % RING;  // stage 0 of this tile is in xa, xb already
    } else {
      slot0 = 0;
      __syncthreads();  // every wave is done with the ring
#pragma unroll
      for (int j = 0; j < RING; ++j) issue(src, min(j, nk - 1), j);
      wait_vm_lds_and_barrier<(RING - 1) * kInstPerWave>();
      read(0, xa, xb);
    }
  }
}

// Tile kernel of the large-batch path: 256 x 256 tiles, 4 waves of 128 x 128, ring of 4
// (128 KB LDS, one workgroup per compute unit).
// Measured and dropped (with 32x32x16 blocks): 8 waves of 128 x 64 (10.55 ms), 256 x 128 tiles
// with a ring of 3 at two workgroups per compute unit (11.8 ms), stages reaching LDS through
// registers (9.65 ms), 64-column stages with one barrier per 64 MFMAs (10.1 ms), 384 x 256 tiles
// (384 accumulators per lane: the compiler spills).
template <bool kTop2>
hipError_t launch_tile(int n_rows, int hidden, int vocab, const void* h, const void* w,
                       Partial* part, float* part2, hipStream_t s) {
  const int n_vtiles = tile_vtiles(vocab);
  const int n_rtiles = (n_rows + kTileBN - 1) / kTileBN;
  const int n_tiles = n_vtiles * n_rtiles;
  const int groups = n_tiles >= kTileGroups ? kTileGroups : n_tiles;
  hipLaunchKernelGGL((lmhead_tile_kernel<kTileBM, kTileRing, kTop2>), dim3(groups), dim3(256), 0,
                     s, static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(w), n_rows,
                     hidden, vocab, n_vtiles, n_rtiles, part, part2);
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
  if (bf16) return tile_vtiles(vocab);
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
