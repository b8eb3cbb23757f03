// Block attention with a prefix KV cache for gfx950.
//
// Every query row of a sequence's active block attends, without a causal mask, to the
// sequence's cached prefix keys followed by the block's own keys.  Grouped-query attention:
// query head h reads key/value head h / G with G = hq / hkv, so one workgroup serves the
// G query heads of one key/value head and its K/V tiles are read once for all of them.
//
// bf16 path: scores are computed transposed, S^T = K Q^T, so each lane owns one query row
// (an MFMA column) and reduces its softmax statistics in registers; the probabilities then
// feed P V directly as the B operand of O^T = V^T P^T.  Head dimension 128 runs
// attn_bf16_d128_kernel (tiles loaded straight into LDS, the next tile's scores interleaved with
// this tile's exponentials); head dimension 64 runs attn_bf16_kernel (tiles staged through
// registers, V stored transposed in LDS).
// Small steps (attn_small_ok) take the 16-row role of attn_small.hpp instead, here as a kernel
// of its own; the decode step runs the same role inside the LM-head launch.
#include <cstdlib>
#include <cstring>

#include "attn_common.hpp"
#include "attn_small.hpp"
#include "eb_common.hpp"
#include "eb_internal.hpp"

namespace eb {
namespace {

constexpr int kThreads = 256;   // 4 waves
constexpr int kRowsPerWg = kAttnRowsPerWg;
constexpr int kKeys = kAttnKeys;
constexpr int kXcdCount = 8;  // XCDs of the chip (workgroups are dealt to them round-robin)


// Two workgroups per compute unit (<= 256 VGPRs per lane, no spills at D = 128), so one
// wave's softmax arithmetic overlaps another wave's MFMAs on the same SIMD (batch 64 at
// D = 128: 1.85 ms with one workgroup per compute unit, 1.07 ms with two).
template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_bf16_kernel(AttnParams p, int row_tiles,
                                                                int units) {
  constexpr int kKRow = D + 8;       // K tile pitch (bf16)
  constexpr int kVRow = kKeys + 8;   // V^T tile pitch (bf16): 144-byte rows, 16-byte aligned
  constexpr int kDSteps = D / 16;    // MFMA k-steps over the head dimension
  constexpr int kDBlocks = D / 32;   // 32-row blocks of O^T
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kKeys * kKRow];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * kVRow];

  // Workgroup id -> (unit, row tile) so that the row tiles of one unit (sequence, K/V head, key
  // range) all run on one XCD, one after another: workgroups are dealt to the 8 XCDs round-robin
  // by id, and the tiles of unit u take ids 8 (row_tiles (u / 8) + tile) + u % 8.  They then read
  // the unit's K/V stages from that XCD's L2 instead of each XCD fetching them.
  const int xcd = blockIdx.x % kXcdCount, j = blockIdx.x / kXcdCount;
  const int unit = kXcdCount * (j / row_tiles) + xcd;
  if (unit >= units) return;  // whole workgroup: padding of the last round
  const int tile = j % row_tiles;
  const int z = unit / p.hkv;
  const int b = z / p.nsplit;
  const int sp = z % p.nsplit;
  const int g = unit % p.hkv;
  const int G = p.group;
  const int bbeg = p.cu_block[b];
  const int len = p.cu_block[b + 1] - bbeg;
  const int pbeg = p.cu_prefix[b];
  const int plen = p.cu_prefix[b + 1] - pbeg;
  const int n_rows = len * G;
  const int row0 = tile * kRowsPerWg;
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
    // V^T: the 16-bit values of keys 2 kp and 2 kp + 1 at one d form one 32-bit word.  Within
    // each 16-key group, key w sits at column 8 ((w / 4) % 2) + 4 (w / 8) + w % 4, so the eight
    // keys one lane contracts over in an MFMA (4 half + 0..3 and 8 + 4 half + 0..3) are
    // contiguous; keys 2 kp and 2 kp + 1 stay adjacent.
    const int w16 = (2 * kp) & 15;
    const int vcol = (2 * kp - w16) + 8 * ((w16 >> 2) & 1) + 4 * (w16 >> 3) + (w16 & 3);
#pragma unroll
    for (int c = 0; c < kVd / 8; ++c)
#pragma unroll
      for (int w4 = 0; w4 < 4; ++w4) {
        const int d = dg * kVd + 8 * c + 2 * w4;
        const uint32_t k0 = vreg[0][c][w4], k1 = vreg[1][c][w4];
        *reinterpret_cast<uint32_t*>(Vt + d * kVRow + vcol) =
            __builtin_amdgcn_perm(k1, k0, 0x05040100u);  // low halves: value at d
        *reinterpret_cast<uint32_t*>(Vt + (d + 1) * kVRow + vcol) =
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
        const int kbase = kb * 32 + 16 * u + 8 * half;  // the lane's 8 keys, contiguous
#pragma unroll
        for (int db = 0; db < kDBlocks; ++db) {
          const bf16x8 va =
              *reinterpret_cast<const bf16x8*>(Vt + (db * 32 + l32) * kVRow + kbase);
          o[db] = mfma32(va, pf, o[db]);
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

// Head dimension 128: the main path of the bf16 block attention.
//
// Staging.  K and V tiles of 64 keys reach LDS by buffer loads straight into LDS (no staging
// registers, no LDS store instructions): waves 0-1 load K tiles, waves 2-3 V tiles, two slots
// each.  K runs one stage ahead of V, so iteration st needs K(st + 1) and V(st) and one barrier
// per iteration suffices: after it, K(st + 2) goes into the slot K(st) left and V(st + 1) into
// the slot V(st - 1) left.  Rows are 256 bytes of 16 sixteen-byte chunks; chunk c of key row r
// sits in slot c ^ (r % 16) for K (the 32-row fragment reads of S^T then touch 16 distinct slots
// per 16 lanes) and in slot c ^ 4 (r % 4) for V (the 4 rows x 4 chunks of a transposing read by
// 16 lanes then touch distinct slots).  A load instruction writes 1 KB, 4 key rows, lane L
// filling slot L % 16 of row L / 16, so each lane fetches the global chunk that lands there.
//
// Schedule.  Iteration st issues the 16 MFMAs of S(st + 1) = K(st + 1) Q^T, each followed by the
// VALU work of one bf16 word (two probabilities) of P(st) from the scores of the previous
// iteration, then the 16 MFMAs of O^T += V(st)^T P(st)^T, each followed by one step of the
// maximum of S(st + 1).  Scheduling barriers keep that interleave, so one wave's exponentials
// run while its matrix pipe works.  V^T fragments come from transposing LDS reads of the
// row-major V tile.  The loop runs two iterations per trip, the score arrays of S(st) and
// S(st + 1) trading places between them, so no scores are copied.
//
// Softmax.  The running maximum m (log2 units) moves only when some row's stage maximum
// exceeds it by more than kAttnSlack, so probabilities 2^(s - m) stay below 2^kAttnSlack and
// O, l are rescaled rarely.  l sums the bf16-rounded probabilities that P V multiplies, two per
// dot instruction.  The final O / l and the split partials (m, l, O) mean the same as in
// attn_bf16_kernel.
constexpr float kAttnSlack = 8.0f;
constexpr int kDmaKeys = 64;  // keys per tile (the schedule pairs 16 S MFMAs with 16 P words)
static_assert(kDmaKeys == kKeys, "stages of the key-split plan");

__global__ __launch_bounds__(kThreads, 2) void attn_bf16_d128_kernel(AttnParams p, int row_tiles,
                                                                     int units) {
  constexpr int D = 128;
  constexpr int kRowBytes = D * 2;
  constexpr int kTileBytes = kDmaKeys * kRowBytes;  // 16 KB
  constexpr int kDSteps = D / 16;                   // MFMA k-steps of S^T over the head dim
  constexpr int kDBlocks = D / 32;                  // 32-row blocks of O^T
  constexpr int kKB = kDmaKeys / 32;                // 32-key blocks per tile
  constexpr int kMfmas = kKB * kDSteps;             // S MFMAs per tile = P V MFMAs per tile
  static_assert(kMfmas == 16 && kKB * 2 * kDBlocks == kMfmas, "schedule");
  constexpr int kInstPerTile = kTileBytes / 1024;            // 1 KB per load instruction
  constexpr int kInstPerWave = 2 * kInstPerTile / (kThreads / 64);
  static_assert(kInstPerTile % kInstPerWave == 0, "a wave loads K or V, not both");
  constexpr int kPreK = 3;  // K fragment reads issued this many MFMAs ahead
  constexpr int kPreV = 3;  // V fragment reads issued this many MFMAs ahead
  // K tiles in slots 0, 1; V tiles in slots 2, 3
  __shared__ __attribute__((aligned(16))) uint8_t smem[4 * kTileBytes];

  // Workgroup id -> (unit, row tile) as in attn_bf16_kernel: the row tiles of one unit run on
  // one XCD, one after another, and share that XCD's L2.
  const int xcd = blockIdx.x % kXcdCount, jx = blockIdx.x / kXcdCount;
  const int unit = kXcdCount * (jx / row_tiles) + xcd;
  if (unit >= units) return;  // whole workgroup: padding of the last round
  const int tile = jx % row_tiles;
  const int z = unit / p.hkv;
  const int b = z / p.nsplit;
  const int sp = z % p.nsplit;
  const int g = unit % p.hkv;
  const int G = p.group;
  const int bbeg = p.cu_block[b];
  const int len = p.cu_block[b + 1] - bbeg;
  const int pbeg = p.cu_prefix[b];
  const int plen = p.cu_prefix[b + 1] - pbeg;
  const int n_rows = len * G;
  const int row0 = tile * kRowsPerWg;
  if (row0 >= n_rows) return;  // whole workgroup: this tile lies past the block
  const int sbeg = p.cu_suffix ? p.cu_suffix[b] : 0;
  const int slen = p.cu_suffix ? p.cu_suffix[b + 1] - sbeg : 0;
  const int n_keys = plen + len + slen;
  const int kbeg = sp * p.kps;
  if (kbeg >= n_keys) return;  // whole workgroup: this key range lies past the sequence
  const int kend = min(n_keys, kbeg + p.kps);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar buffer resources
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

  // Loads: per segment (prefix, block, suffix) a buffer resource at the segment's first key of
  // head g; key j of a segment lies j * key_bytes further.  Instruction i of a wave covers tile
  // rows 4 n .. 4 n + 3, n = (wave * kInstPerWave + i) % kInstPerTile.
  const bool k_wave = wave * kInstPerWave < kInstPerTile;  // wave-uniform
  const uint32_t key_bytes = static_cast<uint32_t>(p.hkv) * kRowBytes;
  // (an empty prefix or suffix segment, never read, takes the block's resource)
  const uint16_t* blk0 = (k_wave ? p.k_blk : p.v_blk) + (static_cast<size_t>(bbeg) * p.hkv + g) * D;
  const __amdgpu_buffer_rsrc_t rs_blk = make_rsrc(blk0);
  const __amdgpu_buffer_rsrc_t rs_pre = make_rsrc(
      plen > 0 ? (k_wave ? p.k_pre : p.v_pre) + (static_cast<size_t>(pbeg) * p.hkv + g) * D : blk0);
  const __amdgpu_buffer_rsrc_t rs_suf = make_rsrc(
      slen > 0 ? (k_wave ? p.k_suf : p.v_suf) + (static_cast<size_t>(sbeg) * p.hkv + g) * D : blk0);
  int lrow[kInstPerWave];       // tile row this lane fills in instruction i
  uint32_t coff[kInstPerWave];  // byte offset of the global chunk it fetches within the row
#pragma unroll
  for (int i = 0; i < kInstPerWave; ++i) {
    const int n = (wave * kInstPerWave + i) % kInstPerTile;
    const int r = 4 * n + (lane >> 4);
    const int swz = k_wave ? (r & 15) : 4 * (r & 3);
    lrow[i] = r;
    coff[i] = 16u * static_cast<uint32_t>((lane & 15) ^ swz);
  }
  // This wave's half (K or V) of the tile of keys kv0 .. kv0 + 63 into dst.  Keys past kend come
  // from a clamped, valid row; their scores are set to -inf.
  auto issue = [&](int kv0, uint8_t* dst) {
    if (kv0 + kDmaKeys <= plen) {  // the whole tile lies in the prefix
#pragma unroll
      for (int i = 0; i < kInstPerWave; ++i) {
        const int n = (wave * kInstPerWave + i) % kInstPerTile;
        buffer_load_to_lds(rs_pre, dst + n * 1024,
                           static_cast<uint32_t>(lrow[i]) * key_bytes + coff[i],
                           static_cast<uint32_t>(kv0) * key_bytes);
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < kInstPerWave; ++i) {
      const int n = (wave * kInstPerWave + i) % kInstPerTile;
      const int j = min(kv0 + lrow[i], kend - 1);
      if (j < plen)
        buffer_load_to_lds(rs_pre, dst + n * 1024, static_cast<uint32_t>(j) * key_bytes + coff[i],
                           0);
      else if (j < plen + len)
        buffer_load_to_lds(rs_blk, dst + n * 1024,
                           static_cast<uint32_t>(j - plen) * key_bytes + coff[i], 0);
      else
        buffer_load_to_lds(rs_suf, dst + n * 1024,
                           static_cast<uint32_t>(j - plen - len) * key_bytes + coff[i], 0);
    }
  };
  auto ktile = [&](int i) { return smem + (i & 1) * kTileBytes; };
  auto vtile = [&](int i) { return smem + (2 + (i & 1)) * kTileBytes; };

  // S^T of tile st into acc (unmasked):
  // acc[kb][r] = S[query l32][key kb*32 + 8(r/4) + 4 half + r%4]
  auto scores = [&](int st, f32x16 (&acc)[kKB]) {
    const uint8_t* Kt = ktile(st);
#pragma unroll
    for (int kb = 0; kb < kKB; ++kb) acc[kb] = f32x16{};
#pragma unroll
    for (int s = 0; s < kDSteps; ++s)
#pragma unroll
      for (int kb = 0; kb < kKB; ++kb) {
        const int r = kb * 32 + l32;
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(
            Kt + r * kRowBytes + 16 * ((2 * s + half) ^ (r & 15)));
        acc[kb] = mfma32(kf, qf[s], acc[kb]);
      }
  };
  // Scores of keys past kend to -inf; returns this lane's maximum over the tile.
  auto mask_max = [&](int st, f32x16 (&acc)[kKB]) {
    const int kv0 = kbeg + st * kDmaKeys;
    float mloc = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < kKB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kv0 + kb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (key >= kend) acc[kb][r] = -INFINITY;
        mloc = fmaxf(mloc, acc[kb][r]);
      }
    return mloc;
  };
  // Running maximum from this lane's tile maximum (both halves of a row agree).
  auto update_max = [&](float mloc) {
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float mcand = mloc * p.scale_log2;  // scale > 0: max(scale s) = scale max(s)
    if (__any(mcand > m_run + kAttnSlack)) {
      const float m_new = fmaxf(m_run, mcand);
      const float alpha = fast_exp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < kDBlocks; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
    }
  };

  const int n_stages = (kend - kbeg + kDmaKeys - 1) / kDmaKeys;
  // prologue: K(0), K(1), V(0); then S(0) and its maximum
  if (k_wave) {
    issue(kbeg, ktile(0));
    if (n_stages > 1) issue(kbeg + kDmaKeys, ktile(1));
  } else {
    issue(kbeg, vtile(0));
  }
  wait_vm_lds_and_barrier<0>();
  f32x16 scur[kKB];
  scores(0, scur);
  update_max(mask_max(0, scur));

  const int q4 = lane & 3, j4 = (lane >> 2) & 3;
  const int d0 = 16 * ((lane >> 4) & 1);
  // Iteration st: S(st + 1) into snxt_ while P(st) comes from scur_.  Two iterations per trip
  // with the two score arrays swapping roles, so the next tile's scores are never copied.
  auto step = [&](int st, f32x16 (&scur_)[kKB], f32x16 (&snxt_)[kKB]) {
    // this wave's loads of K(st + 1) and V(st) have landed; after the barrier every wave's
    // have, and every wave is done with K(st) and V(st - 1)
    wait_vm_lds_and_barrier<0>();
    if (k_wave) {
      if (st + 2 < n_stages) issue(kbeg + (st + 2) * kDmaKeys, ktile(st));
    } else {
      if (st + 1 < n_stages) issue(kbeg + (st + 1) * kDmaKeys, vtile(st + 1));
    }
    const bool more = st + 1 < n_stages;
    // on the last iteration S of a stale K tile is computed and discarded (no branch)
    const uint8_t* Kt = ktile(more ? st + 1 : st);
    const uint8_t* Vt = vtile(st);
    auto kread = [&](int m) {  // K fragment of S MFMA m = 2 s + kb
      const int s = m / kKB, kb = m % kKB, r = kb * 32 + l32;
      return *reinterpret_cast<const bf16x8*>(Kt + r * kRowBytes +
                                              16 * ((2 * s + half) ^ (r & 15)));
    };
    // V^T fragment of P V MFMA n = (2 kb + u) kDBlocks + db: keys kb*32 + 16u + {4 half + 0..3,
    // 8 + 4 half + 0..3} at d = 32 db + l32.  Lane 4 j + q of a 16-lane group addresses key row
    // kbase + j at d = d0 + 4 q .. +3; the transposing read hands lane i of the group
    // d = d0 + i of rows kbase .. kbase + 3.
    auto vread = [&](int n) {
      const int db = n % kDBlocks, u = (n / kDBlocks) % 2, kb = n / (2 * kDBlocks);
      const int c = (32 * db + d0) / 8 + (q4 >> 1);  // 16-byte chunk of columns d0 + 4 q
      v4i16 part[2];
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        const int r = kb * 32 + 16 * u + 8 * x + 4 * half + j4;
        const uint8_t* a = Vt + r * kRowBytes + 16 * (c ^ (4 * (r & 3))) + 8 * (q4 & 1);
        part[x] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(const_cast<uint8_t*>(a)));
      }
      return __builtin_bit_cast(bf16x8,
                                __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7));
    };
#pragma unroll
    for (int kb = 0; kb < kKB; ++kb) snxt_[kb] = f32x16{};
    bf16x8 kf[kMfmas], vf[kMfmas];
    u32x4 pw[2 * kKB];  // P(st) as bf16 pairs: word e of MFMA group 2 kb + u
    float lsum = 0.f;
#pragma unroll
    for (int m = 0; m < kPreK; ++m) kf[m] = kread(m);
    __builtin_amdgcn_sched_barrier(0);
    // S(st + 1), each MFMA followed by the P(st) work of one slot: registers 8u + 2e, 8u + 2e + 1
    // of scur_[kb] are keys kb*32 + 16u + 4 half + ... -- exactly the B operand layout of P V.
    // The P words are software-pipelined over the slots: slot m forms the exponents of word
    // m + 1, the exponentials of word m and the bf16 pair and running sum of word m - 1, so an
    // instruction does not wait on the one just before it (a wave issues in order).
    auto expo = [&](int w, float (&y)[2]) {
      const int kb = w / 8, u = (w / 4) % 2, e = w % 4;
      y[0] = fmaf(scur_[kb][8 * u + 2 * e], p.scale_log2, -m_run);
      y[1] = fmaf(scur_[kb][8 * u + 2 * e + 1], p.scale_log2, -m_run);
    };
    float ya[2][2], ea[2][2];
    auto commit = [&](int w) {
      const uint32_t wd = pack2_bf16(ea[w & 1][0], ea[w & 1][1]);
      pw[w / 4][w % 4] = wd;
      lsum = sum2_bf16(wd, lsum);
    };
    expo(0, ya[0]);
#pragma unroll
    for (int m = 0; m < kMfmas; ++m) {
      if (m + kPreK < kMfmas) kf[m + kPreK] = kread(m + kPreK);
      if (m >= kMfmas - kPreV) vf[m - (kMfmas - kPreV)] = vread(m - (kMfmas - kPreV));
      snxt_[m % kKB] = mfma32(kf[m], qf[m / kKB], snxt_[m % kKB]);
      if (m + 1 < kMfmas) expo(m + 1, ya[(m + 1) & 1]);
      ea[m & 1][0] = fast_exp2(ya[m & 1][0]);
      ea[m & 1][1] = fast_exp2(ya[m & 1][1]);
      if (m >= 1) commit(m - 1);
      __builtin_amdgcn_sched_barrier(0);
    }
    commit(kMfmas - 1);
    // O^T += V^T P^T, each MFMA followed by a step of the maximum of S(st + 1)
    float mx[2] = {-INFINITY, -INFINITY};
#pragma unroll
    for (int n = 0; n < kMfmas; ++n) {
      if (n + kPreV < kMfmas) vf[n + kPreV] = vread(n + kPreV);
      o[n % kDBlocks] =
          mfma32(vf[n], __builtin_bit_cast(bf16x8, pw[n / kDBlocks]), o[n % kDBlocks]);
      mx[n & 1] = fmaxf(mx[n & 1], fmaxf(snxt_[n / 8][2 * (n % 8)], snxt_[n / 8][2 * (n % 8) + 1]));
      asm volatile("" : "+v"(mx[n & 1]));  // keep the step here, between the MFMAs
      __builtin_amdgcn_sched_barrier(0);
    }
    l_run += lsum;
    if (more) {
      float mloc = fmaxf(mx[0], mx[1]);
      if (kbeg + (st + 2) * kDmaKeys > kend) mloc = mask_max(st + 1, snxt_);  // last, partial tile
      update_max(mloc);
    }
  };
  f32x16 salt[kKB];
  for (int st = 0; st < n_stages; st += 2) {
    step(st, scur, salt);
    if (st + 1 < n_stages) step(st + 1, salt, scur);
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!row_ok) return;
  if (p.nsplit > 1) {
    const size_t idx = (static_cast<size_t>(bbeg + pos) * p.hq + g * G + hh) * p.nsplit + sp;
    float* dst = p.o_part + idx * D;
#pragma unroll
    for (int db = 0; db < kDBlocks; ++db)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int d = db * 32 + 8 * q + 4 * half;
        *reinterpret_cast<f32x4*>(dst + d) =
            f32x4{o[db][4 * q + 0], o[db][4 * q + 1], o[db][4 * q + 2], o[db][4 * q + 3]};
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
    for (int q = 0; q < 4; ++q) {
      const int d = db * 32 + 8 * q + 4 * half;
      const u32x2 v{pack2_bf16(o[db][4 * q + 0] * inv, o[db][4 * q + 1] * inv),
                    pack2_bf16(o[db][4 * q + 2] * inv, o[db][4 * q + 3] * inv)};
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

// attn_bf16_d128_kernel addresses a key row by a 32-bit byte offset from its segment's first
// row of the sequence (the buffer range ends at 2^31 - 1): every segment must stay below that.
inline bool attn_dma_offsets_fit(const AttnArgs& a) {
  const long key_bytes = static_cast<long>(a.hkv) * a.head_dim * 2;
  const long longest =
      max(max(a.max_prefix, a.max_block), a.cu_suffix ? a.max_suffix : 0) + kDmaKeys;
  return longest * key_bytes < (1L << 31);
}

// EB_ATTN_STAGED (any value but "0") sends head dimension 128 to attn_bf16_kernel<128>, the
// form the library otherwise keeps for segments too long for 32-bit buffer offsets, so that
// it can be tested at ordinary sizes.
inline bool attn_force_staged() {
  const char* v = getenv("EB_ATTN_STAGED");
  return v && *v && strcmp(v, "0") != 0;
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
    const int row_tiles = static_cast<int>((rows + kRowsPerWg - 1) / kRowsPerWg);
    const int units = a.batch * sp.nsplit * a.hkv;
    const dim3 grid(static_cast<unsigned>(kXcdCount * ((units + kXcdCount - 1) / kXcdCount) *
                                          row_tiles));
    if (a.head_dim == 128 && attn_dma_offsets_fit(a) && !attn_force_staged())
      hipLaunchKernelGGL(attn_bf16_d128_kernel, grid, dim3(kThreads), 0, s, p, row_tiles, units);
    else if (a.head_dim == 128)
      hipLaunchKernelGGL(attn_bf16_kernel<128>, grid, dim3(kThreads), 0, s, p, row_tiles, units);
    else
      hipLaunchKernelGGL(attn_bf16_kernel<64>, grid, dim3(kThreads), 0, s, p, row_tiles, units);
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
