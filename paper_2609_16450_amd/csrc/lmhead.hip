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
#include "eb_common.hpp"
#include "eb_internal.hpp"

namespace eb {
namespace {

// ---------------------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------------------
template <int BM_, int BN_, int BK_, int WM_, int WN_>
struct LmTile {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_;
  static constexpr int kThreads = WM * WN * 64;
  static constexpr int kWaveM = BM / WM;
  static constexpr int kWaveN = BN / WN;
  static constexpr int TM = kWaveM / 32;
  static constexpr int TN = kWaveN / 32;
  static constexpr int kRow = BK + 8;             // LDS row pitch in bf16 (16 B of padding)
  static constexpr int kStage = (BM + BN) * kRow;  // bf16 elements per pipeline stage
  static constexpr int kChunksA = BM * (BK / 8);   // 16-byte chunks per stage
  static constexpr int kChunksB = BN * (BK / 8);
  static constexpr int kPerA = kChunksA / kThreads;
  static constexpr int kPerB = (kChunksB + kThreads - 1) / kThreads;
  static constexpr int kLdsBytes = 2 * kStage * 2;
  static_assert(BM % (32 * WM) == 0 && BN % (32 * WN) == 0, "wave tile must be 32-aligned");
  static_assert(kChunksA % kThreads == 0, "A tile must split evenly over threads");
  static_assert(BK == 32 || BK == 64, "BK");
  static_assert(kLdsBytes <= 65536, "LDS budget");
  static_assert(WM * BN * (int)sizeof(Partial) <= kLdsBytes, "reduction scratch fits in LDS");
};

template <class C>
__global__ __launch_bounds__(C::kThreads) void lmhead_bf16_kernel(
    const uint16_t* __restrict__ h, const uint16_t* __restrict__ w, int n_rows, int hidden,
    int vocab, int n_slices, Partial* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * C::kStage];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % C::WM;
  const int wn = wave / C::WM;
  const int vt = blockIdx.x;
  const int v0 = vt * C::BM;
  const int r0 = blockIdx.y * C::BN;

  // Per-thread 16-byte chunks of each stage: chunk c covers row c / (BK/8), columns
  // 8 * (c % (BK/8)) .. +7.  Rows past the end are clamped to a valid row; their results are
  // discarded in the epilogue.
  constexpr int kCpr = C::BK / 8;
  const uint16_t* ga[C::kPerA];
  int la[C::kPerA];
#pragma unroll
  for (int i = 0; i < C::kPerA; ++i) {
    const int c = tid + i * C::kThreads;
    const int row = c / kCpr, col = (c % kCpr) * 8;
    const int v = min(v0 + row, vocab - 1);
    ga[i] = w + static_cast<size_t>(v) * hidden + col;
    la[i] = row * C::kRow + col;
  }
  const uint16_t* gb[C::kPerB];
  int lb[C::kPerB];
  bool okb[C::kPerB];
#pragma unroll
  for (int i = 0; i < C::kPerB; ++i) {
    const int c = tid + i * C::kThreads;
    okb[i] = c < C::kChunksB;
    const int cc = okb[i] ? c : 0;
    const int row = cc / kCpr, col = (cc % kCpr) * 8;
    const int r = min(r0 + row, n_rows - 1);
    gb[i] = h + static_cast<size_t>(r) * hidden + col;
    lb[i] = C::BM * C::kRow + row * C::kRow + col;
  }

  u32x4 ra[C::kPerA], rb[C::kPerB];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::kPerA; ++i) ra[i] = *reinterpret_cast<const u32x4*>(ga[i] + k0);
#pragma unroll
    for (int i = 0; i < C::kPerB; ++i)
      if (okb[i]) rb[i] = *reinterpret_cast<const u32x4*>(gb[i] + k0);
  };
  auto sstore = [&](int st) {
    uint16_t* base = smem + st * C::kStage;
#pragma unroll
    for (int i = 0; i < C::kPerA; ++i) *reinterpret_cast<u32x4*>(base + la[i]) = ra[i];
#pragma unroll
    for (int i = 0; i < C::kPerB; ++i)
      if (okb[i]) *reinterpret_cast<u32x4*>(base + lb[i]) = rb[i];
  };

  f32x16 acc[C::TM][C::TN];
#pragma unroll
  for (int a = 0; a < C::TM; ++a)
#pragma unroll
    for (int b = 0; b < C::TN; ++b) acc[a][b] = f32x16{};

  // The contraction index inside a stage is permuted so that each lane reads one contiguous
  // run of its row: MFMA step s, lane half hf uses columns (BK/2)*hf + 8*s .. +7 for both
  // operands.  Any permutation applied to both operands leaves W h unchanged.
  const int half = lane >> 5;
  const int l32 = lane & 31;
  const int nk = hidden / C::BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * C::BK);
    const uint16_t* Ab = smem + cur * C::kStage;
    const uint16_t* Bb = Ab + C::BM * C::kRow;
#pragma unroll
    for (int s = 0; s < C::BK / 16; ++s) {
      const int koff = (C::BK / 2) * half + 8 * s;
      bf16x8 a[C::TM], b[C::TN];
#pragma unroll
      for (int tm = 0; tm < C::TM; ++tm)
        a[tm] = *reinterpret_cast<const bf16x8*>(
            Ab + (wm * C::kWaveM + tm * 32 + l32) * C::kRow + koff);
#pragma unroll
      for (int tn = 0; tn < C::TN; ++tn)
        b[tn] = *reinterpret_cast<const bf16x8*>(
            Bb + (wn * C::kWaveN + tn * 32 + l32) * C::kRow + koff);
#pragma unroll
      for (int tm = 0; tm < C::TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < C::TN; ++tn) acc[tm][tn] = mfma32(a[tm], b[tn], acc[tm][tn]);
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // Epilogue: each lane reduces the logits it holds for its column (one block position).
  Partial* red = reinterpret_cast<Partial*>(smem);  // [WM][BN]
#pragma unroll
  for (int tn = 0; tn < C::TN; ++tn) {
    float m = kNegBig;
    int32_t idx = kNoIndex;
#pragma unroll
    for (int tm = 0; tm < C::TM; ++tm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = v0 + wm * C::kWaveM + tm * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        const float z = acc[tm][tn][r];
        if (v < vocab && z > m) {  // ascending v: strict > keeps the lowest index
          m = z;
          idx = v;
        }
      }
    // y = (z - m) log2 e is exactly 0 at the maximum, so s >= 1 and kappa = 1/s <= 1.
    float s = 0.f, t = 0.f;
#pragma unroll
    for (int tm = 0; tm < C::TM; ++tm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = v0 + wm * C::kWaveM + tm * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (v < vocab) {
          const float y = (acc[tm][tn][r] - m) * kLog2e;
          const float e = fast_exp2(y);
          s += e;
          t = fmaf(e, y, t);
        }
      }
    Partial p{m, s, t, idx};
    p = partial_xor_merge(p, 32, lane);
    if (lane < 32) red[wm * C::BN + wn * C::kWaveN + tn * 32 + l32] = p;
  }
  __syncthreads();
  for (int c = tid; c < C::BN; c += C::kThreads) {
    Partial p = red[c];
#pragma unroll
    for (int k = 1; k < C::WM; ++k) p = partial_merge(p, red[k * C::BN + c]);
    const int row = r0 + c;
    if (row < n_rows) part[static_cast<size_t>(row) * n_slices + vt] = p;
  }
}

// Tile shapes: vocabulary rows per workgroup x block positions per workgroup.
using TileNarrow = LmTile<128, 32, 64, 4, 1>;   // n_rows <= 32 (batch-1 step): W streamed once
using TileMid = LmTile<128, 64, 64, 4, 1>;      // n_rows <= 64
using TileWide = LmTile<128, 128, 32, 2, 2>;    // larger batches
constexpr int kBf16SliceRows = 128;             // every bf16 tile shape uses BM = 128
static_assert(TileNarrow::BM == kBf16SliceRows && TileMid::BM == kBf16SliceRows &&
                  TileWide::BM == kBf16SliceRows,
              "slice count depends on BM only");

template <class C>
hipError_t launch_bf16(int n_rows, int hidden, int vocab, const void* h, const void* w,
                       Partial* part, int n_slices, hipStream_t s) {
  dim3 grid(n_slices, (n_rows + C::BN - 1) / C::BN);
  hipLaunchKernelGGL(lmhead_bf16_kernel<C>, grid, dim3(C::kThreads), 0, s,
                     static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(w), n_rows,
                     hidden, vocab, n_slices, part);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// fp32 kernel (small shapes): one thread per vocabulary entry, plain fp32 FMA dot products.
// ---------------------------------------------------------------------------------------
constexpr int kF32SliceRows = 256;

__global__ __launch_bounds__(256) void lmhead_f32_kernel(const float* __restrict__ h,
                                                         const float* __restrict__ w,
                                                         int n_rows, int hidden, int vocab,
                                                         int n_slices,
                                                         Partial* __restrict__ part) {
  __shared__ Partial red[4];
  const int slice = blockIdx.x;
  const int row = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int v = slice * kF32SliceRows + threadIdx.x;
  Partial p = partial_empty();
  if (v < vocab) {
    const float* wr = w + static_cast<size_t>(v) * hidden;
    const float* hr = h + static_cast<size_t>(row) * hidden;
    float z = 0.f;
    for (int k = 0; k < hidden; ++k) z = fmaf(wr[k], hr[k], z);
    p = Partial{z, 1.f, 0.f, v};
  }
  for (int mask = 32; mask >= 1; mask >>= 1) p = partial_xor_merge(p, mask, lane);
  if (lane == 0) red[wave] = p;
  __syncthreads();
  if (threadIdx.x == 0) {
    Partial q = red[0];
    for (int k = 1; k < 4; ++k) q = partial_merge(q, red[k]);
    part[static_cast<size_t>(row) * n_slices + slice] = q;
  }
}

// ---------------------------------------------------------------------------------------
// combine: one wavefront per row, fixed merge order (lane-strided, then butterfly)
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void lmhead_combine_kernel(const Partial* __restrict__ part,
                                                             int n_rows, int n_slices,
                                                             float* __restrict__ conf,
                                                             float* __restrict__ entropy,
                                                             int32_t* __restrict__ argmax,
                                                             float* __restrict__ max_logit) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;  // uniform per wavefront
  const Partial* pr = part + static_cast<size_t>(row) * n_slices;
  Partial p = partial_empty();
  for (int i = lane; i < n_slices; i += 64) p = partial_merge(p, pr[i]);
  for (int mask = 32; mask >= 1; mask >>= 1) p = partial_xor_merge(p, mask, lane);
  if (lane == 0) {
    conf[row] = 1.0f / p.s;
    entropy[row] = logf(p.s) - kLn2 * p.t / p.s;
    argmax[row] = p.idx;
    if (max_logit) max_logit[row] = p.m;
  }
}

}  // namespace

int lmhead_num_slices(bool bf16, int n_rows, int vocab) {
  (void)n_rows;
  const int rows = bf16 ? kBf16SliceRows : kF32SliceRows;
  return (vocab + rows - 1) / rows;
}

size_t lmhead_ws_bytes(bool bf16, int n_rows, int vocab) {
  return static_cast<size_t>(n_rows) * lmhead_num_slices(bf16, n_rows, vocab) * sizeof(Partial);
}

hipError_t lmhead_partials(bool bf16, int n_rows, int hidden, int vocab, const void* h,
                           const void* w, void* ws, hipStream_t s) {
  if (n_rows == 0) return hipSuccess;
  Partial* part = static_cast<Partial*>(ws);
  const int n_slices = lmhead_num_slices(bf16, n_rows, vocab);
  if (!bf16) {
    dim3 grid(n_slices, n_rows);
    hipLaunchKernelGGL(lmhead_f32_kernel, grid, dim3(256), 0, s, static_cast<const float*>(h),
                       static_cast<const float*>(w), n_rows, hidden, vocab, n_slices, part);
    return hipGetLastError();
  }
  if (n_rows <= 32) return launch_bf16<TileNarrow>(n_rows, hidden, vocab, h, w, part, n_slices, s);
  if (n_rows <= 64) return launch_bf16<TileMid>(n_rows, hidden, vocab, h, w, part, n_slices, s);
  return launch_bf16<TileWide>(n_rows, hidden, vocab, h, w, part, n_slices, s);
}

hipError_t lmhead_combine(int n_rows, int n_slices, const void* ws, float* conf,
                          float* entropy, int32_t* argmax, float* max_logit, hipStream_t s) {
  if (n_rows == 0) return hipSuccess;
  hipLaunchKernelGGL(lmhead_combine_kernel, dim3((n_rows + 3) / 4), dim3(256), 0, s,
                     static_cast<const Partial*>(ws), n_rows, n_slices, conf, entropy, argmax,
                     max_logit);
  return hipGetLastError();
}

}  // namespace eb
