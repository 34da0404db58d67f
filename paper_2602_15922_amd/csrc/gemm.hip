// bf16 "NT" GEMM with fused epilogues for gfx950: out = epi(A W^T + bias).
//
// A [M][K] and W [N][K] are both K-contiguous, which is exactly the operand layout
// of the 32x32x16 bf16 MFMA (8 consecutive k per lane for A rows and W rows), so no
// transpose is ever needed.  A workgroup of 4 wavefronts (2x2) computes a BM x BN
// tile; BK=64 slices of A and W are staged through double-buffered LDS (one barrier
// per slice) with the next slice's global loads in flight during the MFMAs.  LDS rows
// are 128 bytes (64 bf16) with 16-byte chunks XOR-swizzled by row, which makes the
// fragment reads (32 rows, same chunk) bank-conflict free.  Tail rows/columns are
// clamped on load and skipped on store; a K tail is zero-filled.
#include "common.h"
#include "kernels.h"

namespace wam {
namespace {

constexpr int BK = 64;

template <int BM, int BN>
struct Cfg {
  static constexpr int WM = 2, WN = 2;               // wave grid
  static constexpr int TM = BM / WM / 32;            // 32x32 tiles per wave, rows
  static constexpr int TN = BN / WN / 32;            // 32x32 tiles per wave, cols
  static constexpr int A_CH = BM * BK / 8 / 256;     // 16-byte chunks per thread (A)
  static constexpr int B_CH = BN * BK / 8 / 256;     // 16-byte chunks per thread (W)
};

WAM_DEV int swz(int row, int ch) { return row * BK + ((ch ^ (row & 7)) << 3); }

// Exact row -> (group, row-in-group) split for a runtime divisor: a float reciprocal
// estimate, corrected by one step (rows < 2^23).
WAM_DEV int64_t group_off(int row, int rows, float inv, int64_t group_stride, int64_t ld) {
  int q = (int)(((float)row + 0.5f) * inv);
  int r = row - q * rows;
  if (r < 0) { q -= 1; r += rows; }
  else if (r >= rows) { q += 1; r -= rows; }
  return (int64_t)q * group_stride + (int64_t)r * ld;
}

// Epilogue of four consecutive columns [col, col+4) of one output row.
template <int EPI>
WAM_DEV void epilogue4(const GemmArgs& g, const float inv_o, const float inv_g, int row, int col, f32x4 v) {
  if (row >= g.M || col >= g.N) return;
  const int64_t orow = group_off(row, g.o_rows, inv_o, g.o_bs, g.ldo);
  if (col + 4 <= g.N) {
    if (g.bias) v += *reinterpret_cast<const f32x4*>(g.bias + col);
    if constexpr (EPI == WAM_EPI_BF16 || EPI == WAM_EPI_GELU_BF16) {
      bf16x4 o;
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = (bf16)(EPI == WAM_EPI_GELU_BF16 ? gelu_tanh_f(v[j]) : v[j]);
      *reinterpret_cast<bf16x4*>(static_cast<bf16*>(g.out) + orow + col) = o;
    } else if constexpr (EPI == WAM_EPI_RESID_F32) {
      f32x4 gt = {1.f, 1.f, 1.f, 1.f};
      if (g.gate_a || g.gate_v) {
        gt = g.gate_a ? *reinterpret_cast<const f32x4*>(g.gate_a + col) : f32x4{0.f, 0.f, 0.f, 0.f};
        if (g.gate_v)
          gt += *reinterpret_cast<const f32x4*>(g.gate_v + group_off(row, g.gate_rows, inv_g, g.gate_stride, 0) + col);
      }
      f32x4* o = reinterpret_cast<f32x4*>(static_cast<float*>(g.out) + orow + col);
      *o = *o + gt * v;
    } else {
      *reinterpret_cast<f32x4*>(static_cast<float*>(g.out) + orow + col) = v;
    }
    return;
  }
  // ragged last columns
  for (int j = 0; j < 4 && col + j < g.N; ++j) {
    float x = v[j] + (g.bias ? g.bias[col + j] : 0.f);
    if constexpr (EPI == WAM_EPI_BF16) {
      static_cast<bf16*>(g.out)[orow + col + j] = (bf16)x;
    } else if constexpr (EPI == WAM_EPI_GELU_BF16) {
      static_cast<bf16*>(g.out)[orow + col + j] = (bf16)gelu_tanh_f(x);
    } else if constexpr (EPI == WAM_EPI_RESID_F32) {
      float gt = 1.f;
      if (g.gate_a || g.gate_v) {
        gt = g.gate_a ? g.gate_a[col + j] : 0.f;
        if (g.gate_v) gt += g.gate_v[group_off(row, g.gate_rows, inv_g, g.gate_stride, 0) + col + j];
      }
      float* o = static_cast<float*>(g.out) + orow + col + j;
      *o = *o + gt * x;
    } else {
      static_cast<float*>(g.out)[orow + col + j] = x;
    }
  }
}

template <int BM, int BN, int EPI>
__global__ __launch_bounds__(256) void gemm_nt(const GemmArgs g, int tiles_m, int tiles_n) {
  using C = Cfg<BM, BN>;
  // one LDS allocation: two A slices, two W slices; reused for epilogue staging
  __shared__ __attribute__((aligned(16))) bf16 smem[2 * (BM + BN) * BK];
  auto As = [&](int buf) { return smem + buf * (BM * BK); };
  auto Bs = [&](int buf) { return smem + 2 * BM * BK + buf * (BN * BK); };

  // XCD-aware remap: the hardware deals workgroups round-robin over 8 XCDs; give each
  // XCD a contiguous range of tiles so tiles that share a W panel share an L2.
  const int nblk = tiles_m * tiles_n;
  const int i = blockIdx.x, x = i & 7, j = i >> 3;
  const int per = nblk >> 3, rem = nblk & 7;
  const int lid = x * per + (x < rem ? x : rem) + j;
  const int tm = lid % tiles_m, tn = lid / tiles_m;  // consecutive tiles share a W panel
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int hh = lane >> 5, l32 = lane & 31;
  const int wm = w / C::WN, wn = w % C::WN;

  const bf16* A = static_cast<const bf16*>(g.A);
  const bf16* W = static_cast<const bf16*>(g.W);

  // per-thread global row offsets (constant over the K loop)
  const int kc = tid & 7;  // 16-byte chunk inside a BK slice
  int64_t a_off[C::A_CH], b_off[C::B_CH];
#pragma unroll
  for (int c = 0; c < C::A_CH; ++c) {
    int r = m0 + (tid >> 3) + 32 * c;
    r = r < g.M ? r : g.M - 1;
    a_off[c] = (int64_t)(r / g.a_rows) * g.a_bs + (int64_t)(r % g.a_rows) * g.lda;
  }
#pragma unroll
  for (int c = 0; c < C::B_CH; ++c) {
    int r = n0 + (tid >> 3) + 32 * c;
    r = r < g.N ? r : g.N - 1;
    b_off[c] = (int64_t)r * g.ldw;
  }

  bf16x8 ra[C::A_CH], rb[C::B_CH];
  auto gload = [&](int k0) {
    const int k = k0 + kc * 8;
    const bool ok = k < g.K;
#pragma unroll
    for (int c = 0; c < C::A_CH; ++c) ra[c] = ok ? load_bf16x8(A + a_off[c] + k) : bf16x8{};
#pragma unroll
    for (int c = 0; c < C::B_CH; ++c) rb[c] = ok ? load_bf16x8(W + b_off[c] + k) : bf16x8{};
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int c = 0; c < C::A_CH; ++c)
      *reinterpret_cast<bf16x8*>(&As(buf)[swz((tid >> 3) + 32 * c, kc)]) = ra[c];
#pragma unroll
    for (int c = 0; c < C::B_CH; ++c)
      *reinterpret_cast<bf16x8*>(&Bs(buf)[swz((tid >> 3) + 32 * c, kc)]) = rb[c];
  };

  f32x16 acc[C::TM][C::TN];
#pragma unroll
  for (int a = 0; a < C::TM; ++a)
#pragma unroll
    for (int b = 0; b < C::TN; ++b) acc[a][b] = f32x16{};

  const int nk = (g.K + BK - 1) / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 fa[C::TM], fb[C::TN];
#pragma unroll
      for (int a = 0; a < C::TM; ++a)
        fa[a] = *reinterpret_cast<const bf16x8*>(
            &As(cur)[swz(wm * (BM / C::WM) + a * 32 + l32, 2 * ks + hh)]);
#pragma unroll
      for (int b = 0; b < C::TN; ++b)
        fb[b] = *reinterpret_cast<const bf16x8*>(
            &Bs(cur)[swz(wn * (BN / C::WN) + b * 32 + l32, 2 * ks + hh)]);
#pragma unroll
      for (int a = 0; a < C::TM; ++a)
#pragma unroll
        for (int b = 0; b < C::TN; ++b) acc[a][b] = mfma32(fa[a], fb[b], acc[a][b]);
    }
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: each wave stages 32 rows x WCOLS of its tile through LDS (reusing
  // the operand buffers) so every lane then owns 4 consecutive columns of one row and
  // the stores are 8/16-byte vectors over contiguous row segments.
  constexpr int WCOLS = BN / C::WN, SROW = WCOLS + 4;
  static_assert(C::WM * C::WN * 32 * SROW * 4 <= 2 * (BM + BN) * BK * 2, "staging does not fit");
  float* stage = reinterpret_cast<float*>(smem) + w * 32 * SROW;
  const float inv_o = 1.0f / (float)g.o_rows, inv_g = 1.0f / (float)g.gate_rows;
  const int row_base = m0 + wm * (BM / C::WM), col_base = n0 + wn * WCOLS;
#pragma unroll
  for (int a = 0; a < C::TM; ++a) {
#pragma unroll
    for (int b = 0; b < C::TN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stage[(8 * (r >> 2) + 4 * hh + (r & 3)) * SROW + b * 32 + l32] = acc[a][b][r];
    __syncthreads();
#pragma unroll
    for (int p = 0; p < 32 * WCOLS / 256; ++p) {
      const int idx = p * 64 + lane;
      const int rloc = idx / (WCOLS / 4), c4 = idx % (WCOLS / 4);
      const f32x4 v = *reinterpret_cast<const f32x4*>(&stage[rloc * SROW + c4 * 4]);
      epilogue4<EPI>(g, inv_o, inv_g, row_base + a * 32 + rloc, col_base + c4 * 4, v);
    }
    __syncthreads();
  }
}

template <int BM, int BN>
hipError_t launch_cfg(const GemmArgs& g, hipStream_t s) {
  const int tm = (g.M + BM - 1) / BM, tn = (g.N + BN - 1) / BN;
  dim3 grid(tm * tn), block(256);
  switch (g.epi) {
    case WAM_EPI_BF16: hipLaunchKernelGGL((gemm_nt<BM, BN, WAM_EPI_BF16>), grid, block, 0, s, g, tm, tn); break;
    case WAM_EPI_GELU_BF16: hipLaunchKernelGGL((gemm_nt<BM, BN, WAM_EPI_GELU_BF16>), grid, block, 0, s, g, tm, tn); break;
    case WAM_EPI_RESID_F32: hipLaunchKernelGGL((gemm_nt<BM, BN, WAM_EPI_RESID_F32>), grid, block, 0, s, g, tm, tn); break;
    default: hipLaunchKernelGGL((gemm_nt<BM, BN, WAM_EPI_F32>), grid, block, 0, s, g, tm, tn); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& gin, hipStream_t s) {
  GemmArgs g = gin;
  if (g.a_rows <= 0) { g.a_rows = g.M; g.a_bs = 0; }
  if (g.o_rows <= 0) { g.o_rows = g.M; g.o_bs = 0; }
  if (g.gate_rows <= 0) { g.gate_rows = g.M; g.gate_stride = 0; }
  // Pick the tile whose rounds of 256 concurrent workgroups cost least, weighting
  // smaller tiles by their lower MFMA efficiency (measured).
  struct Opt { int bm, bn; float eff; };
  const Opt opts[3] = {{256, 256, 1.0f}, {128, 256, 0.85f}, {128, 128, 0.6f}};
  int best = 0;
  float best_cost = 0.f;
  for (int i = 0; i < 3; ++i) {
    const long tiles = (long)((g.M + opts[i].bm - 1) / opts[i].bm) * ((g.N + opts[i].bn - 1) / opts[i].bn);
    const float cost = (float)((tiles + 255) / 256) * opts[i].bm * opts[i].bn / opts[i].eff;
    if (i == 0 || cost < best_cost) { best = i; best_cost = cost; }
  }
  if (best == 0) return launch_cfg<256, 256>(g, s);
  if (best == 1) return launch_cfg<128, 256>(g, s);
  return launch_cfg<128, 128>(g, s);
}

}  // namespace wam
