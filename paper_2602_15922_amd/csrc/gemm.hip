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

template <int EPI>
WAM_DEV void epilogue_store(const GemmArgs& g, int row, int col, float acc) {
  if (row >= g.M || col >= g.N) return;
  float v = acc + (g.bias ? g.bias[col] : 0.f);
  const int64_t orow = (int64_t)(row / g.o_rows) * g.o_bs + (int64_t)(row % g.o_rows) * g.ldo;
  if constexpr (EPI == WAM_EPI_BF16) {
    static_cast<bf16*>(g.out)[orow + col] = (bf16)v;
  } else if constexpr (EPI == WAM_EPI_GELU_BF16) {
    static_cast<bf16*>(g.out)[orow + col] = (bf16)gelu_tanh_f(v);
  } else if constexpr (EPI == WAM_EPI_RESID_F32) {
    float gt = 1.f;
    if (g.gate_a || g.gate_v) {
      gt = g.gate_a ? g.gate_a[col] : 0.f;
      if (g.gate_v) gt += g.gate_v[(int64_t)(row / g.gate_rows) * g.gate_stride + col];
    }
    float* o = static_cast<float*>(g.out) + orow + col;
    *o = *o + gt * v;
  } else {
    static_cast<float*>(g.out)[orow + col] = v;
  }
}

template <int BM, int BN, int EPI>
__global__ __launch_bounds__(256) void gemm_nt(const GemmArgs g, int tiles_m, int tiles_n) {
  using C = Cfg<BM, BN>;
  __shared__ __attribute__((aligned(16))) bf16 As[2][BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * BK];

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
      *reinterpret_cast<bf16x8*>(&As[buf][swz((tid >> 3) + 32 * c, kc)]) = ra[c];
#pragma unroll
    for (int c = 0; c < C::B_CH; ++c)
      *reinterpret_cast<bf16x8*>(&Bs[buf][swz((tid >> 3) + 32 * c, kc)]) = rb[c];
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
            &As[cur][swz(wm * (BM / C::WM) + a * 32 + l32, 2 * ks + hh)]);
#pragma unroll
      for (int b = 0; b < C::TN; ++b)
        fb[b] = *reinterpret_cast<const bf16x8*>(
            &Bs[cur][swz(wn * (BN / C::WN) + b * 32 + l32, 2 * ks + hh)]);
#pragma unroll
      for (int a = 0; a < C::TM; ++a)
#pragma unroll
        for (int b = 0; b < C::TN; ++b) acc[a][b] = mfma32(fa[a], fb[b], acc[a][b]);
    }
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int a = 0; a < C::TM; ++a)
#pragma unroll
    for (int b = 0; b < C::TN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * (BM / C::WM) + a * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
        const int col = n0 + wn * (BN / C::WN) + b * 32 + l32;
        epilogue_store<EPI>(g, row, col, acc[a][b][r]);
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
  // big tiles where they still fill the 256 CUs, smaller ones otherwise
  const long t256 = (long)((g.M + 255) / 256) * ((g.N + 255) / 256);
  if (t256 >= 256) return launch_cfg<256, 256>(g, s);
  return launch_cfg<128, 128>(g, s);
}

}  // namespace wam
