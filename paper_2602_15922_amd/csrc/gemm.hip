// bf16 "NT" GEMM with fused epilogues for gfx950: out = epi(A W^T + bias).
//
// A [M][K] and W [N][K] are both K-contiguous, which is exactly the operand layout
// of the 32x32x16 bf16 MFMA (8 consecutive k per lane for A rows and W rows), so no
// transpose is ever needed.  A workgroup of WM x WN wavefronts computes a BM x BN
// tile.  The large tiles use 8 wavefronts (two per SIMD), so one wavefront's barrier
// and LDS waits overlap the other's MFMAs.  BK-wide slices of A and W are fetched
// with direct global->LDS loads into a ring of STAGES LDS buffers: the loads of slice t+STAGES-1 are issued while slice t
// is consumed, so each load has STAGES-1 slices of MFMA work to land (no staging
// registers, one barrier per slice, waits on the vector-memory counter only for the
// slice about to be used).  Within a slice the fragment reads of the next 16-wide
// k-step are issued before the current step's MFMAs.  LDS rows are BK bf16 with
// 16-byte chunks XOR-swizzled by row so the fragment reads (32 consecutive rows, same
// chunk) are bank-conflict free; since lane l of a direct load lands at LDS unit
// base+l, the swizzle is applied by choosing each lane's source chunk.  Tail
// rows/columns are clamped on load and skipped on store; a K tail is zeroed in LDS
// after it lands.
#include "common.h"
#include "kernels.h"

namespace wam {
namespace {

template <int BM_, int BN_, int BK_, int STAGES_, int WM_, int WN_, int OCC_>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, STAGES = STAGES_;
  static constexpr int WM = WM_, WN = WN_;        // wave grid
  static constexpr int OCC = OCC_;                // wavefronts per SIMD the kernel is built for
  static constexpr int NW = WM * WN, NT = NW * 64;
  static constexpr int TM = BM / WM / 32;         // 32x32 tiles per wave, rows
  static constexpr int TN = BN / WN / 32;         // 32x32 tiles per wave, cols
  static constexpr int CPR = BK / 8;              // 16-byte chunks per LDS row
  static constexpr int NIA = BM * CPR / (NW * 64);  // direct-load instructions per wave (A)
  static constexpr int NIB = BN * CPR / (NW * 64);  // (W)
  static constexpr int STAGE = (BM + BN) * BK;    // elements per stage
  static_assert(NIA * NW * 64 == BM * CPR && NIB * NW * 64 == BN * CPR, "slice not a whole number of wave loads");
  // XOR pattern.  gfx950 LDS serves 256 bytes (64 banks) per cycle, i.e. 16 lanes of a
  // 16-byte read; the 16 consecutive rows those lanes read at one logical chunk must land
  // on 16 distinct 16-byte bank slots.  128-byte rows (8 chunks): two rows share a
  // 256-byte bank line, so XOR the chunk by (row>>1)&7; 64-byte rows (4 chunks): XOR
  // by (row>>2)&3.
  static WAM_DEV int pch(int row, int ch) { return CPR == 8 ? (ch ^ ((row >> 1) & 7)) : (ch ^ ((row >> 2) & 3)); }
  static WAM_DEV int swz(int row, int ch) { return row * BK + (pch(row, ch) << 3); }
};

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

typedef __attribute__((address_space(3))) void lds_void;

// One BK slice of NI*64*4 16-byte units into LDS with direct loads.  Wave w's
// instruction c fills units [(w*NI + c)*64, +64); lane l's unit is read from
// src[c] (its row, already offset to its logical chunk kl[c]) at column k0, or, when
// that chunk lies past K, from the row's last chunk (such units are zeroed once they
// have landed).
template <int NI>
WAM_DEV void fetch_slice(bf16* dst, const bf16* base, const int64_t* src, const int* kl, int k0, int K, int w) {
#pragma unroll
  for (int c = 0; c < NI; ++c) {
    const int k = k0 + kl[c] < K ? k0 : K - 8 - kl[c];
    __builtin_amdgcn_global_load_lds(base + src[c] + k, (lds_void*)(dst + (w * NI + c) * 512), 16, 0, 0);
  }
}

// s_waitcnt on the vector-memory counter only (vmcnt <= n; LDS and export counters
// left unconstrained), gfx9 encoding.
#define WAM_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt((((n) & 15) | (((n) >> 4) << 14)) | (7 << 4) | (15 << 8))
// s_waitcnt on the LDS/scalar counter only (lgkmcnt = 0)
#define WAM_WAIT_LGKMCNT0() __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4))

template <typename C, int EPI>
__global__ __launch_bounds__(C::NT, C::OCC) void gemm_nt(const GemmArgs g, int tiles_m, int tiles_n) {
  constexpr int BM = C::BM, BN = C::BN, BK = C::BK, S = C::STAGES;
  __shared__ __attribute__((aligned(16))) bf16 smem[S * C::STAGE];
  auto As = [&](int buf) { return smem + buf * C::STAGE; };
  auto Bs = [&](int buf) { return smem + buf * C::STAGE + BM * BK; };

  // XCD-aware remap: the hardware deals workgroups round-robin over 8 XCDs; give each
  // XCD a contiguous range of tiles so tiles that share a W panel share an L2.
  const int nblk = tiles_m * tiles_n;
  const int i = blockIdx.x, x = i & 7, j = i >> 3;
  const int per = nblk >> 3, rem = nblk & 7;
  const int lid = x * per + (x < rem ? x : rem) + j;
  const int tm = lid % tiles_m, tn = lid / tiles_m;  // consecutive tiles share a W panel
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;  // w < C::NW
  const int hh = lane >> 5, l32 = lane & 31;
  const int wm = w / C::WN, wn = w % C::WN;

  const bf16* A = static_cast<const bf16*>(g.A);
  const bf16* W = static_cast<const bf16*>(g.W);

  // Direct-load sources (loop-invariant).  Unit u of a slice is row u/CPR, physical
  // chunk u%CPR, which holds logical chunk pch(row, u%CPR) (the XOR is an involution).
  constexpr int RPI = 64 / C::CPR;  // rows covered by one wave instruction
  const int lrow = lane / C::CPR;
  int64_t a_src[C::NIA], b_src[C::NIB];
#pragma unroll
  for (int c = 0; c < C::NIA; ++c) {
    const int row = (w * C::NIA + c) * RPI + lrow;
    int r = m0 + row;
    r = r < g.M ? r : g.M - 1;
    a_src[c] = (int64_t)(r / g.a_rows) * g.a_bs + (int64_t)(r % g.a_rows) * g.lda + C::pch(row, lane % C::CPR) * 8;
  }
#pragma unroll
  for (int c = 0; c < C::NIB; ++c) {
    const int row = (w * C::NIB + c) * RPI + lrow;
    int r = n0 + row;
    r = r < g.N ? r : g.N - 1;
    b_src[c] = (int64_t)r * g.ldw + C::pch(row, lane % C::CPR) * 8;
  }
  // logical column offset of each of the lane's units (for the K-tail test)
  int kla[C::NIA], klb[C::NIB];
#pragma unroll
  for (int c = 0; c < C::NIA; ++c) kla[c] = C::pch((w * C::NIA + c) * RPI + lrow, lane % C::CPR) * 8;
#pragma unroll
  for (int c = 0; c < C::NIB; ++c) klb[c] = C::pch((w * C::NIB + c) * RPI + lrow, lane % C::CPR) * 8;
  auto fetch = [&](int kt) {  // no device builtins in lambdas (they drop the host kernel stub)
    const int buf = kt % S;
    fetch_slice<C::NIA>(As(buf), A, a_src, kla, kt * BK, g.K, w);
    fetch_slice<C::NIB>(Bs(buf), W, b_src, klb, kt * BK, g.K, w);
  };
  auto zero_tail = [&](int kt) {  // only for a slice that runs past K
    const int buf = kt % S;
#pragma unroll
    for (int c = 0; c < C::NIA; ++c)
      if (kt * BK + kla[c] >= g.K) *reinterpret_cast<bf16x8*>(As(buf) + ((w * C::NIA + c) * 64 + lane) * 8) = bf16x8{};
#pragma unroll
    for (int c = 0; c < C::NIB; ++c)
      if (kt * BK + klb[c] >= g.K) *reinterpret_cast<bf16x8*>(Bs(buf) + ((w * C::NIB + c) * 64 + lane) * 8) = bf16x8{};
  };

  f32x16 acc[C::TM][C::TN];
#pragma unroll
  for (int a = 0; a < C::TM; ++a)
#pragma unroll
    for (int b = 0; b < C::TN; ++b) acc[a][b] = f32x16{};

  const int nk = (g.K + BK - 1) / BK;
  constexpr int NI = C::NIA + C::NIB;  // direct-load instructions per slice per wave
#pragma unroll
  for (int p = 0; p < S - 1; ++p)
    if (p < nk) fetch(p);
  for (int kt = 0; kt < nk; ++kt) {
    // slice kt has landed once at most the younger prefetched slices are in flight
    const int younger = (nk - 1 - kt) < (S - 2) ? (nk - 1 - kt) : (S - 2);
    if (younger >= 2) WAM_WAIT_VMCNT(2 * NI);
    else if (younger == 1) WAM_WAIT_VMCNT(NI);
    else WAM_WAIT_VMCNT(0);
    if ((kt + 1) * BK > g.K) {
      zero_tail(kt);
      WAM_WAIT_LGKMCNT0();
    }
    // Slice kt is visible to all waves and slice kt-1's buffer is free once every wave
    // is here: each wave has waited for its own loads of slice kt above, and its reads
    // of slice kt-1 were consumed by its MFMAs.  A plain s_barrier (the __syncthreads
    // fence would also wait for the prefetched slices still in flight).
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (kt + S - 1 < nk) fetch(kt + S - 1);
    const int cur = kt % S;

    // fragments double-buffered in registers: the reads of k-step ks+1 are in flight
    // while the MFMAs of k-step ks run
    bf16x8 fa[2][C::TM], fb[2][C::TN];
    auto read_frags = [&](int ks, int slot) {
#pragma unroll
      for (int a = 0; a < C::TM; ++a)
        fa[slot][a] = *reinterpret_cast<const bf16x8*>(&As(cur)[C::swz(wm * (BM / C::WM) + a * 32 + l32, 2 * ks + hh)]);
#pragma unroll
      for (int b = 0; b < C::TN; ++b)
        fb[slot][b] = *reinterpret_cast<const bf16x8*>(&Bs(cur)[C::swz(wn * (BN / C::WN) + b * 32 + l32, 2 * ks + hh)]);
    };
    read_frags(0, 0);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      if (ks + 1 < BK / 16) read_frags(ks + 1, (ks + 1) & 1);
#pragma unroll
      for (int a = 0; a < C::TM; ++a)
#pragma unroll
        for (int b = 0; b < C::TN; ++b) acc[a][b] = mfma32(fa[ks & 1][a], fb[ks & 1][b], acc[a][b]);
      // fence the k-step: the next step's LDS reads stay in this step's region
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  __syncthreads();  // all waves done with the operand ring before it is reused

  // ---- epilogue: each wave stages 32 rows x WCOLS of its tile through LDS (reusing
  // the operand buffers) so every lane then owns 4 consecutive columns of one row and
  // the stores are 8/16-byte vectors over contiguous row segments.
  // rows padded by 8 floats: the two half-waves (rows 4 apart) use disjoint banks
  constexpr int WCOLS = BN / C::WN, SROW = WCOLS + 8;
  static_assert(C::WM * C::WN * 32 * SROW * 4 <= S * C::STAGE * 2, "staging does not fit");
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

template <typename Cf>
hipError_t launch_cfg(const GemmArgs& g, hipStream_t s) {
  const int tm = (g.M + Cf::BM - 1) / Cf::BM, tn = (g.N + Cf::BN - 1) / Cf::BN;
  dim3 grid(tm * tn), block(Cf::NT);
  switch (g.epi) {
    case WAM_EPI_BF16: hipLaunchKernelGGL((gemm_nt<Cf, WAM_EPI_BF16>), grid, block, 0, s, g, tm, tn); break;
    case WAM_EPI_GELU_BF16: hipLaunchKernelGGL((gemm_nt<Cf, WAM_EPI_GELU_BF16>), grid, block, 0, s, g, tm, tn); break;
    case WAM_EPI_RESID_F32: hipLaunchKernelGGL((gemm_nt<Cf, WAM_EPI_RESID_F32>), grid, block, 0, s, g, tm, tn); break;
    default: hipLaunchKernelGGL((gemm_nt<Cf, WAM_EPI_F32>), grid, block, 0, s, g, tm, tn); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& gin, hipStream_t s) {
  GemmArgs g = gin;
  if (g.a_rows <= 0) { g.a_rows = g.M; g.a_bs = 0; }
  if (g.o_rows <= 0) { g.o_rows = g.M; g.o_bs = 0; }
  if (g.gate_rows <= 0) { g.gate_rows = g.M; g.gate_stride = 0; }
  // Pick the tile whose rounds of concurrent workgroups cost least (per_cu workgroups
  // of a tile fit one CU), weighting tiles by their measured MFMA efficiency.
  struct Opt { int bm, bn, per_cu; float eff; };
  const Opt opts[3] = {{256, 256, 1, 1.0f}, {128, 256, 1, 0.85f}, {128, 128, 2, 0.6f}};
  int best = 0;
  float best_cost = 0.f;
  for (int i = 0; i < 3; ++i) {
    const long tiles = (long)((g.M + opts[i].bm - 1) / opts[i].bm) * ((g.N + opts[i].bn - 1) / opts[i].bn);
    const long slots = 256L * opts[i].per_cu;
    const float cost = (float)((tiles + slots - 1) / slots) * opts[i].bm * opts[i].bn * opts[i].per_cu / opts[i].eff;
    if (i == 0 || cost < best_cost) { best = i; best_cost = cost; }
  }
  if (best == 0) return launch_cfg<Cfg<256, 256, 32, 4, 2, 4, 2>>(g, s);
  if (best == 1) return launch_cfg<Cfg<128, 256, 64, 3, 2, 4, 2>>(g, s);
  return launch_cfg<Cfg<128, 128, 64, 2, 2, 2, 2>>(g, s);
}

}  // namespace wam
