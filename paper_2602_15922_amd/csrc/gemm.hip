// bf16 "NT" GEMM with fused epilogues for gfx950: out = epi(A W^T + bias).
//
// A [M][K] and W [N][K] are both K-contiguous, which is exactly the operand layout
// of the 32x32x16 bf16 MFMA (8 consecutive k per lane for A rows and W rows), so no
// transpose is ever needed.  A workgroup of WM x WN wavefronts computes a BM x BN
// tile.  The large tiles use 8 wavefronts (two per SIMD), so one wavefront's barrier
// and LDS waits overlap the other's MFMAs.  BK-wide slices of A and W are fetched
// with buffer loads straight into LDS (a scalar resource, a loop-invariant 32-bit lane
// offset and a scalar slice offset: no vector ALU work per load) into a ring of STAGES
// LDS buffers; the steady-state loop handles STAGES slices per iteration so each
// stage's LDS offsets are immediates.  One barrier per slice, placed before the
// slice's last k-step: after it, that k-step's MFMAs run while the slice STAGES ahead
// is fetched into the stage just freed and the next slice's first fragments are read,
// so no wave starts a slice waiting on LDS (no staging registers; waits on the
// vector-memory counter only for the slice about to be used).  Within a slice the
// fragment reads of the next 16-wide k-step are issued between the current step's
// MFMAs.  LDS rows are BK bf16 with
// 16-byte chunks XOR-swizzled by row so the fragment reads (32 consecutive rows, same
// chunk) are bank-conflict free; since lane l of a direct load lands at LDS unit
// base+l, the swizzle is applied by choosing each lane's source chunk.  Tail
// rows/columns are clamped on load and skipped on store; a K tail is zeroed in LDS
// after it lands.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace wam {
int cu_count();
namespace {

// EB: operand bytes per element, 2 (bf16: 32x32x16 MFMA) or 1 (FP8 E4M3: the 32x32x64
// f8f6f4 MFMA, scales applied in the epilogue).
template <int BM_, int BN_, int BK_, int STAGES_, int WM_, int WN_, int OCC_, int EB_ = 2>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, STAGES = STAGES_;
  static constexpr int WM = WM_, WN = WN_;        // wave grid
  static constexpr int OCC = OCC_;                // wavefronts per SIMD the kernel is built for
  static constexpr int EB = EB_;
  static constexpr int NW = WM * WN, NT = NW * 64;
  static constexpr int TM = BM / WM / 32;         // 32x32 tiles per wave, rows
  static constexpr int TN = BN / WN / 32;         // 32x32 tiles per wave, cols
  static constexpr int ROWB = BK * EB;            // bytes per LDS row
  static constexpr int CPR = ROWB / 16;           // 16-byte chunks per LDS row
  static constexpr int EPC = 16 / EB;             // elements per chunk
  static constexpr int KCH = EB == 2 ? 2 : 4;     // chunks per MFMA k-step (16 bf16 / 64 fp8)
  static constexpr int FCH = KCH / 2;             // chunks of one lane's fragment
  static constexpr int KS = CPR / KCH;            // MFMA k-steps per slice
  static constexpr int NIA = BM * CPR / (NW * 64);  // direct-load instructions per wave (A)
  static constexpr int NIB = BN * CPR / (NW * 64);  // (W)
  static constexpr int STAGE = (BM + BN) * ROWB;  // bytes per stage
  static constexpr bool MXA = false;              // block-scaled FP8 A (MxA below)
  static constexpr int NI = NIA + NIB;            // vector memory instructions per slice per wave
  static_assert(NIA * NW * 64 == BM * CPR && NIB * NW * 64 == BN * CPR, "slice not a whole number of wave loads");
  // XOR pattern.  gfx950 LDS serves 256 bytes (64 banks) per cycle, i.e. 16 lanes of a
  // 16-byte read; the 16 consecutive rows those lanes read at one logical chunk must land
  // on 16 distinct 16-byte bank slots.  128-byte rows (8 chunks): two rows share a
  // 256-byte bank line, so XOR the chunk by (row>>1)&7; 64-byte rows (4 chunks): XOR
  // by (row>>2)&3.
  static WAM_DEV int pch(int row, int ch) { return CPR == 8 ? (ch ^ ((row >> 1) & 7)) : (ch ^ ((row >> 2) & 3)); }
  static WAM_DEV int swz(int row, int ch) { return row * ROWB + (pch(row, ch) << 4); }  // bytes
};

// Block-scaled FP8 A: every slice also loads, per 32-row tile of the wave, the lane's row's
// exponents of the slice's two 64-column blocks (one coalesced 4-byte load per tile: the
// exponent layout keeps a block pair's rows contiguous, 4 bytes per row, of which the
// MFMA's byte select reads the first two; a 16-bit load would need a zero extension that
// the compiler places at the loop's head, waiting there for the newest loads).
template <typename C>
struct MxA : C {
  static constexpr bool MXA = true;
  static constexpr int NI = C::NIA + C::NIB + C::TM;
};

// The maximum over each row of 16 lanes of a value >= 0, in DPP (no LDS round trips; each
// step folds into the max instruction): the two quad swaps give each lane its quad's
// maximum, the half-row mirror (lane i and 7 - i of each 8) pairs the quads, the row
// mirror (i and 15 - i) the halves.  A source lane that is off reads as 0.  (On the bit
// patterns, whose unsigned order is the order of non-negative floats.)
#define WAM_DPP_MAX(u, ctrl) max(u, (unsigned)__builtin_amdgcn_mov_dpp((int)u, ctrl, 0xF, 0xF, true))
WAM_DEV float row16_max(float v) {
  unsigned u = __float_as_uint(v);
  u = WAM_DPP_MAX(u, 0xB1);   // quad_perm [1, 0, 3, 2]
  u = WAM_DPP_MAX(u, 0x4E);   // quad_perm [2, 3, 0, 1]
  u = WAM_DPP_MAX(u, 0x141);  // row_half_mirror
  u = WAM_DPP_MAX(u, 0x140);  // row_mirror
  return __uint_as_float(u);
}
#undef WAM_DPP_MAX

// Exact row -> (group, row-in-group) split for a runtime divisor: a float reciprocal
// estimate, corrected by one step (rows < 2^23).
WAM_DEV int64_t group_off(int row, int rows, float inv, int64_t group_stride, int64_t ld) {
  int q = (int)(((float)row + 0.5f) * inv);
  int r = row - q * rows;
  if (r < 0) { q -= 1; r += rows; }
  else if (r >= rows) { q += 1; r -= rows; }
  return (int64_t)q * group_stride + (int64_t)r * ld;
}

// Offset of row `row`'s per-group gate vector: its group's stride, plus gate_alt for
// the rows of a group at or past gate_split.
WAM_DEV int64_t gate_off(const GemmArgs& g, int row, float inv) {
  int q = (int)(((float)row + 0.5f) * inv);
  int r = row - q * g.gate_rows;
  if (r < 0) { q -= 1; r += g.gate_rows; }
  else if (r >= g.gate_rows) { q += 1; r -= g.gate_rows; }
  return (int64_t)q * g.gate_stride + (g.gate_split > 0 && r >= g.gate_split ? g.gate_alt : 0);
}

// Epilogue of the last, partial group of columns [col, N) of one output row (col < N <
// col + 4): element by element.
template <int EPI>
WAM_DEV void epilogue_ragged(const GemmArgs& g, const float inv_o, const float inv_g, int row, int col, f32x4 v) {
  if constexpr (EPI == WAM_EPI_ROPE) return;  // N = 3 d with d a multiple of 64: no partial column group
  if constexpr (EPI == WAM_EPI_GELU_MX8) return;  // its N is a multiple of 128: never ragged
  const int64_t orow = group_off(row, g.o_rows, inv_o, g.o_bs, g.ldo);
  if (g.a_scale) v *= g.a_scale[row];  // FP8 operands: per-row and per-column scales
  for (int j = 0; j < 4 && col + j < g.N; ++j) {
    float x = v[j] * (g.w_scale ? g.w_scale[col + j] : 1.f) + (g.bias ? g.bias[col + j] : 0.f);
    if constexpr (EPI == WAM_EPI_BF16) {
      static_cast<bf16*>(g.out)[orow + col + j] = (bf16)x;
    } else if constexpr (EPI == WAM_EPI_GELU_BF16) {
      static_cast<bf16*>(g.out)[orow + col + j] = (bf16)gelu_tanh_f(x);
    } else if constexpr (EPI == WAM_EPI_RESID_F32) {
      float gt = 1.f;
      if (g.gate_a || g.gate_v) {
        gt = g.gate_a ? g.gate_a[col + j] : 0.f;
        if (g.gate_v) gt += g.gate_v[gate_off(g, row, inv_g) + col + j];
      }
      float* o = static_cast<float*>(g.out) + orow + col + j;
      *o = *o + gt * x;
    } else {
      static_cast<float*>(g.out)[orow + col + j] = x;
    }
  }
}

typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt on the vector-memory counter only (vmcnt <= n; LDS and export counters
// left unconstrained), gfx9 encoding.
#define WAM_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt((((n) & 15) | (((n) >> 4) << 14)) | (7 << 4) | (15 << 8))
// s_waitcnt on the LDS/scalar counter only (lgkmcnt = 0)
#define WAM_WAIT_LGKMCNT0() __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4))

// 16 bytes per lane from a buffer straight into LDS (lane l lands at lds + 16*l).  A
// plain function: the builtin's operands must not depend on a template parameter.
WAM_DEV void load_lds16(__amdgpu_buffer_rsrc_t r, char* lds, int voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)lds, 16, voff, soff, 0, 0);
}

// Per-workgroup state of the main loop: the operand base pointers and the lanes'
// loop-invariant byte offsets of their load units and LDS fragment reads.
template <typename C>
struct GemmLane {
  const void *A, *W;
  int a_off[C::NIA], b_off[C::NIB];  // byte offset of the lane's unit (row + logical chunk)
  int kla[C::NIA], klb[C::NIB];      // logical column (elements) of the lane's unit in a slice
  int fa_off[C::KS][C::FCH], fb_off[C::KS][C::FCH];  // LDS byte offsets of the lane's fragment
  int w;
  const uint8_t* ae;  // block-scaled A: exponents, bytes between block pairs, 4 * the lane's rows
  int64_t ae_ld;
  int er[C::TM];
};

// The exponents of slice kt's two 64-column blocks for the lane's rows (block-scaled A).
template <typename C>
WAM_DEV void fetch_exp(const GemmLane<C>& L, int kt, unsigned (&e)[C::TM]) {
  if constexpr (C::MXA) {
#pragma unroll
    for (int a = 0; a < C::TM; ++a) e[a] = *reinterpret_cast<const unsigned*>(L.ae + kt * L.ae_ld + L.er[a]);
  }
}

// One BK slice into ring stage `buf` with buffer loads straight into LDS: lane l of
// wave w's instruction c fills unit (w*NI + c)*64 + l.  Full slices need no per-lane
// work (scalar slice offset + loop-invariant lane offset); in a slice that runs past K
// a unit whose chunk lies past K re-reads the row's last in-range chunk instead (it is
// zeroed in LDS once landed).
// FULL: the caller knows the slice lies inside K (block-scaled A: K a multiple of BK).
template <typename C, bool FULL = false>
WAM_DEV void fetch_slice(char* smem, int buf, const GemmLane<C>& L, int kt, int K) {
  // buffer resources over all of A and W (offsets < 2^31 bytes, checked by the host)
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(L.A), (short)0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(L.W), (short)0, 0x7fffffff, 0x00020000);
  char* As = smem + buf * C::STAGE;
  char* Bs = As + C::BM * C::ROWB;
  const int k0 = kt * C::BK, soff = C::EB * k0;
  if (FULL || k0 + C::BK <= K) {
#pragma unroll
    for (int c = 0; c < C::NIA; ++c)
      load_lds16(ra, As + (L.w * C::NIA + c) * 1024, L.a_off[c], soff);
#pragma unroll
    for (int c = 0; c < C::NIB; ++c)
      load_lds16(rb, Bs + (L.w * C::NIB + c) * 1024, L.b_off[c], soff);
  } else {
#pragma unroll
    for (int c = 0; c < C::NIA; ++c) {
      const int sh = k0 + L.kla[c] < K ? 0 : C::EB * (K - C::EPC - L.kla[c] - k0);
      load_lds16(ra, As + (L.w * C::NIA + c) * 1024, L.a_off[c] + sh, soff);
    }
#pragma unroll
    for (int c = 0; c < C::NIB; ++c) {
      const int sh = k0 + L.klb[c] < K ? 0 : C::EB * (K - C::EPC - L.klb[c] - k0);
      load_lds16(rb, Bs + (L.w * C::NIB + c) * 1024, L.b_off[c] + sh, soff);
    }
  }
}

// Zero the units of a landed slice whose chunks lie past K (only in the last slice).
template <typename C>
WAM_DEV void zero_tail(char* smem, int buf, const GemmLane<C>& L, int kt, int K, int lane) {
  char* As = smem + buf * C::STAGE;
  char* Bs = As + C::BM * C::ROWB;
#pragma unroll
  for (int c = 0; c < C::NIA; ++c)
    if (kt * C::BK + L.kla[c] >= K) *reinterpret_cast<u32x4*>(As + ((L.w * C::NIA + c) * 64 + lane) * 16) = u32x4{};
#pragma unroll
  for (int c = 0; c < C::NIB; ++c)
    if (kt * C::BK + L.klb[c] >= K) *reinterpret_cast<u32x4*>(Bs + ((L.w * C::NIB + c) * 64 + lane) * 16) = u32x4{};
}

// Fragments: bf16 operands are one 16-byte read per 32x32x16 MFMA operand; FP8
// operands are two (32 consecutive k of the lane's row for the 32x32x64 MFMA).
template <typename C>
using Frag = typename std::conditional<C::EB == 2, bf16x8, i32x8>::type;

// The lane's fragments of k-step ks from ring stage `stage` (a compile-time constant in
// the steady state, so every LDS address is a lane offset plus an immediate).
template <typename C>
WAM_DEV void read_frags(const char* smem, int stage, const GemmLane<C>& L, int ks, Frag<C> (&fa)[C::TM],
                        Frag<C> (&fb)[C::TN]) {
  const char* As = smem + stage * C::STAGE;
  const char* Bs = As + C::BM * C::ROWB;
  constexpr int RB = 32 * C::ROWB;  // bytes of 32 LDS rows
  if constexpr (C::EB == 2) {
#pragma unroll
    for (int a = 0; a < C::TM; ++a) fa[a] = *reinterpret_cast<const bf16x8*>(As + L.fa_off[ks][0] + a * RB);
#pragma unroll
    for (int b = 0; b < C::TN; ++b) fb[b] = *reinterpret_cast<const bf16x8*>(Bs + L.fb_off[ks][0] + b * RB);
  } else {
    auto two = [](const char* lo, const char* hi) {
      const u32x4 x = *reinterpret_cast<const u32x4*>(lo), y = *reinterpret_cast<const u32x4*>(hi);
      return i32x8{(int)x[0], (int)x[1], (int)x[2], (int)x[3], (int)y[0], (int)y[1], (int)y[2], (int)y[3]};
    };
#pragma unroll
    for (int a = 0; a < C::TM; ++a) fa[a] = two(As + L.fa_off[ks][0] + a * RB, As + L.fa_off[ks][1] + a * RB);
#pragma unroll
    for (int b = 0; b < C::TN; ++b) fb[b] = two(Bs + L.fb_off[ks][0] + b * RB, Bs + L.fb_off[ks][1] + b * RB);
  }
}

// The TM x TN MFMAs of k-step ks of a slice (block-scaled A: ea[a] holds the exponents
// of the slice's two blocks for tile a's row, k-step ks takes byte ks).
template <typename C>
WAM_DEV void mfma_step(const Frag<C> (&fa)[C::TM], const Frag<C> (&fb)[C::TN], f32x16 (*acc)[C::TN],
                       const unsigned* ea, int ks) {
#pragma unroll
  for (int a = 0; a < C::TM; ++a)
#pragma unroll
    for (int b = 0; b < C::TN; ++b) {
      if constexpr (C::EB == 2) acc[a][b] = mfma32(fa[a], fb[b], acc[a][b]);
      else if constexpr (C::MXA) acc[a][b] = mfma32_fp8_sa(fa[a], fb[b], acc[a][b], (int)ea[a], ks);
      else acc[a][b] = mfma32_fp8(fa[a], fb[b], acc[a][b]);
    }
}

// FP8 tiles: an empty asm that reads and writes every accumulator after a k-step's MFMAs,
// so they stay ahead of what follows in program order.  Without it the compiler sinks
// them below the next k-step's fragment reads and the slice's barrier, keeps three sets
// of 32-byte fragments live and spills (the 256x256 tiles' old loop needed 144 bytes of
// scratch; the 128x256 tiles now take 201 registers instead of 254).
template <typename C>
WAM_DEV void pin_acc(f32x16 (*acc)[C::TN]) {
#pragma unroll
  for (int a = 0; a < C::TM; ++a)
#pragma unroll
    for (int b = 0; b < C::TN; ++b) asm volatile("" : "+v"(acc[a][b]));
}

// Instruction order of one k-step: one LDS read (while any of the NDS are left) and one
// direct global load (while any of the NVM are left) ahead of each of its NMF MFMAs, so
// the reads for the next k-step and the next slice's prefetch issue between the MFMAs.
template <int NMF, int NDS, int NVM>
WAM_DEV void interleave_step() {
#pragma unroll
  for (int i = 0; i < NMF; ++i) {
    if (i < NDS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
    if (i < NVM) __builtin_amdgcn_sched_group_barrier(0x20, 1, 0);   // vector memory read
    __builtin_amdgcn_sched_group_barrier(0x8, 1, 0);                 // MFMA
  }
}

WAM_DEV void block_barrier() {
  // a plain s_barrier: __syncthreads would also wait for the prefetched slices in flight
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Slice t of the steady state, in ring stage CUR; on entry fa/fb[0] hold its k-step 0
// fragments.  Every k-step but the last reads the next k-step's fragments while its
// MFMAs run.  Before the last k-step the wave waits for its reads of this slice and for
// its loads of slice t+1, and the workgroup meets at the slice's only barrier: slice t+1
// is then visible to all, and stage CUR (slice t) is free, so the last k-step's MFMAs
// run while slice t+S is fetched into stage CUR and k-step 0 of slice t+1 is read.  No
// wave waits on an LDS read right after the barrier.
// (Block-scaled A: ering[stage] holds the exponents of the slice in that stage.  Slice
// t+S's exponents are loaded after slice t's last MFMAs, so they take the same registers:
// loaded any earlier, both values are live at once and the compiler moves registers at
// the loop's back edge, each move waiting for its load and so for every slice in flight.)
// (Block-scaled A runs every slice here: past the last slice the prefetch re-reads it into
// the free stage, which is never read; nk is used for that only.)
template <typename C, int CUR>
WAM_DEV void slice_steady(char* smem, const GemmLane<C>& L, int t, int K, f32x16 (*acc)[C::TN],
                          Frag<C> (&fa)[2][C::TM], Frag<C> (&fb)[2][C::TN], unsigned (&ering)[C::STAGES][C::TM],
                          int nk = 0) {
  constexpr int S = C::STAGES, KS = C::KS, NI = C::NI;
  constexpr int NMF = C::TM * C::TN, NR = (C::TM + C::TN) * C::FCH;
#pragma unroll
  for (int ks = 0; ks < KS - 1; ++ks) {
    read_frags<C>(smem, CUR, L, ks + 1, fa[(ks + 1) & 1], fb[(ks + 1) & 1]);
    mfma_step<C>(fa[ks & 1], fb[ks & 1], acc, ering[CUR], ks);
    interleave_step<NMF, NR, 0>();
    if constexpr (C::EB == 1) pin_acc<C>(acc);
    __builtin_amdgcn_sched_barrier(0);
  }
  WAM_WAIT_LGKMCNT0();
  WAM_WAIT_VMCNT((S - 2) * NI);
  block_barrier();
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (C::MXA) fetch_slice<C, true>(smem, CUR, L, t + S < nk ? t + S : nk - 1, K);
  else fetch_slice<C>(smem, CUR, L, t + S, K);
  read_frags<C>(smem, (CUR + 1) % S, L, 0, fa[KS & 1], fb[KS & 1]);
  mfma_step<C>(fa[(KS - 1) & 1], fb[(KS - 1) & 1], acc, ering[CUR], KS - 1);
  interleave_step<NMF, NR, C::NIA + C::NIB>();
  if constexpr (C::EB == 1) pin_acc<C>(acc);
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (C::MXA) {
    fetch_exp<C>(L, t + S < nk ? t + S : nk - 1, ering[CUR]);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <typename C, int CUR>
WAM_DEV void steady_group(char* smem, const GemmLane<C>& L, int t, int K, f32x16 (*acc)[C::TN],
                          Frag<C> (&fa)[2][C::TM], Frag<C> (&fb)[2][C::TN], unsigned (&ering)[C::STAGES][C::TM],
                          int nk = 0) {
  slice_steady<C, CUR>(smem, L, t + CUR, K, acc, fa, fb, ering, nk);
  if constexpr (CUR + 1 < C::STAGES) steady_group<C, CUR + 1>(smem, L, t, K, acc, fa, fb, ering, nk);
}

// A slice after the steady state (the last few: fewer younger slices in flight, the next
// one may run past K and need its tail zeroed, nothing to prefetch past the end), with
// the same order as slice_steady and a runtime stage.
template <typename C>
WAM_DEV void slice_tail(char* smem, const GemmLane<C>& L, int t, int nk, int K, int lane, f32x16 (*acc)[C::TN],
                        Frag<C> (&fa)[2][C::TM], Frag<C> (&fb)[2][C::TN], unsigned (&ering)[C::STAGES][C::TM]) {
  constexpr int S = C::STAGES, KS = C::KS, NI = C::NI;
  static_assert(!C::MXA, "block-scaled A runs every slice in the steady state");
  const int cur = t % S;
  const unsigned* ec = ering[0];
#pragma unroll
  for (int ks = 0; ks < KS - 1; ++ks) {
    read_frags<C>(smem, cur, L, ks + 1, fa[(ks + 1) & 1], fb[(ks + 1) & 1]);
    mfma_step<C>(fa[ks & 1], fb[ks & 1], acc, ec, ks);
    if constexpr (C::EB == 1) pin_acc<C>(acc);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (t + 1 < nk) {
    const int younger = (nk - 2 - t) < (S - 2) ? (nk - 2 - t) : (S - 2);  // slices past t+1 in flight
    WAM_WAIT_LGKMCNT0();
    if (younger >= 2) WAM_WAIT_VMCNT(2 * NI);
    else if (younger == 1) WAM_WAIT_VMCNT(NI);
    else WAM_WAIT_VMCNT(0);
    if ((t + 2) * C::BK > K) {
      zero_tail<C>(smem, (t + 1) % S, L, t + 1, K, lane);
      WAM_WAIT_LGKMCNT0();
    }
    block_barrier();
    if (t + S < nk) fetch_slice<C>(smem, cur, L, t + S, K);
    read_frags<C>(smem, (t + 1) % S, L, 0, fa[KS & 1], fb[KS & 1]);
  }
  mfma_step<C>(fa[(KS - 1) & 1], fb[(KS - 1) & 1], acc, ec, KS - 1);

  if constexpr (C::EB == 1) pin_acc<C>(acc);
  __builtin_amdgcn_sched_barrier(0);
}

// XCD-aware remap: the hardware deals workgroups round-robin over 8 XCDs; give each
// XCD a contiguous range of the nblk tiles so tiles that share a W panel share an L2.
// i is a dispatch slot: the workgroup index, or (persistent workgroups, their count a
// multiple of 8) blockIdx.x + r * gridDim.x for round r, which stays on the same XCD.
WAM_DEV int xcd_tile(int i, int nblk) {
  const int x = i & 7, j = i >> 3;
  const int per = nblk >> 3, rem = nblk & 7;
  return x * per + (x < rem ? x : rem) + j;
}

// The workgroup's LDS: one array per size, so the tiles of two configurations in one
// kernel share it.
template <int BYTES>
WAM_DEV char* lds_ring() {
  __shared__ __attribute__((aligned(16))) char buf[BYTES];
  return buf;
}

// One BM x BN output tile (row tile tm, column tile tn, columns from col0) of g, with
// the operand ring and the epilogue's staging in the first STAGES * STAGE of LBYTES
// bytes of LDS.
// EPI: the epilogue (low 3 bits), or-ed with WAM_EPI_MXA for block-scaled FP8 A.
template <typename C0, int EPI, int LBYTES = C0::STAGES * C0::STAGE>
WAM_DEV void gemm_tile(const GemmArgs g, int tm, int tn, int col0) {
  using C = typename std::conditional<(EPI & WAM_EPI_MXA) != 0, MxA<C0>, C0>::type;
  constexpr int E = EPI & 7;
  static_assert(!C::MXA || C::EB == 1, "block-scaled A is FP8");
  static_assert(E != WAM_EPI_GELU_MX8 || C::EB == 1, "the block-scaled output is an FP8 path's");
  static_assert(E != WAM_EPI_ROPE || C::EB == 2, "RoPE in the epilogue is a bf16 path's");
  static_assert(LBYTES >= C::STAGES * C::STAGE, "operand ring does not fit");
  constexpr int BM = C::BM, BN = C::BN, BK = C::BK, S = C::STAGES;
  char* smem = lds_ring<LBYTES>();
  const int m0 = tm * BM, n0 = col0 + tn * BN;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, w < C::NW
  const int hh = lane >> 5, l32 = lane & 31;
  const int wm = w / C::WN, wn = w % C::WN;

  GemmLane<C> L;
  L.A = g.A;
  L.W = g.W;
  L.w = w;
  // Load units: unit u of a slice is row u/CPR, physical chunk u%CPR, which holds
  // logical chunk pch(row, u%CPR) (the XOR is an involution).
  constexpr int RPI = 64 / C::CPR;  // rows covered by one wave instruction
  const int lrow = lane / C::CPR;
#pragma unroll
  for (int c = 0; c < C::NIA; ++c) {
    const int row = (w * C::NIA + c) * RPI + lrow;
    int r = m0 + row;
    r = r < g.M ? r : g.M - 1;
    L.kla[c] = C::pch(row, lane % C::CPR) * C::EPC;
    L.a_off[c] = (int)(C::EB * ((int64_t)(r / g.a_rows) * g.a_bs + (int64_t)(r % g.a_rows) * g.lda + L.kla[c]));
  }
#pragma unroll
  for (int c = 0; c < C::NIB; ++c) {
    const int row = (w * C::NIB + c) * RPI + lrow;
    int r = n0 + row;
    r = r < g.N ? r : g.N - 1;
    L.klb[c] = C::pch(row, lane % C::CPR) * C::EPC;
    L.b_off[c] = (int)(C::EB * ((int64_t)r * g.ldw + L.klb[c]));
  }
  if constexpr (C::MXA) {  // the exponents of the lane's A rows (clamped to the last row)
    L.ae = g.a_exp;
    L.ae_ld = g.a_lde;
#pragma unroll
    for (int a = 0; a < C::TM; ++a) {
      const int r = m0 + wm * (BM / C::WM) + a * 32 + l32;
      L.er[a] = 4 * (r < g.M ? r : g.M - 1);
    }
  }
  // Fragment reads: rows (wm*BM/WM + a*32 + l32) of A and (wn*BN/WN + b*32 + l32) of W
  // at logical chunks KCH*ks + FCH*hh + f; the XOR only depends on l32 (32-row steps keep it).
#pragma unroll
  for (int ks = 0; ks < C::KS; ++ks)
#pragma unroll
    for (int f = 0; f < C::FCH; ++f) {
      const int ra = wm * (BM / C::WM) + l32, rb = wn * (BN / C::WN) + l32;
      L.fa_off[ks][f] = C::swz(ra, C::KCH * ks + C::FCH * hh + f);
      L.fb_off[ks][f] = C::swz(rb, C::KCH * ks + C::FCH * hh + f);
    }

  f32x16 acc[C::TM][C::TN];
#pragma unroll
  for (int a = 0; a < C::TM; ++a)
#pragma unroll
    for (int b = 0; b < C::TN; ++b) acc[a][b] = f32x16{};

  const int nk = (g.K + BK - 1) / BK;
  constexpr int NI = C::NI;  // loads per slice per wave
  static_assert(C::KS % 2 == 0, "fragment slots alternate per k-step and slice");
  unsigned ering[S][C::TM];  // block-scaled A: exponents of the slice in each stage
  // prologue: the first S slices in flight, slice 0 landed and visible, its k-step 0 read
  if constexpr (C::MXA) {
    // Every stage is fetched (past the last slice, the last slice again, into a stage that
    // is never read; the barrier before the epilogue waits for it), so that no path into
    // the main loop leaves an exponent load unaccounted for: the compiler's wait analysis
    // does not correlate the fetch conditions with the wait's, and would wait inside the
    // loop for the first stage's exponents.
#pragma unroll
    for (int p = 0; p < S; ++p) {
      const int kp = p < nk ? p : nk - 1;
      fetch_slice<C, true>(smem, p, L, kp, g.K);
      fetch_exp<C>(L, kp, ering[p]);
    }
    WAM_WAIT_VMCNT((S - 1) * NI);
    block_barrier();
  } else {
#pragma unroll
    for (int p = 0; p < S; ++p)
      if (p < nk) fetch_slice<C>(smem, p, L, p, g.K);
    const int younger = nk - 1 < S - 1 ? nk - 1 : S - 1;
    if (younger >= 2) WAM_WAIT_VMCNT(2 * NI);
    else if (younger == 1) WAM_WAIT_VMCNT(NI);
    else WAM_WAIT_VMCNT(0);
    if (BK > g.K) {
      zero_tail<C>(smem, 0, L, 0, g.K, lane);
      WAM_WAIT_LGKMCNT0();
    }
    block_barrier();
  }
  Frag<C> fa[2][C::TM], fb[2][C::TN];
  read_frags<C>(smem, 0, L, 0, fa[0], fb[0]);
  int kt = 0;
  // steady state, S slices per iteration so each stage index is a constant: every slice
  // here has a successor, prefetches a slice < nk, and waits for a full slice
  if constexpr (C::MXA) {
    // K is a multiple of the slice: S slices per iteration, then the last nk % S
    for (; kt + S <= nk; kt += S) steady_group<C, 0>(smem, L, kt, g.K, acc, fa, fb, ering, nk);
    if (kt < nk) slice_steady<C, 0>(smem, L, kt, g.K, acc, fa, fb, ering, nk);
    if constexpr (S > 2) {
      if (kt + 1 < nk) slice_steady<C, 1>(smem, L, kt + 1, g.K, acc, fa, fb, ering, nk);
    }
  } else {
    for (; kt + 2 * S + 1 <= nk && (kt + 2 * S + 1) * BK <= g.K; kt += S)
      steady_group<C, 0>(smem, L, kt, g.K, acc, fa, fb, ering);
    for (; kt < nk; ++kt) slice_tail<C>(smem, L, kt, nk, g.K, lane, acc, fa, fb, ering);
  }
  __syncthreads();  // all waves done with the operand ring before it is reused

  // ---- epilogue: each wave stages 32 rows x WCOLS of its tile through LDS (reusing
  // the operand buffers) so every lane then owns 4 consecutive columns of one row and
  // the stores are 8/16-byte vectors over contiguous row segments.  A lane keeps the
  // same four columns for the whole tile, so the per-column operands (scales, bias,
  // shared gate) are loaded once; the per-row ones (row scale, per-group gate, the
  // residual) are loaded for all of a slab's rows before its first store.  Interleaved
  // with the stores, each load would wait for the store before it: the compiler cannot
  // prove that the output does not alias those arrays.
  // rows padded by 8 floats: the two half-waves (rows 4 apart) use disjoint banks
  constexpr int WCOLS = BN / C::WN, SROW = WCOLS + 8;
  constexpr int CG = WCOLS / 4, RP = 64 / CG, NP = 32 / RP;  // column groups, rows per pass, passes
  static_assert(64 % CG == 0 && 32 % RP == 0, "a lane's columns must not change between passes");
  static_assert(C::WM * C::WN * 32 * SROW * 4 <= S * C::STAGE, "staging does not fit");
  constexpr bool RESID = E == WAM_EPI_RESID_F32;
  static_assert(E != WAM_EPI_GELU_MX8 || WCOLS == 64, "a wave's columns of a row are one 64-column block");
  float* stage = reinterpret_cast<float*>(smem) + w * 32 * SROW;
  const float inv_o = 1.0f / (float)g.o_rows, inv_g = 1.0f / (float)g.gate_rows;
  const int row_base = m0 + wm * (BM / C::WM), col_base = n0 + wn * WCOLS;
  const int cl = 4 * (lane % CG), col = col_base + cl, rl = lane / CG;
  const bool col_full = col + 4 <= g.N;
  f32x4 cmul = {1.f, 1.f, 1.f, 1.f}, cadd = {0.f, 0.f, 0.f, 0.f}, cgate = {1.f, 1.f, 1.f, 1.f};
  if (col_full) {
    if (g.w_scale) cmul = *reinterpret_cast<const f32x4*>(g.w_scale + col);
    if (g.bias) cadd = *reinterpret_cast<const f32x4*>(g.bias + col);
    if (RESID && (g.gate_a || g.gate_v))
      cgate = g.gate_a ? *reinterpret_cast<const f32x4*>(g.gate_a + col) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int a = 0; a < C::TM; ++a) {
    // per-row operands of this slab's rows (clamped to the last row; only stored rows use
    // them), in flight while the accumulators go through LDS
    // (raw values only: nothing here waits for a load; the sums and products come after)
    float rmul[NP];
    f32x4 gv[NP], prev[NP];
    int rows[NP];
    float2 rc[NP], rs[NP];  // RoPE: the lane's two rotation pairs' cos and sin for each row
    int64_t kvo[NP];        // RoPE: the row's offset in the K/V cache
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const int row = row_base + a * 32 + p * RP + rl;
      rows[p] = row < g.M ? row : g.M - 1;
      rmul[p] = 1.f;
      gv[p] = prev[p] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    if (col_full) {
      if (g.a_scale) {
#pragma unroll
        for (int p = 0; p < NP; ++p) rmul[p] = g.a_scale[rows[p]];
      }
      if constexpr (RESID) {
        if (g.gate_v) {
#pragma unroll
          for (int p = 0; p < NP; ++p)
            gv[p] = *reinterpret_cast<const f32x4*>(g.gate_v + gate_off(g, rows[p], inv_g) + col);
        }
#pragma unroll
        for (int p = 0; p < NP; ++p)
          prev[p] = *reinterpret_cast<const f32x4*>(static_cast<const float*>(g.out) +
                                                    group_off(rows[p], g.o_rows, inv_o, g.o_bs, g.ldo) + col);
      }
      if constexpr (E == WAM_EPI_ROPE) {
        const float inv_l = 1.0f / (float)g.rope_L;
        const int pair0 = ((col % g.rope_d) % g.rope_Dh) >> 1;
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const int64_t l = group_off(rows[p], g.rope_L, inv_l, 0, 1);
          rc[p] = *reinterpret_cast<const float2*>(g.rope_cos + l * (g.rope_Dh >> 1) + pair0);
          rs[p] = *reinterpret_cast<const float2*>(g.rope_sin + l * (g.rope_Dh >> 1) + pair0);
          kvo[p] = group_off(rows[p], g.rope_L, inv_l, g.rope_Lcap * g.rope_d, g.rope_d) + g.rope_row0 * g.rope_d;
        }
      }
    }
#pragma unroll
    for (int b = 0; b < C::TN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stage[(8 * (r >> 2) + 4 * hh + (r & 3)) * SROW + b * 32 + l32] = acc[a][b][r];
    __syncthreads();
    if (col_full) {
      // One store per pass, all of them after the loads above.  In a slab whose 32 rows
      // are all inside M (every slab but those of the last row tile) the stores are
      // unconditional: with no branch between them each store waits only for its own
      // operands, not for the completion of every earlier store.
      auto store = [&](int p) {
        const int rloc = p * RP + rl;
        f32x4 v = *reinterpret_cast<const f32x4*>(&stage[rloc * SROW + cl]);
        const int64_t orow = group_off(rows[p], g.o_rows, inv_o, g.o_bs, g.ldo);
        v = v * rmul[p] * cmul + cadd;
        if constexpr (E == WAM_EPI_BF16 || E == WAM_EPI_GELU_BF16) {
          bf16x4 o;
#pragma unroll
          for (int j = 0; j < 4; ++j) o[j] = (bf16)(E == WAM_EPI_GELU_BF16 ? gelu_tanh_f(v[j]) : v[j]);
          *reinterpret_cast<bf16x4*>(static_cast<bf16*>(g.out) + orow + col) = o;
        } else if constexpr (E == WAM_EPI_GELU_MX8) {
          // the bf16 GELU values as E4M3 codes of the row's 64-column block, whose 64
          // values are the 4 of each of the CG = 16 lanes that share this row
          float y[4], amax = 0.f;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            y[j] = (float)(bf16)gelu_tanh_f(v[j]);
            amax = fmaxf(amax, fabsf(y[j]));
          }
          static_assert(CG == 16, "one row's columns are a DPP row of 16 lanes");
          amax = row16_max(amax);
          const int eb = mx_exp_biased(amax);
          const float mul = ldexpf(1.0f, 127 - eb);  // |y| * mul <= 448 by the exponent's choice
          int code = __builtin_amdgcn_cvt_pk_fp8_f32(y[0] * mul, y[1] * mul, 0, false);
          code = __builtin_amdgcn_cvt_pk_fp8_f32(y[2] * mul, y[3] * mul, code, true);
          *reinterpret_cast<int*>(static_cast<uint8_t*>(g.out) + orow + col) = code;
          if (cl == 0) {
            const int blk = col_base >> 6;
            g.out_exp[(int64_t)(blk >> 1) * g.o_lde + 4 * rows[p] + (blk & 1)] = (uint8_t)eb;
          }
        } else if constexpr (E == WAM_EPI_ROPE) {
          // rounded to bf16 as the projection's output, then rotated in fp32 (q and k)
          float y[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) y[j] = (float)(bf16)v[j];
          const int sec = col / g.rope_d, c = col - sec * g.rope_d;  // 0 q, 1 k, 2 v (per lane)
          bf16x4 o;
          if (sec < 2) {
            o[0] = (bf16)__builtin_fmaf(y[0], rc[p].x, -(y[1] * rs[p].x));
            o[1] = (bf16)__builtin_fmaf(y[0], rs[p].x, y[1] * rc[p].x);
            o[2] = (bf16)__builtin_fmaf(y[2], rc[p].y, -(y[3] * rs[p].y));
            o[3] = (bf16)__builtin_fmaf(y[2], rs[p].y, y[3] * rc[p].y);
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) o[j] = (bf16)y[j];
          }
          bf16* dst = sec == 0 ? static_cast<bf16*>(g.rope_q) + (int64_t)rows[p] * g.rope_d
                               : static_cast<bf16*>(sec == 1 ? g.rope_k : g.rope_v) + kvo[p];
          *reinterpret_cast<bf16x4*>(dst + c) = o;
        } else if constexpr (RESID) {
          *reinterpret_cast<f32x4*>(static_cast<float*>(g.out) + orow + col) = prev[p] + (cgate + gv[p]) * v;
        } else {
          *reinterpret_cast<f32x4*>(static_cast<float*>(g.out) + orow + col) = v;
        }
      };
      if (row_base + a * 32 + 32 <= g.M) {
#pragma unroll
        for (int p = 0; p < NP; ++p) store(p);
      } else {
#pragma unroll
        for (int p = 0; p < NP; ++p)
          if (row_base + a * 32 + p * RP + rl < g.M) store(p);
      }
    } else if (col < g.N) {  // the matrix's last, partial column group (rare)
#pragma unroll 1
      for (int p = 0; p < NP; ++p) {
        const int rloc = p * RP + rl, row = row_base + a * 32 + rloc;
        const f32x4 v = *reinterpret_cast<const f32x4*>(&stage[rloc * SROW + cl]);
        if (row < g.M) epilogue_ragged<E>(g, inv_o, inv_g, row, col, v);
      }
    }
    __syncthreads();
  }
}

// Tile order within an XCD's contiguous range: ids walk 8 row tiles of one column tile,
// then the same 8 row tiles of the next column tile, so the ~32 tiles an XCD runs at
// once form an 8 x 4 block that shares 8 A panels and 4 W panels in its L2 (instead of
// ~25 A panels and 2 W panels when all row tiles of a column come first; measured
// 0-2.5% faster on the step's projections, interleaved launches).
WAM_DEV void grouped_tile(int slot, int tiles_m, int tiles_n, int& tm, int& tn) {
  constexpr int GM = 8;
  const int lid = xcd_tile(slot, tiles_m * tiles_n);
  const int per = GM * tiles_n, grp = lid / per, first = grp * GM;
  const int gm = tiles_m - first < GM ? tiles_m - first : GM;
  const int r = lid - grp * per;
  tm = first + r % gm;
  tn = r / gm;
}

// The workgroups are persistent: one per resident slot, each taking every gridDim.x-th
// dispatch slot in turn, so a tile's first slices are fetched while the previous tile's
// output stores drain, without a workgroup launch in between.
template <typename C, int EPI>
__global__ __launch_bounds__(C::NT, C::OCC) void gemm_nt(const GemmArgs g, int tiles_m, int tiles_n) {
  if (skip_step(g.skip)) return;
  const int total = tiles_m * tiles_n;
  constexpr int GM = 8;
  for (int slot = blockIdx.x; slot < total; slot += gridDim.x) {
    const int lid = xcd_tile(slot, total);
    const int per = GM * tiles_n, grp = lid / per, first = grp * GM;
    const int gm = tiles_m - first < GM ? tiles_m - first : GM;
    const int r = lid - grp * per;
    gemm_tile<C, EPI>(g, first + r % gm, r / gm, 0);
  }
}

// Two column ranges of one product in one persistent launch: columns [0, tn1 * BN) in
// C1 tiles, the rest in the shorter C2 tiles, dispatch slots of the first range before
// the second's.  A single tile height can leave the last round of tiles partly filled
// (at M = 3152, N = 13824: 702 tiles of 256 rows are 2.74 rounds on 256 CUs, so a third
// of the workgroups idle through the last one); filling it with the cheaper rounds of
// shorter tiles balances the workgroups with no split of the K sum.
template <typename C1, typename C2, int EPI>
__global__ __launch_bounds__(C1::NT, C1::OCC) void gemm_nt2(const GemmArgs g, int tm1, int tn1, int tm2, int tn2) {
  static_assert(C1::NT == C2::NT && C1::OCC == C2::OCC && C1::BN == C2::BN && C1::EB == C2::EB,
                "one workgroup shape for both ranges");
  if (skip_step(g.skip)) return;
  constexpr int L1 = C1::STAGES * C1::STAGE, L2 = C2::STAGES * C2::STAGE, LB = L1 > L2 ? L1 : L2;
  const int t1 = tm1 * tn1, total = t1 + tm2 * tn2;
  for (int slot = blockIdx.x; slot < total; slot += gridDim.x) {
    int tm, tn;
    if (slot < t1) {
      grouped_tile(slot, tm1, tn1, tm, tn);
      gemm_tile<C1, EPI, LB>(g, tm, tn, 0);
    } else {
      // slot - t1 keeps a workgroup's slots on one residue mod 8, i.e. on one XCD range
      grouped_tile(slot - t1, tm2, tn2, tm, tn);
      gemm_tile<C2, EPI, LB>(g, tm, tn, tn1 * C1::BN);
    }
  }
}

// gg.n products of the same shape and A, each with its own W, bias and output: one
// launch whose tiles run group after group (within a group as in gemm_nt).
template <typename C, int EPI>
__global__ __launch_bounds__(C::NT, C::OCC) void gemm_nt_group(const GemmArgs g, int tiles_m, int tiles_n,
                                                               const GemmGroup gg) {
  if (skip_step(g.skip)) return;
  const int per_group = tiles_m * tiles_n, total = per_group * gg.n;
  for (int slot = blockIdx.x; slot < total; slot += gridDim.x) {
    const int lid = xcd_tile(slot, total);
    const int grp = lid / per_group, r = lid - grp * per_group;
    GemmArgs gl = g;
    gl.W = gg.W[grp];
    gl.bias = gg.bias[grp];
    gl.out = gg.out[grp];
    if constexpr (C::EB == 1) gl.w_scale = gg.w_scale[grp];
    gemm_tile<C, EPI>(gl, r % tiles_m, r / tiles_m, 0);
  }
}

// Persistent workgroups: as many as are resident at once (by LDS and by wavefronts per
// SIMD), a multiple of 8 so each keeps its XCD, never more than there are tiles.
template <typename Cf>
int persistent_grid(long tiles) {
  constexpr int LDS = 160 * 1024, by_lds = LDS / (Cf::STAGES * Cf::STAGE);
  constexpr int by_waves = Cf::OCC * 4 / Cf::NW;
  constexpr int per_cu = (by_lds < by_waves ? by_lds : by_waves) > 0 ? (by_lds < by_waves ? by_lds : by_waves) : 1;
  long n = (long)cu_count() * per_cu;
  if (n >= 8) n &= ~7L;
  return (int)(tiles < n ? tiles : n);
}

template <typename Cf>
hipError_t launch_cfg(const GemmArgs& g, const GemmGroup* gg, hipStream_t s) {
  const int tm = (g.M + Cf::BM - 1) / Cf::BM, tn = (g.N + Cf::BN - 1) / Cf::BN;
  dim3 block(Cf::NT);
  if (gg) {  // grouped: the bf16 epilogue only
    if (g.epi != WAM_EPI_BF16) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_nt_group<Cf, WAM_EPI_BF16>), dim3(persistent_grid<Cf>((long)tm * tn * gg->n)), block, 0,
                       s, g, tm, tn, *gg);
    return hipGetLastError();
  }
  dim3 grid(persistent_grid<Cf>((long)tm * tn));
  if constexpr (Cf::EB == 1) {  // the block-scaled FP8 variants
    constexpr int MXB = WAM_EPI_MXA | WAM_EPI_BF16, MXR = WAM_EPI_MXA | WAM_EPI_RESID_F32;
    switch (g.epi) {
      case WAM_EPI_GELU_MX8: hipLaunchKernelGGL((gemm_nt<Cf, WAM_EPI_GELU_MX8>), grid, block, 0, s, g, tm, tn); break;
      case MXB: hipLaunchKernelGGL((gemm_nt<Cf, MXB>), grid, block, 0, s, g, tm, tn); break;
      case MXR: hipLaunchKernelGGL((gemm_nt<Cf, MXR>), grid, block, 0, s, g, tm, tn); break;
      default: break;
    }
    if (g.epi == WAM_EPI_GELU_MX8 || g.epi == MXB || g.epi == MXR) return hipGetLastError();
  }
  if (g.epi == WAM_EPI_ROPE) {  // bf16 operands only
    if constexpr (Cf::EB == 2) hipLaunchKernelGGL((gemm_nt<Cf, WAM_EPI_ROPE>), grid, block, 0, s, g, tm, tn);
    else return hipErrorInvalidValue;
    return hipGetLastError();
  }
  switch (g.epi) {
    case WAM_EPI_BF16: hipLaunchKernelGGL((gemm_nt<Cf, WAM_EPI_BF16>), grid, block, 0, s, g, tm, tn); break;
    case WAM_EPI_GELU_BF16: hipLaunchKernelGGL((gemm_nt<Cf, WAM_EPI_GELU_BF16>), grid, block, 0, s, g, tm, tn); break;
    case WAM_EPI_RESID_F32: hipLaunchKernelGGL((gemm_nt<Cf, WAM_EPI_RESID_F32>), grid, block, 0, s, g, tm, tn); break;
    default: hipLaunchKernelGGL((gemm_nt<Cf, WAM_EPI_F32>), grid, block, 0, s, g, tm, tn); break;
  }
  return hipGetLastError();
}

// Columns [0, c1 * 256) in Ca tiles, the rest in Cb tiles (both 256 wide).
template <typename Ca, typename Cb>
hipError_t launch_cfg2(const GemmArgs& g, int c1, hipStream_t s) {
  const int tm1 = (g.M + Ca::BM - 1) / Ca::BM, tm2 = (g.M + Cb::BM - 1) / Cb::BM;
  const int tn2 = (g.N - c1 * Ca::BN + Cb::BN - 1) / Cb::BN;
  const long t = (long)tm1 * c1 + (long)tm2 * tn2;
  const int ga = persistent_grid<Ca>(t), gb = persistent_grid<Cb>(t);
  dim3 grid(ga < gb ? ga : gb), block(Ca::NT);
  if constexpr (Ca::EB == 1) {  // the block-scaled FP8 variants
    constexpr int MXB = WAM_EPI_MXA | WAM_EPI_BF16, MXR = WAM_EPI_MXA | WAM_EPI_RESID_F32;
    switch (g.epi) {
      case WAM_EPI_GELU_MX8:
        hipLaunchKernelGGL((gemm_nt2<Ca, Cb, WAM_EPI_GELU_MX8>), grid, block, 0, s, g, tm1, c1, tm2, tn2);
        break;
      case MXB: hipLaunchKernelGGL((gemm_nt2<Ca, Cb, MXB>), grid, block, 0, s, g, tm1, c1, tm2, tn2); break;
      case MXR: hipLaunchKernelGGL((gemm_nt2<Ca, Cb, MXR>), grid, block, 0, s, g, tm1, c1, tm2, tn2); break;
      default: break;
    }
    if (g.epi == WAM_EPI_GELU_MX8 || g.epi == MXB || g.epi == MXR) return hipGetLastError();
  }
  if (g.epi == WAM_EPI_ROPE) {  // bf16 operands only
    if constexpr (Ca::EB == 2)
      hipLaunchKernelGGL((gemm_nt2<Ca, Cb, WAM_EPI_ROPE>), grid, block, 0, s, g, tm1, c1, tm2, tn2);
    else return hipErrorInvalidValue;
    return hipGetLastError();
  }
  switch (g.epi) {
    case WAM_EPI_BF16: hipLaunchKernelGGL((gemm_nt2<Ca, Cb, WAM_EPI_BF16>), grid, block, 0, s, g, tm1, c1, tm2, tn2); break;
    case WAM_EPI_GELU_BF16:
      hipLaunchKernelGGL((gemm_nt2<Ca, Cb, WAM_EPI_GELU_BF16>), grid, block, 0, s, g, tm1, c1, tm2, tn2);
      break;
    case WAM_EPI_RESID_F32:
      hipLaunchKernelGGL((gemm_nt2<Ca, Cb, WAM_EPI_RESID_F32>), grid, block, 0, s, g, tm1, c1, tm2, tn2);
      break;
    default: hipLaunchKernelGGL((gemm_nt2<Ca, Cb, WAM_EPI_F32>), grid, block, 0, s, g, tm1, c1, tm2, tn2); break;
  }
  return hipGetLastError();
}

}  // namespace

// Compute units of the current device (queried once per device).
int cu_count() {
  static int cus[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    cus[dev] = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0 ? n : 256;
  }
  return cus[dev];
}

namespace {
hipError_t launch_any(const GemmArgs& gin, const GemmGroup* gg, hipStream_t s) {
  GemmArgs g = gin;
  if (g.a_rows <= 0) { g.a_rows = g.M; g.a_bs = 0; }
  if (g.o_rows <= 0) { g.o_rows = g.M; g.o_bs = 0; }
  if (g.gate_rows <= 0) { g.gate_rows = g.M; g.gate_stride = 0; }
  // 128x256 tiles (8 wavefronts, 3-stage ring, one workgroup per CU) on every shape that
  // fills the chip; below one round of them (e.g. the 512-row text projections) 128x128
  // tiles, two workgroups per CU, spread the work wider.
  const long cus = cu_count();
  const long ng = gg ? gg->n : 1;
  const long tiles = ng * ((g.M + 127) / 128) * ((g.N + 255) / 256);
  if (tiles < cus) {
    if (g.fp8) return launch_cfg<Cfg<128, 128, 128, 2, 2, 2, 2, 1>>(g, gg, s);
    return launch_cfg<Cfg<128, 128, 64, 2, 2, 2, 2>>(g, gg, s);
  }
  // Cost of a round of tiles (one per CU), from launches at K = 5120 whose weights are not
  // in the last-level cache (as in a model step, where every block brings its own):
  // 128x256 tiles (8 wavefronts of 64x64, 3-stage ring) ~72 us, 192x256 (8 of 96x64, 2
  // stages) ~110 us, 256x256 (8 of 128x64, 2 stages) ~124 us.  With warm weights the
  // 192-row tiles cost ~10% less, which once made them look best for QKV; with cold ones
  // a tile that holds only one slice in flight waits on HBM more often, and the 3-stage
  // ring and the taller tiles (fewer re-reads per flop) lose less.  One workgroup per CU
  // for all three, so a workgroup that runs n tiles of one height costs n times its
  // figure, and the launch costs what its busiest workgroup does: take the least of that
  // over the three heights and over the splits of the columns into a taller range and a
  // shorter one (gemm_nt2, whose first workgroup is always among the busiest: slots are
  // dealt in order and the taller range comes first).  At M = 3152: QKV (60 column
  // tiles) 19 columns of 256-row tiles and 41 of 128-row ones (124 + 4 x 72 = 412 against
  // 440 for 192 rows alone: 416 against 441 us measured, cold); FFN1 (54 column tiles) 39
  // columns of 256-row tiles and 15 of 192-row ones (2 x 124 + 110 = 358 against 372 for
  // 256 rows alone: 369 against 383 us); O, cross-Q, cross-O and FFN2 (20 column tiles)
  // 128-row tiles (500 in 2 rounds).  FP8 takes the same tiles with 128-wide slices (the
  // bytes of a 64-wide bf16 slice).
  constexpr int NH = 3;
  const int height[NH] = {128, 192, 256}, cost[NH] = {72, 110, 124};
  const long ncol = (g.N + 255) / 256;
  auto tiles_m = [&](int h) { return (g.M + h - 1) / h; };
  auto ceil_div = [](long a, long b) { return (a + b - 1) / b; };
  long one[NH];  // one height for all columns
  for (int a = 0; a < NH; ++a) one[a] = cost[a] * ceil_div(ng * tiles_m(height[a]) * ncol, cus);
  int best_a = one[2] < one[0] && one[2] <= one[1] ? 2 : one[1] < one[0] ? 1 : 0, best_b = -1, best_c1 = 0;
  long best = one[best_a];
  if (!gg) {  // a split must beat one height by 3%; among equal splits, the least total work
    long best2 = 0, work2 = 0;
    for (int a = 1; a < NH; ++a)
      for (int b = 0; b < a; ++b)
        for (long c1 = 1; c1 < ncol; ++c1) {
          const long t1 = tiles_m(height[a]) * c1, t2 = tiles_m(height[b]) * (ncol - c1);
          const long n1 = ceil_div(t1, cus), n2 = ceil_div(t1 + t2, cus) - n1;
          const long c = cost[a] * n1 + cost[b] * n2, work = cost[a] * t1 + cost[b] * t2;
          if (100 * c < 97 * best && (best_b < 0 || c < best2 || (c == best2 && work < work2))) {
            best2 = c; work2 = work; best_a = a; best_b = b; best_c1 = (int)c1;
          }
        }
  }
  if (best_b >= 0) {
    if (g.fp8) {
      if (best_a == 2 && best_b == 1) return launch_cfg2<Cfg<256, 256, 128, 2, 2, 4, 2, 1>, Cfg<192, 256, 128, 2, 2, 4, 2, 1>>(g, best_c1, s);
      if (best_a == 2) return launch_cfg2<Cfg<256, 256, 128, 2, 2, 4, 2, 1>, Cfg<128, 256, 128, 3, 2, 4, 2, 1>>(g, best_c1, s);
      return launch_cfg2<Cfg<192, 256, 128, 2, 2, 4, 2, 1>, Cfg<128, 256, 128, 3, 2, 4, 2, 1>>(g, best_c1, s);
    }
    if (best_a == 2 && best_b == 1) return launch_cfg2<Cfg<256, 256, 64, 2, 2, 4, 2>, Cfg<192, 256, 64, 2, 2, 4, 2>>(g, best_c1, s);
    if (best_a == 2) return launch_cfg2<Cfg<256, 256, 64, 2, 2, 4, 2>, Cfg<128, 256, 64, 3, 2, 4, 2>>(g, best_c1, s);
    return launch_cfg2<Cfg<192, 256, 64, 2, 2, 4, 2>, Cfg<128, 256, 64, 3, 2, 4, 2>>(g, best_c1, s);
  }
  if (best_a == 2) {
    if (g.fp8) return launch_cfg<Cfg<256, 256, 128, 2, 2, 4, 2, 1>>(g, gg, s);
    return launch_cfg<Cfg<256, 256, 64, 2, 2, 4, 2>>(g, gg, s);
  }
  if (best_a == 1) {
    if (g.fp8) return launch_cfg<Cfg<192, 256, 128, 2, 2, 4, 2, 1>>(g, gg, s);
    return launch_cfg<Cfg<192, 256, 64, 2, 2, 4, 2>>(g, gg, s);
  }
  if (g.fp8) return launch_cfg<Cfg<128, 256, 128, 3, 2, 4, 2, 1>>(g, gg, s);
  return launch_cfg<Cfg<128, 256, 64, 3, 2, 4, 2>>(g, gg, s);
}
}  // namespace

hipError_t launch_gemm(const GemmArgs& g, hipStream_t s) { return launch_any(g, nullptr, s); }

hipError_t launch_gemm_group(const GemmArgs& g, const GemmGroup& gg, hipStream_t s) {
  if (gg.n < 1 || gg.n > WAM_GEMM_GROUP_MAX || g.epi != WAM_EPI_BF16) return hipErrorInvalidValue;
  return launch_any(g, &gg, s);
}

}  // namespace wam
