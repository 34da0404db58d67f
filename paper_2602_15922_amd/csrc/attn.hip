// Flash-style block-causal attention for gfx950 (bf16 MFMA, fp32 online softmax).
//
// A query of chunk c sees the key prefix [0, kend(c)): every cached, clean earlier
// chunk and its own chunk (section 3.1; Appendix C, Figure 10b).  Key tiles past the
// largest prefix of a query tile are never visited; only tiles that straddle a
// query row's prefix end are masked.
//
// Work split: a workgroup of 4 wavefronts owns 128 query rows of one (batch, head),
// 32 rows per wavefront, so a wavefront's whole state (Q fragments, score tile,
// probabilities and the fp32 output accumulators) stays in ordinary VGPRs and two
// wavefronts share each SIMD: one's softmax overlaps the other's MFMAs.  Key tiles of
// 64 keys are double-buffered in LDS and fetched with buffer loads straight into LDS
// (no staging registers; a scalar resource descriptor, a loop-invariant 32-bit lane
// offset and a scalar per-tile offset, so the fetch costs no vector ALU work): the next
// tile is in flight while the current one is consumed, with one barrier per tile.  The
// main loop handles two tiles per iteration, one per LDS buffer, so every LDS operand
// address is a lane base plus an immediate.  The score
// tile is computed transposed, S^T = K Q^T, so a lane owns one query and its softmax
// statistics stay in the lane (plus the partner lane l^32 holding the other half of
// the keys); the output is accumulated transposed as well, O^T = V^T P^T, so the
// rescale is lane-local too.  V stays row-major in LDS and its transposed MFMA
// operand is read with the gfx950 transposing LDS load (ds_read_b64_tr_b16, issued as
// asm two MFMAs ahead so it waits on nothing but its own LDS reads).  The
// reference maximum is only raised when a tile exceeds it by more than 2^8 in the
// exp2 domain, which leaves the result exact (o = acc / l for any reference) and skips
// almost every accumulator rescale.  Both tiles are XOR-swizzled in 16-byte chunks so
// the operand reads are bank-conflict free (kswz/vswz below), applied on the load side
// by choosing each lane's source chunk.
#include "common.h"
#include "kernels.h"

namespace wam {
namespace {

constexpr int BM = 128;  // query rows per workgroup
constexpr int BN = 64;   // keys per tile
constexpr int NT = 256;  // threads per workgroup
constexpr float RESCALE_LOG2 = 8.0f;  // allowed growth of exp2 arguments before a rescale

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

// The value held by lane l ^ 32 (the lane with the same query and the other half of the
// keys): one v_permlane32_swap, which exchanges the upper half of its first operand with
// the lower half of its second, instead of a round trip through LDS (ds_bpermute).
WAM_DEV float other_half(float v) {
  const unsigned u = __float_as_uint(v);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}

WAM_DEV int kend_of(const AttnArgs& a, int row) {
  int e = a.kend[a.n_q_chunks - 1];
  for (int i = a.n_q_chunks - 1; i >= 0; --i)
    if (row < a.q_off[i + 1]) e = a.kend[i];
  return e;
}

// One K tile and one V tile (BN keys from key kb) into LDS with direct global->LDS
// loads: 16 bytes per lane, lane l of a wave instruction landing at LDS unit base + l.
// Rows past Lk are clamped to the last key (their scores are masked, so their values
// never count).  koff/voff are the lanes' loop-invariant source offsets.
// LDS swizzles (XOR of the 16-byte chunk index).  gfx950 LDS serves 256 bytes (64
// banks) per cycle: 16 lanes of a 16-byte read, 32 lanes of an 8-byte read.
//  K: the fragment read has 16 lanes on 16 consecutive rows at one logical chunk;
//     with 256-byte rows (Dh=128) XOR by row&15, with 128-byte rows by (row>>1)&7.
//  V: a transposing read covers 4 consecutive rows x 64 bytes per 32 lanes, so the
//     4 rows' 64-byte groups must fall in different quarters of the 256-byte line:
//     XOR by 4*(row&3) (Dh=128) or 4*((row>>1)&1) (Dh=64, two rows per line).
template <int DH>
WAM_DEV int kswz(int row, int ch) { return DH == 128 ? (ch ^ (row & 15)) : (ch ^ ((row >> 1) & 7)); }
template <int DH>
WAM_DEV int vswz(int row, int ch) { return DH == 128 ? (ch ^ (4 * (row & 3))) : (ch ^ (4 * ((row >> 1) & 1))); }

template <int DH>
WAM_DEV void fetch_tile(bf16* Ks, __amdgpu_buffer_rsrc_t kr, __amdgpu_buffer_rsrc_t vr, int kv_tsb, int Lk,
                        int kb, int w, const int* koff, const int* voff, const int* krow) {
  constexpr int KCH = BN * (DH / 8) / NT;
  bf16* Vs = Ks + BN * DH;
  const int soff = kb * kv_tsb;  // wave-uniform byte offset of the tile's first key row
  if (kb + BN <= Lk) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int base = (w * KCH + i) * 64;  // wave-uniform first unit of this instruction
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (lds_void*)(Ks + base * 8), 16, koff[i], soff, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_void*)(Vs + base * 8), 16, voff[i], soff, 0, 0);
    }
  } else {
    // ragged last tile: rows past Lk re-read the last key row (their scores are masked)
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int base = (w * KCH + i) * 64;
      const int over = kb + krow[i] - (Lk - 1);
      const int shift = over > 0 ? -over * kv_tsb : 0;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (lds_void*)(Ks + base * 8), 16, koff[i] + shift, soff, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_void*)(Vs + base * 8), 16, voff[i] + shift, soff, 0, 0);
    }
  }
}

// V^T fragments through inline asm.  The compiler cannot prove that these LDS reads miss
// the direct-to-LDS prefetch of the next tile still in flight, so before its own form of
// the transposing read it waits for all outstanding vector memory, i.e. for the next
// tile's loads, every tile.  Issued as asm, the reads wait only on the LDS counter, which
// the code below sets itself: the reads of P.V MFMA i+2 are issued before MFMA i, which
// then waits until at most the 4 younger reads are outstanding (LDS reads complete in
// order).  The asm results are tied through the wait so nothing reads them earlier.
template <int OFF>
WAM_DEV s16x4 tr16(unsigned addr) {
  s16x4 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}
WAM_DEV unsigned lds_addr(const void* p) {
  return (unsigned)(uintptr_t)(const __attribute__((address_space(3))) char*)(p);
}
template <int N>
WAM_DEV void wait_lgkm(s16x4& a, s16x4& b) {
  asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(a), "+v"(b) : "i"(N));
}

// the two reads of P.V MFMA i = (mt, nt, hf): keys 32 nt + 16 hf + (0..7, 8..15) of dims
// 32 mt + (lane's 4), from the lane's base address of output tile mt
template <int DH, int I>
WAM_DEV void vread(const unsigned* va, s16x4* lo, s16x4* hi) {
  constexpr int ROWB = DH * 2, mt = I >> 2, nt = (I >> 1) & 1, hf = I & 1, off = (32 * nt + 16 * hf) * ROWB;
  lo[I % 3] = tr16<off>(va[mt]);
  hi[I % 3] = tr16<off + 8 * ROWB>(va[mt]);
}

template <int DH, int I>
WAM_DEV void pv_steps(const unsigned* va, s16x4* lo, s16x4* hi, const bf16x8 (*pb)[2], f32x16* acc) {
  constexpr int NMF = DH / 8, mt = I >> 2, nt = (I >> 1) & 1, hf = I & 1;  // NMF = 4 MT MFMAs
  if constexpr (I + 2 < NMF) {
    vread<DH, I + 2>(va, lo, hi);
    wait_lgkm<4>(lo[I % 3], hi[I % 3]);
  } else if constexpr (I + 1 < NMF) {
    wait_lgkm<2>(lo[I % 3], hi[I % 3]);
  } else {
    wait_lgkm<0>(lo[I % 3], hi[I % 3]);
  }
  const s16x4 v8[2] = {lo[I % 3], hi[I % 3]};
  acc[mt] = mfma32(*reinterpret_cast<const bf16x8*>(v8), pb[nt][hf], acc[mt]);
  if constexpr (I + 1 < NMF) pv_steps<DH, I + 1>(va, lo, hi, pb, acc);
}

// K fragments of the score MFMAs, likewise as asm: the compiler's schedule issued each
// read one MFMA ahead of its use, exposing the LDS latency once the tile's other stall was
// gone; here the read of score MFMA i+3 is issued before MFMA i (measured best of 2, 3, 5
// and 7 ahead).  Score MFMA i = (ks = i/2, nt = i%2) alternates the two accumulators.
constexpr int KAHEAD = 3;
template <int OFF>
WAM_DEV bf16x8 kread(unsigned addr) {
  bf16x8 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}
template <int N>
WAM_DEV void wait_k(bf16x8& a) {
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(a) : "i"(N));
}
template <int DH, int I>
WAM_DEV void kload(const unsigned* ka, bf16x8* kf) {
  constexpr int ks = I >> 1, nt = I & 1;
  kf[I % (KAHEAD + 1)] = kread<nt * 32 * DH * 2>(ka[ks]);
}
template <int DH, int I>
WAM_DEV void score_steps(const unsigned* ka, bf16x8* kf, const bf16x8* qf, f32x16* s) {
  constexpr int NS = DH / 8, ks = I >> 1, nt = I & 1;  // NS = 2 KS score MFMAs
  if constexpr (I + KAHEAD < NS) {
    kload<DH, I + KAHEAD>(ka, kf);
    wait_k<KAHEAD>(kf[I % (KAHEAD + 1)]);
  } else {
    wait_k<NS - 1 - I>(kf[I % (KAHEAD + 1)]);
  }
  s[nt] = mfma32(kf[I % (KAHEAD + 1)], qf[ks], s[nt]);
  if constexpr (I + 1 < NS) score_steps<DH, I + 1>(ka, kf, qf, s);
}
template <int DH, int I>
WAM_DEV void kloads(const unsigned* ka, bf16x8* kf) {
  kload<DH, I>(ka, kf);
  if constexpr (I + 1 < KAHEAD) kloads<DH, I + 1>(ka, kf);
}
// S^T = K Q^T for one tile (keys 0..31 into s[0], 32..63 into s[1])
template <int DH>
WAM_DEV void scores_tile(const char* Ks, const int* kofs, const bf16x8* qf, f32x16* s) {
  constexpr int KS = DH / 16;
  unsigned ka[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) ka[ks] = lds_addr(Ks + kofs[ks]);
  bf16x8 kf[KAHEAD + 1];
  kloads<DH, 0>(ka, kf);
  score_steps<DH, 0>(ka, kf, qf, s);
}

// O^T += V^T P^T for one tile: 4 MT MFMAs, each with its two transposing V reads
template <int DH>
WAM_DEV void pv_tile(const char* Vs, const int* vofs, const bf16x8 (*pb)[2], f32x16* acc) {
  constexpr int MT = DH / 32;
  unsigned va[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) va[mt] = lds_addr(Vs + vofs[mt]);
  s16x4 lo[3], hi[3];
  vread<DH, 0>(va, lo, hi);
  vread<DH, 1>(va, lo, hi);
  pv_steps<DH, 0>(va, lo, hi, pb, acc);
}

// One 64-key tile for one wavefront's 32 queries: S^T = K Q^T, optional prefix mask,
// online softmax with a lazily raised reference, O^T += V^T P^T.  Ks/Vs are the tile's
// LDS buffers; kofs[ks] is the lane's byte offset of its K fragment for k-step ks
// (keys 0..31; +32 rows for the second sub-tile), vofs[mt] the lane's byte offset of
// its transposing V read for output tile mt (row groups added as constants).
template <int DH, bool MASK>
WAM_DEV void attn_tile(const char* Ks, const char* Vs, const bf16x8* qf, f32x16* acc, float& m_ref,
                       float& l_part, const int* kofs, const int* vofs, float c, float thr, int kb,
                       int row_kend, int hh) {
  constexpr int MT = DH / 32;
  f32x16 s[2] = {f32x16{}, f32x16{}};
  // The wave raises its issue priority for the score MFMAs only: while it runs them, the
  // SIMD's other wave, in its softmax or P.V, fills the gaps of this chain instead of
  // delaying it, and the scores the softmax waits on come out sooner.  Measured with
  // launches interleaved, outputs bit for bit equal: 980 -> 934 us alone, 0.953 -> 0.918 ms
  // per launch inside the step.  Held through the softmax as well: 1.7% faster alone; two
  // levels (scores 2, P.V 1): 1.3% faster; raised for P.V only: 0.4% slower; for the
  // scores and P.V: 0.9% slower.
  __builtin_amdgcn_s_setprio(1);
  scores_tile<DH>(Ks, kofs, qf, s);
  __builtin_amdgcn_s_setprio(0);
  if (MASK) {
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kb + 32 * nt + 8 * (r >> 2) + 4 * hh + (r & 3);
        if (key >= row_kend) s[nt][r] = -INFINITY;
      }
  }
  float mx = s[0][0];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[nt][r]);
  mx = fmaxf(mx, other_half(mx));
  const bool raise = mx > m_ref + thr || (m_ref == -INFINITY && mx != -INFINITY);
  if (__any(raise)) {
    const float m_new = raise ? mx : m_ref;
    const float alpha = m_ref == -INFINITY ? 0.f : exp2_fast((m_ref - m_new) * c);
    m_ref = m_new;
    l_part *= alpha;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] *= alpha;
  }
  const float ms = m_ref == -INFINITY ? 0.f : m_ref * c;
  bf16x8 pb[2][2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
#pragma unroll
    for (int r = 0; r < 16; ++r) pb[nt][r >> 3][r & 7] = (bf16)exp2_fast(__builtin_fmaf(s[nt][r], c, -ms));
  // row sum of exactly the bf16 probabilities the PV product uses, two per dot2
  const bf16x2 ones = {(bf16)1.0f, (bf16)1.0f};
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16x2 pr = {pb[nt][hf][2 * e], pb[nt][hf][2 * e + 1]};
        l_part = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, l_part, false);
      }
  pv_tile<DH>(Vs, vofs, pb, acc);
}

// Wait for this wave's direct loads of the next tile, then sync the workgroup.
WAM_DEV void tile_sync() {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

// Key tile t from LDS buffer `cur` (a compile-time constant in the main loop), with tile
// t+1 fetched into the other buffer meanwhile.
template <int DH, bool MASK>
WAM_DEV void attn_step(bf16* smem, int cur, __amdgpu_buffer_rsrc_t kr, __amdgpu_buffer_rsrc_t vr, int kv_tsb,
                       int Lk, int t, int ntiles, int w, const int* koff, const int* voff, const int* krow,
                       const bf16x8* qf, f32x16* acc, float& m_ref, float& l_part, const int* kofs,
                       const int* vofs, float c, float thr, int row_kend, int hh) {
  constexpr int TILE = 2 * BN * DH;
  const int kb = t * BN;
  if (t + 1 < ntiles) fetch_tile<DH>(smem + (cur ^ 1) * TILE, kr, vr, kv_tsb, Lk, kb + BN, w, koff, voff, krow);
  const char* Ks = reinterpret_cast<const char*>(smem + cur * TILE);
  attn_tile<DH, MASK>(Ks, Ks + BN * DH * 2, qf, acc, m_ref, l_part, kofs, vofs, c, thr, kb, row_kend, hh);
  tile_sync();
}

// CHUNKED: the keys form more than one chunk (cached chunks plus the current one), so a
// query's visible prefix is looked up from its chunk; otherwise (cross-attention to the
// text, or a single chunk) every query sees all Lk keys and only the ragged last tile
// is masked.
// MX8: the output written block-scaled (store_attn_row_mx8; Dh = 128): E4M3 codes at a.o
// (strides in bytes), for output row m = b * Lq + query and head h the exponents of dims
// 0-63 and 64-127 at o_exp[h * o_lde + 4 m + {0, 1}].  (Kernel arguments rather than
// AttnArgs fields, so that the other instantiations keep their argument layout and code.)
template <int DH, bool CHUNKED, bool MX8 = false>
__global__ __launch_bounds__(NT, 2) void attn_fwd(const AttnArgs a, int nqt, uint8_t* o_exp, int64_t o_lde) {
  static_assert(!MX8 || DH == 128, "the block-scaled output is for Dh = 128");
  constexpr int KS = DH / 16;         // MFMA k-steps over the head dim
  constexpr int MT = DH / 32;         // 32-row tiles of the transposed output
  constexpr int CPR = DH / 8;         // 16-byte chunks per K/V row
  constexpr int KCH = BN * CPR / NT;  // 16-byte chunks of K (and of V) per thread
  constexpr int TILE = 2 * BN * DH;   // K tile + V tile, elements
  __shared__ __attribute__((aligned(16))) bf16 smem[2 * TILE];
  if (skip_step(a.skip)) return;

  // XCD-aware mapping: give each XCD a contiguous range of (q-tile, head) pairs so
  // the workgroups sharing a head's K/V share an L2.
  const int nblk = gridDim.x, bi = blockIdx.x, xcd = bi & 7, slot = bi >> 3;
  const int per = nblk >> 3, rem = nblk & 7;
  const int lid = xcd * per + (xcd < rem ? xcd : rem) + slot;
  const int qt = lid % nqt, hb = lid / nqt, h = hb % a.H, b = hb / a.H;
  const int q0 = qt * BM;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, in a scalar register
  const int hh = lane >> 5, l32 = lane & 31;

  const int qrow = q0 + 32 * w + l32;
  const int qrow_c = qrow < a.Lq ? qrow : a.Lq - 1;
  const int row_kend = CHUNKED ? kend_of(a, qrow_c) : a.Lk;
  bf16x8 qf[KS];
  {
    const bf16* qp = static_cast<const bf16*>(a.q) + b * a.q_bs + (int64_t)qrow_c * a.q_ts + h * DH + 8 * hh;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = load_bf16x8(qp + 16 * ks);
  }
  const int last = (q0 + BM < a.Lq ? q0 + BM : a.Lq) - 1;
  const int kend_max = CHUNKED ? kend_of(a, last) : a.Lk;
  const int kend_min = CHUNKED ? kend_of(a, q0) : a.Lk;

  // buffer resources over this (batch, head)'s keys: every offset the kernel forms is
  // below Lk * row bytes (< 2^31, checked by the host), so the range check never fires
  const bf16* kp = static_cast<const bf16*>(a.k) + b * a.kv_bs + h * DH;
  const bf16* vp = static_cast<const bf16*>(a.v) + b * a.kv_bs + h * DH;
  const int kv_tsb = 2 * (int)a.kv_ts;  // bytes per key row
  const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc((void*)kp, (short)0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc((void*)vp, (short)0, 0x7fffffff, 0x00020000);

  // ---- per-lane byte offsets of the tile fetch (loop-invariant)
  int koff[KCH], voff[KCH], krow[KCH];
#pragma unroll
  for (int i = 0; i < KCH; ++i) {
    const int u = (w * KCH + i) * 64 + lane, row = u / CPR, pch = u % CPR;
    krow[i] = row;
    koff[i] = row * kv_tsb + kswz<DH>(row, pch) * 16;
    voff[i] = row * kv_tsb + vswz<DH>(row, pch) * 16;
  }

  // ---- per-lane LDS operand offsets (bytes, loop-invariant)
  // K fragment of k-step ks: row l32, logical chunk 2*ks + hh (the swizzle of rows
  // l32 and l32 + 32 is the same).
  int kofs[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) kofs[ks] = l32 * DH * 2 + kswz<DH>(l32, 2 * ks + hh) * 16;
  // V^T: in each 16-lane group, lane j points at row (rb + j/4), dims (db + 4*(j%4)
  // .. +3); the transposing load then hands lane i the four keys rb..rb+3 of dim db+i.
  // Row group rb = 32*nt + 16*hf + 4*(grp>>1) (+8 for the second half), dims of output
  // tile mt at db = 32*mt + 16*(grp&1).  The swizzle only depends on the lane.
  const int grp = lane >> 4, j16 = lane & 15;
  int vofs[MT];
  {
    const int r0 = 4 * (grp >> 1) + (j16 >> 2);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int col = 32 * mt + 16 * (grp & 1) + 4 * (j16 & 3);
      vofs[mt] = r0 * DH * 2 + vswz<DH>(r0, col >> 3) * 16 + 8 * ((col >> 2) & 1);
    }
  }

  f32x16 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x16{};
  float m_ref = -INFINITY, l_part = 0.f;
  const float c = a.c, thr = RESCALE_LOG2 / c;

  const int ntiles = (kend_max + BN - 1) / BN;
  const int n_plain = kend_min / BN < ntiles ? kend_min / BN : ntiles;  // tiles no row masks
  fetch_tile<DH>(smem, kr, vr, kv_tsb, a.Lk, 0, w, koff, voff, krow);
  tile_sync();
  // unmasked tiles in pairs (tile t in buffer 0, t+1 in buffer 1)
  int t = 0;
  for (; t + 2 <= n_plain; t += 2) {
    attn_step<DH, false>(smem, 0, kr, vr, kv_tsb, a.Lk, t, ntiles, w, koff, voff, krow, qf, acc, m_ref, l_part,
                         kofs, vofs, c, thr, row_kend, hh);
    attn_step<DH, false>(smem, 1, kr, vr, kv_tsb, a.Lk, t + 1, ntiles, w, koff, voff, krow, qf, acc, m_ref,
                         l_part, kofs, vofs, c, thr, row_kend, hh);
  }
  // the rest (at most one unmasked tile, then the tiles that straddle a prefix end),
  // masked: the mask is a no-op on keys every row sees
  for (; t < ntiles; ++t)
    attn_step<DH, true>(smem, t & 1, kr, vr, kv_tsb, a.Lk, t, ntiles, w, koff, voff, krow, qf, acc, m_ref, l_part,
                        kofs, vofs, c, thr, row_kend, hh);

  const float l = l_part + other_half(l_part);
  if constexpr (MX8) {
    uint8_t* o8 = static_cast<uint8_t*>(a.o) + b * a.o_bs + (int64_t)qrow * a.o_ts + h * DH;
    uint8_t* oe = o_exp + h * o_lde + 4 * ((int64_t)b * a.Lq + qrow);
    store_attn_row_mx8(o8, oe, acc, 1.0f / l, hh, qrow < a.Lq);
  } else if (qrow < a.Lq) {
    const float inv = 1.0f / l;
    bf16* ob = static_cast<bf16*>(a.o) + b * a.o_bs + (int64_t)qrow * a.o_ts + h * DH;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        bf16x4 v4 = {(bf16)(acc[mt][4 * rr + 0] * inv), (bf16)(acc[mt][4 * rr + 1] * inv),
                     (bf16)(acc[mt][4 * rr + 2] * inv), (bf16)(acc[mt][4 * rr + 3] * inv)};
        *reinterpret_cast<bf16x4*>(ob + 32 * mt + 8 * rr + 4 * hh) = v4;
      }
  }
}

}  // namespace

hipError_t launch_attn(const AttnArgs& a, hipStream_t s, uint8_t* o_exp, int64_t o_lde) {
  const int nqt = (a.Lq + BM - 1) / BM;
  const dim3 grid((unsigned)((long)nqt * a.H * a.B)), block(NT);
  const bool chunked = a.n_k_chunks > 1;
  uint8_t* const z = nullptr;
  if (o_exp) {  // block-scaled output (Dh = 128, checked by the host)
    if (chunked) hipLaunchKernelGGL((attn_fwd<128, true, true>), grid, block, 0, s, a, nqt, o_exp, o_lde);
    else hipLaunchKernelGGL((attn_fwd<128, false, true>), grid, block, 0, s, a, nqt, o_exp, o_lde);
  } else if (a.Dh == 128) {
    if (chunked) hipLaunchKernelGGL((attn_fwd<128, true>), grid, block, 0, s, a, nqt, z, (int64_t)0);
    else hipLaunchKernelGGL((attn_fwd<128, false>), grid, block, 0, s, a, nqt, z, (int64_t)0);
  } else {
    if (chunked) hipLaunchKernelGGL((attn_fwd<64, true>), grid, block, 0, s, a, nqt, z, (int64_t)0);
    else hipLaunchKernelGGL((attn_fwd<64, false>), grid, block, 0, s, a, nqt, z, (int64_t)0);
  }
  return hipGetLastError();
}

}  // namespace wam
