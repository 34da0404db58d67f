// FP8 (E4M3) block-causal attention for gfx950: the softmax attention of attn.hip with
// q, k, v and the probabilities in FP8 (the paper runs QKV and the softmax in FP8 in its
// deployment, section 3.2.4 and Appendix D.2), on the 32x32x64 FP8 MFMA with block scales.
//
// Operands.  q and k carry one power-of-two scale per 32 dims of a head (an 8-bit biased
// exponent, four per (token, head) at Dh = 128, packed in one uint32); the MFMA applies
// them itself.  Its scale blocks interleave the lane halves: block 0 of a 64-wide k step
// is bytes 0-15 of lanes l and l+32 (scale from lane l), block 1 their bytes 16-31 (scale
// from lane l+32), checked on the GPU with an in-bounds probe.  So lane half hh holds dims
// [64 ks + 16 hh, +16) and [64 ks + 32 + 16 hh, +16), and supplies block 2 ks + hh's scale.
// v has one scale for the whole tensor, applied with 1/l at the end.  The probabilities
// are rounded to E4M3 as
// p = 2^(s c - m c + 6): the reference maximum m is raised whenever a tile exceeds it by
// 2^2, so p <= 2^8 stays inside E4M3's range and small probabilities keep 6 more binary
// orders of magnitude above E4M3's smallest subnormal.  The row sum l comes from one more
// MFMA of the rounded probabilities, so the normaliser adds exactly the values the output
// product used: a 16x16x128 one (half the cycles of the 32x32x64 shape) whose A operand is
// E4M3 1.0 in two rows only, chosen by lane so that row 0 sums the keys of queries 0-15 and
// row 4 those of queries 16-31 (below).
//
// Layout and schedule follow the bf16 kernel: 4 wavefronts x 32 queries of one (batch,
// head), S^T = K Q^T and O^T = V^T P^T so a lane owns one query, 64-key tiles of K codes,
// V codes and K exponents double-buffered in LDS and fetched with direct global->LDS
// loads.  V^T fragments come from the transposing LDS read ds_read_b64_tr_b8: in each
// 16-lane group, lane i receives byte i%8 of the 8-byte chunks addressed by lanes
// 2e + i/8 (e = 0..7), i.e. 8 keys of one dim, with the keys chosen by the addressing
// lanes; each lane's 32 keys are the keys its score registers hold.
#include "common.h"
#include "kernels.h"

namespace wam {
namespace {

constexpr int BM = 128;    // query rows per workgroup
constexpr int BN = 64;     // keys per tile
constexpr int NT = 256;    // threads per workgroup
constexpr int DH = 128;    // head dim (the only one this kernel takes)
constexpr int ROWB = DH;   // bytes per K/V code row
constexpr int KT = BN * ROWB;         // bytes of one K (or V) code tile
constexpr int STAGE = 2 * KT + BN * 4;  // K codes, V codes, K exponents
constexpr float RESCALE_LOG2 = 2.0f;  // allowed growth of exp2 arguments before a rescale
constexpr float P_SHIFT = 6.0f;       // probabilities are stored as p * 2^6 (<= 256)

typedef int v2i __attribute__((ext_vector_type(2)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v2i lds_v2i;
typedef __attribute__((address_space(3))) void lds_void;

WAM_DEV f32x16 mfma_f8(i32x8 a, i32x8 b, f32x16 c, int sa, int sb) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, sa, 0, sb);
}
WAM_DEV f32x4 mfma_f8_16(i32x8 a, i32x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 127, 0, 127);
}

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

// LDS swizzles of the 16-byte chunk index of a 128-byte code row (gfx950 LDS: 256 bytes
// per cycle).  K: a fragment read covers 16 consecutive rows at one logical chunk, i.e.
// two rows per 256-byte line, so XOR by (row >> 1) & 7.  V: a transposing read of 32
// lanes covers rows {0,1,2,3,8,9,10,11} (+4, +16k) x 32 bytes; XOR the 32-byte segment by
// ((row >> 1) & 1) | ((row >> 3) & 1) << 1 so those rows fall in distinct segments.
WAM_DEV int kswz(int row, int ch) { return ch ^ ((row >> 1) & 7); }
WAM_DEV int vswz(int row, int ch) { return ch ^ (2 * (((row >> 1) & 1) | (((row >> 3) & 1) << 1))); }

// One tile (K codes, V codes, K exponents of BN keys from key kb) into LDS.  Rows past Lk
// re-read the last key row (their scores are masked).
WAM_DEV void fetch_tile(char* st, __amdgpu_buffer_rsrc_t kr, __amdgpu_buffer_rsrc_t vr, __amdgpu_buffer_rsrc_t er,
                        int kv_tsb, int e_tsb, int Lk, int kb, int w, int lane, const int* koff, const int* voff,
                        const int* krow) {
  constexpr int KCH = BN * (ROWB / 16) / NT;
  char* Vs = st + KT;
  char* Es = st + 2 * KT;
  const int soff = kb * kv_tsb, esoff = kb * e_tsb;
  if (kb + BN <= Lk) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int base = (w * KCH + i) * 64;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (lds_void*)(st + base * 16), 16, koff[i], soff, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_void*)(Vs + base * 16), 16, voff[i], soff, 0, 0);
    }
    if (w == 0) __builtin_amdgcn_raw_ptr_buffer_load_lds(er, (lds_void*)Es, 4, lane * e_tsb, esoff, 0, 0);
  } else {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int base = (w * KCH + i) * 64;
      const int over = kb + krow[i] - (Lk - 1);
      const int shift = over > 0 ? -over * kv_tsb : 0;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (lds_void*)(st + base * 16), 16, koff[i] + shift, soff, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_void*)(Vs + base * 16), 16, voff[i] + shift, soff, 0, 0);
    }
    if (w == 0) {
      const int row = kb + lane < Lk ? lane : Lk - 1 - kb;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(er, (lds_void*)Es, 4, row * e_tsb, esoff, 0, 0);
    }
  }
}

WAM_DEV v4i lds16(const char* p) { return *reinterpret_cast<const v4i*>(p); }

// V^T fragments through inline asm, as in the bf16 kernel: in the compiler's form each
// tile's first transposing read waits for all outstanding vector memory, i.e. for the next
// tile's loads (the compiler cannot prove the direct-to-LDS prefetch misses them).  Issued
// as asm, the reads of P.V MFMA mt+1 go out before MFMA mt, which waits only until its own
// four reads are done (LDS reads complete in order); the results are tied through the wait.
template <int OFF>
WAM_DEV v2i tr8(unsigned addr) {
  v2i r;
  asm volatile("ds_read_b64_tr_b8 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}
template <int N>
WAM_DEV void wait_lgkm4(v2i& a, v2i& b, v2i& c, v2i& d) {
  asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d) : "i"(N));
}
WAM_DEV unsigned lds_addr(const void* p) {
  return (unsigned)(uintptr_t)(const __attribute__((address_space(3))) char*)(p);
}
// the four reads of P.V MFMA mt: keys 16 k + (the lane's 8) for k = 0..3
WAM_DEV void vreads(unsigned a, v2i* r) {
  r[0] = tr8<0>(a);
  r[1] = tr8<16 * ROWB>(a);
  r[2] = tr8<32 * ROWB>(a);
  r[3] = tr8<48 * ROWB>(a);
}

// One 64-key tile for one wavefront's 32 queries.
template <bool MASK>
WAM_DEV void attn_tile(const char* st, const i32x8* qf, const int* qsc, f32x16* acc, f32x4& accl, const i32x8& sel,
                       float& m_ref,
                       const int* kofs, const int* vofs, float c, float thr, int kb, int row_kend, int hh, int l32) {
  const char* Vs = st + KT;
  const char* Es = st + 2 * KT;
  f32x16 s[2] = {f32x16{}, f32x16{}};
  // The wave raises its issue priority for the score MFMAs only (as the bf16 kernel does):
  // 0.645 -> 0.635 ms per launch inside the FP8 step, against the priority raised for the
  // row sum and P.V as well (0.69 -> 0.67 ms against none).
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const unsigned kw = *reinterpret_cast<const unsigned*>(Es + (32 * nt + l32) * 4);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const v4i lo = lds16(st + kofs[2 * ks] + nt * 32 * ROWB);
      const v4i hi = lds16(st + kofs[2 * ks + 1] + nt * 32 * ROWB);
      const i32x8 kf = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      const int ksc = (int)((kw >> (8 * (2 * ks + hh))) & 0xffu);
      s[nt] = mfma_f8(kf, qf[ks], s[nt], ksc, qsc[ks]);
    }
  }
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
    accl *= alpha;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) acc[mt] *= alpha;
  }
  const float ms = m_ref == -INFINITY ? 0.f : m_ref * c - P_SHIFT;
  // probabilities as E4M3 codes, byte 16*nt + r of the operand = score register r of nt
  i32x8 pk;
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float p0 = exp2_fast(__builtin_fmaf(s[nt][4 * q + 0], c, -ms));
      const float p1 = exp2_fast(__builtin_fmaf(s[nt][4 * q + 1], c, -ms));
      const float p2 = exp2_fast(__builtin_fmaf(s[nt][4 * q + 2], c, -ms));
      const float p3 = exp2_fast(__builtin_fmaf(s[nt][4 * q + 3], c, -ms));
      int wd = __builtin_amdgcn_cvt_pk_fp8_f32(p0, p1, 0, false);
      wd = __builtin_amdgcn_cvt_pk_fp8_f32(p2, p3, wd, true);
      pk[4 * nt + q] = wd;
    }
  accl = mfma_f8_16(sel, pk, accl);
  unsigned va[4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) va[mt] = lds_addr(Vs + vofs[mt]);
  v2i r[2][4];
  vreads(va[0], r[0]);
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
    v2i* c = r[mt & 1];
    if (mt + 1 < 4) {
      vreads(va[mt + 1], r[(mt + 1) & 1]);
      wait_lgkm4<4>(c[0], c[1], c[2], c[3]);
    } else {
      wait_lgkm4<0>(c[0], c[1], c[2], c[3]);
    }
    const i32x8 vf = {c[0][0], c[0][1], c[1][0], c[1][1], c[2][0], c[2][1], c[3][0], c[3][1]};
    acc[mt] = mfma_f8(vf, pk, acc[mt], 127, 127);
  }
}

WAM_DEV void tile_sync() {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

// MX8: the output written block-scaled, laid out as attn_fwd's.
template <bool CHUNKED, bool MX8 = false>
__global__ __launch_bounds__(NT, 2) void attn_fwd_fp8(const AttnFp8Args f, int nqt, uint8_t* o_exp, int64_t o_lde) {
  constexpr int CPR = ROWB / 16;       // 16-byte chunks per code row
  constexpr int KCH = BN * CPR / NT;   // chunks of K (and of V) per thread
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE];
  const AttnArgs& a = f.a;
  if (skip_step(a.skip)) return;

  const int nblk = gridDim.x, bi = blockIdx.x, xcd = bi & 7, slot = bi >> 3;
  const int per = nblk >> 3, rem = nblk & 7;
  const int lid = xcd * per + (xcd < rem ? xcd : rem) + slot;
  const int qt = lid % nqt, hb = lid / nqt, h = hb % a.H, b = hb / a.H;
  const int q0 = qt * BM;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = lane >> 5, l32 = lane & 31;

  const int qrow = q0 + 32 * w + l32;
  const int qrow_c = qrow < a.Lq ? qrow : a.Lq - 1;
  const int row_kend = CHUNKED ? kend_of(a, qrow_c) : a.Lk;
  // Q^T operand: dims [64 ks + 16 hh, +16) and [64 ks + 32 + 16 hh, +16) of this lane's
  // query, and the scales of blocks 2 ks + hh
  i32x8 qf[2];
  int qsc[2];
  {
    const char* qp = static_cast<const char*>(a.q) + b * a.q_bs + (int64_t)qrow_c * a.q_ts + h * DH + 16 * hh;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const v4i lo = *reinterpret_cast<const v4i*>(qp + 64 * ks);
      const v4i hi = *reinterpret_cast<const v4i*>(qp + 64 * ks + 32);
      qf[ks] = i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
    const unsigned qw = static_cast<const unsigned*>(f.q_exp)[b * f.qe_bs + (int64_t)qrow_c * f.qe_ts + h];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) qsc[ks] = (int)((qw >> (8 * (2 * ks + hh))) & 0xffu);
  }
  const int last = (q0 + BM < a.Lq ? q0 + BM : a.Lq) - 1;
  const int kend_max = CHUNKED ? kend_of(a, last) : a.Lk;
  const int kend_min = CHUNKED ? kend_of(a, q0) : a.Lk;

  // buffer resources over this (batch, head)'s keys (offsets below 2^31, checked by the host)
  const char* kp = static_cast<const char*>(a.k) + b * a.kv_bs + h * DH;
  const char* vp = static_cast<const char*>(a.v) + b * a.kv_bs + h * DH;
  const char* ep = reinterpret_cast<const char*>(static_cast<const unsigned*>(f.k_exp) + b * f.ke_bs + h);
  const int kv_tsb = (int)a.kv_ts, e_tsb = 4 * (int)f.ke_ts;
  const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc((void*)kp, (short)0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc((void*)vp, (short)0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t er = __builtin_amdgcn_make_buffer_rsrc((void*)ep, (short)0, 0x7fffffff, 0x00020000);

  int koff[KCH], voff[KCH], krow[KCH];
#pragma unroll
  for (int i = 0; i < KCH; ++i) {
    const int u = (w * KCH + i) * 64 + lane, row = u / CPR, pch = u % CPR;
    krow[i] = row;
    koff[i] = row * kv_tsb + kswz(row, pch) * 16;
    voff[i] = row * kv_tsb + vswz(row, pch) * 16;
  }
  // K fragment of k-step ks: row l32, logical chunks 4 ks + hh and 4 ks + 2 + hh (the
  // same dims as the Q operand's)
  int kofs[4];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int j = 0; j < 2; ++j) kofs[2 * ks + j] = l32 * ROWB + kswz(l32, 4 * ks + 2 * j + hh) * 16;
  // V^T: lane (group g, index i16 = 2e + half) addresses key row 8(e>>2) + 4hh + (e&3)
  // (+16 per read), dims 32 mt + 16 (g&1) + 8 half; the row's segment swizzle only
  // depends on e.
  int vofs[4];
  {
    const int g = lane >> 4, i16 = lane & 15, e = i16 >> 1, half = i16 & 1;
    const int row = 8 * (e >> 2) + 4 * hh + (e & 3);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const int ch = 2 * mt + (g & 1);  // logical 16-byte chunk of the dims
      vofs[mt] = row * ROWB + vswz(row, ch) * 16 + 8 * half;
    }
  }

  f32x16 acc[4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) acc[mt] = f32x16{};
  // Row sums.  Read as a 16x16x128 operand, the probabilities of lane l are column l % 16
  // of k-chunk l / 16: chunks 0 and 2 hold the keys of queries 0-15 (lanes 0-15, 32-47),
  // chunks 1 and 3 those of queries 16-31.  A is E4M3 1.0 in lanes 0 and 32 (row 0, chunks
  // 0 and 2) and 20 and 52 (row 4, chunks 1 and 3), zero elsewhere, so row 0 of the result
  // is the sums of queries 0-15 and row 4 those of 16-31, i.e. register 0 of lane l < 32
  // holds query l's sum (lanes 32-63 hold zeros).
  const int sw = ((lane & 15) == 0 && !(lane & 16)) || ((lane & 15) == 4 && (lane & 16)) ? 0x38383838 : 0;
  const i32x8 sel = {sw, sw, sw, sw, sw, sw, sw, sw};
  f32x4 accl = f32x4{};
  float m_ref = -INFINITY;
  const float c = a.c, thr = RESCALE_LOG2 / c;

  const int ntiles = (kend_max + BN - 1) / BN;
  const int n_plain = kend_min / BN < ntiles ? kend_min / BN : ntiles;
  fetch_tile(smem, kr, vr, er, kv_tsb, e_tsb, a.Lk, 0, w, lane, koff, voff, krow);
  tile_sync();
  int t = 0;
  for (; t + 2 <= n_plain; t += 2) {
#pragma unroll
    for (int cur = 0; cur < 2; ++cur) {
      const int tt = t + cur;
      if (tt + 1 < ntiles)
        fetch_tile(smem + (cur ^ 1) * STAGE, kr, vr, er, kv_tsb, e_tsb, a.Lk, (tt + 1) * BN, w, lane, koff, voff,
                   krow);
      attn_tile<false>(smem + cur * STAGE, qf, qsc, acc, accl, sel, m_ref, kofs, vofs, c, thr, tt * BN, row_kend, hh,
                       l32);
      tile_sync();
    }
  }
  for (; t < ntiles; ++t) {
    const int cur = t & 1;
    if (t + 1 < ntiles)
      fetch_tile(smem + (cur ^ 1) * STAGE, kr, vr, er, kv_tsb, e_tsb, a.Lk, (t + 1) * BN, w, lane, koff, voff, krow);
    attn_tile<true>(smem + cur * STAGE, qf, qsc, acc, accl, sel, m_ref, kofs, vofs, c, thr, t * BN, row_kend, hh, l32);
    tile_sync();
  }

  const float lsum = accl[0] + other_half(accl[0]);  // one of the two is zero
  if constexpr (MX8) {
    uint8_t* o8 = static_cast<uint8_t*>(a.o) + b * a.o_bs + (int64_t)qrow * a.o_ts + h * DH;
    uint8_t* oe = o_exp + h * o_lde + 4 * ((int64_t)b * a.Lq + qrow);
    store_attn_row_mx8(o8, oe, acc, f.v_scale / lsum, hh, qrow < a.Lq);
  } else if (qrow < a.Lq) {
    const float inv = f.v_scale / lsum;
    bf16* ob = static_cast<bf16*>(a.o) + b * a.o_bs + (int64_t)qrow * a.o_ts + h * DH;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        bf16x4 v4 = {(bf16)(acc[mt][4 * rr + 0] * inv), (bf16)(acc[mt][4 * rr + 1] * inv),
                     (bf16)(acc[mt][4 * rr + 2] * inv), (bf16)(acc[mt][4 * rr + 3] * inv)};
        *reinterpret_cast<bf16x4*>(ob + 32 * mt + 8 * rr + 4 * hh) = v4;
      }
  }
}

}  // namespace

hipError_t launch_attn_fp8(const AttnFp8Args& f, hipStream_t s, uint8_t* o_exp, int64_t o_lde) {
  const AttnArgs& a = f.a;
  const int nqt = (a.Lq + BM - 1) / BM;
  const dim3 grid((unsigned)((long)nqt * a.H * a.B)), block(NT);
  const bool chunked = a.n_k_chunks > 1;
  if (o_exp) {  // block-scaled output
    if (chunked) hipLaunchKernelGGL((attn_fwd_fp8<true, true>), grid, block, 0, s, f, nqt, o_exp, o_lde);
    else hipLaunchKernelGGL((attn_fwd_fp8<false, true>), grid, block, 0, s, f, nqt, o_exp, o_lde);
  } else {
    uint8_t* const z = nullptr;
    if (chunked) hipLaunchKernelGGL((attn_fwd_fp8<true>), grid, block, 0, s, f, nqt, z, (int64_t)0);
    else hipLaunchKernelGGL((attn_fwd_fp8<false>), grid, block, 0, s, f, nqt, z, (int64_t)0);
  }
  return hipGetLastError();
}

}  // namespace wam
