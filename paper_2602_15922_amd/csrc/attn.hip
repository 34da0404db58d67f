// Flash-style block-causal attention for gfx950 (bf16 MFMA, fp32 online softmax).
//
// A query of chunk c sees the key prefix [0, kend(c)): every cached, clean earlier
// chunk and its own chunk (section 3.1; Appendix C, Figure 10b).  Key tiles past the
// largest prefix of a query tile are never visited; only tiles that straddle a
// query row's prefix end are masked.
//
// Work split: one workgroup = 4 wavefronts = 128 query rows of one (batch, head);
// each wavefront owns 32 query rows and walks all visible key tiles of 64 keys.
// The score tile is computed transposed, S^T = K Q^T, so that a lane owns one
// query and the softmax row statistics stay inside the lane (plus one exchange
// with the partner lane l^32).  The output is accumulated transposed as well,
// O^T = V^T P^T, so the per-query rescale is again lane-local.  K tiles sit in LDS
// row-major, V tiles transposed ([dh][key]); both XOR-swizzled so the MFMA operand
// reads are bank-conflict free.
#include "common.h"
#include "kernels.h"

namespace wam {
namespace {

constexpr int BM = 128;  // query rows per workgroup
constexpr int BN = 64;   // keys per tile

WAM_DEV int kend_of(const AttnArgs& a, int row) {
  int e = a.kend[a.n_q_chunks - 1];
  for (int i = a.n_q_chunks - 1; i >= 0; --i)
    if (row < a.q_off[i + 1]) e = a.kend[i];
  return e;
}

template <int DH>
__global__ __launch_bounds__(256) void attn_fwd(const AttnArgs a) {
  constexpr int KS = DH / 16;  // MFMA k-steps over the head dim
  constexpr int MT = DH / 32;  // 32-row tiles of the transposed output
  constexpr int CPR = DH / 8;  // 16-byte chunks per K row
  __shared__ __attribute__((aligned(16))) bf16 Ks[BN * DH];
  __shared__ __attribute__((aligned(16))) bf16 Vt[DH * BN];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int hh = lane >> 5, l32 = lane & 31;
  const int b = blockIdx.z, h = blockIdx.y, q0 = blockIdx.x * BM;

  const int qrow = q0 + 32 * w + l32;
  const int qrow_c = qrow < a.Lq ? qrow : a.Lq - 1;
  const int row_kend = kend_of(a, qrow_c);
  const int last = (q0 + BM < a.Lq ? q0 + BM : a.Lq) - 1;
  const int kend_max = kend_of(a, last);
  const int kend_min = kend_of(a, q0);

  const bf16* qb = static_cast<const bf16*>(a.q) + b * a.q_bs + (int64_t)qrow_c * a.q_ts + h * DH + 8 * hh;
  bf16x8 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qf[ks] = load_bf16x8(qb + 16 * ks);

  const bf16* kb_ptr = static_cast<const bf16*>(a.k) + b * a.kv_bs + h * DH;
  const bf16* vb_ptr = static_cast<const bf16*>(a.v) + b * a.kv_bs + h * DH;

  f32x16 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x16{};
  float m_i = -INFINITY, l_i = 0.f;
  const float c = a.c;

  const int ntiles = (kend_max + BN - 1) / BN;
  for (int t = 0; t < ntiles; ++t) {
    const int kb = t * BN;
    __syncthreads();
    // ---- K tile -> LDS, row-major [key][dh], 16-byte chunks swizzled by key
#pragma unroll
    for (int i = 0; i < (BN * CPR) / 256; ++i) {
      const int cidx = tid + 256 * i;
      const int key = cidx / CPR, ch = cidx % CPR;
      const int gk = kb + key;
      bf16x8 val = {};
      if (gk < a.Lk) val = load_bf16x8(kb_ptr + (int64_t)gk * a.kv_ts + ch * 8);
      *reinterpret_cast<bf16x8*>(&Ks[key * DH + ((ch ^ (key & 7)) * 8)]) = val;
    }
    // ---- V tile -> LDS transposed [dh][key]; a thread moves 4 keys x 8 dims
    if (tid < (BN / 4) * CPR) {
      const int kg = tid % (BN / 4), c8 = tid / (BN / 4);
      bf16x8 r[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int gk = kb + 4 * kg + i;
        r[i] = gk < a.Lk ? load_bf16x8(vb_ptr + (int64_t)gk * a.kv_ts + c8 * 8) : bf16x8{};
      }
#pragma unroll
      for (int dd = 0; dd < 8; ++dd) {
        const int dh = 8 * c8 + dd;
        bf16x4 col = {r[0][dd], r[1][dd], r[2][dd], r[3][dd]};
        *reinterpret_cast<bf16x4*>(&Vt[dh * BN + ((kg ^ (dh & 15)) * 4)]) = col;
      }
    }
    __syncthreads();

    // ---- S^T = K Q^T for two 32-key sub-tiles
    f32x16 s[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      s[nt] = f32x16{};
      const int key = 32 * nt + l32;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Ks[key * DH + (((2 * ks + hh) ^ (key & 7)) * 8)]);
        s[nt] = mfma32(kf, qf[ks], s[nt]);
      }
    }
    // ---- mask keys past this query's visible prefix (only on straddling tiles)
    if (kb + BN > kend_min) {
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kb + 32 * nt + 8 * (r >> 2) + 4 * hh + (r & 3);
          if (key >= row_kend) s[nt][r] = -INFINITY;
        }
    }
    // ---- online softmax (lane-local for its query, plus the partner lane)
    float mx = -INFINITY;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[nt][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_i, mx);
    const float ms = (m_new == -INFINITY) ? 0.f : m_new * c;
    const float alpha = exp2_fast(m_i * c - ms);
    float rs = 0.f;
    bf16x8 pb[2][2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2_fast(s[nt][r] * c - ms);
        rs += p;
        pb[nt][r >> 3][r & 7] = (bf16)p;
      }
    rs += __shfl_xor(rs, 32, 64);
    l_i = l_i * alpha + rs;
    m_i = m_new;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] *= alpha;

    // ---- O^T += V^T P^T
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int dh = 32 * mt + l32;
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int u0 = (32 * nt + 16 * hf + 4 * hh) >> 2;
          bf16x4 lo = *reinterpret_cast<const bf16x4*>(&Vt[dh * BN + ((u0 ^ (dh & 15)) * 4)]);
          bf16x4 hi = *reinterpret_cast<const bf16x4*>(&Vt[dh * BN + (((u0 + 2) ^ (dh & 15)) * 4)]);
          bf16x8 vf = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          acc[mt] = mfma32(vf, pb[nt][hf], acc[mt]);
        }
    }
  }

  if (qrow < a.Lq) {
    const float inv = 1.0f / l_i;
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

hipError_t launch_attn(const AttnArgs& a, hipStream_t s) {
  dim3 grid((a.Lq + BM - 1) / BM, a.H, a.B);
  if (a.Dh == 128)
    hipLaunchKernelGGL(attn_fwd<128>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(attn_fwd<64>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace wam
