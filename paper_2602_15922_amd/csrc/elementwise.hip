// HBM-bound and small kernels of the DiT step for gfx950: AdaLN LayerNorm+modulate,
// 3D RoPE with KV-cache append, time-embedding GEMV and sinusoid, patchify and
// unpatchify.  All loads and stores are 16-byte vectors over contiguous rows.
#include "common.h"
#include "kernels.h"

namespace wam {
namespace {

// ---------------------------------------------------------------------------------
// LayerNorm (biased variance, eps) of fp32 rows, then the optional affine and the
// AdaLN modulation, to bf16.  Both are folded into one per-column affine,
//   y = LN(x) * P + Q,  P = gamma (1 + scale),  Q = beta (1 + scale) + shift,
// computed once per workgroup into LDS (2*d floats): a workgroup owns LN_ROWS rows of
// one sample and one row segment (a sample's rows may form two segments with their own
// per-sample modulation: video and action tokens at their own timesteps), so the
// modulation vectors are read once per LN_ROWS rows.  One wavefront
// per row, so a 3152-row call keeps ~3150 rows in flight at once; the row stays in
// registers (NV float4 per lane, NV = d/256) between the mean, variance and output
// passes, so x is read from HBM once.  Each wavefront issues its row's loads before the
// workgroup builds P and Q, and the barrier after that waits for the LDS writes only,
// so the row is in flight while the modulation vectors are read.
// ---------------------------------------------------------------------------------
constexpr int LN_ROWS = 8;  // rows (= wavefronts) per workgroup

template <int NV>
// (4 wavefronts per SIMD up to d = 5120: a row, 80 VGPRs, fits with the rest in 128)
__global__ __launch_bounds__(LN_ROWS * 64, NV <= 20 ? 4 : 2) void ln_mod_kernel(const LnArgs a, int blocks_per_batch, int seg,
                                                              int seg_blocks) {
  extern __shared__ __attribute__((aligned(16))) float PQ[];  // [2][d]
  if (skip_step(a.skip)) return;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int b = blockIdx.x / blocks_per_batch, j = blockIdx.x % blocks_per_batch;
  // a workgroup's rows lie in one segment: [0, seg) or [seg, rows_per_batch)
  const bool second = j >= seg_blocks;
  const int rloc = second ? seg + (j - seg_blocks) * LN_ROWS + w : j * LN_ROWS + w;
  const int rend = second ? a.rows_per_batch : seg;
  const int d = a.d, nv = d >> 8;
  const int64_t mb = (int64_t)b * a.mod_stride + (second ? a.alt_off : 0);
  const bool active = rloc < rend;
  const int64_t row = (int64_t)b * a.rows_per_batch + (active ? rloc : rend - 1);
  const float* xr = a.x + row * d;
  f32x4 v[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i)
    if (i < nv) v[i] = *reinterpret_cast<const f32x4*>(xr + (i * 64 + lane) * 4);
  float* P = PQ;
  float* Q = PQ + d;
  for (int c = threadIdx.x * 4; c < d; c += LN_ROWS * 256) {
    f32x4 g = {1.f, 1.f, 1.f, 1.f}, bt = {0.f, 0.f, 0.f, 0.f}, sc = {0.f, 0.f, 0.f, 0.f}, sh = {0.f, 0.f, 0.f, 0.f};
    if (a.gamma) g = *reinterpret_cast<const f32x4*>(a.gamma + c);
    if (a.beta) bt = *reinterpret_cast<const f32x4*>(a.beta + c);
    if (a.scale_a) sc += *reinterpret_cast<const f32x4*>(a.scale_a + c);
    if (a.scale_v) sc += *reinterpret_cast<const f32x4*>(a.scale_v + mb + c);
    if (a.shift_a) sh += *reinterpret_cast<const f32x4*>(a.shift_a + c);
    if (a.shift_v) sh += *reinterpret_cast<const f32x4*>(a.shift_v + mb + c);
    const f32x4 one = {1.f, 1.f, 1.f, 1.f};
    *reinterpret_cast<f32x4*>(P + c) = g * (one + sc);
    *reinterpret_cast<f32x4*>(Q + c) = bt * (one + sc) + sh;
  }
  // LDS writes visible to the workgroup (the row loads stay in flight)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));  // lgkmcnt(0) only
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  if (!active) return;
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i)
    if (i < nv) s += (v[i][0] + v[i][1]) + (v[i][2] + v[i][3]);
  const float mean = wave_sum(s) / (float)d;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i)
    if (i < nv) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float t = v[i][j] - mean;
        q += t * t;
      }
    }
  const float rstd = rsqrtf(wave_sum(q) / (float)d + a.eps);
  bf16* hr = static_cast<bf16*>(a.h) + row * d;
#pragma unroll
  for (int i = 0; i < NV; ++i)
    if (i < nv) {
      const int col = (i * 64 + lane) * 4;
      const f32x4 pp = *reinterpret_cast<const f32x4*>(P + col);
      const f32x4 qq = *reinterpret_cast<const f32x4*>(Q + col);
      bf16x4 o;
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = (bf16)((v[i][j] - mean) * rstd * pp[j] + qq[j]);
      *reinterpret_cast<bf16x4*>(hr + col) = o;
    }
}

// The same with 8 consecutive columns per lane (d a multiple of 512): two adjacent 16-byte
// loads and one 16-byte store of 8 bf16 per lane and chunk, half the store instructions.
// With Q8 the row is not stored in bf16: its bf16 values are quantized to E4M3 codes with
// one scale per row (the maximum over the row's bf16 values / 448), the arithmetic of
// quant_rows_kernel applied to the row this kernel would have stored, and 8 codes per lane
// and chunk are stored (half the bytes of the bf16 row).
template <int NC, bool Q8>
__global__ __launch_bounds__(LN_ROWS * 64, NC <= 10 ? 4 : 2) void ln_mod8_kernel(const LnArgs a, int blocks_per_batch,
                                                                             int seg, int seg_blocks) {
  // Q8: d is exactly 512 NC (no chunk of the row is conditional)
  extern __shared__ __attribute__((aligned(16))) float PQ[];  // [2][d]
  if (skip_step(a.skip)) return;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int b = blockIdx.x / blocks_per_batch, j = blockIdx.x % blocks_per_batch;
  const bool second = j >= seg_blocks;
  const int rloc = second ? seg + (j - seg_blocks) * LN_ROWS + w : j * LN_ROWS + w;
  const int rend = second ? a.rows_per_batch : seg;
  const int d = a.d, nc = Q8 ? NC : d >> 9;
  const int64_t mb = (int64_t)b * a.mod_stride + (second ? a.alt_off : 0);
  const bool active = rloc < rend;
  const int64_t row = (int64_t)b * a.rows_per_batch + (active ? rloc : rend - 1);
  const float* xr = a.x + row * d;
  f32x4 v[NC][2];
#pragma unroll
  for (int i = 0; i < NC; ++i)
    if (i < nc) {
      const float* p = xr + (i * 64 + lane) * 8;
      v[i][0] = *reinterpret_cast<const f32x4*>(p);
      v[i][1] = *reinterpret_cast<const f32x4*>(p + 4);
    }
  float* P = PQ;
  float* Q = PQ + d;
  for (int c = threadIdx.x * 4; c < d; c += LN_ROWS * 256) {
    f32x4 g = {1.f, 1.f, 1.f, 1.f}, bt = {0.f, 0.f, 0.f, 0.f}, sc = {0.f, 0.f, 0.f, 0.f}, sh = {0.f, 0.f, 0.f, 0.f};
    if (a.gamma) g = *reinterpret_cast<const f32x4*>(a.gamma + c);
    if (a.beta) bt = *reinterpret_cast<const f32x4*>(a.beta + c);
    if (a.scale_a) sc += *reinterpret_cast<const f32x4*>(a.scale_a + c);
    if (a.scale_v) sc += *reinterpret_cast<const f32x4*>(a.scale_v + mb + c);
    if (a.shift_a) sh += *reinterpret_cast<const f32x4*>(a.shift_a + c);
    if (a.shift_v) sh += *reinterpret_cast<const f32x4*>(a.shift_v + mb + c);
    const f32x4 one = {1.f, 1.f, 1.f, 1.f};
    *reinterpret_cast<f32x4*>(P + c) = g * (one + sc);
    *reinterpret_cast<f32x4*>(Q + c) = bt * (one + sc) + sh;
  }
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));  // lgkmcnt(0) only
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  if (!active) return;
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NC; ++i)
    if (i < nc)
#pragma unroll
      for (int h = 0; h < 2; ++h) s += (v[i][h][0] + v[i][h][1]) + (v[i][h][2] + v[i][h][3]);
  const float mean = wave_sum(s) / (float)d;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < NC; ++i)
    if (i < nc)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const float t = v[i][h][k] - mean;
          q += t * t;
        }
  const float rstd = rsqrtf(wave_sum(q) / (float)d + a.eps);
  float amax = 0.f;  // Q8: the largest |bf16 output| of the row
#pragma unroll
  for (int i = 0; i < NC; ++i)
    if (i < nc) {
      const int col = (i * 64 + lane) * 8;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const f32x4 pp = *reinterpret_cast<const f32x4*>(P + col + 4 * h);
        const f32x4 qq = *reinterpret_cast<const f32x4*>(Q + col + 4 * h);
#pragma unroll
        for (int k = 0; k < 4; ++k) v[i][h][k] = (v[i][h][k] - mean) * rstd * pp[k] + qq[k];
      }
      bf16x8 o;
#pragma unroll
      for (int k = 0; k < 8; ++k) o[k] = (bf16)v[i][k >> 2][k & 3];
      if constexpr (Q8) {  // keep the bf16 values (as fp32) for the second pass
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          v[i][k >> 2][k & 3] = (float)o[k];
          amax = fmaxf(amax, fabsf((float)o[k]));
        }
      } else {
        *reinterpret_cast<bf16x8*>(static_cast<bf16*>(a.h) + row * d + col) = o;
      }
    }
  if constexpr (Q8) {
    amax = wave_max_nonneg(amax);
    const float inv = amax > 0.f ? 448.0f / amax : 1.0f;
    if (lane == 0) a.q_scale[row] = amax > 0.f ? amax / 448.0f : 1.0f;
    uint8_t* qr = a.q8 + row * a.ldq;
#pragma unroll
    for (int i = 0; i < NC; ++i)
      if (i < nc) {
        float f[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) f[k] = fminf(fmaxf(v[i][k >> 2][k & 3] * inv, -448.0f), 448.0f);
        int lo = 0, hi = 0;
        lo = __builtin_amdgcn_cvt_pk_fp8_f32(f[0], f[1], lo, false);
        lo = __builtin_amdgcn_cvt_pk_fp8_f32(f[2], f[3], lo, true);
        hi = __builtin_amdgcn_cvt_pk_fp8_f32(f[4], f[5], hi, false);
        hi = __builtin_amdgcn_cvt_pk_fp8_f32(f[6], f[7], hi, true);
        *reinterpret_cast<u32x2*>(qr + (i * 64 + lane) * 8) = u32x2{(uint32_t)lo, (uint32_t)hi};
      }
  }
}

// One thread per 4 columns of one (layer, norm, sample, segment): the shift and scale
// sums of the AdaLN modulation (the same fp32 additions the LayerNorm performs).
__global__ __launch_bounds__(256) void adaln_fold_kernel(const AdalnFoldArgs a) {
  if (skip_step(a.skip)) return;
  const int d4 = a.d >> 2;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t n = (int64_t)a.n_layers * 2 * a.B * a.nseg * d4;
  if (i >= n) return;
  int64_t t = i;
  const int c = (int)(t % d4) * 4; t /= d4;
  const int g = (int)(t % a.nseg); t /= a.nseg;
  const int b = (int)(t % a.B); t /= a.B;
  const int k = (int)(t % 2);
  const int l = (int)(t / 2);
  const float* m6 = a.mod6[l];
  const float* e0 = a.e0 + (int64_t)b * a.e0_stride + (g ? a.alt : 0);
  float* o = a.out + (int64_t)l * a.layer_stride + ((((int64_t)k * a.B + b) * a.nseg + g) * 2) * a.d;
  const int sh = 3 * k, sc = 3 * k + 1;
  *reinterpret_cast<f32x4*>(o + c) =
      *reinterpret_cast<const f32x4*>(m6 + sh * a.d + c) + *reinterpret_cast<const f32x4*>(e0 + sh * a.d + c);
  *reinterpret_cast<f32x4*>(o + a.d + c) =
      *reinterpret_cast<const f32x4*>(m6 + sc * a.d + c) + *reinterpret_cast<const f32x4*>(e0 + sc * a.d + c);
}

// ---------------------------------------------------------------------------------
// Per-row E4M3 quantization for the FP8 GEMMs: one wavefront per row of K bf16 values,
// amax over the row, inv = 448 / amax (fp32), q = E4M3(x * inv) rounded to nearest even
// (|x * inv| <= 448 by construction), scale = amax / 448 (1 for an all-zero row).
// Each lane converts 8 consecutive values per step into one 8-byte store.
// ---------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void quant_rows_kernel(int M, int K, const bf16* __restrict__ x, int64_t ldx,
                                                         uint8_t* __restrict__ q, int64_t ldq,
                                                         float* __restrict__ scale, const int32_t* skip) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + w;
  if (row >= M || skip_step(skip)) return;
  const bf16* xr = x + (int64_t)row * ldx;
  float amax = 0.f;
  for (int k = lane * 8; k < K; k += 512) {
    const bf16x8 v = load_bf16x8(xr + k);
#pragma unroll
    for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf((float)v[j]));
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
  const float inv = amax > 0.f ? 448.0f / amax : 1.0f;
  if (lane == 0) scale[row] = amax > 0.f ? amax / 448.0f : 1.0f;
  uint8_t* qr = q + (int64_t)row * ldq;
  for (int k = lane * 8; k < K; k += 512) {
    const bf16x8 v = load_bf16x8(xr + k);
    float f[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) f[j] = fminf(fmaxf((float)v[j] * inv, -448.0f), 448.0f);
    int lo = 0, hi = 0;
    lo = __builtin_amdgcn_cvt_pk_fp8_f32(f[0], f[1], lo, false);
    lo = __builtin_amdgcn_cvt_pk_fp8_f32(f[2], f[3], lo, true);
    hi = __builtin_amdgcn_cvt_pk_fp8_f32(f[4], f[5], hi, false);
    hi = __builtin_amdgcn_cvt_pk_fp8_f32(f[6], f[7], hi, true);
    *reinterpret_cast<u32x2*>(qr + k) = u32x2{(uint32_t)lo, (uint32_t)hi};
  }
}

// The same for rows of at most 512 * NC values: the row is held in registers (NC 16-byte
// loads per lane, all issued before the first is used) and read from memory once.
template <int NC>
__global__ __launch_bounds__(256) void quant_rows_reg_kernel(int M, int K, const bf16* __restrict__ x, int64_t ldx,
                                                             uint8_t* __restrict__ q, int64_t ldq,
                                                             float* __restrict__ scale, const int32_t* skip) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + w;
  if (row >= M || skip_step(skip)) return;
  const bf16* xr = x + (int64_t)row * ldx;
  bf16x8 v[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int k = c * 512 + lane * 8;
    v[c] = k < K ? load_bf16x8(xr + k) : bf16x8{};
  }
  float amax = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf((float)v[c][j]));
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
  const float inv = amax > 0.f ? 448.0f / amax : 1.0f;
  if (lane == 0) scale[row] = amax > 0.f ? amax / 448.0f : 1.0f;
  uint8_t* qr = q + (int64_t)row * ldq;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int k = c * 512 + lane * 8;
    if (k < K) {
      float f[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) f[j] = fminf(fmaxf((float)v[c][j] * inv, -448.0f), 448.0f);
      int lo = 0, hi = 0;
      lo = __builtin_amdgcn_cvt_pk_fp8_f32(f[0], f[1], lo, false);
      lo = __builtin_amdgcn_cvt_pk_fp8_f32(f[2], f[3], lo, true);
      hi = __builtin_amdgcn_cvt_pk_fp8_f32(f[4], f[5], hi, false);
      hi = __builtin_amdgcn_cvt_pk_fp8_f32(f[6], f[7], hi, true);
      *reinterpret_cast<u32x2*>(qr + k) = u32x2{(uint32_t)lo, (uint32_t)hi};
    }
  }
}

// ---------------------------------------------------------------------------------
// FP8 operands of the attention.  MX-style blocks: 32 consecutive elements share the
// scale 2^e, e the smallest integer with max|x| <= 448 * 2^e (clamped to [-127, 127];
// 0 for a zero block), stored biased by 127 in one byte; codes E4M3(x * 2^-e), exact
// scaling and round to nearest even.  One thread converts 8 elements; the 4 threads of
// a block (consecutive lanes) share its maximum through two lane exchanges.
// ---------------------------------------------------------------------------------
WAM_DEV u32x2 e4m3x8(const float* f, float mul) {
  float y[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) y[j] = fminf(fmaxf(f[j] * mul, -448.0f), 448.0f);
  int lo = __builtin_amdgcn_cvt_pk_fp8_f32(y[0], y[1], 0, false);
  lo = __builtin_amdgcn_cvt_pk_fp8_f32(y[2], y[3], lo, true);
  int hi = __builtin_amdgcn_cvt_pk_fp8_f32(y[4], y[5], 0, false);
  hi = __builtin_amdgcn_cvt_pk_fp8_f32(y[6], y[7], hi, true);
  return u32x2{(uint32_t)lo, (uint32_t)hi};
}

// 8 values of one 32-element block -> 8 codes; returns the block's biased exponent.
WAM_DEV int mx_encode8(const float* f, u32x2& codes) {
  float amax = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf(f[j]));
  amax = fmaxf(amax, __shfl_xor(amax, 1, 64));
  amax = fmaxf(amax, __shfl_xor(amax, 2, 64));
  const int eb = mx_exp_biased(amax);
  codes = e4m3x8(f, ldexpf(1.0f, 127 - eb));
  return eb;
}

__global__ __launch_bounds__(256) void quant_mx_kernel(int rows, int cols, const bf16* __restrict__ x, int64_t ldx,
                                                       uint8_t* __restrict__ q, int64_t ldq,
                                                       uint8_t* __restrict__ ex) {
  const int c8 = cols >> 3;
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (id >= (int64_t)rows * c8) return;  // rows * c8 is a multiple of 4: whole blocks
  const int64_t r = id / c8;
  const int c = (int)(id - r * c8) * 8;
  const bf16x8 v = load_bf16x8(x + r * ldx + c);
  float f[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = (float)v[j];
  u32x2 codes;
  const int eb = mx_encode8(f, codes);
  *reinterpret_cast<u32x2*>(q + r * ldq + c) = codes;
  if ((c & 31) == 0) ex[r * (cols >> 5) + (c >> 5)] = (uint8_t)eb;
}

// One-scale codes E4M3(x * inv), 8 elements per thread.
__global__ __launch_bounds__(256) void quant_scaled_kernel(int64_t n8, const bf16* __restrict__ x, float inv,
                                                           uint8_t* __restrict__ q) {
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (id >= n8) return;
  const bf16x8 v = load_bf16x8(x + id * 8);
  float f[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = (float)v[j];
  *reinterpret_cast<u32x2*>(q + id * 8) = e4m3x8(f, inv);
}

// ---------------------------------------------------------------------------------
// 3D RoPE + KV append.  A thread owns 8 consecutive dims (4 rotation pairs) of one
// head of one token and moves the q, k and v slices of the fused QKV row: q rotated
// to q_out, k rotated and v copied into the cache rows [row0, row0 + L).
// ---------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void rope_qkv_kernel(const RopeArgs a) {
  const int d = a.H * a.Dh, d8 = d >> 3;
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (id >= (int64_t)a.B * a.L * d8 || skip_step(a.skip)) return;
  const int c = (int)(id % d8);
  const int64_t bl = id / d8;
  const int l = (int)(bl % a.L), b = (int)(bl / a.L);
  const int col = c * 8;            // column inside the d-wide q/k/v slice
  const int pair0 = (col % a.Dh) >> 1;  // first rotation pair inside the head
  const bf16* src = static_cast<const bf16*>(a.qkv) + bl * 3 * d + col;
  const bf16x8 qv = a.q_out ? load_bf16x8(src) : bf16x8{};
  const bf16x8 kv = load_bf16x8(src + d), vv = load_bf16x8(src + 2 * d);
  const f32x4 cs = *reinterpret_cast<const f32x4*>(a.cos_t + (int64_t)l * (a.Dh >> 1) + pair0);
  const f32x4 sn = *reinterpret_cast<const f32x4*>(a.sin_t + (int64_t)l * (a.Dh >> 1) + pair0);
  bf16x8 qo, ko;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const float q0 = (float)qv[2 * p], q1 = (float)qv[2 * p + 1];
    const float k0 = (float)kv[2 * p], k1 = (float)kv[2 * p + 1];
    // the rotation in this fma form wherever it is applied (the QKV epilogue too)
    qo[2 * p] = (bf16)__builtin_fmaf(q0, cs[p], -(q1 * sn[p]));
    qo[2 * p + 1] = (bf16)__builtin_fmaf(q0, sn[p], q1 * cs[p]);
    ko[2 * p] = (bf16)__builtin_fmaf(k0, cs[p], -(k1 * sn[p]));
    ko[2 * p + 1] = (bf16)__builtin_fmaf(k0, sn[p], k1 * cs[p]);
  }
  if (a.q_out) *reinterpret_cast<bf16x8*>(static_cast<bf16*>(a.q_out) + bl * d + col) = qo;
  const int64_t crow = ((int64_t)b * a.Lcap + a.row0 + l) * d + col;
  *reinterpret_cast<bf16x8*>(static_cast<bf16*>(a.k_cache) + crow) = ko;
  *reinterpret_cast<bf16x8*>(static_cast<bf16*>(a.v_cache) + crow) = vv;
}

// RoPE + KV append with FP8 outputs for the FP8 attention: the rotated q and k (fp32)
// are encoded in 32-dim blocks into q8 / the K code cache with their exponents (one
// byte per block, four per (token, head) at Dh = 128), v as E4M3(v * v_inv) into the
// V code cache.  Same thread layout as rope_qkv_kernel: the 4 threads of a 32-dim
// block are consecutive lanes.
__global__ __launch_bounds__(256) void rope_qkv_fp8_kernel(const RopeFp8Args f) {
  const RopeArgs& a = f.r;
  const int d = a.H * a.Dh, d8 = d >> 3, d32 = d >> 5;
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (id >= (int64_t)a.B * a.L * d8 || skip_step(a.skip)) return;  // whole 4-thread blocks
  const int c = (int)(id % d8);
  const int64_t bl = id / d8;
  const int l = (int)(bl % a.L), b = (int)(bl / a.L);
  const int col = c * 8;
  const int pair0 = (col % a.Dh) >> 1;
  const bf16* src = static_cast<const bf16*>(a.qkv) + bl * 3 * d + col;
  const bf16x8 qv = a.q_out ? load_bf16x8(src) : bf16x8{};
  const bf16x8 kv = load_bf16x8(src + d), vv = load_bf16x8(src + 2 * d);
  const f32x4 cs = *reinterpret_cast<const f32x4*>(a.cos_t + (int64_t)l * (a.Dh >> 1) + pair0);
  const f32x4 sn = *reinterpret_cast<const f32x4*>(a.sin_t + (int64_t)l * (a.Dh >> 1) + pair0);
  float qo[8], ko[8], vo[8];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const float q0 = (float)qv[2 * p], q1 = (float)qv[2 * p + 1];
    const float k0 = (float)kv[2 * p], k1 = (float)kv[2 * p + 1];
    qo[2 * p] = q0 * cs[p] - q1 * sn[p];
    qo[2 * p + 1] = q0 * sn[p] + q1 * cs[p];
    ko[2 * p] = k0 * cs[p] - k1 * sn[p];
    ko[2 * p + 1] = k0 * sn[p] + k1 * cs[p];
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) vo[j] = (float)vv[j];
  const bool lead = (col & 31) == 0;
  if (a.q_out) {  // uniform over the launch
    u32x2 codes;
    const int eb = mx_encode8(qo, codes);
    *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(a.q_out) + bl * d + col) = codes;
    if (lead) static_cast<uint8_t*>(f.q_exp)[bl * d32 + (col >> 5)] = (uint8_t)eb;
  }
  const int64_t crow = (int64_t)b * a.Lcap + a.row0 + l;
  u32x2 codes;
  const int eb = mx_encode8(ko, codes);
  *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(a.k_cache) + crow * d + col) = codes;
  if (lead) static_cast<uint8_t*>(f.k_exp)[crow * d32 + (col >> 5)] = (uint8_t)eb;
  *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(a.v_cache) + crow * d + col) = e4m3x8(vo, f.v_inv);
}

// ---------------------------------------------------------------------------------
// Small-batch GEMV for the time MLP (B <= 8): a workgroup of 4 wavefronts owns
// GEMV_ROWS output features, GEMV_WROWS per wavefront, for every sample b.  The input
// (after its activation, evaluated once per workgroup instead of once per feature) is
// staged in LDS (all of it, or passes of up to GEMV_LDS floats); each lane then reads 8 consecutive
// k of each of its wavefront's W rows per 16-byte load, so W streams from HBM once with
// GEMV_WROWS loads in flight per lane.  Lane l sums k = 8 l + 512 i (+0..7), the same
// order for any pass length (passes are multiples of 512 columns).
// ---------------------------------------------------------------------------------
constexpr int GEMV_MAXB = 8;
constexpr int GEMV_WROWS = 4;
constexpr int GEMV_ROWS = 4 * GEMV_WROWS;
constexpr int GEMV_LDS = 16384;

template <int B>
__global__ __launch_bounds__(256, 2) void gemv_kernel(int N, int K, int kc, const float* __restrict__ x,
                                                   int act, const bf16* __restrict__ W,
                                                   const float* __restrict__ bias, float* __restrict__ out,
                                                   const int32_t* skip) {
  extern __shared__ __attribute__((aligned(16))) float xs[];  // B * kc floats
  if (skip_step(skip)) return;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n0 = blockIdx.x * GEMV_ROWS + w * GEMV_WROWS;
  float acc[B][GEMV_WROWS];
#pragma unroll
  for (int b = 0; b < B; ++b)
#pragma unroll
    for (int r = 0; r < GEMV_WROWS; ++r) acc[b][r] = 0.f;
  for (int k0 = 0; k0 < K; k0 += kc) {
    const int kn = K - k0 < kc ? K - k0 : kc;
    __syncthreads();
    // 4 floats per load, a thread's loads issued in groups of 8 before any is used (B * kn
    // <= GEMV_LDS: at most GEMV_LDS / 1024 per thread; kn is a multiple of 8)
    {
      const int kn4 = kn >> 2, n4 = B * kn4;
#pragma unroll
      for (int j0 = 0; j0 < GEMV_LDS / 1024; j0 += 8) {
        f32x4 v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int i = threadIdx.x + 256 * (j0 + j);
          if (i < n4) {
            const int b = i / kn4, k = (i - b * kn4) * 4;
            v[j] = *reinterpret_cast<const f32x4*>(x + (int64_t)b * K + k0 + k);
          }
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int i = threadIdx.x + 256 * (j0 + j);
          if (i < n4) {
            const int b = i / kn4, k = (i - b * kn4) * 4;
            f32x4 u = v[j];
            if (act == GEMV_ACT_SILU)
#pragma unroll
              for (int e = 0; e < 4; ++e) u[e] = silu_f(u[e]);
            *reinterpret_cast<f32x4*>(xs + b * kn + k) = u;
          }
        }
      }
    }
    __syncthreads();
    for (int kk = lane * 8; kk < kn; kk += 512) {
      bf16x8 wv[GEMV_WROWS];
#pragma unroll
      for (int r = 0; r < GEMV_WROWS; ++r)
        wv[r] = n0 + r < N ? load_bf16x8(W + (int64_t)(n0 + r) * K + k0 + kk) : bf16x8{};
#pragma unroll
      for (int b = 0; b < B; ++b) {
          const f32x4 x0 = *reinterpret_cast<const f32x4*>(xs + b * kn + kk);
          const f32x4 x1 = *reinterpret_cast<const f32x4*>(xs + b * kn + kk + 4);
          const float xv[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
#pragma unroll
          for (int r = 0; r < GEMV_WROWS; ++r)
#pragma unroll
            for (int j = 0; j < 8; ++j) acc[b][r] += xv[j] * (float)wv[r][j];
        }
    }
  }
#pragma unroll
  for (int b = 0; b < B; ++b)
#pragma unroll
      for (int r = 0; r < GEMV_WROWS; ++r) {
        const float s = wave_sum(acc[b][r]);
        if (lane == 0 && n0 + r < N) out[(int64_t)b * N + n0 + r] = s + (bias ? bias[n0 + r] : 0.f);
      }
}

// [cos(1000 t w_k), sin(1000 t w_k)], w_k = 10000^(-k/half); evaluated in double so the
// large arguments (up to 1000 rad) keep full fp32 accuracy.
__global__ void sinusoid_kernel(int B, int fd, const float* t, float* out, const int32_t* skip) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * fd || skip_step(skip)) return;
  const int b = i / fd, k = i % fd, half = fd / 2;
  const int kk = k < half ? k : k - half;
  const double omega = pow(10000.0, -(double)kk / (double)half);
  const double arg = 1000.0 * (double)t[b] * omega;
  out[i] = (float)(k < half ? cos(arg) : sin(arg));
}

// token (f, r, s) feature (c, ph, pw) <- z[b][c][f][2r+ph][2s+pw]
__global__ void patchify_kernel(int B, int C, int F, int Hl, int Wl, const bf16* z, bf16* tok,
                                const int32_t* skip) {
  const int Hg = Hl / 2, Wg = Wl / 2, P = C * 4;
  const int64_t n = (int64_t)B * F * Hg * Wg * P;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n || skip_step(skip)) return;
  const int fe = (int)(i % P);
  int64_t t = i / P;
  const int s = (int)(t % Wg); t /= Wg;
  const int r = (int)(t % Hg); t /= Hg;
  const int f = (int)(t % F);
  const int b = (int)(t / F);
  const int c = fe / 4, ph = (fe / 2) & 1, pw = fe & 1;
  tok[i] = z[((((int64_t)b * C + c) * F + f) * Hl + 2 * r + ph) * Wl + 2 * s + pw];
}

__global__ void unpatchify_kernel(int B, int C, int F, int Hl, int Wl, const float* tok, float* out,
                                  const int32_t* skip) {
  const int Hg = Hl / 2, Wg = Wl / 2;
  const int64_t n = (int64_t)B * C * F * Hl * Wl;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n || skip_step(skip)) return;
  int64_t t = i;
  const int xw = (int)(t % Wl); t /= Wl;
  const int y = (int)(t % Hl); t /= Hl;
  const int f = (int)(t % F); t /= F;
  const int c = (int)(t % C);
  const int b = (int)(t / C);
  const int64_t token = ((int64_t)b * F + f) * Hg * Wg + (y / 2) * Wg + xw / 2;
  out[i] = tok[token * (C * 4) + c * 4 + (y & 1) * 2 + (xw & 1)];
}

}  // namespace

hipError_t launch_ln_mod(const LnArgs& a, hipStream_t s) {
  if (a.rows == 0) return hipSuccess;
  const int B = a.rows / a.rows_per_batch;
  const int seg = a.seg_rows > 0 && a.seg_rows < a.rows_per_batch ? a.seg_rows : a.rows_per_batch;
  const int sb0 = (seg + LN_ROWS - 1) / LN_ROWS;
  const int bpb = sb0 + (a.rows_per_batch - seg + LN_ROWS - 1) / LN_ROWS;
  const dim3 grid((unsigned)(B * bpb)), block(LN_ROWS * 64);
  const size_t lds = (size_t)2 * a.d * sizeof(float);  // d <= 8192: at most 64 KB
  const int nv = a.d / 256;
  if (a.q8) {  // FP8 output: one kernel per row width
    if (!ln_fp8_supported(a.d)) return hipErrorInvalidValue;
    switch (a.d / 512) {
      case 1: hipLaunchKernelGGL((ln_mod8_kernel<1, true>), grid, block, lds, s, a, bpb, seg, sb0); break;
      case 2: hipLaunchKernelGGL((ln_mod8_kernel<2, true>), grid, block, lds, s, a, bpb, seg, sb0); break;
      case 3: hipLaunchKernelGGL((ln_mod8_kernel<3, true>), grid, block, lds, s, a, bpb, seg, sb0); break;
      case 4: hipLaunchKernelGGL((ln_mod8_kernel<4, true>), grid, block, lds, s, a, bpb, seg, sb0); break;
      case 5: hipLaunchKernelGGL((ln_mod8_kernel<5, true>), grid, block, lds, s, a, bpb, seg, sb0); break;
      case 6: hipLaunchKernelGGL((ln_mod8_kernel<6, true>), grid, block, lds, s, a, bpb, seg, sb0); break;
      case 7: hipLaunchKernelGGL((ln_mod8_kernel<7, true>), grid, block, lds, s, a, bpb, seg, sb0); break;
      case 8: hipLaunchKernelGGL((ln_mod8_kernel<8, true>), grid, block, lds, s, a, bpb, seg, sb0); break;
      case 9: hipLaunchKernelGGL((ln_mod8_kernel<9, true>), grid, block, lds, s, a, bpb, seg, sb0); break;
      default: hipLaunchKernelGGL((ln_mod8_kernel<10, true>), grid, block, lds, s, a, bpb, seg, sb0); break;
    }
    return hipGetLastError();
  }
  if (a.d % 512 == 0 && a.d <= 5120) {  // 8 columns per lane (d up to 5120: 80 values per lane)
    if (a.d <= 2048) hipLaunchKernelGGL((ln_mod8_kernel<4, false>), grid, block, lds, s, a, bpb, seg, sb0);
    else hipLaunchKernelGGL((ln_mod8_kernel<10, false>), grid, block, lds, s, a, bpb, seg, sb0);
    return hipGetLastError();
  }
  if (nv <= 2) hipLaunchKernelGGL(ln_mod_kernel<2>, grid, block, lds, s, a, bpb, seg, sb0);
  else if (nv <= 8) hipLaunchKernelGGL(ln_mod_kernel<8>, grid, block, lds, s, a, bpb, seg, sb0);
  else if (nv <= 20) hipLaunchKernelGGL(ln_mod_kernel<20>, grid, block, lds, s, a, bpb, seg, sb0);
  else hipLaunchKernelGGL(ln_mod_kernel<32>, grid, block, lds, s, a, bpb, seg, sb0);
  return hipGetLastError();
}

hipError_t launch_adaln_fold(const AdalnFoldArgs& a, hipStream_t s) {
  const int64_t n = (int64_t)a.n_layers * 2 * a.B * a.nseg * (a.d / 4);
  if (n == 0) return hipSuccess;
  if (a.n_layers > ADALN_FOLD_MAX_LAYERS || a.d % 4 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(adaln_fold_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_quant_rows(int32_t M, int32_t K, const void* x, int64_t ldx, void* q, int64_t ldq, float* scale,
                             hipStream_t s, const int32_t* skip) {
  if (M == 0) return hipSuccess;
  const dim3 grid((unsigned)((M + 3) / 4)), block(256);
  const bf16* xb = static_cast<const bf16*>(x);
  uint8_t* qb = static_cast<uint8_t*>(q);
  // register tiers: up to 2048 / 4096 / 6144 / 14336 values per row (the 14B model's
  // projection inputs are 5120 and 13824 wide); longer rows take the two-pass kernel
  if (K <= 2048) hipLaunchKernelGGL(quant_rows_reg_kernel<4>, grid, block, 0, s, M, K, xb, ldx, qb, ldq, scale, skip);
  else if (K <= 4096) hipLaunchKernelGGL(quant_rows_reg_kernel<8>, grid, block, 0, s, M, K, xb, ldx, qb, ldq, scale, skip);
  else if (K <= 6144) hipLaunchKernelGGL(quant_rows_reg_kernel<12>, grid, block, 0, s, M, K, xb, ldx, qb, ldq, scale, skip);
  else if (K <= 14336) hipLaunchKernelGGL(quant_rows_reg_kernel<28>, grid, block, 0, s, M, K, xb, ldx, qb, ldq, scale, skip);
  else hipLaunchKernelGGL(quant_rows_kernel, grid, block, 0, s, M, K, xb, ldx, qb, ldq, scale, skip);
  return hipGetLastError();
}

hipError_t launch_rope_qkv(const RopeArgs& a, hipStream_t s) {
  const int64_t n = (int64_t)a.B * a.L * (a.H * a.Dh / 8);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(rope_qkv_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gemv(int32_t B, int32_t N, int32_t K, const float* x, int32_t act, const void* W,
                       const float* bias, float* out, hipStream_t s, const int32_t* skip) {
  if (B <= 0 || N <= 0) return hipSuccess;
  if (B > GEMV_MAXB || K % 8 != 0) return hipErrorInvalidValue;
  // columns per pass: all of K when B x K floats fit, else a multiple of 512 (B <= 8: at
  // least 2048); the LDS is sized to the pass, so small inputs leave room for more
  // workgroups per CU
  const int kc = (int64_t)B * K <= GEMV_LDS ? K : (GEMV_LDS / B) & ~511;
  const dim3 grid((N + GEMV_ROWS - 1) / GEMV_ROWS), block(256);
  const size_t lds = (size_t)B * kc * sizeof(float);
  const bf16* w = static_cast<const bf16*>(W);
  switch (B) {
    case 1: hipLaunchKernelGGL(gemv_kernel<1>, grid, block, lds, s, N, K, kc, x, act, w, bias, out, skip); break;
    case 2: hipLaunchKernelGGL(gemv_kernel<2>, grid, block, lds, s, N, K, kc, x, act, w, bias, out, skip); break;
    case 3: hipLaunchKernelGGL(gemv_kernel<3>, grid, block, lds, s, N, K, kc, x, act, w, bias, out, skip); break;
    case 4: hipLaunchKernelGGL(gemv_kernel<4>, grid, block, lds, s, N, K, kc, x, act, w, bias, out, skip); break;
    case 5: hipLaunchKernelGGL(gemv_kernel<5>, grid, block, lds, s, N, K, kc, x, act, w, bias, out, skip); break;
    case 6: hipLaunchKernelGGL(gemv_kernel<6>, grid, block, lds, s, N, K, kc, x, act, w, bias, out, skip); break;
    case 7: hipLaunchKernelGGL(gemv_kernel<7>, grid, block, lds, s, N, K, kc, x, act, w, bias, out, skip); break;
    default: hipLaunchKernelGGL(gemv_kernel<8>, grid, block, lds, s, N, K, kc, x, act, w, bias, out, skip); break;
  }
  return hipGetLastError();
}

hipError_t launch_sinusoid(int32_t B, int32_t fd, const float* t, float* out, hipStream_t s, const int32_t* skip) {
  hipLaunchKernelGGL(sinusoid_kernel, dim3((B * fd + 255) / 256), dim3(256), 0, s, B, fd, t, out, skip);
  return hipGetLastError();
}

hipError_t launch_patchify(int32_t B, int32_t C, int32_t F, int32_t Hl, int32_t Wl, const void* z,
                           void* tok, hipStream_t s, const int32_t* skip) {
  const int64_t n = (int64_t)B * F * (Hl / 2) * (Wl / 2) * C * 4;
  hipLaunchKernelGGL(patchify_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, B, C, F,
                     Hl, Wl, static_cast<const bf16*>(z), static_cast<bf16*>(tok), skip);
  return hipGetLastError();
}

hipError_t launch_unpatchify(int32_t B, int32_t C, int32_t F, int32_t Hl, int32_t Wl, const float* tok,
                             float* out, hipStream_t s, const int32_t* skip) {
  const int64_t n = (int64_t)B * C * F * Hl * Wl;
  hipLaunchKernelGGL(unpatchify_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, B, C, F,
                     Hl, Wl, tok, out, skip);
  return hipGetLastError();
}

hipError_t launch_quant_mx(int32_t rows, int32_t cols, const void* x, int64_t ldx, void* q, int64_t ldq, void* ex,
                           hipStream_t s) {
  const int64_t n = (int64_t)rows * (cols / 8);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(quant_mx_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, rows, cols,
                     static_cast<const bf16*>(x), ldx, static_cast<uint8_t*>(q), ldq, static_cast<uint8_t*>(ex));
  return hipGetLastError();
}

hipError_t launch_quant_scaled(int64_t n, const void* x, float inv, void* q, hipStream_t s) {
  const int64_t n8 = n / 8;
  if (n8 == 0) return hipSuccess;
  hipLaunchKernelGGL(quant_scaled_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, s, n8,
                     static_cast<const bf16*>(x), inv, static_cast<uint8_t*>(q));
  return hipGetLastError();
}

hipError_t launch_rope_qkv_fp8(const RopeFp8Args& f, hipStream_t s) {
  const RopeArgs& a = f.r;
  const int64_t n = (int64_t)a.B * a.L * (a.H * a.Dh / 8);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(rope_qkv_fp8_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, f);
  return hipGetLastError();
}

}  // namespace wam
