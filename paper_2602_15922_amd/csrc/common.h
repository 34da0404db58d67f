// Shared device-side definitions for the gfx950 kernels of libwamdit.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

#define WAM_DEV __device__ __forceinline__

// 32x32x16 bf16 MFMA (gfx950).  Lane l, half h = l/32:
//   A operand: A[m = l%32][k = 8h .. 8h+7]      (8 consecutive k of one row)
//   B operand: B[k = 8h .. 8h+7][n = l%32]      (8 consecutive k of one column)
//   C/D:       register r holds D[m = 8*(r/4) + 4h + r%4][n = l%32]
WAM_DEV f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// 32x32x64 FP8 (E4M3 x E4M3) MFMA (gfx950), unit block scales.  Lane l, h = l/32, holds
// 32 bytes of row m = l%32 of A (column n = l%32 of B); A's and B's bytes at the same
// lane half and position are multiplied together.  With unit scales any k order shared
// by both operands gives the product; block scales group bytes 0-15 of both halves
// (scale from half 0) and bytes 16-31 of both halves (scale from half 1).
//   C/D:       as for mfma32
WAM_DEV f32x16 mfma32_fp8(i32x8 a, i32x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 127, 0, 127);
}

// The same with A scaled: byte sel (0 or 1, a constant after inlining) of sa is the biased
// exponent (scale 2^(byte - 127)) of the lane's row; the two lanes of a row hold the same
// byte, so both of the instruction's scale blocks take it.  W unscaled.
WAM_DEV f32x16 mfma32_fp8_sa(i32x8 a, i32x8 b, f32x16 c, int sa, int sel) {
  if (sel == 0) return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, sa, 0, 127);
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 1, sa, 0, 127);
}

// The value of lane l ^ 32 (the other half of the wavefront).
WAM_DEV float half_swap(float v) {
  const unsigned u = __float_as_uint(v);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}

WAM_DEV int mx_exp_biased(float amax);

// One query row of an attention output (Dh = 128) as block-scaled E4M3: acc[mt][r] holds
// dims 32 mt + 8 (r / 4) + 4 hh + r % 4 of the lane's query (lane l ^ 32 the other hh),
// o = acc * inv.  The output is rounded to bf16 first, as the bf16 store writes it; dims
// 0-63 (mt 0, 1) and 64-127 (mt 2, 3) are the two 64-element blocks, each with the exponent
// of mx_exp_biased.  Codes go to o8 (the head's 128 bytes of the row), the two exponents
// to oe[0] and oe[1].  Every lane calls it (the block maximum takes the other half's);
// only rows with valid set store.
WAM_DEV void store_attn_row_mx8(uint8_t* o8, uint8_t* oe, const f32x16* acc, float inv, int hh, bool valid) {
  float y[4][16], am[2] = {0.f, 0.f};
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      y[mt][r] = (float)(bf16)(acc[mt][r] * inv);
      am[mt >> 1] = fmaxf(am[mt >> 1], fabsf(y[mt][r]));
    }
#pragma unroll
  for (int k = 0; k < 2; ++k) am[k] = fmaxf(am[k], half_swap(am[k]));
  const int e0 = mx_exp_biased(am[0]), e1 = mx_exp_biased(am[1]);
  const float mul[2] = {ldexpf(1.0f, 127 - e0), ldexpf(1.0f, 127 - e1)};  // |y| * mul <= 448
  if (!valid) return;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const float k = mul[mt >> 1];
      int code = __builtin_amdgcn_cvt_pk_fp8_f32(y[mt][4 * rr] * k, y[mt][4 * rr + 1] * k, 0, false);
      code = __builtin_amdgcn_cvt_pk_fp8_f32(y[mt][4 * rr + 2] * k, y[mt][4 * rr + 3] * k, code, true);
      *reinterpret_cast<int*>(o8 + 32 * mt + 8 * rr + 4 * hh) = code;
    }
  if (hh == 0) *reinterpret_cast<uint16_t*>(oe) = (uint16_t)(e0 | (e1 << 8));
}

// Biased (127) exponent of an MX block with largest magnitude amax (finite, >= 0): the
// smallest e with amax <= 448 * 2^e, clamped to [-127, 127]; 0 (byte 127) for a zero
// block.  From the bits: amax = m 2^E' with m in [1, 2) takes e = E' - 8 if m <= 1.75
// (448 = 1.75 * 2^8), else E' - 7; below 2^-126 the clamp gives -127 (byte 0), and a finite
// amax never reaches the upper clamp.
WAM_DEV int mx_exp_biased(float amax) {
  if (!(amax > 0.f)) return 127;
  const unsigned u = __float_as_uint(amax);
  const int eb = (int)(u >> 23) - 8 + ((u & 0x7fffffu) > 0x600000u ? 1 : 0);
  return eb < 0 ? 0 : eb;
}

// The denoising loop launches a step's kernels with a device flag: while it is > 0 the
// step reuses an earlier velocity and every workgroup returns at entry.
WAM_DEV bool skip_step(const int32_t* skip) { return skip != nullptr && *skip > 0; }

WAM_DEV float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

WAM_DEV bf16x8 load_bf16x8(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

WAM_DEV float gelu_tanh_f(float u) {
  // 0.5 u (1 + tanh(y)) with y = sqrt(2/pi) (u + 0.044715 u^3) equals u * sigmoid(2y)
  // = u / (1 + 2^(-2 y log2 e)); evaluated with the hardware exp2 and reciprocal.
  const float k0 = 0.7978845608028654f * 2.0f * 1.4426950408889634f, k1 = 0.044715f;
  const float z = -k0 * (u + k1 * u * u * u);
  return u * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z));
}

WAM_DEV float silu_f(float u) { return u / (1.0f + __expf(-u)); }

// 64-lane wavefront reductions (every lane active), with no LDS round trips: within each row
// of 16 lanes by DPP (the two quad swaps, then the half-row mirror, lane i and 7 - i of each
// 8, and the row mirror, i and 15 - i), then the four rows' values by readlane.  Every lane
// gets the same value (each step adds the same two partial values in either lane).
#define WAM_DPP_F(v, ctrl) __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), ctrl, 0xF, 0xF, true))
WAM_DEV float wave_sum(float v) {
  v += WAM_DPP_F(v, 0xB1);   // quad_perm [1, 0, 3, 2]
  v += WAM_DPP_F(v, 0x4E);   // quad_perm [2, 3, 0, 1]
  v += WAM_DPP_F(v, 0x141);  // row_half_mirror
  v += WAM_DPP_F(v, 0x140);  // row_mirror
  const float a0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float a1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float a2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float a3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (a0 + a1) + (a2 + a3);
}
// the largest of v >= 0 over the wavefront (on the bit patterns: same order as the floats)
WAM_DEV float wave_max_nonneg(float v) {
  unsigned u = __float_as_uint(v);
  u = max(u, (unsigned)__builtin_amdgcn_mov_dpp((int)u, 0xB1, 0xF, 0xF, true));
  u = max(u, (unsigned)__builtin_amdgcn_mov_dpp((int)u, 0x4E, 0xF, 0xF, true));
  u = max(u, (unsigned)__builtin_amdgcn_mov_dpp((int)u, 0x141, 0xF, 0xF, true));
  u = max(u, (unsigned)__builtin_amdgcn_mov_dpp((int)u, 0x140, 0xF, 0xF, true));
  const unsigned r0 = __builtin_amdgcn_readlane((int)u, 0), r1 = __builtin_amdgcn_readlane((int)u, 16);
  const unsigned r2 = __builtin_amdgcn_readlane((int)u, 32), r3 = __builtin_amdgcn_readlane((int)u, 48);
  return __uint_as_float(max(max(r0, r1), max(r2, r3)));
}
#undef WAM_DPP_F
