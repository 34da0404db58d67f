// Internal launchers of the gfx950 kernels.  Arguments are validated by the C-ABI
// layer (capi.hip) before any of these is called; the launchers assume valid input.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/wamdit.h"

namespace wam {

struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  int64_t q_ts, q_bs, kv_ts, kv_bs, o_ts, o_bs;
  int32_t B, H, Dh, Lq, Lk;
  float c;  // softmax scale * log2(e)
  int32_t n_k_chunks;
  int32_t n_q_chunks;
  int32_t q_off[WAM_MAX_CHUNKS + 1];
  int32_t kend[WAM_MAX_CHUNKS];  // visible key prefix [0, kend) of each query chunk
  // device flag of the denoising loop: while *skip > 0 every workgroup exits at entry (NULL: never)
  const int32_t* skip;
};
// o_exp non-NULL (Dh = 128): the output as block-scaled E4M3 (codes at a.o, strides in bytes;
// for output row m = b * Lq + query and head h the exponents of dims 0-63 and 64-127 at
// o_exp[h * o_lde + 4 m + {0, 1}]), the bf16-rounded values quantized by the MX rule.
hipError_t launch_attn(const AttnArgs& a, hipStream_t s, uint8_t* o_exp = nullptr, int64_t o_lde = 0);

// FP8 attention (Dh = 128): a.q / a.k / a.v point at E4M3 codes (strides in bytes), a.o
// at bf16 output; q_exp / k_exp hold one uint32 per (token, head), byte j the biased
// exponent (scale 2^(byte - 127)) of dims [32 j, 32 j + 32), strides in uint32 units;
// v = code * v_scale.
struct AttnFp8Args {
  AttnArgs a;
  const void *q_exp, *k_exp;
  int64_t qe_ts, qe_bs, ke_ts, ke_bs;
  float v_scale;
};
hipError_t launch_attn_fp8(const AttnFp8Args& f, hipStream_t s, uint8_t* o_exp = nullptr, int64_t o_lde = 0);

struct GemmArgs {
  int32_t M, N, K, epi;
  const void* A;
  int64_t lda, a_bs;
  int32_t a_rows;
  const void* W;
  int64_t ldw;
  const float* bias;
  void* out;
  int64_t ldo, o_bs;
  int32_t o_rows;
  const float* gate_a;
  const float* gate_v;
  int64_t gate_stride;
  int32_t gate_rows;
  // rows r >= gate_split of a gate group (0: none) read gate_v + gate_alt instead
  int32_t gate_split;
  int64_t gate_alt;
  // FP8 operands (E4M3 A and W, one byte per element): acc * a_scale[m] * w_scale[n]
  int32_t fp8;
  const float *a_scale, *w_scale;
  // Block-scaled FP8 A (epi | WAM_EPI_MXA, a_scale NULL): one power-of-two scale per 64
  // columns of a row, an 8-bit exponent biased by 127; block kb of row m at
  // a_exp[(kb / 2) * a_lde + 4 m + kb % 2] (pairs of blocks, rows contiguous, 4 bytes
  // per row of which 2 are used; a_lde a multiple of 4)
  const uint8_t* a_exp;
  int64_t a_lde;
  // epi WAM_EPI_GELU_MX8: the bf16-rounded GELU output as E4M3 codes in out (row stride
  // ldo bytes) with one exponent per 64 columns in out_exp, laid out as a_exp (o_lde)
  uint8_t* out_exp;
  int64_t o_lde;
  // device flag of the denoising loop: while *skip > 0 every workgroup exits at entry (NULL: never)
  const int32_t* skip;
  // epi WAM_EPI_ROPE (N = 3 d, d = H * Dh a multiple of 64; row r = b * rope_L + l): the
  // bf16-rounded q|k|v row with q and k rotated as rope_qkv_kernel does, q into rope_q
  // [M][d], k and v into rope_k / rope_v row b * rope_Lcap + rope_row0 + l ([.][d])
  const float *rope_cos, *rope_sin;
  void *rope_q, *rope_k, *rope_v;
  int32_t rope_L, rope_Dh, rope_d;
  int64_t rope_Lcap, rope_row0;
};
// Internal epilogue codes beyond the public ones: the GELU output written as block-scaled
// E4M3, (or-ed in) block-scaled FP8 A, and RoPE with the K/V append (bf16 operands).
constexpr int WAM_EPI_GELU_MX8 = 4;
constexpr int WAM_EPI_ROPE = 5;
constexpr int WAM_EPI_MXA = 8;
hipError_t launch_gemm(const GemmArgs& g, hipStream_t s);
// n products sharing A (and, for FP8 operands, its row scales) and every size and stride,
// each with its own W, bias, output and (FP8) column scales, in one launch; bf16 epilogue.
constexpr int WAM_GEMM_GROUP_MAX = 48;
struct GemmGroup {
  int32_t n;
  const void* W[WAM_GEMM_GROUP_MAX];
  const float* bias[WAM_GEMM_GROUP_MAX];
  void* out[WAM_GEMM_GROUP_MAX];
  const float* w_scale[WAM_GEMM_GROUP_MAX];
};
hipError_t launch_gemm_group(const GemmArgs& g, const GemmGroup& gg, hipStream_t s);

struct LnArgs {
  int32_t rows, rows_per_batch, d;
  float eps;
  const float* x;
  const float *gamma, *beta, *shift_a, *shift_v, *scale_a, *scale_v;
  int64_t mod_stride;
  void* h;
  // rows >= seg_rows of a sample (seg_rows <= 0 or >= rows_per_batch: none) take their
  // per-sample modulation from shift_v / scale_v + alt_off
  int32_t seg_rows;
  int64_t alt_off;
  // device flag of the denoising loop: while *skip > 0 every workgroup exits at entry (NULL: never)
  const int32_t* skip;
  // FP8 output (q8 non-null; d a multiple of 512, at most 5120): instead of h, the E4M3
  // codes of the bf16 output rows (row stride ldq bytes) and their row scales, exactly as
  // launch_quant_rows would make them from h
  uint8_t* q8 = nullptr;
  int64_t ldq = 0;
  float* q_scale = nullptr;
};
hipError_t launch_ln_mod(const LnArgs& a, hipStream_t s);
// whether launch_ln_mod takes FP8 output for rows of d values
inline bool ln_fp8_supported(int d) { return d % 512 == 0 && d >= 512 && d <= 5120; }

// The combined AdaLN modulation of every block's two modulated LayerNorms, formed once per
// step: for layer l, norm k (0: shift/scale rows 0/1 of the six, 1: rows 3/4), sample b and
// segment g, out[l][k][b][g][0] = mod6_l[3k] + e0_b[3k] (shift) and [1] = mod6_l[3k+1] +
// e0_b[3k+1] (scale), d floats each; segment 1 reads e0 at +alt.  A LayerNorm given the
// shift and scale rows as its per-sample vectors (stride nseg*2*d, segment offset 2*d) then
// forms exactly the sums it forms from the four vectors.
constexpr int ADALN_FOLD_MAX_LAYERS = 64;
struct AdalnFoldArgs {
  int32_t n_layers, d, B, nseg;
  const float* e0;
  int64_t e0_stride, alt;
  const float* mod6[ADALN_FOLD_MAX_LAYERS];
  float* out;
  int64_t layer_stride;  // floats per layer: 2 * B * nseg * 2 * d
  const int32_t* skip;
};
hipError_t launch_adaln_fold(const AdalnFoldArgs& a, hipStream_t s);

struct RopeArgs {
  int32_t B, L, H, Dh, Lcap, row0;
  const void* qkv;
  const float *cos_t, *sin_t;
  void *q_out, *k_cache, *v_cache;  // q_out NULL: q is neither rotated nor stored
  // device flag of the denoising loop: while *skip > 0 every workgroup exits at entry (NULL: never)
  const int32_t* skip;
};
hipError_t launch_rope_qkv(const RopeArgs& a, hipStream_t s);

// RoPE + append for the FP8 attention (Dh = 128): r.q_out -> q codes [B*L][d] bytes with
// q_exp [B*L][d/32] bytes, r.k_cache / r.v_cache -> E4M3 code caches [B][Lcap][d] bytes
// with k_exp [B][Lcap][d/32] bytes (32-dim blocks, biased exponents); v codes E4M3(v * v_inv).
struct RopeFp8Args {
  RopeArgs r;
  void *q_exp, *k_exp;
  float v_inv;
};
hipError_t launch_rope_qkv_fp8(const RopeFp8Args& f, hipStream_t s);
// MX-style E4M3 codes of bf16 rows [rows][ldx] (cols % 32 == 0): q [rows][ldq] bytes,
// ex [rows][cols/32] biased block exponents.
hipError_t launch_quant_mx(int32_t rows, int32_t cols, const void* x, int64_t ldx, void* q, int64_t ldq, void* ex,
                           hipStream_t s);
// One-scale E4M3 codes q[i] = E4M3(x[i] * inv) of n bf16 values (n % 8 == 0).
hipError_t launch_quant_scaled(int64_t n, const void* x, float inv, void* q, hipStream_t s);

// out[b][n] = act(x[b][:]) . W[n][:] + bias[n]  (fp32 in/out, bf16 W [N][K])
enum { GEMV_ACT_NONE = 0, GEMV_ACT_SILU = 1 };
hipError_t launch_gemv(int32_t B, int32_t N, int32_t K, const float* x, int32_t act,
                       const void* W, const float* bias, float* out, hipStream_t s, const int32_t* skip = nullptr);
// [B][freq_dim] sinusoid of 1000*t
hipError_t launch_sinusoid(int32_t B, int32_t freq_dim, const float* t, float* out, hipStream_t s,
                           const int32_t* skip = nullptr);
// latent [B][C][F][Hl][Wl] bf16 -> tokens [B][F*Hg*Wg][C*4] bf16
hipError_t launch_patchify(int32_t B, int32_t C, int32_t F, int32_t Hl, int32_t Wl,
                           const void* z, void* tok, hipStream_t s, const int32_t* skip = nullptr);
// tokens [B][Lv][C*4] fp32 -> video [B][C][F][Hl][Wl] fp32
hipError_t launch_unpatchify(int32_t B, int32_t C, int32_t F, int32_t Hl, int32_t Wl,
                             const float* tok, float* out, hipStream_t s, const int32_t* skip = nullptr);

// Per-row E4M3 quantization of bf16 rows [M][K] (K % 8 == 0): q [M][ldq] bytes, scale [M].
hipError_t launch_quant_rows(int32_t M, int32_t K, const void* x, int64_t ldx, void* q, int64_t ldq, float* scale,
                             hipStream_t s, const int32_t* skip = nullptr);

// Solver step of the denoising loop over one chunk.  State x [nx][n_video + n_action]
// fp32 (nx = 1 with guidance, else B); velocity from the step outputs v_video [B][n_video]
// and v_action [B][n_action] (guidance: sample 0 cond, 1 uncond) or directly from v_in
// [nx][n]; both NULL: x unchanged.  With skip set, the device flag chooses: v_in while
// *skip > 0, else the step outputs.  v_out (optional) receives the effective velocity;
// z_next [B][n_video] / a_next [B][n_action] bf16 receive round(x) for every step sample.
struct FlowArgs {
  int32_t B, cfg;
  float cfg_scale, dt;
  int64_t n_video, n_action;
  const float *v_video, *v_action, *v_in;
  float *x, *v_out;
  void *z_next, *a_next;
  const int32_t* skip;
};
hipError_t launch_flow_step(const FlowArgs& a, hipStream_t s);
// One UniPC step over the same state: the data prediction m = x + s_v v_eff, the
// corrector (when `correct`) x_c = c_x x_last + c_new m + sum_j c_m[j] m_hist[j], then the
// predictor x <- p_x x_c + p_new m + sum_j p_m[j] m_hist[j]; x_last <- x_c, m_out <- m.
// m_hist[j] holds the data prediction j + 1 steps back (NULL where its weights are 0).
struct UnipcArgs {
  FlowArgs f;          // velocities, guidance, x, v_out, model inputs, skip flag (dt unused)
  float* x_last;
  float* m_out;
  const float* m_hist[3];
  float s_v;
  int32_t correct;
  float c_x, c_new, c_m[3];
  float p_x, p_new, p_m[2];
};
hipError_t launch_unipc_step(const UnipcArgs& a, hipStream_t s);
// cosine similarity of x and y (n floats) into out[0]; ws of cosine_workspace_bytes()
size_t cosine_workspace_bytes();
// the current device's copy of the allocation-free cosine's static scratch
// (cosine_static_scratch_bytes() bytes), its address looked up on first use
size_t cosine_static_scratch_bytes();
hipError_t cosine_static_scratch(void** ptr);
hipError_t launch_cosine(const float* x, const float* y, int64_t n, void* ws, float* out, hipStream_t s,
                         const int32_t* skip = nullptr);
// p[0..n) = v for n <= 64
hipError_t launch_fill(float* p, int n, float v, hipStream_t s);

// The loop's DiT-caching state on the device, three int32: [0] steps still to reuse
// (the flag every kernel of a step reads), [1] computed steps so far, [2] 1 if the
// latest step was computed.  init zeroes it; decide runs after step i's solver update:
// a reused step counts [0] down, a computed one (the cosine similarity cs of its velocity
// with the previous computed one, valid when [1] >= 1) sets [0] = window when cs > tau;
// computed[i] (optional) receives [2].  copy_if copies n floats while *flag != 0.
hipError_t launch_loop_init(int32_t* state, hipStream_t s);
hipError_t launch_loop_decide(int32_t* state, const float* cs, float tau, int32_t window, int32_t* computed,
                              int32_t i, hipStream_t s);
hipError_t launch_copy_if(const int32_t* flag, const float* src, float* dst, int64_t n, hipStream_t s);

}  // namespace wam
