/*
 * libwamdit — one denoising step of a block-causal video/action diffusion
 * transformer (DiT) on AMD Instinct MI355X (gfx950).
 *
 * The step is the velocity call u_theta([z_t, a_t]; KV, c, t) of the paper's
 * closed-loop inference (Appendix C, Algorithm 2, the denoising forward with
 * update=False): a chunk of K=2 latent video frames plus its action tokens
 * attends to a KV cache of earlier, clean chunks and to itself (section 3.1,
 * Model Inference; Appendix C, Figure 10b).  The KV cache is passed in and out
 * explicitly, never held by the library (Appendix D.2, the functional KV cache
 * used for graph capture).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Ownership  The caller owns every buffer, stream and event.  Tensor pointers are
 *            DEVICE pointers unless a comment says HOST.  The library allocates no
 *            memory, creates no stream and never synchronises; every call only
 *            validates its arguments on the host and enqueues kernels on `stream`.
 *            It keeps no state between calls, so calls on different streams with
 *            different workspaces may run concurrently.
 * Errors     Every entry point returns a wam_status.  All argument checks happen on
 *            the host before the first launch; on failure nothing is enqueued and
 *            wam_last_error() (thread-local) describes the problem.  WAM_EHIP means
 *            a launch was rejected by the HIP runtime (work enqueued before it in
 *            the same call may have run).  Kernel faults surface asynchronously at
 *            the caller's next synchronisation, as with any HIP kernel.
 * Dtypes     "bf16" = bfloat16 storage, round-to-nearest-even; every product is
 *            accumulated in fp32.  Weight matrices, activations, q/k/v/o, the KV
 *            cache and the text context are bf16.  The residual stream x, biases,
 *            modulation tables, LayerNorm affine, RoPE tables, timesteps and the
 *            output velocities are fp32.
 * Layouts    Row-major, token-major.  A [B][L][H][Dh] tensor is the same memory as
 *            [B][L][d] with d = H*Dh, head h at columns [h*Dh, (h+1)*Dh).  Weight
 *            matrices are PyTorch Linear layout [out][in].  Strides are in ELEMENTS.
 * Alignment  Device pointers must be 16-byte aligned; bf16 row strides must be
 *            multiples of 8 elements.
 */
#ifndef WAMDIT_H
#define WAMDIT_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WAM_ABI_VERSION 7
#define WAM_MAX_CHUNKS 16

typedef enum {
  WAM_OK = 0,
  WAM_EINVAL = 1,        /* bad argument: null/misaligned pointer, inconsistent sizes */
  WAM_EUNSUPPORTED = 2,  /* well-formed but outside what the kernels implement      */
  WAM_EWORKSPACE = 3,    /* workspace missing or smaller than the query function says */
  WAM_EHIP = 4           /* the HIP runtime rejected a launch                          */
} wam_status;

/* Thread-local, human-readable detail of the last non-OK status of this thread. */
const char* wam_last_error(void);
int32_t wam_abi_version(void);

/* ------------------------------------------------------------------------------
 * Chunk layout of one attention call (Appendix C, Figure 10b; section 3.1).
 *
 * Key rows are grouped into chunks in order: key chunk j holds key rows
 * [k_off[j], k_off[j+1]).  Query rows are grouped likewise into query chunks; query
 * chunk i holds query rows [q_off[i], q_off[i+1]) and carries the global chunk id
 * q_chunk_id[i].  A query of chunk id c sees exactly the keys of key chunks j <= c:
 * the clean cached chunks before it and its own chunk; attention inside a chunk is
 * bidirectional.  So the visible keys of a query form the prefix [0, k_off[c+1]).
 *
 * Requirements (else WAM_EINVAL): 1 <= n_k_chunks, n_q_chunks <= WAM_MAX_CHUNKS;
 * k_off[0] = 0, non-decreasing, k_off[n_k_chunks] = Lk; q_off[0] = 0,
 * non-decreasing, q_off[n_q_chunks] = Lq; 0 <= q_chunk_id[i] < n_k_chunks,
 * non-decreasing in i; every non-empty query chunk sees at least one key.
 *
 * Cached denoising (one query chunk that is the last key chunk) masks nothing.
 * ------------------------------------------------------------------------------ */
typedef struct {
  int32_t n_k_chunks;
  int32_t k_off[WAM_MAX_CHUNKS + 1];
  int32_t n_q_chunks;
  int32_t q_off[WAM_MAX_CHUNKS + 1];
  int32_t q_chunk_id[WAM_MAX_CHUNKS];
} wam_chunks;

/* ------------------------------------------------------------------------------
 * wam_attn_blockcausal — block-causal softmax attention (the rule above).
 *
 *   o[b, i, h, :] = sum_j softmax_j(scale * q[b,i,h,:] . k[b,j,h,:]) v[b,j,h,:]
 *                   over the keys j visible to query i.
 *
 * q: [B] x [Lq] tokens x [H][Dh] bf16, token stride q_tok_stride, batch stride
 * q_batch_stride; k, v: [B] x [Lk] x [H][Dh] bf16 sharing kv_tok_stride and
 * kv_batch_stride (k and v may be two halves of one [.., 2*d] buffer); o: written,
 * [B] x [Lq] x [H][Dh] bf16.  scale <= 0 selects 1/sqrt(Dh).  Dh must be 64 or 128.
 * Lq = 0 or B = 0 is a no-op.  o must not overlap q, k or v.  One sample's keys
 * must span less than 2 GiB (Lk * kv_tok_stride * 2 bytes < 2^31; else
 * WAM_EUNSUPPORTED).  Deterministic: the same inputs give bitwise the same output
 * (no atomics, no split-K).
 * ------------------------------------------------------------------------------ */
typedef struct {
  int32_t B, H, Dh, Lq, Lk;
  int64_t q_tok_stride, q_batch_stride;
  int64_t kv_tok_stride, kv_batch_stride;
  int64_t o_tok_stride, o_batch_stride;
  float scale;
  wam_chunks ch;
} wam_attn_desc;

wam_status wam_attn_blockcausal(const wam_attn_desc* desc, const void* q, const void* k,
                                const void* v, void* o, hipStream_t stream);

/* ------------------------------------------------------------------------------
 * FP8 attention operands (section 3.2.4 and Appendix D.2 run QKV and the softmax in FP8;
 * the formats below are this library's reading).  E4M3 is the OCP 8-bit float (bias 7,
 * largest 448, no infinities), rounded to nearest even.
 *   MX blocks (q, k): 32 consecutive elements share a power-of-two scale 2^e with e the
 *     smallest integer such that max|x| <= 448 * 2^e (clamped to [-127, 127]; 0 for a
 *     zero block), stored as the byte e + 127; codes E4M3(x * 2^-e).  A head of Dh = 128
 *     has four blocks, so its exponents form one uint32 (byte j: dims [32j, 32j+32)).
 *   One scale (v): codes E4M3(fp32(x * fp32(1 / scale))), saturating at +-448.
 *
 * wam_quantize_mx_fp8 — MX codes of bf16 rows x [rows][ldx] (cols % 32 == 0, ldx % 8 ==
 *   0, x 16-byte aligned): q8 [rows][ldq] bytes (ldq % 8 == 0, 8-byte aligned), exps
 *   [rows][cols/32] bytes, contiguous.
 * wam_quantize_scaled_fp8 — one-scale codes of n bf16 values (n % 8 == 0).
 * ------------------------------------------------------------------------------ */
wam_status wam_quantize_mx_fp8(int32_t rows, int32_t cols, const void* x, int64_t ldx, void* q8,
                               int64_t ldq, void* exps, hipStream_t stream);
wam_status wam_quantize_scaled_fp8(int64_t n, const void* x, float scale, void* q8,
                                   hipStream_t stream);

/* wam_attn_blockcausal_fp8 — the attention of wam_attn_blockcausal (same chunk rule and
 * descriptor) on FP8 operands, Dh = 128 only:
 *   q8, k8, v8  E4M3 codes addressed like the bf16 operands with one byte per element
 *               (strides in bytes, multiples of 128; 16-byte aligned);
 *   q_exp, k_exp  uint32 block exponents of q and k, one per (token, head), addressed
 *               with the code strides divided by 128 (4-byte aligned);
 *   v_scale     v = code * v_scale;  o  bf16 as in wam_attn_blockcausal.
 * Scores use the exact products of the decoded q and k (fp32 accumulation); the
 * probabilities are rounded to E4M3 before the value product, relative to a running
 * maximum that is raised whenever a tile exceeds it by 2^2 in the exp2 domain (so they
 * stay below 2^8 after a fixed 2^6 scaling), and the normaliser is the sum of those
 * rounded probabilities.  Deterministic. */
wam_status wam_attn_blockcausal_fp8(const wam_attn_desc* desc, const void* q8, const void* q_exp,
                                    const void* k8, const void* k_exp, const void* v8, float v_scale,
                                    void* o, hipStream_t stream);

/* ------------------------------------------------------------------------------
 * Model dimensions.  d = H*Dh, d % 256 == 0, Dh in {64, 128}; latent_ch*4 patch
 * features per token (1x2x2 patches); act_dim action features; text_dim text
 * feature width; freq_dim sinusoid width (even); eps the LayerNorm epsilon.
 * ------------------------------------------------------------------------------ */
typedef struct {
  int32_t d, H, Dh, ffn, n_layers, latent_ch, act_dim, text_dim, freq_dim;
  float eps;
} wam_dims;

/* Per-block weights.  Matrices bf16 [out][in]:
 *   w_qkv [3d][d] (rows: q | k | v), w_o [d][d], w_cq [d][d], w_ckv [2d][d] (k | v),
 *   w_co [d][d], w_f1 [ffn][d], w_f2 [d][ffn].
 * Vectors fp32: every b_* of its matrix's out size (NULL = zero bias); mod6 [6][d]
 * the block's modulation table added to the per-sample time modulation e0, rows
 * (shift1, scale1, gate1, shift2, scale2, gate2); lnc_gamma, lnc_beta [d] the affine
 * of the cross-attention LayerNorm (NULL = 1 and 0). */
typedef struct wam_block_fp8 wam_block_fp8;
typedef struct {
  const void *w_qkv, *w_o, *w_cq, *w_ckv, *w_co, *w_f1, *w_f2;
  const float *b_qkv, *b_o, *b_cq, *b_ckv, *b_co, *b_f1, *b_f2;
  const float* mod6;
  const float *lnc_gamma, *lnc_beta;
  const wam_block_fp8* fp8;  /* optional FP8 copies of the seven projections (below) */
} wam_block_weights;

/* FP8 copies of a block's projections: E4M3 [out][in] contiguous (each bf16 matrix's rows
 * quantized with wam_quantize_rows_fp8) with their per-output-channel scales.  When a
 * block's weights carry them, its seven projections (QKV, O, cross-Q, cross-K|V, cross-O,
 * FFN1, FFN2) run as FP8 GEMMs: every activation is quantized per row into the workspace
 * right before its projection; LayerNorm, RoPE, both attentions, the epilogues and the
 * fp32 residual are unchanged (the bf16 matrices are then not read). */
struct wam_block_fp8 {
  const void *w_qkv, *w_o, *w_cq, *w_ckv, *w_co, *w_f1, *w_f2;
  const float *s_qkv, *s_o, *s_cq, *s_ckv, *s_co, *s_f1, *s_f2;
};

/* ------------------------------------------------------------------------------
 * wam_dit_block_fwd — one DiT block over the current rows (in place on x).
 *
 *   m = mod6 + e0[b];  (sh1, sc1, g1, sh2, sc2, g2) = rows of m
 *   qkv = (LN(x)(1+sc1)+sh1) W_qkv^T + b_qkv;  q, k <- 3D RoPE (tables rope_cos/sin)
 *   k, v of the current rows -> cache rows [cache_len, cache_len + L)
 *   x += g1 * (Attn(q, cache rows [0, cache_len+L), chunks ch) W_o^T + b_o)
 *   x += Attn((LN(x)*gamma+beta) W_cq^T + b_cq, ctx W_ckv^T + b_ckv) W_co^T + b_co
 *   x += g2 * (gelu_tanh((LN(x)(1+sc2)+sh2) W_f1^T + b_f1) W_f2^T + b_f2)
 *
 * x      [B][L][d] fp32 residual, read and updated in place.
 * e0     [B][6][d] fp32 per-sample time modulation.
 * rope_cos, rope_sin  [L][Dh/2] fp32, built with wam_rope_tables for the rows'
 *        positions (all samples share positions).
 * k_cache, v_cache  [B][Lcap][H][Dh] bf16, K stored after RoPE.  Rows
 *        [0, cache_len) are read; rows [cache_len, cache_len+L) are overwritten with
 *        the current rows' K and V.  The caller advances cache_len by L only for a
 *        cache-update pass; a denoising step leaves it, so the next step overwrites
 *        the same rows.  cache_len + L <= Lcap.
 * ch     key/query chunks of the self-attention: Lk = cache_len + L, Lq = L.
 * ctx    [B][Lc][d] bf16 projected text; or ctx_kv [B][Lc][2d] bf16 its cross K|V
 *        already projected with this block's w_ckv (then ctx may be NULL and w_ckv
 *        is not read).
 * ws     device workspace of at least wam_block_workspace_bytes(...) bytes,
 *        256-byte aligned; its contents on entry do not matter.
 * ------------------------------------------------------------------------------ */
typedef struct {
  float* x;
  const float* e0;
  const float *rope_cos, *rope_sin;
  void *k_cache, *v_cache;
  int32_t Lcap, cache_len;
  wam_chunks ch;
  const void* ctx;
  const void* ctx_kv;
  int32_t B, L, Lc;
  void* k_exp;     /* optional: an FP8 KV cache (Dh = 128): k_cache / v_cache then hold E4M3 */
  float v_scale;   /* codes [B][Lcap][H][Dh] bytes, k_exp [B][Lcap][H] uint32 the K block  */
                   /* exponents, v = code * v_scale; the self-attention runs in FP8        */
} wam_block_io;

size_t wam_block_workspace_bytes(const wam_dims* dims, int32_t B, int32_t L, int32_t Lc);
wam_status wam_dit_block_fwd(const wam_dims* dims, const wam_block_weights* w,
                             const wam_block_io* io, void* ws, size_t ws_bytes,
                             hipStream_t stream);

/* ------------------------------------------------------------------------------
 * Model-level weights (bf16 [out][in] matrices, fp32 vectors, NULL bias = 0):
 *   time MLP   w_t1 [d][freq_dim], w_t2 [d][d], w_t6 [6d][d]
 *              e = W_t2 silu(W_t1 sinusoid(t) + b_t1) + b_t2;  e0 = W_t6 silu(e) + b_t6
 *   text proj  w_x1 [d][text_dim], w_x2 [d][d]:  ctx = W_x2 gelu_tanh(W_x1 text + b_x1) + b_x2
 *   embed      w_patch [d][latent_ch*4] on patchified latents, w_ain [d][act_dim]
 *   head       head_mod2 [2][d] (shift, scale) added to e;
 *              w_hv [latent_ch*4][d] (unpatchified), w_ha [act_dim][d]
 * blocks is a HOST array of n_layers block weight sets.
 * ------------------------------------------------------------------------------ */
typedef struct {
  wam_dims dims;
  const wam_block_weights* blocks;
  const void *w_t1, *w_t2, *w_t6, *w_x1, *w_x2, *w_patch, *w_ain, *w_hv, *w_ha;
  const float *b_t1, *b_t2, *b_t6, *b_x1, *b_x2, *b_patch, *b_ain, *b_hv, *b_ha;
  const float* head_mod2;
} wam_model;

/* ------------------------------------------------------------------------------
 * wam_dit_step_fwd — one denoising step u_theta([z_t, a_t]; KV, c, t) of one chunk
 * (Algorithm 2, the forward inside the denoising loop).
 *
 * z_t      [B][latent_ch][F][Hl][Wl] bf16 noisy latents (Hl, Wl even); the chunk's
 *          video tokens are its 1x2x2 patches, frame-major, then row, then column
 *          (Lv = F*Hl/2*Wl/2), followed by its A action tokens: L = Lv + A.
 * a_t      [B][A][act_dim] bf16 noisy actions.
 * t        [B] fp32 timestep per sample (one per chunk, section 3.1).
 * text     [B][Lc][text_dim] bf16 text features.
 * k_cache, v_cache  HOST arrays of n_layers device pointers, each [B][Lcap][H][Dh]
 *          bf16, semantics as in wam_dit_block_fwd.
 * ctx_kv   optional HOST array of n_layers device pointers [B][Lc][2d] bf16 holding
 *          each block's precomputed cross K|V of this text (NULL: computed here, for
 *          every block before the first one, into the workspace: n_layers*B*Lc*2d bf16
 *          of the size wam_step_workspace_bytes reports; the same products as one GEMM
 *          per block, batched so that they fill the GPU).
 * rope_cos, rope_sin  [L][Dh/2] fp32 tables of the rows' positions.
 * ch       self-attention chunks (Lk = cache_len + L, Lq = L).
 * v_video  written, [B][latent_ch][F][Hl][Wl] fp32;  v_action  written, [B][A][act_dim] fp32.
 * attn_events  optional HOST array of 2*n_layers hipEvent_t: when non-NULL,
 *          events[2l] and events[2l+1] are recorded on `stream` just before and just
 *          after block l's self-attention kernel (for per-kernel timing).
 * block_events optional HOST array of 2*WAM_BLOCK_EVENTS*n_layers hipEvent_t: when
 *          non-NULL, events[(l*WAM_BLOCK_EVENTS + k)*2] and [.. + 1] are recorded just
 *          before and just after launch k (wam_block_event) of block l.  A projection
 *          with FP8 weights includes its activation quantization.  Recording ~24 events
 *          per block adds launch gaps: meant for profiling steps, not timed ones.
 * t_action optional [B] fp32 device: the action tokens' own timestep (DreamZero-Flash,
 *          Appendix D.3).  When non-NULL (and A > 0) the action rows' AdaLN modulation,
 *          gates and head modulation come from t_action's time embedding and the video
 *          rows' from t's; NULL: every row uses t.
 * ------------------------------------------------------------------------------ */
/* The launches of a block, in order, that wam_step_io.block_events brackets. */
typedef enum {
  WAM_EV_LN1 = 0,        /* AdaLN #1                                   */
  WAM_EV_QKV = 1,        /* fused QKV projection (bf16 operands and cache, d % 64 == 0:
                            with RoPE and the KV-cache append in its epilogue) */
  WAM_EV_ROPE = 2,       /* 3D RoPE + KV-cache append (brackets no launch when the QKV
                            projection applies them)                          */
  WAM_EV_SELF_ATTN = 3,  /* block-causal self-attention                */
  WAM_EV_O = 4,          /* output projection + gated residual         */
  WAM_EV_LNC = 5,        /* cross-attention LayerNorm                  */
  WAM_EV_CQ = 6,         /* cross-attention query projection           */
  WAM_EV_CROSS_ATTN = 7, /* cross-attention over the text              */
  WAM_EV_CO = 8,         /* cross-attention output projection + residual */
  WAM_EV_LN2 = 9,        /* AdaLN #2                                   */
  WAM_EV_FFN1 = 10,      /* FFN up-projection + tanh-GELU              */
  WAM_EV_FFN2 = 11,      /* FFN down-projection + gated residual       */
  WAM_BLOCK_EVENTS = 12
} wam_block_event;

typedef struct {
  const void* z_t;
  const void* a_t;
  const float* t;
  const void* text;
  void* const* k_cache;
  void* const* v_cache;
  const void* const* ctx_kv;
  const float *rope_cos, *rope_sin;
  int32_t B, F, Hl, Wl, A, Lc, Lcap, cache_len;
  wam_chunks ch;
  float* v_video;
  float* v_action;
  hipEvent_t* attn_events;
  const float* t_action;
  void* const* k_exp;     /* optional HOST array of n_layers FP8 K exponent caches (then   */
  const float* v_scale;   /* k_cache / v_cache hold E4M3 codes; v_scale HOST [n_layers]),  */
                          /* as in wam_block_io                                            */
  hipEvent_t* block_events;
} wam_step_io;

size_t wam_step_workspace_bytes(const wam_model* m, const wam_step_io* io);
wam_status wam_dit_step_fwd(const wam_model* m, const wam_step_io* io, void* ws,
                            size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------------
 * wam_dit_update_fwd — the cache-update pass u_theta([z, a]; KV, c, t, update=True)
 * (Algorithm 2: the context prefill, and the injection of each real observation after
 * a chunk is executed).
 *
 * Same wam_step_io as wam_dit_step_fwd, with z_t holding CLEAN latents and t the
 * timestep the caller uses for clean content (the library does not interpret t).
 * Algorithm 2 passes no actions (A = 0); A > 0 is accepted and appends the action
 * rows too.  The call writes, for every layer l, the K (after RoPE) and V of the
 * L = Lv + A current rows into rows [cache_len, cache_len + L) of k_cache[l] and
 * v_cache[l]; no other cache row and no output buffer is written (v_video and
 * v_action are ignored and may be NULL).  The caller then advances its cache_len by L.
 *
 * Several chunks may be appended in one call: z_t holds their frames back to back,
 * ch lists them as query chunks (each row sees the cached chunks and the current rows
 * of its own and earlier chunks, Figure 10b) and rope_cos/rope_sin give every row its
 * own position.  The head is skipped and the last layer stops after its K/V
 * projection (nothing downstream reads the rest).  Validation, errors and
 * asynchronous semantics are those of wam_dit_step_fwd; attn_events, when non-NULL,
 * holds 2*n_layers events of which the last layer's pair is left unrecorded.
 * ------------------------------------------------------------------------------ */
size_t wam_update_workspace_bytes(const wam_model* m, const wam_step_io* io);
wam_status wam_dit_update_fwd(const wam_model* m, const wam_step_io* io, void* ws,
                              size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------------
 * The denoising loop around the step (Algorithm 2): the noisy chunk moves along the
 * straight path of Eq. 2 from t = 0 (noise) to t = 1 (clean) by explicit Euler steps
 * x <- x + (t_next - t) v, or by UniPC (below), optionally with classifier-free guidance
 * v = v_u + s (v_c - v_u) and DiT caching (Appendix D.1).
 *
 * The state x is fp32 [nx][n_video + n_action] per chunk: the latent elements
 * (latent_ch*F*Hl*Wl, in z_t's order) followed by the action elements (A*act_dim);
 * nx = 1 with guidance (the pair shares one state), else B.
 * ------------------------------------------------------------------------------ */
typedef struct {
  int32_t B;          /* samples per network call (the step's batch) */
  int32_t cfg;        /* 1: guidance pair, B == 2, sample 0 conditional, sample 1 unconditional */
  float cfg_scale;    /* s */
  int64_t n_video;    /* latent elements per sample */
  int64_t n_action;   /* action elements per sample */
} wam_flow_dims;

/* One solver step: v_eff from the step outputs v_video [B][n_video] / v_action
 * [B][n_action] (fp32, device), combined by guidance when cfg, or taken directly from
 * v_in [nx][n] (a cached velocity; then v_video / v_action are ignored); all three NULL
 * leaves x unchanged.  x += (t_next - t) v_eff in place; v_out (optional, [nx][n])
 * receives v_eff; z_next [B][n_video] and a_next [B][n_action] (bf16, the next step's
 * z_t / a_t) receive round-to-nearest-even(x) for every sample (both halves of a
 * guidance pair).  Asynchronous; no workspace. */
wam_status wam_flow_step(const wam_flow_dims* d, const float* v_video, const float* v_action,
                         const float* v_in, float* x, float* v_out, float t, float t_next,
                         void* z_next, void* a_next, hipStream_t stream);

/* UniPC, the multistep predictor-corrector solver the paper deploys (Flow-UniPC; its
 * formulas are those of Zhao et al., 2023, in the data-prediction form with
 * B(h) = e^h - 1), on the straight path: alpha_t = t, sigma_t = 1 - t,
 * lambda = log(t / (1 - t)), and the data prediction of velocity v at state x and time t
 * is m = x + (1 - t) v.  Step i (from t_i to t_(i+1)) first corrects the state at t_i
 * with the new prediction m_i (every step after the first; no extra network call), then
 * predicts the state at t_(i+1) from m_i and up to two earlier predictions.  The order
 * warms up as min(order, i + 1) and is 1 for a step that ends at t = 1 (which returns
 * its data prediction); UniPC of order p converges at order p + 1.  The schedule must
 * satisfy 0 < t_0 < t_1 < ... < t_N <= 1.
 *
 * wam_unipc_plan (HOST, no GPU work) writes one wam_unipc_coef per step: the step's
 * weights, computed in double precision and stored as fp32.  wam_unipc_step applies
 * step `step` to the state (device, fp32 [nx][n], as wam_flow_step):
 *   m     = x + s_v v_eff                       (v_eff as in wam_flow_step)
 *   x_c   = correct ? c_x x_last + c_new m + sum_q c_m[q] m_(step-1-q) : x
 *   x     = p_x x_c + p_new m + sum_q p_m[q] m_(step-1-q)
 *   x_last = x_c;  m_ring[step % 4] = m;  z_next / a_next = bf16(x) as in wam_flow_step
 * m_ring: 4 device buffers of nx*n fp32 owned by the caller; m_j lives in m_ring[j % 4],
 * so steps must be applied in order on one stream.  x_last: one more such buffer.
 * Errors: WAM_EINVAL for a bad schedule or order, NULL buffers a step needs, or a
 * correcting first step. */
typedef struct {
  float s_v;          /* 1 - t_i */
  int32_t correct;    /* 1: apply the corrector */
  float c_x, c_new;   /* corrector weights of x_last and m_i */
  float c_m[3];       /* corrector weights of m_(i-1), m_(i-2), m_(i-3) */
  float p_x, p_new;   /* predictor weights of x_c and m_i */
  float p_m[2];       /* predictor weights of m_(i-1), m_(i-2) */
} wam_unipc_coef;
wam_status wam_unipc_plan(const float* t_sched, int32_t n_steps, int32_t order,
                          wam_unipc_coef* out);
wam_status wam_unipc_step(const wam_flow_dims* d, const float* v_video, const float* v_action,
                          const float* v_in, float* x, float* x_last, float* const* m_ring,
                          int32_t step, const wam_unipc_coef* c, float* v_out, void* z_next,
                          void* a_next, hipStream_t stream);

/* Cosine similarity <a, b> / (|a| |b|) of n fp32 values into out[0] (device; 0 when a
 * norm is 0), accumulated in fp64 in a fixed order (deterministic).  ws of
 * wam_cosine_workspace_bytes() device bytes. */
size_t wam_cosine_workspace_bytes(void);
wam_status wam_cosine_similarity(const float* a, const float* b, int64_t n, void* ws,
                                 size_t ws_bytes, float* out, hipStream_t stream);

/* wam_cosine_similarity without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses that forbid
 * hipMalloc): the same kernels and the same result, bit for bit, with the partial sums
 * in a static device array of the library (12 KiB per GPU, the fixed 512 x 3 fp64
 * partials of the reduction whatever n is; each GPU the library runs on holds its copy
 * until the process ends).  Nothing in it needs clearing: every call writes all
 * partials before reading them.  The call allocates nothing and uses the current
 * device's copy (its address looked up on the first call on that device), so `stream`
 * must belong to the current device.  Every call on one GPU shares that copy: calls that
 * overlap in time on one GPU (on different streams, or from different threads without
 * ordering) race and may return wrong values; calls ordered on one stream do not.
 * WAM_EWORKSPACE if the library's partials outgrow the array (a build mismatch). */
wam_status wam_cosine_similarity_noalloc(const float* a, const float* b, int64_t n,
                                         float* out, hipStream_t stream);

typedef struct {
  int32_t n_steps;        /* N >= 1 solver steps */
  const float* t_sched;   /* HOST [N + 1] scheduler times t_0 .. t_N */
  int32_t cfg;            /* guidance pair (io->B == 2) */
  float cfg_scale;
  float cache_tau;        /* DiT caching: after a computed step whose velocity has cosine  */
  int32_t cache_window;   /* similarity > cache_tau with the previous computed one, the next */
                          /* cache_window steps reuse it; cache_window = 0: caching off     */
  float* x;               /* device fp32 state [nx][n_video + n_action]: noise in, x_N out */
  int32_t* computed;      /* optional DEVICE [N] int32: 1 where step i called the network    */
  int32_t solver;         /* WAM_SOLVER_EULER or WAM_SOLVER_UNIPC                            */
  int32_t solver_order;   /* UniPC order 1..3 (ignored by Euler)                             */
} wam_denoise_params;
#define WAM_SOLVER_EULER 0
#define WAM_SOLVER_UNIPC 1

/* wam_denoise_chunk — the N-step denoising loop of one chunk: per step, the network
 * call wam_dit_step_fwd(io) at t_i (io->t [B] is written by the loop; io->z_t and
 * io->a_t are rewritten from x before every call; io->v_video / v_action receive the
 * step's raw velocities), then wam_flow_step (or wam_unipc_step, with the weights of
 * wam_unipc_plan and the history buffers in the workspace: 5 * nx * n fp32 more).  A
 * reused step's velocity enters UniPC like a computed one.  The cache rows [cache_len, cache_len+L)
 * are rewritten by every computed step, as by a single step.  The text conditions every
 * step alike, so when io->ctx_kv is NULL the loop projects the text and each block's
 * cross-attention K|V once, before the first step, into its workspace (n_layers * B *
 * Lc * 2d bf16 more) and every step reads them; results are those of independent
 * steps.  DiT caching is decided on the device: after each computed step the cosine
 * similarity of its velocity with the previous computed one is reduced on the GPU, and a
 * reused step's kernels read that decision from the workspace and return at entry.  The
 * loop never synchronizes or allocates, so a caller can capture a whole call in a graph
 * (the schedule t_sched is read on the host when the call is made, or captured).  Same
 * validation and errors as wam_dit_step_fwd, plus the loop's own parameters. */
size_t wam_denoise_workspace_bytes(const wam_model* m, const wam_step_io* io,
                                   const wam_denoise_params* p);
wam_status wam_denoise_chunk(const wam_model* m, const wam_step_io* io, const wam_denoise_params* p,
                             void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------------
 * Pieces of the step, exported for testing each kernel on its own.
 * ------------------------------------------------------------------------------ */

/* Time embedding: e [B][d] and e0 [B][6][d] (fp32) from t [B].  ws >= B*(freq_dim+d)*4 bytes. */
size_t wam_time_embed_workspace_bytes(const wam_dims* dims, int32_t B);
wam_status wam_time_embed_fwd(const wam_model* m, int32_t B, const float* t, float* e,
                              float* e0, void* ws, size_t ws_bytes, hipStream_t stream);

/* Text projection: ctx [B*Lc][d] bf16 from text [B*Lc][text_dim] bf16.
 * ws >= B*Lc*d*2 bytes (the GELU hidden). */
size_t wam_text_proj_workspace_bytes(const wam_dims* dims, int32_t B, int32_t Lc);
wam_status wam_text_proj_fwd(const wam_model* m, int32_t B, int32_t Lc, const void* text,
                             void* ctx, void* ws, size_t ws_bytes, hipStream_t stream);

/* LayerNorm over rows of d fp32 values, then optional affine and modulation, to bf16:
 *   h[b,r,:] = ((x - mean)/sqrt(var + eps) * gamma + beta) * (1 + scale_b) + shift_b
 * with shift_b = shift_a + shift_v[b*mod_stride .. ] (likewise scale).  Rows are
 * [B][rows_per_batch] with row stride d (x) and d (h).  gamma/beta NULL = 1/0; a
 * NULL shift_a/shift_v (scale_a/scale_v) contributes 0. */
wam_status wam_adaln_ln_mod(int32_t B, int32_t rows_per_batch, int32_t d, float eps,
                            const float* x, const float* gamma, const float* beta,
                            const float* shift_a, const float* shift_v,
                            const float* scale_a, const float* scale_v, int64_t mod_stride,
                            void* h, hipStream_t stream);

/* 3D RoPE on a fused QKV projection and KV-cache append.
 * qkv [B][L][3][H][Dh] bf16 (q | k | v per token); rope_cos/sin [L][Dh/2] fp32.
 * Writes q_out [B][L][H][Dh] (rotated q), rotated k into k_cache rows
 * [row0, row0+L) and v into v_cache rows [row0, row0+L) of [B][Lcap][H][Dh]. */
wam_status wam_rope_qkv(int32_t B, int32_t L, int32_t H, int32_t Dh, const void* qkv,
                        const float* rope_cos, const float* rope_sin, void* q_out,
                        void* k_cache, void* v_cache, int32_t Lcap, int32_t row0,
                        hipStream_t stream);

/* wam_rope_qkv_fp8 — the same rotation and append into an FP8 cache (Dh = 128): the
 * rotated q (fp32) as MX codes q8 [B][L][H][Dh] bytes with exponents q_exp [B][L][H]
 * uint32 (both NULL: q is not written), the rotated k as MX codes into rows
 * [row0, row0+L) of k8_cache [B][Lcap][H][Dh] bytes and k_exp [B][Lcap][H] uint32, v as
 * one-scale codes (v_scale) into v8_cache.  Formats as for wam_quantize_mx_fp8. */
wam_status wam_rope_qkv_fp8(int32_t B, int32_t L, int32_t H, int32_t Dh, const void* qkv,
                            const float* rope_cos, const float* rope_sin, void* q8, void* q_exp,
                            void* k8_cache, void* k_exp, void* v8_cache, float v_scale,
                            int32_t Lcap, int32_t row0, hipStream_t stream);

/* GEMM with fused epilogue: acc[m][n] = sum_k A[m][k] W[n][k] (bf16 in, fp32 acc),
 * v = acc + bias[n] (bias NULL = 0), then by epilogue:
 *   WAM_EPI_BF16         out_bf16[m][n] = v
 *   WAM_EPI_GELU_BF16    out_bf16[m][n] = gelu_tanh(v)
 *   WAM_EPI_RESID_F32    out_f32[m][n] += g * v, g = gate_a[n] + gate_v[(m / gate_rows)*gate_stride + n]
 *                        (both gate pointers NULL: g = 1)
 *   WAM_EPI_F32          out_f32[m][n] = v
 * Row m of A is at A + (m / a_rows)*a_batch_stride + (m % a_rows)*lda and row m of
 * out at out + (m / out_rows)*out_batch_stride + (m % out_rows)*ldo (a_rows or
 * out_rows = 0: plain, i.e. row m at m*lda / m*ldo).  K % 8 == 0; lda, ldw and
 * a_batch_stride multiples of 8; ldo, out_batch_stride and gate_stride multiples of 4;
 * bias and gate pointers 16-byte aligned.  The rows of A read and all of W must each
 * span less than 2 GiB from their base pointer (else WAM_EUNSUPPORTED). */
enum { WAM_EPI_BF16 = 0, WAM_EPI_GELU_BF16 = 1, WAM_EPI_RESID_F32 = 2, WAM_EPI_F32 = 3 };
typedef struct {
  int32_t M, N, K, epilogue;
  const void* A;
  int64_t lda, a_batch_stride;
  int32_t a_rows;
  const void* W;
  int64_t ldw;
  const float* bias;
  void* out;
  int64_t ldo, out_batch_stride;
  int32_t out_rows;
  const float *gate_a, *gate_v;
  int64_t gate_stride;
  int32_t gate_rows;
} wam_gemm_desc;

wam_status wam_gemm_bf16(const wam_gemm_desc* g, hipStream_t stream);

/* ------------------------------------------------------------------------------
 * FP8 (E4M3) operands.  The paper's deployment quantizes to FP8 E4M3 (Appendix D.2);
 * here E4M3 is the OCP 8-bit float (bias 7, 3 mantissa bits, largest 448, no
 * infinities).
 *
 * wam_quantize_rows_fp8: per-row quantization of bf16 x [M][K] (row stride ldx, K and
 * ldx multiples of 8): scale[m] = max_k |x[m][k]| / 448 (1 for an all-zero row) and
 * q[m][k] = E4M3(x[m][k] * (448 / max_k |x[m][k]|)) rounded to nearest, ties to even
 * (fp32 arithmetic); q has row stride ldq bytes (a multiple of 16).  Used for
 * activations (per token) and for weights (per output channel, rows of W [N][K]).
 *
 * wam_gemm_fp8: the GEMM of wam_gemm_bf16 with E4M3 operands: A [M][K] and W [N][K]
 * bytes (lda, ldw, a_batch_stride and K multiples of 16), fp32 accumulation of the
 * exact products, then v = acc * a_scale[m] * w_scale[n] + bias[n] and the same
 * epilogues.  a_scale [M] and w_scale [N] fp32 device arrays are required.
 * ------------------------------------------------------------------------------ */
wam_status wam_quantize_rows_fp8(int32_t M, int32_t K, const void* x, int64_t ldx, void* q,
                                 int64_t ldq, float* scale, hipStream_t stream);

/* wam_adaln_ln_mod_fp8: the LayerNorm of wam_adaln_ln_mod (same arguments and arithmetic)
 * whose bf16 output rows are not stored but quantized as wam_quantize_rows_fp8 would
 * quantize them: the E4M3 codes into q [B*rows_per_batch][ldq bytes] (ldq >= d, a multiple
 * of 16) and the row scales into scale [B*rows_per_batch], bit for bit the two calls' result,
 * in one pass that writes a byte per element.  This is how an FP8 projection's input is
 * made when the LayerNorm output feeds nothing else (the paper quantizes the DiT's
 * projections to FP8 for deployment, Section 3.2.4, Appendix D.2).  d must be a multiple of
 * 512 in [512, 5120] (else WAM_EUNSUPPORTED). */
wam_status wam_adaln_ln_mod_fp8(int32_t B, int32_t rows_per_batch, int32_t d, float eps,
                                const float* x, const float* gamma, const float* beta,
                                const float* shift_a, const float* shift_v,
                                const float* scale_a, const float* scale_v, int64_t mod_stride,
                                void* q, int64_t ldq, float* scale, hipStream_t stream);
wam_status wam_gemm_fp8(const wam_gemm_desc* g, const float* a_scale, const float* w_scale,
                        hipStream_t stream);

/* wam_gemm_fp8_mx: wam_gemm_fp8 with block-scaled activations on one side of it, for a
 * projection whose input another projection produces (the FFN's hidden activations; the
 * paper's deployment runs the DiT's projections in FP8, Section 3.2.4, Appendix D.2).  A
 * block is 64 consecutive columns of a row with one power-of-two scale 2^(e - 127), e an
 * 8-bit exponent, chosen as for wam_quantize_mx_fp8 (the smallest with max|block| <= 448 *
 * 2^(e-127)); the exponents of blocks kb of row m sit at exps[(kb / 2) * lde + 4 m + kb % 2]
 * (per pair of blocks all rows in order, 4 bytes per row of which the first 2 are used;
 * lde a multiple of 4, >= 4 M; exps 4-byte aligned).
 *   a_exp (a_scale NULL): A's E4M3 codes are block-scaled, acc[m][n] = sum_k A[m][k]
 *     2^(e(m, k / 64) - 127) W[n][k] (fp32 accumulation of exact products), v = acc *
 *     w_scale[n] + bias[n], epilogue WAM_EPI_BF16 or WAM_EPI_RESID_F32; K % 128 == 0,
 *     a_rows == 0.  (Otherwise a_scale as for wam_gemm_fp8.)
 *   out_exp (epilogue WAM_EPI_GELU_BF16, with a_scale): the GELU output, rounded to bf16 as
 *     that epilogue stores it, is written block-scaled instead: E4M3 codes into out (one
 *     byte per element, row stride ldo bytes, 4-byte aligned) and the exponents into
 *     out_exp (stride o_lde), bit for bit wam_quantize_mx_fp8's rule over 64-column
 *     blocks of the bf16 output; N % 128 == 0, out_rows == 0.
 * Both a_exp and out_exp: WAM_EUNSUPPORTED. */
wam_status wam_gemm_fp8_mx(const wam_gemm_desc* g, const float* a_scale, const void* a_exp, int64_t a_lde,
                           const float* w_scale, void* out_exp, int64_t o_lde, hipStream_t stream);

/* wam_attn_blockcausal_mx / wam_attn_blockcausal_fp8_mx: the attentions above (same
 * arguments and arithmetic, Dh = 128) with the output written block-scaled for the FP8
 * projection that reads it (the attention output projection, Section 3.2.4, Appendix D.2):
 * each row's output is rounded to bf16 as the plain entry point stores it, then each head's
 * dims 0-63 and 64-127 are a block quantized by wam_gemm_fp8_mx's rule.  o8 receives the
 * E4M3 codes (one byte per element; o_tok_stride and o_batch_stride in bytes, o_batch_stride
 * = Lq * o_tok_stride when B > 1; 4-byte aligned); for output row m = b * Lq + query the
 * exponents of head h's two blocks are at o_exp[h * o_lde + 4 m + {0, 1}] (o_lde a multiple
 * of 4, >= 4 B Lq; o_exp 4-byte aligned), i.e. the a_exp layout of wam_gemm_fp8_mx with K =
 * H * 128. */
wam_status wam_attn_blockcausal_mx(const wam_attn_desc* desc, const void* q, const void* k, const void* v,
                                   void* o8, void* o_exp, int64_t o_lde, hipStream_t stream);
wam_status wam_attn_blockcausal_fp8_mx(const wam_attn_desc* desc, const void* q8, const void* q_exp,
                                       const void* k8, const void* k_exp, const void* v8, float v_scale,
                                       void* o8, void* o_exp, int64_t o_lde, hipStream_t stream);

/* Patch and action embedding into the fp32 residual x [B][Lv+A][d]. */
size_t wam_embed_workspace_bytes(const wam_dims* dims, int32_t B, int32_t F, int32_t Hl, int32_t Wl);
wam_status wam_embed_fwd(const wam_model* m, int32_t B, int32_t F, int32_t Hl, int32_t Wl,
                         int32_t A, const void* z_t, const void* a_t, float* x, void* ws,
                         size_t ws_bytes, hipStream_t stream);

/* Output head from x [B][Lv+A][d] and e [B][d]: v_video [B][latent_ch][F][Hl][Wl] and
 * v_action [B][A][act_dim], both fp32. */
size_t wam_head_workspace_bytes(const wam_dims* dims, int32_t B, int32_t F, int32_t Hl, int32_t Wl, int32_t A);
wam_status wam_head_fwd(const wam_model* m, int32_t B, int32_t F, int32_t Hl, int32_t Wl,
                        int32_t A, const float* x, const float* e, float* v_video,
                        float* v_action, void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------------
 * Host helpers (HOST memory, no GPU work).
 * ------------------------------------------------------------------------------ */

/* RoPE positions of chunk c: video token (f, r, s) of its F frames at (F*c + f, r, s),
 * frame-major then row then column over an Hg x Wg grid; action token j after the
 * last frame at (F*c + F + j, 0, 0).  pos: HOST [(F*Hg*Wg + A)][3]. */
wam_status wam_chunk_positions(int32_t c, int32_t F, int32_t Hg, int32_t Wg, int32_t A,
                               int32_t* pos);

/* RoPE tables for L positions pos [L][3] (HOST): the head vector splits into
 * contiguous (t, h, w) segments of (Dh - 4*floor(Dh/6), 2*floor(Dh/6), 2*floor(Dh/6))
 * dims; pair i of a segment with D_a dims at position p rotates by
 * p * theta^(-2i/D_a).  Computed in double, rounded to fp32:
 * cos_out, sin_out HOST [L][Dh/2]. */
wam_status wam_rope_tables(const int32_t* pos, int32_t L, int32_t Dh, double theta,
                           float* cos_out, float* sin_out);

#ifdef __cplusplus
}
#endif
#endif /* WAMDIT_H */
