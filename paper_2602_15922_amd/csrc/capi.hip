// C ABI of libwamdit: host-side validation, workspace planning and the launch
// sequences of the DiT block and denoising step.  No memory is allocated and no
// stream is synchronised here; every entry point validates all arguments before its
// first launch (the multi-launch sequences by a dry pass over the whole sequence).
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "kernels.h"

using namespace wam;

namespace {

thread_local std::string g_err;

// Inside the denoising loop with DiT caching, every kernel of a step is launched with
// the loop's device flag (a reused step's kernels return at entry; the decision stays
// on the device).  Set by SkipScope around one step; NULL everywhere else.
thread_local const int32_t* t_skip = nullptr;
struct SkipScope {
  explicit SkipScope(const int32_t* f) { t_skip = f; }
  ~SkipScope() { t_skip = nullptr; }
};
template <class Args>
const Args& pred(Args& a) {
  a.skip = t_skip;
  return a;
}

wam_status fail(wam_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define CHECK(cond, st, ...) \
  do {                       \
    if (!(cond)) return fail(st, __VA_ARGS__); \
  } while (0)

#define HIPCHECK(expr)                                                              \
  do {                                                                              \
    hipError_t e_ = (expr);                                                         \
    if (e_ != hipSuccess) return fail(WAM_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

#define TRY(expr)                      \
  do {                                 \
    wam_status s_ = (expr);            \
    if (s_ != WAM_OK) return s_;       \
  } while (0)

// A launch sequence (block, step, update pass, loop) first runs dry: every descriptor of
// every launch is built and validated, nothing is launched or recorded.  Only if that
// pass returns WAM_OK does the same sequence run for real, so an invalid argument found
// deep in the sequence never leaves the caller's buffers partly updated.
thread_local bool t_dry = false;
struct DryScope {
  DryScope() { t_dry = true; }
  ~DryScope() { t_dry = false; }
};
#define LAUNCH(expr)          \
  do {                        \
    if (!t_dry) HIPCHECK(expr); \
  } while (0)

bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }
bool al4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3) == 0; }

wam_status need_ptr(const void* p, const char* name) {
  if (!p) return fail(WAM_EINVAL, "%s is NULL", name);
  if (!al16(p)) return fail(WAM_EINVAL, "%s is not 16-byte aligned", name);
  return WAM_OK;
}
wam_status opt_ptr(const void* p, const char* name) {
  if (p && !al16(p)) return fail(WAM_EINVAL, "%s is not 16-byte aligned", name);
  return WAM_OK;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Validate a chunk layout for Lq query rows and Lk key rows; on success fill the
// per-query-chunk visible key prefix.
wam_status check_chunks(const wam_chunks& c, int32_t Lq, int32_t Lk, int32_t* kend) {
  CHECK(c.n_k_chunks >= 1 && c.n_k_chunks <= WAM_MAX_CHUNKS, WAM_EINVAL,
        "n_k_chunks=%d outside [1,%d]", c.n_k_chunks, WAM_MAX_CHUNKS);
  CHECK(c.n_q_chunks >= 1 && c.n_q_chunks <= WAM_MAX_CHUNKS, WAM_EINVAL,
        "n_q_chunks=%d outside [1,%d]", c.n_q_chunks, WAM_MAX_CHUNKS);
  CHECK(c.k_off[0] == 0 && c.k_off[c.n_k_chunks] == Lk, WAM_EINVAL,
        "k_off must run from 0 to Lk=%d (got %d..%d)", Lk, c.k_off[0], c.k_off[c.n_k_chunks]);
  for (int j = 0; j < c.n_k_chunks; ++j)
    CHECK(c.k_off[j] <= c.k_off[j + 1], WAM_EINVAL, "k_off not non-decreasing at %d", j);
  CHECK(c.q_off[0] == 0 && c.q_off[c.n_q_chunks] == Lq, WAM_EINVAL,
        "q_off must run from 0 to Lq=%d (got %d..%d)", Lq, c.q_off[0], c.q_off[c.n_q_chunks]);
  for (int i = 0; i < c.n_q_chunks; ++i) {
    CHECK(c.q_off[i] <= c.q_off[i + 1], WAM_EINVAL, "q_off not non-decreasing at %d", i);
    CHECK(c.q_chunk_id[i] >= 0 && c.q_chunk_id[i] < c.n_k_chunks, WAM_EINVAL,
          "q_chunk_id[%d]=%d outside [0,%d)", i, c.q_chunk_id[i], c.n_k_chunks);
    CHECK(i == 0 || c.q_chunk_id[i] >= c.q_chunk_id[i - 1], WAM_EINVAL,
          "q_chunk_id not non-decreasing at %d", i);
    kend[i] = c.k_off[c.q_chunk_id[i] + 1];
    CHECK(c.q_off[i] == c.q_off[i + 1] || kend[i] > 0, WAM_EINVAL,
          "query chunk %d sees no key", i);
  }
  return WAM_OK;
}

wam_status check_dims(const wam_dims& D) {
  CHECK(D.Dh == 64 || D.Dh == 128, WAM_EUNSUPPORTED, "Dh=%d (supported: 64, 128)", D.Dh);
  CHECK(D.H >= 1 && D.H * D.Dh == D.d, WAM_EINVAL, "H*Dh=%d != d=%d", D.H * D.Dh, D.d);
  CHECK(D.d % 256 == 0 && D.d <= 8192, WAM_EUNSUPPORTED, "d=%d must be a multiple of 256, <= 8192", D.d);
  CHECK(D.ffn >= 8 && D.ffn % 8 == 0, WAM_EUNSUPPORTED, "ffn=%d must be a positive multiple of 8", D.ffn);
  CHECK(D.eps > 0.f, WAM_EINVAL, "eps must be > 0");
  return WAM_OK;
}

// ---------------------------------------------------------------------------------
// attention
// ---------------------------------------------------------------------------------
// o_exp non-NULL: the output block-scaled (codes at o, one byte per element, strides in
// bytes; exponents at o_exp, see wam_attn_blockcausal_mx).
wam_status attn_out_blocks_check(const wam_attn_desc& d, const void* o, const void* o_exp, int64_t o_lde) {
  CHECK(d.Dh == 128, WAM_EUNSUPPORTED, "a block-scaled attention output needs Dh=128 (got %d)", d.Dh);
  CHECK(d.B <= 1 || d.o_batch_stride == (int64_t)d.Lq * d.o_tok_stride, WAM_EINVAL,
        "a block-scaled output takes plain rows (o_batch_stride = Lq * o_tok_stride)");
  CHECK(o_lde % 4 == 0 && o_lde >= 4 * (int64_t)d.B * d.Lq, WAM_EINVAL, "o_lde must be a multiple of 4, >= 4*B*Lq");
  CHECK(al4(o) && al4(o_exp), WAM_EINVAL, "o and o_exp must be 4-byte aligned");
  return WAM_OK;
}

wam_status attn_checked(const wam_attn_desc& d, const void* q, const void* k, const void* v, void* o,
                        hipStream_t s, void* o_exp = nullptr, int64_t o_lde = 0) {
  CHECK(d.Dh == 64 || d.Dh == 128, WAM_EUNSUPPORTED, "Dh=%d (supported: 64, 128)", d.Dh);
  CHECK(d.B >= 0 && d.H >= 1 && d.Lq >= 0 && d.Lk >= 0, WAM_EINVAL, "negative size (B=%d H=%d Lq=%d Lk=%d)",
        d.B, d.H, d.Lq, d.Lk);
  AttnArgs a{};
  TRY(check_chunks(d.ch, d.Lq, d.Lk, a.kend));
  if (d.B == 0 || d.Lq == 0) return WAM_OK;
  TRY(need_ptr(q, "q"));
  TRY(need_ptr(k, "k"));
  TRY(need_ptr(v, "v"));
  TRY(need_ptr(o, "o"));
  const int64_t hd = (int64_t)d.H * d.Dh;
  CHECK(d.q_tok_stride >= hd && d.kv_tok_stride >= hd && d.o_tok_stride >= hd, WAM_EINVAL,
        "token strides must be >= H*Dh=%lld", (long long)hd);
  CHECK(d.q_tok_stride % 8 == 0 && d.kv_tok_stride % 8 == 0 && d.o_tok_stride % 8 == 0 &&
            d.q_batch_stride % 8 == 0 && d.kv_batch_stride % 8 == 0 && d.o_batch_stride % 8 == 0,
        WAM_EINVAL, "strides must be multiples of 8 elements");
  CHECK(d.B == 1 || (d.q_batch_stride >= (int64_t)d.Lq * d.q_tok_stride &&
                     d.o_batch_stride >= (int64_t)d.Lq * d.o_tok_stride &&
                     d.kv_batch_stride >= (int64_t)d.Lk * d.kv_tok_stride),
        WAM_EINVAL, "batch strides smaller than one sample");
  CHECK((int64_t)d.Lk * d.kv_tok_stride * 2 <= INT32_MAX, WAM_EUNSUPPORTED,
        "one sample's keys span %lld bytes (Lk * kv_tok_stride * 2 must stay below 2^31)",
        (long long)d.Lk * d.kv_tok_stride * 2);
  a.q = q; a.k = k; a.v = v; a.o = o;
  a.q_ts = d.q_tok_stride; a.q_bs = d.q_batch_stride;
  a.kv_ts = d.kv_tok_stride; a.kv_bs = d.kv_batch_stride;
  a.o_ts = d.o_tok_stride; a.o_bs = d.o_batch_stride;
  a.B = d.B; a.H = d.H; a.Dh = d.Dh; a.Lq = d.Lq; a.Lk = d.Lk;
  const float scale = d.scale > 0.f ? d.scale : 1.0f / std::sqrt((float)d.Dh);
  a.c = scale * 1.4426950408889634f;
  a.n_k_chunks = d.ch.n_k_chunks;
  a.n_q_chunks = d.ch.n_q_chunks;
  for (int i = 0; i <= d.ch.n_q_chunks; ++i) a.q_off[i] = d.ch.q_off[i];
  if (o_exp) TRY(attn_out_blocks_check(d, o, o_exp, o_lde));
  LAUNCH(launch_attn(pred(a), s, static_cast<uint8_t*>(o_exp), o_lde));
  return WAM_OK;
}


// FP8 attention (Dh = 128): codes addressed like the bf16 operands with one byte per
// element; each (token, head) has one uint32 of block exponents, so the exponent arrays'
// strides are the code strides / Dh.
wam_status attn_fp8_checked(const wam_attn_desc& d, const void* q, const void* qe, const void* k, const void* ke,
                            const void* v, float v_scale, void* o, hipStream_t s, void* o_exp = nullptr,
                            int64_t o_lde = 0) {
  CHECK(d.Dh == 128, WAM_EUNSUPPORTED, "FP8 attention needs Dh=128 (got %d)", d.Dh);
  CHECK(d.B >= 0 && d.H >= 1 && d.Lq >= 0 && d.Lk >= 0, WAM_EINVAL, "negative size (B=%d H=%d Lq=%d Lk=%d)",
        d.B, d.H, d.Lq, d.Lk);
  CHECK(std::isfinite(v_scale) && v_scale > 0.f, WAM_EINVAL, "v_scale=%g must be positive and finite",
        (double)v_scale);
  AttnFp8Args f{};
  AttnArgs& a = f.a;
  TRY(check_chunks(d.ch, d.Lq, d.Lk, a.kend));
  if (d.B == 0 || d.Lq == 0) return WAM_OK;
  TRY(need_ptr(q, "q8")); TRY(need_ptr(qe, "q_exp")); TRY(need_ptr(k, "k8")); TRY(need_ptr(ke, "k_exp"));
  TRY(need_ptr(v, "v8")); TRY(need_ptr(o, "o"));
  CHECK(al16(q) && al16(k) && al16(v) && al16(o) && al4(qe) && al4(ke), WAM_EINVAL,
        "q8/k8/v8/o must be 16-byte and q_exp/k_exp 4-byte aligned");
  const int64_t hd = (int64_t)d.H * d.Dh;
  CHECK(d.q_tok_stride >= hd && d.kv_tok_stride >= hd && d.o_tok_stride >= hd, WAM_EINVAL,
        "token strides must be >= H*Dh=%lld", (long long)hd);
  CHECK(d.q_tok_stride % 128 == 0 && d.kv_tok_stride % 128 == 0 && d.q_batch_stride % 128 == 0 &&
            d.kv_batch_stride % 128 == 0,
        WAM_EINVAL, "q and k/v strides must be multiples of Dh=128 bytes");
  CHECK(d.o_tok_stride % 8 == 0 && d.o_batch_stride % 8 == 0, WAM_EINVAL, "o strides must be multiples of 8");
  CHECK(d.B == 1 || (d.q_batch_stride >= (int64_t)d.Lq * d.q_tok_stride &&
                     d.o_batch_stride >= (int64_t)d.Lq * d.o_tok_stride &&
                     d.kv_batch_stride >= (int64_t)d.Lk * d.kv_tok_stride),
        WAM_EINVAL, "batch strides smaller than one sample");
  CHECK((int64_t)d.Lk * d.kv_tok_stride <= INT32_MAX, WAM_EUNSUPPORTED,
        "one sample's keys span %lld bytes (must stay below 2^31)", (long long)d.Lk * d.kv_tok_stride);
  a.q = q; a.k = k; a.v = v; a.o = o;
  a.q_ts = d.q_tok_stride; a.q_bs = d.q_batch_stride;
  a.kv_ts = d.kv_tok_stride; a.kv_bs = d.kv_batch_stride;
  a.o_ts = d.o_tok_stride; a.o_bs = d.o_batch_stride;
  a.B = d.B; a.H = d.H; a.Dh = d.Dh; a.Lq = d.Lq; a.Lk = d.Lk;
  const float scale = d.scale > 0.f ? d.scale : 1.0f / std::sqrt((float)d.Dh);
  a.c = scale * 1.4426950408889634f;
  a.n_k_chunks = d.ch.n_k_chunks;
  a.n_q_chunks = d.ch.n_q_chunks;
  for (int i = 0; i <= d.ch.n_q_chunks; ++i) a.q_off[i] = d.ch.q_off[i];
  a.skip = t_skip;
  f.q_exp = qe; f.k_exp = ke;
  f.qe_ts = d.q_tok_stride / 128; f.qe_bs = d.q_batch_stride / 128;
  f.ke_ts = d.kv_tok_stride / 128; f.ke_bs = d.kv_batch_stride / 128;
  f.v_scale = v_scale;
  if (o_exp) TRY(attn_out_blocks_check(d, o, o_exp, o_lde));
  LAUNCH(launch_attn_fp8(f, s, static_cast<uint8_t*>(o_exp), o_lde));
  return WAM_OK;
}

wam_chunks single_chunk(int32_t Lq, int32_t Lk) {
  wam_chunks c{};
  c.n_k_chunks = 1; c.k_off[0] = 0; c.k_off[1] = Lk;
  c.n_q_chunks = 1; c.q_off[0] = 0; c.q_off[1] = Lq; c.q_chunk_id[0] = 0;
  return c;
}

// ---------------------------------------------------------------------------------
// GEMM
// ---------------------------------------------------------------------------------
// fp8: A and W are E4M3 bytes with per-row a_scale [M] and per-column w_scale [N].
// Validate one GEMM descriptor and fill its launch arguments (a.M = 0: nothing to run).
wam_status gemm_prep(const wam_gemm_desc& g, GemmArgs& a, int32_t gate_split = 0, int64_t gate_alt = 0,
                     const float* a_scale = nullptr, const float* w_scale = nullptr, bool a_blocks = false) {
  a = GemmArgs{};
  const bool fp8 = a_scale != nullptr || a_blocks;
  const int eb = fp8 ? 1 : 2, epc = 16 / eb;  // bytes per element, elements per 16 bytes
  CHECK(g.M >= 0 && g.N >= 1 && g.K >= epc && g.K % epc == 0, WAM_EINVAL,
        "GEMM sizes M=%d N=%d K=%d (need N>=1, K>=%d, K%%%d==0)", g.M, g.N, g.K, epc, epc);
  CHECK(g.epilogue >= WAM_EPI_BF16 && g.epilogue <= WAM_EPI_F32, WAM_EINVAL, "unknown epilogue %d", g.epilogue);
  if (g.M == 0) return WAM_OK;
  TRY(need_ptr(g.A, "A"));
  TRY(need_ptr(g.W, "W"));
  TRY(need_ptr(g.out, "out"));
  CHECK(g.lda >= g.K && g.lda % epc == 0 && g.ldw >= g.K && g.ldw % epc == 0, WAM_EINVAL,
        "lda/ldw must be >= K and multiples of %d", epc);
  CHECK(g.ldo >= g.N, WAM_EINVAL, "ldo < N");
  CHECK(g.a_rows >= 0 && g.out_rows >= 0 && g.gate_rows >= 0, WAM_EINVAL, "negative row groups");
  CHECK(g.a_batch_stride % epc == 0, WAM_EINVAL, "a_batch_stride must be a multiple of %d", epc);
  if (fp8) {
    if (!a_blocks) TRY(need_ptr(a_scale, "a_scale"));
    TRY(need_ptr(w_scale, "w_scale"));
  }
  CHECK(g.ldo % 4 == 0 && g.out_batch_stride % 4 == 0 && g.gate_stride % 4 == 0, WAM_EINVAL,
        "ldo, out_batch_stride and gate_stride must be multiples of 4");
  TRY(opt_ptr(g.bias, "bias"));
  TRY(opt_ptr(g.gate_a, "gate_a"));
  TRY(opt_ptr(g.gate_v, "gate_v"));
  {
    // the kernels address A and W with 32-bit byte offsets from their base pointers
    const int64_t ar = g.a_rows > 0 ? g.a_rows : g.M;
    const int64_t a_end = (g.a_rows > 0 ? (int64_t)(g.M - 1) / ar * g.a_batch_stride : 0) +
                          (std::min<int64_t>(ar, g.M) - 1) * g.lda + g.K;
    const int64_t w_end = (int64_t)(g.N - 1) * g.ldw + g.K;
    CHECK(eb * a_end <= INT32_MAX && eb * w_end <= INT32_MAX, WAM_EUNSUPPORTED,
          "A or W spans 2 GiB or more (A %lld bytes, W %lld bytes)", (long long)(eb * a_end),
          (long long)(eb * w_end));
  }
  a.M = g.M; a.N = g.N; a.K = g.K; a.epi = g.epilogue;
  a.A = g.A; a.lda = g.lda; a.a_bs = g.a_batch_stride; a.a_rows = g.a_rows;
  a.W = g.W; a.ldw = g.ldw; a.bias = g.bias;
  a.out = g.out; a.ldo = g.ldo; a.o_bs = g.out_batch_stride; a.o_rows = g.out_rows;
  a.gate_a = g.gate_a; a.gate_v = g.gate_v; a.gate_stride = g.gate_stride; a.gate_rows = g.gate_rows;
  a.gate_split = gate_split; a.gate_alt = gate_alt;
  a.fp8 = fp8 ? 1 : 0; a.a_scale = a_scale; a.w_scale = w_scale;
  return WAM_OK;
}

wam_status gemm_checked(const wam_gemm_desc& g, hipStream_t s, int32_t gate_split = 0, int64_t gate_alt = 0,
                        const float* a_scale = nullptr, const float* w_scale = nullptr) {
  GemmArgs a;
  TRY(gemm_prep(g, a, gate_split, gate_alt, a_scale, w_scale));
  if (a.M == 0) return WAM_OK;
  LAUNCH(launch_gemm(pred(a), s));
  return WAM_OK;
}

// The FP8 GEMM with block-scaled operands on either side (see wam_gemm_fp8_mx): a_exp
// (instead of a_scale) the exponents of A's 64-column blocks; out_exp (GELU epilogue) the
// output written as E4M3 codes with the exponents of its 64-column blocks.
wam_status gemm_fp8_blocks(const wam_gemm_desc& g, const float* a_scale, const void* a_exp, int64_t a_lde,
                           const float* w_scale, void* out_exp, int64_t o_lde, hipStream_t s,
                           int32_t gate_split = 0, int64_t gate_alt = 0) {
  CHECK((a_scale != nullptr) != (a_exp != nullptr), WAM_EINVAL, "exactly one of a_scale and a_exp is required");
  CHECK(!(a_exp && out_exp), WAM_EUNSUPPORTED, "block-scaled A with a block-scaled output");
  GemmArgs a;
  TRY(gemm_prep(g, a, gate_split, gate_alt, a_scale, w_scale, a_exp != nullptr));
  if (a_exp) {
    CHECK(g.K % 128 == 0, WAM_EUNSUPPORTED, "block-scaled A needs K %% 128 == 0 (K=%d)", g.K);
    CHECK(g.epilogue == WAM_EPI_BF16 || g.epilogue == WAM_EPI_RESID_F32, WAM_EUNSUPPORTED,
          "block-scaled A takes the bf16 or the residual epilogue");
    CHECK(g.a_rows == 0, WAM_EUNSUPPORTED, "block-scaled A takes plain rows (a_rows = 0)");
    CHECK(a_lde % 4 == 0 && a_lde >= 4 * (int64_t)g.M, WAM_EINVAL, "a_lde must be a multiple of 4, >= 4*M");
    CHECK(g.M == 0 || al4(a_exp), WAM_EINVAL, "a_exp must be 4-byte aligned");
  }
  if (out_exp) {
    CHECK(g.epilogue == WAM_EPI_GELU_BF16, WAM_EUNSUPPORTED, "a block-scaled output takes the GELU epilogue");
    CHECK(g.N % 128 == 0, WAM_EUNSUPPORTED, "a block-scaled output needs N %% 128 == 0 (N=%d)", g.N);
    CHECK(g.out_rows == 0, WAM_EUNSUPPORTED, "a block-scaled output takes plain rows (out_rows = 0)");
    CHECK(o_lde % 4 == 0 && o_lde >= 4 * (int64_t)g.M, WAM_EINVAL, "o_lde must be a multiple of 4, >= 4*M");
    CHECK(g.M == 0 || al4(g.out), WAM_EINVAL, "out must be 4-byte aligned");
  }
  if (a.M == 0) return WAM_OK;
  if (a_exp) {
    a.epi |= WAM_EPI_MXA;
    a.a_exp = static_cast<const uint8_t*>(a_exp);
    a.a_lde = a_lde;
  }
  if (out_exp) {
    a.epi = WAM_EPI_GELU_MX8;
    a.out_exp = static_cast<uint8_t*>(out_exp);
    a.o_lde = o_lde;
  }
  LAUNCH(launch_gemm(pred(a), s));
  return WAM_OK;
}

wam_gemm_desc gemm(int M, int N, int K, int epi, const void* A, int64_t lda, const void* W,
                   const float* bias, void* out, int64_t ldo) {
  wam_gemm_desc g{};
  g.M = M; g.N = N; g.K = K; g.epilogue = epi;
  g.A = A; g.lda = lda; g.W = W; g.ldw = K; g.bias = bias; g.out = out; g.ldo = ldo;
  return g;
}

// ---------------------------------------------------------------------------------
// block
// ---------------------------------------------------------------------------------
struct BlockWs {
  size_t h, big, q, o, ckv, q8, qs, total;
};
// q8 / qs: an activation quantized to E4M3 for an FP8 projection and its row scales.
BlockWs block_ws(const wam_dims& D, int32_t B, int32_t L, int32_t Lc) {
  const size_t M = (size_t)B * L, d = D.d;
  const size_t wide = (size_t)(3 * D.d > D.ffn ? 3 * D.d : D.ffn);
  const size_t rows = std::max(M, (size_t)B * Lc), kmax = (size_t)std::max(D.d, (D.ffn + 15) / 16 * 16);
  BlockWs w{};
  size_t off = 0;
  w.h = off; off += align256(M * d * 2);
  w.big = off; off += align256(M * wide * 2);
  w.q = off; off += align256(M * d * 2);
  w.o = off; off += align256(M * d * 2);
  w.ckv = off; off += align256((size_t)B * Lc * 2 * d * 2);
  w.q8 = off; off += align256(rows * kmax);
  w.qs = off; off += align256(rows * 4);
  w.total = off;
  return w;
}

// One projection of a block: the bf16 GEMM, or, with FP8 weights w8 / s8, the
// activation rows quantized to E4M3 into q8 / qs and the FP8 GEMM.
wam_status proj(const wam_gemm_desc& g0, const void* w8, const float* s8, char* q8, float* qs, hipStream_t s,
                int32_t gate_split = 0, int64_t gate_alt = 0) {
  if (!w8) return gemm_checked(g0, s, gate_split, gate_alt);
  const int64_t ldq = (g0.K + 15) / 16 * 16;
  LAUNCH(launch_quant_rows(g0.M, g0.K, g0.A, g0.lda, q8, ldq, qs, s, t_skip));
  wam_gemm_desc g = g0;
  g.A = q8; g.lda = ldq; g.a_rows = 0; g.a_batch_stride = 0;
  g.W = w8; g.ldw = g0.K;
  return gemm_checked(g, s, gate_split, gate_alt, qs, s8);
}

// An FP8 projection whose activation rows the LayerNorm before it already wrote as E4M3
// codes (row stride K rounded up to 16) and row scales.
wam_status proj_q8(const wam_gemm_desc& g0, const void* w8, const float* s8, char* q8, float* qs, hipStream_t s) {
  wam_gemm_desc g = g0;
  g.A = q8; g.lda = (g0.K + 15) / 16 * 16; g.a_rows = 0; g.a_batch_stride = 0;
  g.W = w8; g.ldw = g0.K;
  return gemm_checked(g, s, 0, 0, qs, s8);
}

// The QKV projection with RoPE and the K/V append of rope_qkv_kernel in its epilogue (bf16
// operands and cache; H * Dh a multiple of 64): the same output bits, without the q|k|v
// round trip through memory.
wam_status qkv_rope(const wam_gemm_desc& g, const RopeArgs& r, hipStream_t s) {
  GemmArgs a;
  TRY(gemm_prep(g, a));
  if (a.M == 0) return WAM_OK;
  a.epi = WAM_EPI_ROPE;
  a.rope_cos = r.cos_t; a.rope_sin = r.sin_t;
  a.rope_q = r.q_out; a.rope_k = r.k_cache; a.rope_v = r.v_cache;
  a.rope_L = r.L; a.rope_Dh = r.Dh; a.rope_d = r.H * r.Dh;
  a.rope_Lcap = r.Lcap; a.rope_row0 = r.row0;
  LAUNCH(launch_gemm(pred(a), s));
  return WAM_OK;
}

// A LayerNorm that feeds only an FP8 projection writes E4M3 codes and row scales directly.
void ln_to_fp8(LnArgs& ln, char* q8, float* qs) {
  ln.q8 = reinterpret_cast<uint8_t*>(q8);
  ln.ldq = (ln.d + 15) / 16 * 16;
  ln.q_scale = qs;
}

wam_status check_block_weights(const wam_block_weights& w) {
  if (!w.fp8) {  // with FP8 copies the bf16 matrices are not read
    TRY(need_ptr(w.w_qkv, "w_qkv")); TRY(need_ptr(w.w_o, "w_o")); TRY(need_ptr(w.w_cq, "w_cq"));
    TRY(need_ptr(w.w_co, "w_co")); TRY(need_ptr(w.w_f1, "w_f1")); TRY(need_ptr(w.w_f2, "w_f2"));
  }
  TRY(need_ptr(w.mod6, "mod6"));
  TRY(opt_ptr(w.w_ckv, "w_ckv"));
  TRY(opt_ptr(w.b_qkv, "b_qkv")); TRY(opt_ptr(w.b_o, "b_o")); TRY(opt_ptr(w.b_cq, "b_cq"));
  TRY(opt_ptr(w.b_ckv, "b_ckv")); TRY(opt_ptr(w.b_co, "b_co")); TRY(opt_ptr(w.b_f1, "b_f1"));
  TRY(opt_ptr(w.b_f2, "b_f2")); TRY(opt_ptr(w.lnc_gamma, "lnc_gamma")); TRY(opt_ptr(w.lnc_beta, "lnc_beta"));
  if (w.fp8) {
    const wam_block_fp8& f = *w.fp8;
    TRY(need_ptr(f.w_qkv, "fp8 w_qkv")); TRY(need_ptr(f.w_o, "fp8 w_o")); TRY(need_ptr(f.w_cq, "fp8 w_cq"));
    TRY(need_ptr(f.w_co, "fp8 w_co")); TRY(need_ptr(f.w_f1, "fp8 w_f1")); TRY(need_ptr(f.w_f2, "fp8 w_f2"));
    TRY(need_ptr(f.s_qkv, "fp8 s_qkv")); TRY(need_ptr(f.s_o, "fp8 s_o")); TRY(need_ptr(f.s_cq, "fp8 s_cq"));
    TRY(need_ptr(f.s_co, "fp8 s_co")); TRY(need_ptr(f.s_f1, "fp8 s_f1")); TRY(need_ptr(f.s_f2, "fp8 s_f2"));
    TRY(opt_ptr(f.w_ckv, "fp8 w_ckv")); TRY(opt_ptr(f.s_ckv, "fp8 s_ckv"));
  }
  return WAM_OK;
}

wam_status check_block_io(const wam_dims& D, const wam_block_weights& w, const wam_block_io& io) {
  CHECK(io.B >= 1 && io.L >= 1 && io.Lc >= 1, WAM_EINVAL, "B=%d L=%d Lc=%d must be >= 1", io.B, io.L, io.Lc);
  CHECK(io.B <= 8, WAM_EUNSUPPORTED, "B=%d > 8", io.B);
  CHECK(io.cache_len >= 0 && (int64_t)io.cache_len + io.L <= io.Lcap, WAM_EINVAL,
        "cache_len=%d + L=%d exceeds Lcap=%d", io.cache_len, io.L, io.Lcap);
  int32_t kend[WAM_MAX_CHUNKS];
  TRY(check_chunks(io.ch, io.L, io.cache_len + io.L, kend));
  TRY(need_ptr(io.x, "x")); TRY(need_ptr(io.e0, "e0"));
  TRY(need_ptr(io.rope_cos, "rope_cos")); TRY(need_ptr(io.rope_sin, "rope_sin"));
  TRY(need_ptr(io.k_cache, "k_cache")); TRY(need_ptr(io.v_cache, "v_cache"));
  if (io.k_exp) {
    CHECK(D.Dh == 128, WAM_EUNSUPPORTED, "an FP8 KV cache needs Dh=128 (got %d)", D.Dh);
    CHECK(std::isfinite(io.v_scale) && io.v_scale > 0.f, WAM_EINVAL, "v_scale=%g must be positive and finite",
          (double)io.v_scale);
    CHECK(al16(io.k_cache) && al16(io.v_cache) && al4(io.k_exp), WAM_EINVAL, "FP8 cache pointers misaligned");
  }
  if (io.ctx_kv) {
    TRY(need_ptr(io.ctx_kv, "ctx_kv"));
  } else {
    TRY(need_ptr(io.ctx, "ctx"));
    if (w.fp8) { TRY(need_ptr(w.fp8->w_ckv, "fp8 w_ckv")); TRY(need_ptr(w.fp8->s_ckv, "fp8 s_ckv")); }
    else TRY(need_ptr(w.w_ckv, "w_ckv"));
  }
  return WAM_OK;
}

// The launch sequence of one block; arguments already validated.
// seg/alt: rows >= seg of a sample (0: none) take their per-sample modulation (e0) from
// e0 + alt (the action tokens' own timestep).
// ev: NULL, or 2*WAM_BLOCK_EVENTS events recorded around the block's launches (its
// self-attention pair doubles as the step's attn_events pair).
struct BlockEvents {
  const hipEvent_t* ev = nullptr;  // [WAM_BLOCK_EVENTS][2]
  hipEvent_t attn0 = nullptr, attn1 = nullptr;
};
wam_status mark(const BlockEvents& e, int kind, int end, hipStream_t s) {
  if (kind == WAM_EV_SELF_ATTN) {
    hipEvent_t a = end ? e.attn1 : e.attn0;
    if (a) LAUNCH(hipEventRecord(a, s));
  }
  if (e.ev) LAUNCH(hipEventRecord(e.ev[2 * kind + end], s));
  return WAM_OK;
}

// pq: this block's folded AdaLN shift/scale rows (AdalnFoldArgs layout, nseg segments), or
// NULL to sum the block's and the sample's rows in each LayerNorm
wam_status block_run(const wam_dims& D, const wam_block_weights& W, const wam_block_io& io, char* ws,
                     hipStream_t s, const BlockEvents& ev = BlockEvents{}, int32_t seg = 0, int64_t alt = 0,
                     const float* pq = nullptr, int32_t nseg = 1) {
  const int d = D.d, B = io.B, L = io.L, M = B * L;
  const BlockWs lay = block_ws(D, B, L, io.Lc);
  void* h = ws + lay.h;
  void* big = ws + lay.big;
  void* q = ws + lay.q;
  void* o = ws + lay.o;
  void* ckv = ws + lay.ckv;
  char* q8 = ws + lay.q8;
  float* qs = reinterpret_cast<float*>(ws + lay.qs);
  const wam_block_fp8* F8 = W.fp8;
  const float* m6 = W.mod6;
  const float* e0 = io.e0;
  const int64_t ms = 6 * (int64_t)d;

  // 1. AdaLN: h = LN(x)(1 + scale1) + shift1
  LnArgs ln{M, L, d, D.eps, io.x, nullptr, nullptr, m6 + 0 * d, e0 + 0 * d, m6 + 1 * d, e0 + 1 * d, ms, h, seg, alt};
  const int64_t pq_ms = (int64_t)nseg * 2 * d, pq_alt = 2 * (int64_t)d, pq_norm = (int64_t)B * pq_ms;
  if (pq) ln = LnArgs{M, L, d, D.eps, io.x, nullptr, nullptr, nullptr, pq, nullptr, pq + d, pq_ms, h, seg, pq_alt};
  // FP8 projections after the three LayerNorms: the LayerNorm writes the E4M3 rows itself
  const bool ln8 = F8 && ln_fp8_supported(d);
  if (ln8) ln_to_fp8(ln, q8, qs);
  TRY(mark(ev, WAM_EV_LN1, 0, s));
  LAUNCH(launch_ln_mod(pred(ln), s));
  TRY(mark(ev, WAM_EV_LN1, 1, s));
  // 2. fused QKV projection; 3. RoPE on q, k; k, v appended to the cache rows of this chunk
  // (with an FP8 cache: q and k encoded in 32-dim blocks, q into the q buffer with its
  // exponents behind it).  With bf16 operands and cache, step 3 runs in step 2's epilogue
  // and the RoPE events bracket no launch.
  void* qe = static_cast<char*>(q) + (size_t)M * d;
  RopeArgs ra{B, L, D.H, D.Dh, io.Lcap, io.cache_len, big, io.rope_cos, io.rope_sin, q, io.k_cache, io.v_cache};
  const bool rope_epi = !F8 && !io.k_exp && d % 64 == 0;
  TRY(mark(ev, WAM_EV_QKV, 0, s));
  if (ln8) TRY(proj_q8(gemm(M, 3 * d, d, WAM_EPI_BF16, h, d, W.w_qkv, W.b_qkv, big, 3 * d), F8->w_qkv, F8->s_qkv, q8, qs, s));
  else if (rope_epi) TRY(qkv_rope(gemm(M, 3 * d, d, WAM_EPI_BF16, h, d, W.w_qkv, W.b_qkv, big, 3 * d), ra, s));
  else TRY(proj(gemm(M, 3 * d, d, WAM_EPI_BF16, h, d, W.w_qkv, W.b_qkv, big, 3 * d), F8 ? F8->w_qkv : nullptr,
                F8 ? F8->s_qkv : nullptr, q8, qs, s));
  TRY(mark(ev, WAM_EV_QKV, 1, s));
  TRY(mark(ev, WAM_EV_ROPE, 0, s));
  if (io.k_exp) {
    RopeFp8Args rf{pred(ra), qe, io.k_exp, 1.0f / io.v_scale};
    LAUNCH(launch_rope_qkv_fp8(rf, s));
  } else if (!rope_epi) {
    LAUNCH(launch_rope_qkv(pred(ra), s));
  }
  TRY(mark(ev, WAM_EV_ROPE, 1, s));
  // 4. block-causal self-attention over cache rows [0, cache_len + L)
  wam_attn_desc ad{};
  ad.B = B; ad.H = D.H; ad.Dh = D.Dh; ad.Lq = L; ad.Lk = io.cache_len + L;
  ad.q_tok_stride = d; ad.q_batch_stride = (int64_t)L * d;
  ad.kv_tok_stride = d; ad.kv_batch_stride = (int64_t)io.Lcap * d;
  ad.o_tok_stride = d; ad.o_batch_stride = (int64_t)L * d;
  ad.ch = io.ch;
  // With FP8 weights both attentions write their output block-scaled: E4M3 codes [M][d] at
  // o, behind them the exponents of each row's 64-dim blocks (4 bytes per row per head), and
  // the O and cross-O projections read it as it is, with no quantization pass before them.
  const bool attn_blocks = F8 && D.Dh == 128;
  char* oe = static_cast<char*>(o) + align256((size_t)M * d);
  const int64_t oe_ld = 4 * (int64_t)M;
  void* const oe_or_null = attn_blocks ? oe : nullptr;
  TRY(mark(ev, WAM_EV_SELF_ATTN, 0, s));
  if (io.k_exp) TRY(attn_fp8_checked(ad, q, qe, io.k_cache, io.k_exp, io.v_cache, io.v_scale, o, s, oe_or_null, oe_ld));
  else TRY(attn_checked(ad, q, io.k_cache, io.v_cache, o, s, oe_or_null, oe_ld));
  TRY(mark(ev, WAM_EV_SELF_ATTN, 1, s));
  // 5. x += gate1 * (o W_o^T + b_o)
  {
    wam_gemm_desc g = gemm(M, d, d, WAM_EPI_RESID_F32, o, d, W.w_o, W.b_o, io.x, d);
    g.gate_a = m6 + 2 * d; g.gate_v = e0 + 2 * d; g.gate_stride = ms; g.gate_rows = L;
    TRY(mark(ev, WAM_EV_O, 0, s));
    if (attn_blocks) {
      g.W = F8->w_o; g.ldw = d;
      TRY(gemm_fp8_blocks(g, nullptr, oe, oe_ld, F8->s_o, nullptr, 0, s, seg, alt));
    } else {
      TRY(proj(g, F8 ? F8->w_o : nullptr, F8 ? F8->s_o : nullptr, q8, qs, s, seg, alt));
    }
    TRY(mark(ev, WAM_EV_O, 1, s));
  }
  // 6. cross-attention LayerNorm (affine, no modulation)
  LnArgs lc{M, L, d, D.eps, io.x, W.lnc_gamma, W.lnc_beta, nullptr, nullptr, nullptr, nullptr, 0, h};
  if (ln8) ln_to_fp8(lc, q8, qs);
  TRY(mark(ev, WAM_EV_LNC, 0, s));
  LAUNCH(launch_ln_mod(pred(lc), s));
  TRY(mark(ev, WAM_EV_LNC, 1, s));
  // 7. cross query
  TRY(mark(ev, WAM_EV_CQ, 0, s));
  if (ln8) TRY(proj_q8(gemm(M, d, d, WAM_EPI_BF16, h, d, W.w_cq, W.b_cq, q, d), F8->w_cq, F8->s_cq, q8, qs, s));
  else TRY(proj(gemm(M, d, d, WAM_EPI_BF16, h, d, W.w_cq, W.b_cq, q, d), F8 ? F8->w_cq : nullptr,
                F8 ? F8->s_cq : nullptr, q8, qs, s));
  TRY(mark(ev, WAM_EV_CQ, 1, s));
  // 8. cross K|V of the text (unless precomputed for this block)
  const void* kv = io.ctx_kv;
  if (!kv) {
    TRY(proj(gemm(B * io.Lc, 2 * d, d, WAM_EPI_BF16, io.ctx, d, W.w_ckv, W.b_ckv, ckv, 2 * d),
             F8 ? F8->w_ckv : nullptr, F8 ? F8->s_ckv : nullptr, q8, qs, s));
    kv = ckv;
  }
  // 9. cross-attention: every text token visible
  wam_attn_desc cd{};
  cd.B = B; cd.H = D.H; cd.Dh = D.Dh; cd.Lq = L; cd.Lk = io.Lc;
  cd.q_tok_stride = d; cd.q_batch_stride = (int64_t)L * d;
  cd.kv_tok_stride = 2 * d; cd.kv_batch_stride = (int64_t)io.Lc * 2 * d;
  cd.o_tok_stride = d; cd.o_batch_stride = (int64_t)L * d;
  cd.ch = single_chunk(L, io.Lc);
  TRY(mark(ev, WAM_EV_CROSS_ATTN, 0, s));
  TRY(attn_checked(cd, q, kv, static_cast<const char*>(kv) + (size_t)d * 2, o, s, oe_or_null, oe_ld));
  TRY(mark(ev, WAM_EV_CROSS_ATTN, 1, s));
  // 10. x += o W_co^T + b_co (no gate)
  TRY(mark(ev, WAM_EV_CO, 0, s));
  if (attn_blocks) {
    wam_gemm_desc g = gemm(M, d, d, WAM_EPI_RESID_F32, o, d, F8->w_co, W.b_co, io.x, d);
    TRY(gemm_fp8_blocks(g, nullptr, oe, oe_ld, F8->s_co, nullptr, 0, s));
  } else {
    TRY(proj(gemm(M, d, d, WAM_EPI_RESID_F32, o, d, W.w_co, W.b_co, io.x, d), F8 ? F8->w_co : nullptr,
             F8 ? F8->s_co : nullptr, q8, qs, s));
  }
  TRY(mark(ev, WAM_EV_CO, 1, s));
  // 11. AdaLN #2
  LnArgs l2{M, L, d, D.eps, io.x, nullptr, nullptr, m6 + 3 * d, e0 + 3 * d, m6 + 4 * d, e0 + 4 * d, ms, h, seg, alt};
  if (pq)
    l2 = LnArgs{M, L, d, D.eps, io.x, nullptr, nullptr, nullptr, pq + pq_norm, nullptr, pq + pq_norm + d, pq_ms, h,
                seg, pq_alt};
  if (ln8) ln_to_fp8(l2, q8, qs);
  TRY(mark(ev, WAM_EV_LN2, 0, s));
  LAUNCH(launch_ln_mod(pred(l2), s));
  TRY(mark(ev, WAM_EV_LN2, 1, s));
  // 12. FFN up-projection with tanh-GELU.  With FP8 weights (ffn a multiple of 128) its
  // output goes to FFN2 block-scaled: E4M3 codes [M][ffn] at big, behind them the
  // exponents of each row's 64-column blocks (4 bytes per row per pair of blocks), so the
  // hidden activations are written once, as bytes, and FFN2 needs no quantization pass.
  const bool ffn_blocks = F8 && D.ffn % 128 == 0;
  char* u8 = static_cast<char*>(big);
  char* ue = u8 + align256((size_t)M * D.ffn);
  const int64_t ue_ld = 4 * (int64_t)M;
  TRY(mark(ev, WAM_EV_FFN1, 0, s));
  if (ffn_blocks) {
    wam_gemm_desc g = gemm(M, D.ffn, d, WAM_EPI_GELU_BF16, h, d, W.w_f1, W.b_f1, u8, D.ffn);
    g.W = F8->w_f1; g.ldw = d;
    if (ln8) {
      g.A = q8; g.lda = (d + 15) / 16 * 16;
    } else {
      const int64_t ldq = (d + 15) / 16 * 16;
      LAUNCH(launch_quant_rows(M, d, h, d, q8, ldq, qs, s, t_skip));
      g.A = q8; g.lda = ldq;
    }
    TRY(gemm_fp8_blocks(g, qs, nullptr, 0, F8->s_f1, ue, ue_ld, s));
  } else if (ln8) {
    TRY(proj_q8(gemm(M, D.ffn, d, WAM_EPI_GELU_BF16, h, d, W.w_f1, W.b_f1, big, D.ffn), F8->w_f1, F8->s_f1, q8, qs, s));
  } else {
    TRY(proj(gemm(M, D.ffn, d, WAM_EPI_GELU_BF16, h, d, W.w_f1, W.b_f1, big, D.ffn), F8 ? F8->w_f1 : nullptr,
             F8 ? F8->s_f1 : nullptr, q8, qs, s));
  }
  TRY(mark(ev, WAM_EV_FFN1, 1, s));
  // 13. x += gate2 * (u W_f2^T + b_f2)
  {
    wam_gemm_desc g = gemm(M, d, D.ffn, WAM_EPI_RESID_F32, big, D.ffn, W.w_f2, W.b_f2, io.x, d);
    g.gate_a = m6 + 5 * d; g.gate_v = e0 + 5 * d; g.gate_stride = ms; g.gate_rows = L;
    TRY(mark(ev, WAM_EV_FFN2, 0, s));
    if (ffn_blocks) {
      g.A = u8; g.lda = D.ffn; g.W = F8->w_f2; g.ldw = D.ffn;
      TRY(gemm_fp8_blocks(g, nullptr, ue, ue_ld, F8->s_f2, nullptr, 0, s, seg, alt));
    } else {
      TRY(proj(g, F8 ? F8->w_f2 : nullptr, F8 ? F8->s_f2 : nullptr, q8, qs, s, seg, alt));
    }
    TRY(mark(ev, WAM_EV_FFN2, 1, s));
  }
  return WAM_OK;
}

// The part of a block that an update pass needs from its last layer: AdaLN #1, the K|V
// columns of the QKV projection, and RoPE on k with the cache append.
wam_status block_kv_run(const wam_dims& D, const wam_block_weights& W, const wam_block_io& io, char* ws,
                        hipStream_t s, int32_t seg = 0, int64_t alt = 0, const float* pq = nullptr,
                        int32_t nseg = 1) {
  const int d = D.d, B = io.B, L = io.L, M = B * L;
  const BlockWs lay = block_ws(D, B, L, io.Lc);
  void* h = ws + lay.h;
  char* big = ws + lay.big;  // [M][3d] bf16
  const float* m6 = W.mod6;
  const float* e0 = io.e0;
  const int64_t ms = 6 * (int64_t)d;
  LnArgs ln{M, L, d, D.eps, io.x, nullptr, nullptr, m6 + 0 * d, e0 + 0 * d, m6 + 1 * d, e0 + 1 * d, ms, h, seg, alt};
  if (pq)
    ln = LnArgs{M, L, d, D.eps, io.x, nullptr, nullptr, nullptr, pq, nullptr, pq + d, (int64_t)nseg * 2 * d, h, seg,
                2 * (int64_t)d};
  const wam_block_fp8* F8 = W.fp8;
  char* q8 = ws + lay.q8;
  float* qs = reinterpret_cast<float*>(ws + lay.qs);
  const bool ln8 = F8 && ln_fp8_supported(d);
  if (ln8) ln_to_fp8(ln, q8, qs);
  LAUNCH(launch_ln_mod(pred(ln), s));
  // rows d..3d of W_qkv (the k and v outputs) into columns d..3d of the [M][3d] buffer
  const char* wkv = F8 ? nullptr : static_cast<const char*>(W.w_qkv) + (size_t)d * d * 2;
  const float* bkv = W.b_qkv ? W.b_qkv + d : nullptr;
  const wam_gemm_desc gkv = gemm(M, 2 * d, d, WAM_EPI_BF16, h, d, wkv, bkv, big + (size_t)d * 2, 3 * d);
  if (ln8) TRY(proj_q8(gkv, static_cast<const char*>(F8->w_qkv) + (size_t)d * d, F8->s_qkv + d, q8, qs, s));
  else TRY(proj(gkv, F8 ? static_cast<const char*>(F8->w_qkv) + (size_t)d * d : nullptr, F8 ? F8->s_qkv + d : nullptr,
                q8, qs, s));
  RopeArgs ra{B, L, D.H, D.Dh, io.Lcap, io.cache_len, big, io.rope_cos, io.rope_sin, nullptr, io.k_cache,
              io.v_cache};
  if (io.k_exp) {
    RopeFp8Args rf{pred(ra), nullptr, io.k_exp, 1.0f / io.v_scale};
    LAUNCH(launch_rope_qkv_fp8(rf, s));
  } else {
    LAUNCH(launch_rope_qkv(pred(ra), s));
  }
  return WAM_OK;
}

// ---------------------------------------------------------------------------------
// model-level pieces
// ---------------------------------------------------------------------------------
wam_status check_model_common(const wam_model& m) {
  TRY(check_dims(m.dims));
  CHECK(m.dims.freq_dim >= 2 && m.dims.freq_dim % 8 == 0, WAM_EUNSUPPORTED, "freq_dim=%d must be a multiple of 8",
        m.dims.freq_dim);
  CHECK(m.dims.text_dim >= 8 && m.dims.text_dim % 8 == 0, WAM_EUNSUPPORTED, "text_dim=%d must be a multiple of 8",
        m.dims.text_dim);
  CHECK(m.dims.act_dim >= 8 && m.dims.act_dim % 8 == 0, WAM_EUNSUPPORTED, "act_dim=%d must be a multiple of 8",
        m.dims.act_dim);
  CHECK(m.dims.latent_ch >= 2 && m.dims.latent_ch % 2 == 0, WAM_EUNSUPPORTED,
        "latent_ch=%d must be even (patch features a multiple of 8)", m.dims.latent_ch);
  return WAM_OK;
}

size_t time_ws(const wam_dims& D, int32_t B) { return align256((size_t)B * (D.freq_dim + D.d) * 4); }

wam_status time_run(const wam_model& m, int32_t B, const float* t, float* e, float* e0, char* ws, hipStream_t s) {
  const wam_dims& D = m.dims;
  float* sinus = reinterpret_cast<float*>(ws);
  float* hid = sinus + (size_t)B * D.freq_dim;
  LAUNCH(launch_sinusoid(B, D.freq_dim, t, sinus, s, t_skip));
  LAUNCH(launch_gemv(B, D.d, D.freq_dim, sinus, GEMV_ACT_NONE, m.w_t1, m.b_t1, hid, s, t_skip));
  LAUNCH(launch_gemv(B, D.d, D.d, hid, GEMV_ACT_SILU, m.w_t2, m.b_t2, e, s, t_skip));
  LAUNCH(launch_gemv(B, 6 * D.d, D.d, e, GEMV_ACT_SILU, m.w_t6, m.b_t6, e0, s, t_skip));
  return WAM_OK;
}

size_t text_ws(const wam_dims& D, int32_t B, int32_t Lc) { return align256((size_t)B * Lc * D.d * 2); }

wam_status text_run(const wam_model& m, int32_t B, int32_t Lc, const void* text, void* ctx, char* ws,
                    hipStream_t s) {
  const wam_dims& D = m.dims;
  TRY(gemm_checked(gemm(B * Lc, D.d, D.text_dim, WAM_EPI_GELU_BF16, text, D.text_dim, m.w_x1, m.b_x1, ws, D.d), s));
  TRY(gemm_checked(gemm(B * Lc, D.d, D.d, WAM_EPI_BF16, ws, D.d, m.w_x2, m.b_x2, ctx, D.d), s));
  return WAM_OK;
}

size_t embed_ws(const wam_dims& D, int32_t B, int32_t F, int32_t Hl, int32_t Wl) {
  return align256((size_t)B * F * (Hl / 2) * (Wl / 2) * D.latent_ch * 4 * 2);
}

wam_status embed_run(const wam_model& m, int32_t B, int32_t F, int32_t Hl, int32_t Wl, int32_t A, const void* z,
                     const void* a, float* x, char* ws, hipStream_t s) {
  const wam_dims& D = m.dims;
  const int P = D.latent_ch * 4, Lv = F * (Hl / 2) * (Wl / 2), L = Lv + A;
  LAUNCH(launch_patchify(B, D.latent_ch, F, Hl, Wl, z, ws, s, t_skip));
  wam_gemm_desc g = gemm(B * Lv, D.d, P, WAM_EPI_F32, ws, P, m.w_patch, m.b_patch, x, D.d);
  g.out_rows = Lv; g.out_batch_stride = (int64_t)L * D.d;
  TRY(gemm_checked(g, s));
  if (A > 0) {
    wam_gemm_desc ga = gemm(B * A, D.d, D.act_dim, WAM_EPI_F32, a, D.act_dim, m.w_ain, m.b_ain,
                            x + (size_t)Lv * D.d, D.d);
    ga.out_rows = A; ga.out_batch_stride = (int64_t)L * D.d;
    TRY(gemm_checked(ga, s));
  }
  return WAM_OK;
}

struct HeadWs {
  size_t h, tok, total;
};
HeadWs head_ws(const wam_dims& D, int32_t B, int32_t F, int32_t Hl, int32_t Wl, int32_t A) {
  const size_t Lv = (size_t)F * (Hl / 2) * (Wl / 2), M = (size_t)B * (Lv + A);
  HeadWs w{};
  w.h = 0;
  w.tok = align256(M * D.d * 2);
  w.total = w.tok + align256((size_t)B * Lv * D.latent_ch * 4 * 4);
  return w;
}

// e_alt: the action rows' embedding is e + e_alt (0: the same as the video rows')
wam_status head_run(const wam_model& m, int32_t B, int32_t F, int32_t Hl, int32_t Wl, int32_t A, const float* x,
                    const float* e, float* v_video, float* v_action, char* ws, hipStream_t s, int64_t e_alt = 0) {
  const wam_dims& D = m.dims;
  const int d = D.d, P = D.latent_ch * 4, Lv = F * (Hl / 2) * (Wl / 2), L = Lv + A;
  const HeadWs lay = head_ws(D, B, F, Hl, Wl, A);
  char* h = ws + lay.h;
  float* tok = reinterpret_cast<float*>(ws + lay.tok);
  LnArgs ln{B * L, L, d, D.eps, x, nullptr, nullptr, m.head_mod2, e, m.head_mod2 + d, e, d, h,
            e_alt ? Lv : 0, e_alt};
  LAUNCH(launch_ln_mod(pred(ln), s));
  wam_gemm_desc gv = gemm(B * Lv, P, d, WAM_EPI_F32, h, d, m.w_hv, m.b_hv, tok, P);
  gv.a_rows = Lv; gv.a_batch_stride = (int64_t)L * d;
  TRY(gemm_checked(gv, s));
  LAUNCH(launch_unpatchify(B, D.latent_ch, F, Hl, Wl, tok, v_video, s, t_skip));
  if (A > 0) {
    wam_gemm_desc ga = gemm(B * A, D.act_dim, d, WAM_EPI_F32, h + (size_t)Lv * d * 2, d, m.w_ha, m.b_ha,
                            v_action, D.act_dim);
    ga.a_rows = A; ga.a_batch_stride = (int64_t)L * d;
    TRY(gemm_checked(ga, s));
  }
  return WAM_OK;
}

// Every block's cross-attention K|V of the projected text ctx (B*Lc rows, the same input
// for every block) into kv + l*kv_layer for the first n blocks, in grouped launches of up
// to WAM_GEMM_GROUP_MAX blocks: the tiles and arithmetic of one launch per block, but the
// 512-row products fill the chip together instead of ~1.25 rounds each.  Blocks with bf16
// weights and blocks with FP8 weights form separate groups; for the FP8 ones the text is
// quantized once (per-row scales, as for any FP8 projection) and shared.
wam_status cross_kv_run(const wam_model& m, int32_t B, int32_t Lc, const void* ctx, char* kv, size_t kv_layer,
                        int n, char* q8, float* qs, hipStream_t s) {
  const wam_dims& D = m.dims;
  const int M = B * Lc, N = 2 * D.d, K = D.d;
  const int64_t ldq = (K + 15) / 16 * 16;
  std::vector<GemmArgs> members(n);
  bool any_fp8 = false;
  for (int l = 0; l < n; ++l) {  // validate every member before the first launch
    const wam_block_weights& W = m.blocks[l];
    wam_gemm_desc g = gemm(M, N, K, WAM_EPI_BF16, ctx, K, W.w_ckv, W.b_ckv, kv + (size_t)l * kv_layer, N);
    if (W.fp8) {
      g.A = q8; g.lda = ldq; g.W = W.fp8->w_ckv; g.ldw = K;
      TRY(gemm_prep(g, members[l], 0, 0, qs, W.fp8->s_ckv));
      any_fp8 = true;
    } else {
      TRY(gemm_prep(g, members[l]));
    }
  }
  if (M == 0 || n == 0) return WAM_OK;
  if (any_fp8) LAUNCH(launch_quant_rows(M, K, ctx, K, q8, ldq, qs, s, t_skip));
  for (int fp8 = 0; fp8 < 2; ++fp8) {
    GemmGroup gg{};
    GemmArgs first{};
    for (int l = 0; l < n; ++l) {
      if ((m.blocks[l].fp8 != nullptr) != (fp8 == 1)) continue;
      const GemmArgs& a = members[l];
      if (gg.n == 0) first = a;
      gg.W[gg.n] = a.W;
      gg.bias[gg.n] = a.bias;
      gg.out[gg.n] = a.out;
      gg.w_scale[gg.n] = a.w_scale;
      if (++gg.n == WAM_GEMM_GROUP_MAX) {
        LAUNCH(launch_gemm_group(pred(first), gg, s));
        gg.n = 0;
      }
    }
    if (gg.n > 0) LAUNCH(launch_gemm_group(pred(first), gg, s));
  }
  return WAM_OK;
}

struct StepWs {
  size_t x, e, e0, ctx, piece, block, pq, pq_layer, kv, kv_layer, total;
  int32_t nseg;
};
StepWs step_ws(const wam_model& m, const wam_step_io& io) {
  const wam_dims& D = m.dims;
  const size_t Lv = (size_t)io.F * (io.Hl / 2) * (io.Wl / 2), L = Lv + io.A, M = (size_t)io.B * L;
  StepWs w{};
  size_t off = 0;
  w.x = off; off += align256(M * D.d * 4);
  // time embeddings of t, then (DreamZero-Flash) of t_action
  w.e = off; off += align256((size_t)2 * io.B * D.d * 4);
  w.e0 = off; off += align256((size_t)2 * io.B * 6 * D.d * 4);
  w.ctx = off; off += align256((size_t)io.B * io.Lc * D.d * 2);
  // scratch for the time MLP, text projection, embedding and head (used one at a time)
  size_t piece = time_ws(D, io.B);
  piece = std::max(piece, text_ws(D, io.B, io.Lc));
  piece = std::max(piece, embed_ws(D, io.B, io.F, io.Hl, io.Wl));
  piece = std::max(piece, head_ws(D, io.B, io.F, io.Hl, io.Wl, io.A).total);
  w.piece = off; off += align256(piece);
  w.block = off; off += block_ws(D, io.B, (int32_t)L, io.Lc).total;
  // every block's folded AdaLN rows (two norms x B samples x segments x shift/scale)
  w.nseg = io.t_action != nullptr && io.A > 0 ? 2 : 1;
  w.pq_layer = (size_t)2 * io.B * w.nseg * 2 * D.d;  // floats
  w.pq = off; off += align256((size_t)std::max(D.n_layers, 0) * w.pq_layer * 4);
  // without ctx_kv: every block's cross K|V, projected before the first block.  Last, so
  // every other offset is the same with and without it.
  w.kv_layer = io.ctx_kv ? 0 : align256((size_t)io.B * io.Lc * 2 * D.d * 2);
  w.kv = off; off += (size_t)std::max(D.n_layers, 0) * w.kv_layer;
  w.total = off;
  return w;
}

wam_status check_ws(const void* ws, size_t have, size_t need) {
  CHECK(ws != nullptr, WAM_EWORKSPACE, "workspace is NULL (need %zu bytes)", need);
  CHECK((reinterpret_cast<uintptr_t>(ws) & 255) == 0, WAM_EWORKSPACE, "workspace must be 256-byte aligned");
  CHECK(have >= need, WAM_EWORKSPACE, "workspace %zu bytes < %zu needed", have, need);
  return WAM_OK;
}

wam_status check_step(const wam_model& m, const wam_step_io& io, bool head) {
  TRY(check_model_common(m));
  const wam_dims& D = m.dims;
  CHECK(D.n_layers >= 0, WAM_EINVAL, "n_layers < 0");
  CHECK(io.B >= 1 && io.B <= 8, WAM_EUNSUPPORTED, "B=%d outside [1,8]", io.B);
  CHECK(io.F >= 1 && io.Hl >= 2 && io.Wl >= 2 && io.Hl % 2 == 0 && io.Wl % 2 == 0, WAM_EINVAL,
        "latent F=%d Hl=%d Wl=%d (Hl, Wl even)", io.F, io.Hl, io.Wl);
  CHECK(io.A >= 0 && io.Lc >= 1, WAM_EINVAL, "A=%d Lc=%d", io.A, io.Lc);
  const int64_t L = (int64_t)io.F * (io.Hl / 2) * (io.Wl / 2) + io.A;
  CHECK(L < (1 << 30), WAM_EINVAL, "chunk too long");
  CHECK(io.cache_len >= 0 && io.cache_len + L <= io.Lcap, WAM_EINVAL, "cache_len=%d + L=%lld exceeds Lcap=%d",
        io.cache_len, (long long)L, io.Lcap);
  int32_t kend[WAM_MAX_CHUNKS];
  TRY(check_chunks(io.ch, (int32_t)L, (int32_t)(io.cache_len + L), kend));
  TRY(need_ptr(io.z_t, "z_t")); TRY(need_ptr(io.t, "t")); TRY(need_ptr(io.text, "text"));
  if (io.A > 0) TRY(need_ptr(io.a_t, "a_t"));
  if (io.A > 0 && head) TRY(need_ptr(io.v_action, "v_action"));
  TRY(need_ptr(io.rope_cos, "rope_cos")); TRY(need_ptr(io.rope_sin, "rope_sin"));
  if (head) TRY(need_ptr(io.v_video, "v_video"));
  TRY(need_ptr(m.w_t1, "w_t1")); TRY(need_ptr(m.w_t2, "w_t2")); TRY(need_ptr(m.w_t6, "w_t6"));
  TRY(need_ptr(m.w_x1, "w_x1")); TRY(need_ptr(m.w_x2, "w_x2")); TRY(need_ptr(m.w_patch, "w_patch"));
  if (head) { TRY(need_ptr(m.w_hv, "w_hv")); TRY(need_ptr(m.head_mod2, "head_mod2")); }
  if (io.A > 0) TRY(need_ptr(m.w_ain, "w_ain"));
  if (io.A > 0 && head) TRY(need_ptr(m.w_ha, "w_ha"));
  if (D.n_layers > 0) {
    CHECK(m.blocks != nullptr, WAM_EINVAL, "blocks is NULL");
    CHECK(io.k_cache != nullptr && io.v_cache != nullptr, WAM_EINVAL, "k_cache/v_cache arrays are NULL");
  }
  for (int l = 0; l < D.n_layers; ++l) {
    wam_status st = check_block_weights(m.blocks[l]);
    if (st != WAM_OK) return fail(st, "block %d: %s", l, g_err.c_str());
    CHECK(io.k_cache[l] && io.v_cache[l] && al16(io.k_cache[l]) && al16(io.v_cache[l]), WAM_EINVAL,
          "k_cache/v_cache[%d] NULL or misaligned", l);
    if (io.k_exp) {
      CHECK(D.Dh == 128, WAM_EUNSUPPORTED, "an FP8 KV cache needs Dh=128 (got %d)", D.Dh);
      CHECK(io.v_scale != nullptr, WAM_EINVAL, "k_exp given without v_scale");
      CHECK(io.k_exp[l] && al4(io.k_exp[l]), WAM_EINVAL, "k_exp[%d] NULL or misaligned", l);
      CHECK(std::isfinite(io.v_scale[l]) && io.v_scale[l] > 0.f, WAM_EINVAL, "v_scale[%d]=%g must be positive", l,
            (double)io.v_scale[l]);
    }
    if (io.ctx_kv) {
      CHECK(io.ctx_kv[l] && al16(io.ctx_kv[l]), WAM_EINVAL, "ctx_kv[%d] NULL or misaligned", l);
    } else if (m.blocks[l].fp8) {
      TRY(need_ptr(m.blocks[l].fp8->w_ckv, "fp8 w_ckv")); TRY(need_ptr(m.blocks[l].fp8->s_ckv, "fp8 s_ckv"));
    } else {
      TRY(need_ptr(m.blocks[l].w_ckv, "w_ckv"));
    }
  }
  return WAM_OK;
}

BlockEvents block_events(const wam_step_io& io, int l) {
  BlockEvents e;
  if (io.attn_events) {
    e.attn0 = io.attn_events[2 * l];
    e.attn1 = io.attn_events[2 * l + 1];
  }
  if (io.block_events) e.ev = io.block_events + (size_t)l * 2 * WAM_BLOCK_EVENTS;
  return e;
}

// Every block's combined AdaLN rows for this step's time embeddings (e0, and at alt_e0 the
// action rows' own), in chunks of at most ADALN_FOLD_MAX_LAYERS layers per launch.
wam_status fold_run(const wam_model& m, int32_t B, const float* e0, int64_t alt_e0, const StepWs& lay, char* w,
                    hipStream_t s) {
  const wam_dims& D = m.dims;
  for (int l0 = 0; l0 < D.n_layers; l0 += ADALN_FOLD_MAX_LAYERS) {
    AdalnFoldArgs a{};
    a.n_layers = std::min(D.n_layers - l0, ADALN_FOLD_MAX_LAYERS);
    a.d = D.d; a.B = B; a.nseg = lay.nseg;
    a.e0 = e0; a.e0_stride = 6 * (int64_t)D.d; a.alt = alt_e0;
    for (int i = 0; i < a.n_layers; ++i) a.mod6[i] = m.blocks[l0 + i].mod6;
    a.out = reinterpret_cast<float*>(w + lay.pq) + (size_t)l0 * lay.pq_layer;
    a.layer_stride = (int64_t)lay.pq_layer;
    a.skip = t_skip;
    LAUNCH(launch_adaln_fold(a, s));
  }
  return WAM_OK;
}

// The launch sequence of one step; arguments already validated.
wam_status step_run(const wam_model& m, const wam_step_io& io, char* w, hipStream_t stream) {
  const StepWs lay = step_ws(m, io);
  const wam_dims& D = m.dims;
  float* x = reinterpret_cast<float*>(w + lay.x);
  float* e = reinterpret_cast<float*>(w + lay.e);
  float* e0 = reinterpret_cast<float*>(w + lay.e0);
  void* ctx = w + lay.ctx;
  char* piece = w + lay.piece;
  const int32_t Lv = io.F * (io.Hl / 2) * (io.Wl / 2), L = Lv + io.A;

  TRY(time_run(m, io.B, io.t, e, e0, piece, stream));
  // DreamZero-Flash: the action rows' modulation comes from their own timestep
  const bool flash = io.t_action != nullptr && io.A > 0;
  const int64_t alt_e = flash ? (int64_t)io.B * D.d : 0, alt_e0 = flash ? (int64_t)io.B * 6 * D.d : 0;
  if (flash) TRY(time_run(m, io.B, io.t_action, e + alt_e, e0 + alt_e0, piece, stream));
  TRY(fold_run(m, io.B, e0, alt_e0, lay, w, stream));
  if (!io.ctx_kv) {
    TRY(text_run(m, io.B, io.Lc, io.text, ctx, piece, stream));
    const BlockWs bl = block_ws(D, io.B, L, io.Lc);
    TRY(cross_kv_run(m, io.B, io.Lc, ctx, w + lay.kv, lay.kv_layer, D.n_layers, w + lay.block + bl.q8,
                     reinterpret_cast<float*>(w + lay.block + bl.qs), stream));
  }
  TRY(embed_run(m, io.B, io.F, io.Hl, io.Wl, io.A, io.z_t, io.a_t, x, piece, stream));
  for (int l = 0; l < D.n_layers; ++l) {
    wam_block_io b{};
    b.x = x; b.e0 = e0; b.rope_cos = io.rope_cos; b.rope_sin = io.rope_sin;
    b.k_cache = io.k_cache[l]; b.v_cache = io.v_cache[l]; b.Lcap = io.Lcap; b.cache_len = io.cache_len;
    b.ch = io.ch; b.ctx = ctx; b.ctx_kv = io.ctx_kv ? io.ctx_kv[l] : w + lay.kv + (size_t)l * lay.kv_layer;
    b.B = io.B; b.L = L; b.Lc = io.Lc;
    b.k_exp = io.k_exp ? io.k_exp[l] : nullptr; b.v_scale = io.v_scale ? io.v_scale[l] : 1.0f;
    TRY(block_run(D, m.blocks[l], b, w + lay.block, stream, block_events(io, l), flash ? Lv : 0, alt_e0,
                  reinterpret_cast<const float*>(w + lay.pq) + (size_t)l * lay.pq_layer, lay.nseg));
  }
  TRY(head_run(m, io.B, io.F, io.Hl, io.Wl, io.A, x, e, io.v_video, io.v_action, piece, stream, alt_e));
  return WAM_OK;
}

// ---------------------------------------------------------------------------------
// denoising loop
// ---------------------------------------------------------------------------------
wam_status check_flow_dims(const wam_flow_dims& d) {
  CHECK(d.B >= 1 && d.n_video >= 0 && d.n_action >= 0, WAM_EINVAL, "flow dims B=%d n_video=%lld n_action=%lld",
        d.B, (long long)d.n_video, (long long)d.n_action);
  CHECK(!d.cfg || d.B == 2, WAM_EINVAL, "guidance needs a pair (B == 2), got B=%d", d.B);
  return WAM_OK;
}

FlowArgs flow_args(const wam_flow_dims& d) {
  FlowArgs f{};
  f.B = d.B; f.cfg = d.cfg ? 1 : 0; f.cfg_scale = d.cfg_scale;
  f.n_video = d.n_video; f.n_action = d.n_action;
  return f;
}

// UniPC on the straight path (alpha_t = t, sigma_t = 1 - t, lambda = log(alpha/sigma)).
// The exact solution from t_s is x_t = (sigma_t/sigma_s) x_s + sigma_t times the integral
// of e^lambda m over [lambda_s, lambda_t], m = x + (1 - t) v the data prediction.
// Expanding m in lambda turns the integral into alpha_t sum_k m^(k) I_k(h), with
// I_0 = 1 - e^-h and I_k = h^k/k! - I_(k-1).  An update with K other predictions m_j (at
// lambda_s + r_j h) uses the divided differences (m_j - m_s)/r_j, weighted by the
// solution a of sum_j a_j r_j^(k-1) = k! I_k / (h^k I_0), k = 1..K, so that it is exact
// for m of degree <= K in lambda.  The update as weights on x_s, m_s and the m_j:
struct UnipcW {
  double x, s, m[3];
};

double unipc_lambda(double t) { return std::log(t) - std::log1p(-t); }

// Solve the K x K system R a = b (K <= 3) by Gaussian elimination with partial pivoting.
bool solve_small(double R[3][3], double* b, int K, double* a) {
  for (int c = 0; c < K; ++c) {
    int piv = c;
    for (int r = c + 1; r < K; ++r)
      if (std::fabs(R[r][c]) > std::fabs(R[piv][c])) piv = r;
    if (!(std::fabs(R[piv][c]) > 0.0)) return false;
    if (piv != c) {
      for (int q = 0; q < K; ++q) std::swap(R[c][q], R[piv][q]);
      std::swap(b[c], b[piv]);
    }
    for (int r = c + 1; r < K; ++r) {
      const double f = R[r][c] / R[c][c];
      for (int q = c; q < K; ++q) R[r][q] -= f * R[c][q];
      b[r] -= f * b[c];
    }
  }
  for (int c = K - 1; c >= 0; --c) {
    double v = b[c];
    for (int q = c + 1; q < K; ++q) v -= R[c][q] * a[q];
    a[c] = v / R[c][c];
  }
  return true;
}

bool unipc_weights(double ts, double t, const double* tp, int K, UnipcW& w) {
  const double e = (ts * (1.0 - t)) / ((1.0 - ts) * t);  // e^-h (0 at t = 1)
  const double i0 = 1.0 - e;
  w.x = (1.0 - t) / (1.0 - ts);
  w.s = t * i0;
  w.m[0] = w.m[1] = w.m[2] = 0.0;
  if (K == 0) return true;
  const double h = unipc_lambda(t) - unipc_lambda(ts);
  double ik = i0, fact = 1.0, hk = 1.0, rhs[3], r[3], R[3][3], a[3];
  for (int k = 1; k <= K; ++k) {
    fact *= k;
    hk *= h;
    ik = hk / fact - ik;
    rhs[k - 1] = fact * ik / (hk * i0);
  }
  for (int j = 0; j < K; ++j) r[j] = (unipc_lambda(tp[j]) - unipc_lambda(ts)) / h;
  for (int k = 0; k < K; ++k)
    for (int j = 0; j < K; ++j) R[k][j] = std::pow(r[j], k);
  if (!solve_small(R, rhs, K, a)) return false;
  for (int j = 0; j < K; ++j) {
    w.m[j] = t * i0 * a[j] / r[j];
    w.s -= w.m[j];
  }
  return std::isfinite(w.x) && std::isfinite(w.s) && std::isfinite(w.m[0]) && std::isfinite(w.m[1]) &&
         std::isfinite(w.m[2]);
}

// The weights of every step of a schedule: step i corrects the state at t_i (after the
// first step) with the order of the predictor that produced it, then predicts t_(i+1) at
// order min(order, i + 1), or 1 when t_(i+1) = 1 (lambda is infinite there).
wam_status unipc_plan(const float* t_sched, int32_t n, int32_t order, wam_unipc_coef* out) {
  CHECK(t_sched != nullptr && out != nullptr, WAM_EINVAL, "NULL schedule or output");
  CHECK(n >= 1, WAM_EINVAL, "n_steps=%d must be >= 1", n);
  CHECK(order >= 1 && order <= 3, WAM_EINVAL, "UniPC order %d not in 1..3", order);
  CHECK(t_sched[0] > 0.f && t_sched[n] <= 1.f, WAM_EINVAL, "UniPC needs 0 < t_0 and t_N <= 1 (got %g, %g)",
        (double)t_sched[0], (double)t_sched[n]);
  for (int i = 0; i < n; ++i)
    CHECK(t_sched[i] < t_sched[i + 1], WAM_EINVAL, "schedule not increasing at %d (%g, %g)", i,
          (double)t_sched[i], (double)t_sched[i + 1]);
  int p_prev = 0;
  for (int i = 0; i < n; ++i) {
    const double t = t_sched[i], tn = t_sched[i + 1];
    wam_unipc_coef c{};
    c.s_v = (float)(1.0 - t);
    double tp[3];
    UnipcW w;
    if (i > 0) {  // corrector: from t_(i-1) with m_(i-2) .. m_(i-p_prev) and the new m_i
      for (int k = 1; k < p_prev; ++k) tp[k - 1] = t_sched[i - 1 - k];
      tp[p_prev - 1] = t;
      CHECK(unipc_weights(t_sched[i - 1], t, tp, p_prev, w), WAM_EINVAL, "UniPC weights of step %d not finite", i);
      c.correct = 1;
      c.c_x = (float)w.x;
      c.c_m[0] = (float)w.s;
      for (int k = 1; k < p_prev; ++k) c.c_m[k] = (float)w.m[k - 1];
      c.c_new = (float)w.m[p_prev - 1];
    }
    const int p = t_sched[i + 1] == 1.f ? 1 : std::min(order, i + 1);
    for (int k = 1; k < p; ++k) tp[k - 1] = t_sched[i - k];
    CHECK(unipc_weights(t, tn, tp, p - 1, w), WAM_EINVAL, "UniPC weights of step %d not finite", i);
    c.p_x = (float)w.x;
    c.p_new = (float)w.s;
    for (int k = 1; k < p; ++k) c.p_m[k - 1] = (float)w.m[k - 1];
    out[i] = c;
    p_prev = p;
  }
  return WAM_OK;
}

// One UniPC step's launch arguments; m_ring[j % 4] holds the data prediction of step j.
wam_status unipc_args(const wam_flow_dims& d, float* x, float* x_last, float* const* m_ring, int32_t step,
                      const wam_unipc_coef& c, UnipcArgs& u) {
  CHECK(step >= 0, WAM_EINVAL, "step %d < 0", step);
  CHECK(!c.correct || step >= 1, WAM_EINVAL, "the first step has nothing to correct");
  TRY(need_ptr(x, "x"));
  TRY(need_ptr(x_last, "x_last"));
  CHECK(m_ring != nullptr && m_ring[step % 4] != nullptr, WAM_EINVAL, "m_ring[%d] is NULL", step % 4);
  u = UnipcArgs{};
  u.f = flow_args(d);
  u.f.x = x;
  u.x_last = x_last;
  u.m_out = m_ring[step % 4];
  for (int q = 0; q < 3; ++q) {
    const bool used = (c.correct && c.c_m[q] != 0.f) || (q < 2 && c.p_m[q] != 0.f);
    if (!used) continue;
    CHECK(step - 1 - q >= 0, WAM_EINVAL, "step %d has no data prediction %d steps back", step, q + 1);
    CHECK(m_ring[(step - 1 - q) % 4] != nullptr, WAM_EINVAL, "m_ring[%d] is NULL", (step - 1 - q) % 4);
    u.m_hist[q] = m_ring[(step - 1 - q) % 4];
  }
  u.s_v = c.s_v;
  u.correct = c.correct;
  u.c_x = c.c_x;
  u.c_new = c.c_new;
  for (int q = 0; q < 3; ++q) u.c_m[q] = c.c_m[q];
  u.p_x = c.p_x;
  u.p_new = c.p_new;
  for (int q = 0; q < 2; ++q) u.p_m[q] = c.p_m[q];
  return WAM_OK;
}

struct DenoiseWs {
  size_t step, va, vb, cos, cos_out, state, xl, ring, total;
};
DenoiseWs denoise_ws(const wam_model& m, const wam_step_io& io, const wam_denoise_params& p) {
  const int64_t nx = p.cfg ? 1 : io.B;
  const int64_t n = (int64_t)m.dims.latent_ch * io.F * io.Hl * io.Wl + (int64_t)io.A * m.dims.act_dim;
  DenoiseWs w{};
  size_t off = 0;
  w.step = off; off += step_ws(m, io).total;
  w.va = off; off += align256((size_t)nx * n * 4);
  w.vb = off; off += align256((size_t)nx * n * 4);
  w.cos = off; off += align256(cosine_workspace_bytes());
  w.cos_out = off; off += 256;
  w.state = off; off += 256;
  // UniPC: the corrected state of the previous step and a ring of 4 data predictions
  const bool unipc = p.solver == WAM_SOLVER_UNIPC;
  w.xl = off; off += unipc ? align256((size_t)nx * n * 4) : 0;
  w.ring = off; off += unipc ? 4 * align256((size_t)nx * n * 4) : 0;
  w.total = off;
  return w;
}

// The update pass's launch sequence; arguments already validated.
wam_status update_run(const wam_model* m, const wam_step_io* io, void* ws, hipStream_t stream) {
  const StepWs lay = step_ws(*m, *io);
  const wam_dims& D = m->dims;
  char* w = static_cast<char*>(ws);
  float* x = reinterpret_cast<float*>(w + lay.x);
  float* e = reinterpret_cast<float*>(w + lay.e);
  float* e0 = reinterpret_cast<float*>(w + lay.e0);
  void* ctx = w + lay.ctx;
  char* piece = w + lay.piece;
  const int32_t Lv = io->F * (io->Hl / 2) * (io->Wl / 2), L = Lv + io->A;

  TRY(time_run(*m, io->B, io->t, e, e0, piece, stream));
  const bool flash = io->t_action != nullptr && io->A > 0;
  const int64_t alt_e0 = flash ? (int64_t)io->B * 6 * D.d : 0;
  if (flash) TRY(time_run(*m, io->B, io->t_action, e + (int64_t)io->B * D.d, e0 + alt_e0, piece, stream));
  TRY(fold_run(*m, io->B, e0, alt_e0, lay, w, stream));
  // the last block only projects its K/V, so the cross K|V of the others
  if (!io->ctx_kv && D.n_layers > 1) {
    TRY(text_run(*m, io->B, io->Lc, io->text, ctx, piece, stream));
    const BlockWs bl = block_ws(D, io->B, L, io->Lc);
    TRY(cross_kv_run(*m, io->B, io->Lc, ctx, w + lay.kv, lay.kv_layer, D.n_layers - 1, w + lay.block + bl.q8,
                     reinterpret_cast<float*>(w + lay.block + bl.qs), stream));
  }
  TRY(embed_run(*m, io->B, io->F, io->Hl, io->Wl, io->A, io->z_t, io->a_t, x, piece, stream));
  for (int l = 0; l < D.n_layers; ++l) {
    wam_block_io b{};
    b.x = x; b.e0 = e0; b.rope_cos = io->rope_cos; b.rope_sin = io->rope_sin;
    b.k_cache = io->k_cache[l]; b.v_cache = io->v_cache[l]; b.Lcap = io->Lcap; b.cache_len = io->cache_len;
    b.ch = io->ch; b.ctx = ctx;
    b.ctx_kv = io->ctx_kv ? io->ctx_kv[l] : w + lay.kv + (size_t)l * lay.kv_layer;
    b.B = io->B; b.L = L; b.Lc = io->Lc;
    b.k_exp = io->k_exp ? io->k_exp[l] : nullptr; b.v_scale = io->v_scale ? io->v_scale[l] : 1.0f;
    const float* pq = reinterpret_cast<const float*>(w + lay.pq) + (size_t)l * lay.pq_layer;
    if (l + 1 == D.n_layers) {
      TRY(block_kv_run(D, m->blocks[l], b, w + lay.block, stream, flash ? Lv : 0, alt_e0, pq, lay.nseg));
    } else {
      TRY(block_run(D, m->blocks[l], b, w + lay.block, stream, block_events(*io, l), flash ? Lv : 0, alt_e0, pq,
                    lay.nseg));
    }
  }
  return WAM_OK;
}

}  // namespace

// =================================================================================
// exported entry points
// =================================================================================
extern "C" {

const char* wam_last_error(void) { return g_err.c_str(); }
int32_t wam_abi_version(void) { return WAM_ABI_VERSION; }

wam_status wam_attn_blockcausal(const wam_attn_desc* desc, const void* q, const void* k, const void* v, void* o,
                                hipStream_t stream) {
  CHECK(desc != nullptr, WAM_EINVAL, "desc is NULL");
  return attn_checked(*desc, q, k, v, o, stream);
}

wam_status wam_attn_blockcausal_mx(const wam_attn_desc* desc, const void* q, const void* k, const void* v, void* o8,
                                   void* o_exp, int64_t o_lde, hipStream_t stream) {
  CHECK(desc != nullptr, WAM_EINVAL, "desc is NULL");
  CHECK(o_exp != nullptr || desc->B == 0 || desc->Lq == 0, WAM_EINVAL, "o_exp is NULL");
  return attn_checked(*desc, q, k, v, o8, stream, o_exp, o_lde);
}

wam_status wam_gemm_bf16(const wam_gemm_desc* g, hipStream_t stream) {
  CHECK(g != nullptr, WAM_EINVAL, "desc is NULL");
  return gemm_checked(*g, stream);
}

wam_status wam_gemm_fp8(const wam_gemm_desc* g, const float* a_scale, const float* w_scale, hipStream_t stream) {
  CHECK(g != nullptr, WAM_EINVAL, "NULL descriptor");
  CHECK(a_scale != nullptr && w_scale != nullptr, WAM_EINVAL, "a_scale and w_scale are required");
  return gemm_checked(*g, stream, 0, 0, a_scale, w_scale);
}

wam_status wam_gemm_fp8_mx(const wam_gemm_desc* g, const float* a_scale, const void* a_exp, int64_t a_lde,
                           const float* w_scale, void* out_exp, int64_t o_lde, hipStream_t stream) {
  CHECK(g != nullptr, WAM_EINVAL, "NULL descriptor");
  CHECK(w_scale != nullptr, WAM_EINVAL, "w_scale is required");
  return gemm_fp8_blocks(*g, a_scale, a_exp, a_lde, w_scale, out_exp, o_lde, stream);
}

wam_status wam_quantize_rows_fp8(int32_t M, int32_t K, const void* x, int64_t ldx, void* q, int64_t ldq,
                                 float* scale, hipStream_t stream) {
  CHECK(M >= 0 && K >= 8 && K % 8 == 0, WAM_EINVAL, "M=%d K=%d (need K >= 8, K %% 8 == 0)", M, K);
  CHECK(ldx >= K && ldx % 8 == 0 && ldq >= K && ldq % 16 == 0, WAM_EINVAL,
        "ldx must be >= K and a multiple of 8; ldq >= K and a multiple of 16");
  if (M == 0) return WAM_OK;
  TRY(need_ptr(x, "x")); TRY(need_ptr(q, "q")); TRY(need_ptr(scale, "scale"));
  HIPCHECK(launch_quant_rows(M, K, x, ldx, q, ldq, scale, stream));
  return WAM_OK;
}

wam_status wam_adaln_ln_mod(int32_t B, int32_t rows_per_batch, int32_t d, float eps, const float* x,
                            const float* gamma, const float* beta, const float* shift_a, const float* shift_v,
                            const float* scale_a, const float* scale_v, int64_t mod_stride, void* h,
                            hipStream_t stream) {
  CHECK(B >= 0 && rows_per_batch >= 0, WAM_EINVAL, "negative sizes");
  CHECK(d % 256 == 0 && d >= 256 && d <= 8192, WAM_EUNSUPPORTED, "d=%d must be a multiple of 256 in [256, 8192]", d);
  CHECK(eps > 0.f, WAM_EINVAL, "eps must be > 0");
  if ((int64_t)B * rows_per_batch == 0) return WAM_OK;
  CHECK((int64_t)B * rows_per_batch < (1ll << 31), WAM_EINVAL, "too many rows");
  TRY(need_ptr(x, "x")); TRY(need_ptr(h, "h"));
  TRY(opt_ptr(gamma, "gamma")); TRY(opt_ptr(beta, "beta"));
  TRY(opt_ptr(shift_a, "shift_a")); TRY(opt_ptr(shift_v, "shift_v"));
  TRY(opt_ptr(scale_a, "scale_a")); TRY(opt_ptr(scale_v, "scale_v"));
  CHECK(mod_stride % 4 == 0, WAM_EINVAL, "mod_stride must be a multiple of 4");
  LnArgs a{B * rows_per_batch, rows_per_batch, d, eps, x, gamma, beta, shift_a, shift_v, scale_a, scale_v,
           mod_stride, h};
  HIPCHECK(launch_ln_mod(a, stream));
  return WAM_OK;
}

wam_status wam_adaln_ln_mod_fp8(int32_t B, int32_t rows_per_batch, int32_t d, float eps, const float* x,
                                const float* gamma, const float* beta, const float* shift_a, const float* shift_v,
                                const float* scale_a, const float* scale_v, int64_t mod_stride, void* q,
                                int64_t ldq, float* scale, hipStream_t stream) {
  CHECK(B >= 0 && rows_per_batch >= 0, WAM_EINVAL, "negative sizes");
  CHECK(ln_fp8_supported(d), WAM_EUNSUPPORTED, "d=%d must be a multiple of 512 in [512, 5120]", d);
  CHECK(eps > 0.f, WAM_EINVAL, "eps must be > 0");
  CHECK(ldq >= d && ldq % 16 == 0, WAM_EINVAL, "ldq must be >= d and a multiple of 16");
  if ((int64_t)B * rows_per_batch == 0) return WAM_OK;
  CHECK((int64_t)B * rows_per_batch < (1ll << 31), WAM_EINVAL, "too many rows");
  TRY(need_ptr(x, "x")); TRY(need_ptr(q, "q")); TRY(need_ptr(scale, "scale"));
  TRY(opt_ptr(gamma, "gamma")); TRY(opt_ptr(beta, "beta"));
  TRY(opt_ptr(shift_a, "shift_a")); TRY(opt_ptr(shift_v, "shift_v"));
  TRY(opt_ptr(scale_a, "scale_a")); TRY(opt_ptr(scale_v, "scale_v"));
  CHECK(mod_stride % 4 == 0, WAM_EINVAL, "mod_stride must be a multiple of 4");
  LnArgs a{B * rows_per_batch, rows_per_batch, d, eps, x, gamma, beta, shift_a, shift_v, scale_a, scale_v,
           mod_stride, nullptr};
  a.q8 = static_cast<uint8_t*>(q);
  a.ldq = ldq;
  a.q_scale = scale;
  HIPCHECK(launch_ln_mod(a, stream));
  return WAM_OK;
}

wam_status wam_rope_qkv(int32_t B, int32_t L, int32_t H, int32_t Dh, const void* qkv, const float* rope_cos,
                        const float* rope_sin, void* q_out, void* k_cache, void* v_cache, int32_t Lcap,
                        int32_t row0, hipStream_t stream) {
  CHECK(Dh == 64 || Dh == 128, WAM_EUNSUPPORTED, "Dh=%d (supported: 64, 128)", Dh);
  CHECK(B >= 0 && L >= 0 && H >= 1, WAM_EINVAL, "bad sizes B=%d L=%d H=%d", B, L, H);
  CHECK(row0 >= 0 && (int64_t)row0 + L <= Lcap, WAM_EINVAL, "row0=%d + L=%d exceeds Lcap=%d", row0, L, Lcap);
  if ((int64_t)B * L == 0) return WAM_OK;
  TRY(need_ptr(qkv, "qkv")); TRY(need_ptr(rope_cos, "rope_cos")); TRY(need_ptr(rope_sin, "rope_sin"));
  TRY(need_ptr(q_out, "q_out")); TRY(need_ptr(k_cache, "k_cache")); TRY(need_ptr(v_cache, "v_cache"));
  RopeArgs a{B, L, H, Dh, Lcap, row0, qkv, rope_cos, rope_sin, q_out, k_cache, v_cache};
  HIPCHECK(launch_rope_qkv(a, stream));
  return WAM_OK;
}

wam_status wam_attn_blockcausal_fp8(const wam_attn_desc* desc, const void* q8, const void* q_exp, const void* k8,
                                    const void* k_exp, const void* v8, float v_scale, void* o, hipStream_t stream) {
  CHECK(desc != nullptr, WAM_EINVAL, "NULL descriptor");
  return attn_fp8_checked(*desc, q8, q_exp, k8, k_exp, v8, v_scale, o, stream);
}

wam_status wam_attn_blockcausal_fp8_mx(const wam_attn_desc* desc, const void* q8, const void* q_exp, const void* k8,
                                       const void* k_exp, const void* v8, float v_scale, void* o8, void* o_exp,
                                       int64_t o_lde, hipStream_t stream) {
  CHECK(desc != nullptr, WAM_EINVAL, "NULL descriptor");
  CHECK(o_exp != nullptr || desc->B == 0 || desc->Lq == 0, WAM_EINVAL, "o_exp is NULL");
  return attn_fp8_checked(*desc, q8, q_exp, k8, k_exp, v8, v_scale, o8, stream, o_exp, o_lde);
}

wam_status wam_quantize_mx_fp8(int32_t rows, int32_t cols, const void* x, int64_t ldx, void* q8, int64_t ldq,
                               void* exps, hipStream_t stream) {
  CHECK(rows >= 0 && cols >= 0 && cols % 32 == 0, WAM_EINVAL, "rows=%d cols=%d (cols a multiple of 32)", rows,
        cols);
  CHECK(ldx >= cols && ldx % 8 == 0 && ldq >= cols && ldq % 8 == 0, WAM_EINVAL,
        "ldx=%lld ldq=%lld must be >= cols and multiples of 8", (long long)ldx, (long long)ldq);
  if ((int64_t)rows * cols == 0) return WAM_OK;
  TRY(need_ptr(x, "x")); TRY(need_ptr(q8, "q8")); TRY(need_ptr(exps, "exps"));
  CHECK(al16(x) && (reinterpret_cast<uintptr_t>(q8) & 7) == 0, WAM_EINVAL, "x must be 16-byte, q8 8-byte aligned");
  HIPCHECK(launch_quant_mx(rows, cols, x, ldx, q8, ldq, exps, stream));
  return WAM_OK;
}

wam_status wam_quantize_scaled_fp8(int64_t n, const void* x, float scale, void* q8, hipStream_t stream) {
  CHECK(n >= 0 && n % 8 == 0, WAM_EINVAL, "n=%lld must be a non-negative multiple of 8", (long long)n);
  CHECK(std::isfinite(scale) && scale > 0.f, WAM_EINVAL, "scale=%g must be positive and finite", (double)scale);
  if (n == 0) return WAM_OK;
  TRY(need_ptr(x, "x")); TRY(need_ptr(q8, "q8"));
  CHECK(al16(x) && (reinterpret_cast<uintptr_t>(q8) & 7) == 0, WAM_EINVAL, "x must be 16-byte, q8 8-byte aligned");
  HIPCHECK(launch_quant_scaled(n, x, 1.0f / scale, q8, stream));
  return WAM_OK;
}

wam_status wam_rope_qkv_fp8(int32_t B, int32_t L, int32_t H, int32_t Dh, const void* qkv, const float* rope_cos,
                            const float* rope_sin, void* q8, void* q_exp, void* k8_cache, void* k_exp,
                            void* v8_cache, float v_scale, int32_t Lcap, int32_t row0, hipStream_t stream) {
  CHECK(Dh == 128, WAM_EUNSUPPORTED, "the FP8 append needs Dh=128 (got %d)", Dh);
  CHECK(B >= 0 && L >= 0 && H >= 1, WAM_EINVAL, "bad sizes B=%d L=%d H=%d", B, L, H);
  CHECK(row0 >= 0 && (int64_t)row0 + L <= Lcap, WAM_EINVAL, "row0=%d + L=%d exceeds Lcap=%d", row0, L, Lcap);
  CHECK(std::isfinite(v_scale) && v_scale > 0.f, WAM_EINVAL, "v_scale=%g must be positive and finite",
        (double)v_scale);
  CHECK((q8 == nullptr) == (q_exp == nullptr), WAM_EINVAL, "q8 and q_exp must both be given or both be NULL");
  if ((int64_t)B * L == 0) return WAM_OK;
  TRY(need_ptr(qkv, "qkv")); TRY(need_ptr(rope_cos, "rope_cos")); TRY(need_ptr(rope_sin, "rope_sin"));
  TRY(need_ptr(k8_cache, "k8_cache")); TRY(need_ptr(k_exp, "k_exp")); TRY(need_ptr(v8_cache, "v8_cache"));
  CHECK(al16(qkv) && (reinterpret_cast<uintptr_t>(k8_cache) & 7) == 0 &&
            (reinterpret_cast<uintptr_t>(v8_cache) & 7) == 0 && (!q8 || (reinterpret_cast<uintptr_t>(q8) & 7) == 0),
        WAM_EINVAL, "qkv must be 16-byte, code buffers 8-byte aligned");
  RopeArgs a{B, L, H, Dh, Lcap, row0, qkv, rope_cos, rope_sin, q8, k8_cache, v8_cache};
  RopeFp8Args f{a, q_exp, k_exp, 1.0f / v_scale};
  HIPCHECK(launch_rope_qkv_fp8(f, stream));
  return WAM_OK;
}

size_t wam_block_workspace_bytes(const wam_dims* dims, int32_t B, int32_t L, int32_t Lc) {
  if (!dims || B < 0 || L < 0 || Lc < 0) return 0;
  return block_ws(*dims, B, L, Lc).total;
}

wam_status wam_dit_block_fwd(const wam_dims* dims, const wam_block_weights* w, const wam_block_io* io, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  CHECK(dims && w && io, WAM_EINVAL, "NULL dims/weights/io");
  TRY(check_dims(*dims));
  TRY(check_block_weights(*w));
  TRY(check_block_io(*dims, *w, *io));
  TRY(check_ws(ws, ws_bytes, block_ws(*dims, io->B, io->L, io->Lc).total));
  {
    DryScope dry;
    TRY(block_run(*dims, *w, *io, static_cast<char*>(ws), stream));
  }
  return block_run(*dims, *w, *io, static_cast<char*>(ws), stream);
}

size_t wam_time_embed_workspace_bytes(const wam_dims* dims, int32_t B) {
  if (!dims || B < 0) return 0;
  return time_ws(*dims, B);
}

wam_status wam_time_embed_fwd(const wam_model* m, int32_t B, const float* t, float* e, float* e0, void* ws,
                              size_t ws_bytes, hipStream_t stream) {
  CHECK(m != nullptr, WAM_EINVAL, "model is NULL");
  TRY(check_model_common(*m));
  CHECK(B >= 1 && B <= 8, WAM_EUNSUPPORTED, "B=%d outside [1,8]", B);
  TRY(need_ptr(t, "t")); TRY(need_ptr(e, "e")); TRY(need_ptr(e0, "e0"));
  TRY(need_ptr(m->w_t1, "w_t1")); TRY(need_ptr(m->w_t2, "w_t2")); TRY(need_ptr(m->w_t6, "w_t6"));
  TRY(check_ws(ws, ws_bytes, time_ws(m->dims, B)));
  return time_run(*m, B, t, e, e0, static_cast<char*>(ws), stream);
}

size_t wam_text_proj_workspace_bytes(const wam_dims* dims, int32_t B, int32_t Lc) {
  if (!dims || B < 0 || Lc < 0) return 0;
  return text_ws(*dims, B, Lc);
}

wam_status wam_text_proj_fwd(const wam_model* m, int32_t B, int32_t Lc, const void* text, void* ctx, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  CHECK(m != nullptr, WAM_EINVAL, "model is NULL");
  TRY(check_model_common(*m));
  CHECK(B >= 1 && Lc >= 1, WAM_EINVAL, "B=%d Lc=%d", B, Lc);
  TRY(need_ptr(text, "text")); TRY(need_ptr(ctx, "ctx"));
  TRY(need_ptr(m->w_x1, "w_x1")); TRY(need_ptr(m->w_x2, "w_x2"));
  TRY(check_ws(ws, ws_bytes, text_ws(m->dims, B, Lc)));
  return text_run(*m, B, Lc, text, ctx, static_cast<char*>(ws), stream);
}

size_t wam_embed_workspace_bytes(const wam_dims* dims, int32_t B, int32_t F, int32_t Hl, int32_t Wl) {
  if (!dims || B < 0 || F < 0 || Hl < 0 || Wl < 0) return 0;
  return embed_ws(*dims, B, F, Hl, Wl);
}

wam_status wam_embed_fwd(const wam_model* m, int32_t B, int32_t F, int32_t Hl, int32_t Wl, int32_t A,
                         const void* z_t, const void* a_t, float* x, void* ws, size_t ws_bytes,
                         hipStream_t stream) {
  CHECK(m != nullptr, WAM_EINVAL, "model is NULL");
  TRY(check_model_common(*m));
  CHECK(B >= 1 && F >= 1 && Hl >= 2 && Wl >= 2 && Hl % 2 == 0 && Wl % 2 == 0 && A >= 0, WAM_EINVAL,
        "bad latent/action sizes");
  TRY(need_ptr(z_t, "z_t")); TRY(need_ptr(x, "x")); TRY(need_ptr(m->w_patch, "w_patch"));
  if (A > 0) { TRY(need_ptr(a_t, "a_t")); TRY(need_ptr(m->w_ain, "w_ain")); }
  TRY(check_ws(ws, ws_bytes, embed_ws(m->dims, B, F, Hl, Wl)));
  return embed_run(*m, B, F, Hl, Wl, A, z_t, a_t, x, static_cast<char*>(ws), stream);
}

size_t wam_head_workspace_bytes(const wam_dims* dims, int32_t B, int32_t F, int32_t Hl, int32_t Wl, int32_t A) {
  if (!dims || B < 0 || F < 0 || Hl < 0 || Wl < 0 || A < 0) return 0;
  return head_ws(*dims, B, F, Hl, Wl, A).total;
}

wam_status wam_head_fwd(const wam_model* m, int32_t B, int32_t F, int32_t Hl, int32_t Wl, int32_t A,
                        const float* x, const float* e, float* v_video, float* v_action, void* ws,
                        size_t ws_bytes, hipStream_t stream) {
  CHECK(m != nullptr, WAM_EINVAL, "model is NULL");
  TRY(check_model_common(*m));
  CHECK(B >= 1 && B <= 8 && F >= 1 && Hl >= 2 && Wl >= 2 && Hl % 2 == 0 && Wl % 2 == 0 && A >= 0, WAM_EINVAL,
        "bad latent/action sizes");
  TRY(need_ptr(x, "x")); TRY(need_ptr(e, "e")); TRY(need_ptr(v_video, "v_video"));
  TRY(need_ptr(m->w_hv, "w_hv")); TRY(need_ptr(m->head_mod2, "head_mod2"));
  if (A > 0) { TRY(need_ptr(v_action, "v_action")); TRY(need_ptr(m->w_ha, "w_ha")); }
  TRY(check_ws(ws, ws_bytes, head_ws(m->dims, B, F, Hl, Wl, A).total));
  return head_run(*m, B, F, Hl, Wl, A, x, e, v_video, v_action, static_cast<char*>(ws), stream);
}

size_t wam_step_workspace_bytes(const wam_model* m, const wam_step_io* io) {
  if (!m || !io || io->B < 0 || io->F < 0 || io->Hl < 0 || io->Wl < 0 || io->A < 0 || io->Lc < 0) return 0;
  return step_ws(*m, *io).total;
}

wam_status wam_dit_step_fwd(const wam_model* m, const wam_step_io* io, void* ws, size_t ws_bytes,
                            hipStream_t stream) {
  CHECK(m && io, WAM_EINVAL, "NULL model/io");
  TRY(check_step(*m, *io, true));
  TRY(check_ws(ws, ws_bytes, step_ws(*m, *io).total));
  {
    DryScope dry;
    TRY(step_run(*m, *io, static_cast<char*>(ws), stream));
  }
  return step_run(*m, *io, static_cast<char*>(ws), stream);
}

size_t wam_update_workspace_bytes(const wam_model* m, const wam_step_io* io) {
  return wam_step_workspace_bytes(m, io);
}

wam_status wam_dit_update_fwd(const wam_model* m, const wam_step_io* io, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  CHECK(m && io, WAM_EINVAL, "NULL model/io");
  TRY(check_step(*m, *io, false));
  TRY(check_ws(ws, ws_bytes, step_ws(*m, *io).total));
  {
    DryScope dry;
    TRY(update_run(m, io, ws, stream));
  }
  return update_run(m, io, ws, stream);
}

wam_status wam_flow_step(const wam_flow_dims* d, const float* v_video, const float* v_action, const float* v_in,
                         float* x, float* v_out, float t, float t_next, void* z_next, void* a_next,
                         hipStream_t stream) {
  CHECK(d != nullptr, WAM_EINVAL, "NULL dims");
  TRY(check_flow_dims(*d));
  TRY(need_ptr(x, "x"));
  if (d->n_video > 0) TRY(need_ptr(z_next, "z_next"));
  if (d->n_action > 0) TRY(need_ptr(a_next, "a_next"));
  if (!v_in && (v_video || v_action)) {
    if (d->n_video > 0) TRY(need_ptr(v_video, "v_video"));
    if (d->n_action > 0) TRY(need_ptr(v_action, "v_action"));
  }
  FlowArgs f = flow_args(*d);
  f.dt = t_next - t;
  f.v_in = v_in;
  if (!v_in) { f.v_video = v_video; f.v_action = v_action; }
  f.x = x; f.v_out = v_out; f.z_next = z_next; f.a_next = a_next;
  HIPCHECK(launch_flow_step(f, stream));
  return WAM_OK;
}

wam_status wam_unipc_plan(const float* t_sched, int32_t n_steps, int32_t order, wam_unipc_coef* out) {
  return unipc_plan(t_sched, n_steps, order, out);
}

wam_status wam_unipc_step(const wam_flow_dims* d, const float* v_video, const float* v_action, const float* v_in,
                          float* x, float* x_last, float* const* m_ring, int32_t step, const wam_unipc_coef* c,
                          float* v_out, void* z_next, void* a_next, hipStream_t stream) {
  CHECK(d != nullptr && c != nullptr, WAM_EINVAL, "NULL dims or coefficients");
  TRY(check_flow_dims(*d));
  if (d->n_video > 0) TRY(need_ptr(z_next, "z_next"));
  if (d->n_action > 0) TRY(need_ptr(a_next, "a_next"));
  if (!v_in) {
    if (d->n_video > 0) TRY(need_ptr(v_video, "v_video"));
    if (d->n_action > 0) TRY(need_ptr(v_action, "v_action"));
  }
  UnipcArgs u;
  TRY(unipc_args(*d, x, x_last, m_ring, step, *c, u));
  u.f.v_in = v_in;
  if (!v_in) { u.f.v_video = v_video; u.f.v_action = v_action; }
  u.f.v_out = v_out; u.f.z_next = z_next; u.f.a_next = a_next;
  HIPCHECK(launch_unipc_step(u, stream));
  return WAM_OK;
}

size_t wam_cosine_workspace_bytes(void) { return cosine_workspace_bytes(); }

wam_status wam_cosine_similarity(const float* a, const float* b, int64_t n, void* ws, size_t ws_bytes, float* out,
                                 hipStream_t stream) {
  CHECK(n >= 0, WAM_EINVAL, "n < 0");
  TRY(need_ptr(out, "out"));
  if (n > 0) { TRY(need_ptr(a, "a")); TRY(need_ptr(b, "b")); }
  CHECK(ws != nullptr && ws_bytes >= cosine_workspace_bytes(), WAM_EWORKSPACE, "workspace %zu < %zu bytes", ws_bytes,
        cosine_workspace_bytes());
  HIPCHECK(launch_cosine(a, b, n, ws, out, stream));
  return WAM_OK;
}

wam_status wam_cosine_similarity_noalloc(const float* a, const float* b, int64_t n, float* out,
                                         hipStream_t stream) {
  CHECK(n >= 0, WAM_EINVAL, "n < 0");
  TRY(need_ptr(out, "out"));
  if (n > 0) { TRY(need_ptr(a, "a")); TRY(need_ptr(b, "b")); }
  CHECK(cosine_workspace_bytes() <= cosine_static_scratch_bytes(), WAM_EWORKSPACE,
        "the partial sums need %zu bytes, the static scratch holds %zu", cosine_workspace_bytes(),
        cosine_static_scratch_bytes());
  void* part = nullptr;
  HIPCHECK(cosine_static_scratch(&part));
  HIPCHECK(launch_cosine(a, b, n, part, out, stream));
  return WAM_OK;
}

size_t wam_denoise_workspace_bytes(const wam_model* m, const wam_step_io* io, const wam_denoise_params* p) {
  if (!m || !io || !p || io->B < 0 || io->F < 0 || io->Hl < 0 || io->Wl < 0 || io->A < 0 || io->Lc < 0) return 0;
  return denoise_ws(*m, *io, *p).total;
}

wam_status wam_denoise_chunk(const wam_model* m, const wam_step_io* io, const wam_denoise_params* p, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  CHECK(m && io && p, WAM_EINVAL, "NULL model/io/params");
  TRY(check_step(*m, *io, true));
  CHECK(p->n_steps >= 1, WAM_EINVAL, "n_steps=%d must be >= 1", p->n_steps);
  CHECK(p->t_sched != nullptr, WAM_EINVAL, "t_sched is NULL");
  CHECK(p->cache_window >= 0, WAM_EINVAL, "cache_window < 0");
  CHECK(io->t_action == nullptr, WAM_EUNSUPPORTED, "the loop runs one schedule for both modalities (t_action must be NULL)");
  CHECK(p->solver == WAM_SOLVER_EULER || p->solver == WAM_SOLVER_UNIPC, WAM_EINVAL, "unknown solver %d", p->solver);
  TRY(need_ptr(p->x, "x"));
  const bool unipc = p->solver == WAM_SOLVER_UNIPC;
  std::vector<wam_unipc_coef> plan(unipc ? p->n_steps : 0);
  if (unipc) TRY(unipc_plan(p->t_sched, p->n_steps, p->solver_order, plan.data()));
  wam_flow_dims fd{};
  fd.B = io->B; fd.cfg = p->cfg; fd.cfg_scale = p->cfg_scale;
  fd.n_video = (int64_t)m->dims.latent_ch * io->F * io->Hl * io->Wl;
  fd.n_action = (int64_t)io->A * m->dims.act_dim;
  TRY(check_flow_dims(fd));
  const DenoiseWs lay = denoise_ws(*m, *io, *p);
  TRY(check_ws(ws, ws_bytes, lay.total));
  char* w = static_cast<char*>(ws);
  // vcur: the latest computed velocity (what a reused step applies), vprev: the one before
  float* vcur = reinterpret_cast<float*>(w + lay.va);
  float* vprev = reinterpret_cast<float*>(w + lay.vb);
  float* cs_dev = reinterpret_cast<float*>(w + lay.cos_out);
  int32_t* st = reinterpret_cast<int32_t*>(w + lay.state);
  void* z = const_cast<void*>(io->z_t);
  void* a = const_cast<void*>(io->a_t);
  float* t_dev = const_cast<float*>(io->t);
  const int64_t n = (int64_t)(p->cfg ? 1 : io->B) * (fd.n_video + fd.n_action);
  const bool caching = p->cache_window > 0;
  float* xl = reinterpret_cast<float*>(w + lay.xl);
  float* ring[4];
  for (int q = 0; q < 4; ++q) ring[q] = reinterpret_cast<float*>(w + lay.ring + q * align256((size_t)n * 4));
  std::vector<UnipcArgs> uargs(plan.size());
  for (size_t i = 0; i < plan.size(); ++i) TRY(unipc_args(fd, p->x, xl, ring, (int32_t)i, plan[i], uargs[i]));

  {  // every launch of a step validated before the first launch of the loop
    DryScope dry;
    TRY(step_run(*m, *io, w + lay.step, stream));
  }

  // The text and so every block's cross-attention K|V are the same at every step of
  // the chunk: unless the caller supplied them, project them once here, into the step
  // workspace's cross K|V region (the last region, so the step's other offsets are the
  // same with ctx_kv given), and let each step read them (the same GEMMs a step would
  // run, so the results are unchanged).
  wam_step_io sio = *io;
  std::vector<const void*> kv_ptrs;
  if (!io->ctx_kv && m->dims.n_layers > 0) {
    const wam_dims& D = m->dims;
    const StepWs sl = step_ws(*m, *io);
    char* sw = w + lay.step;
    const int32_t L = io->F * (io->Hl / 2) * (io->Wl / 2) + io->A;
    const BlockWs bl = block_ws(D, io->B, L, io->Lc);
    void* ctx = sw + sl.ctx;
    TRY(text_run(*m, io->B, io->Lc, io->text, ctx, sw + sl.piece, stream));
    TRY(cross_kv_run(*m, io->B, io->Lc, ctx, sw + sl.kv, sl.kv_layer, D.n_layers, sw + sl.block + bl.q8,
                     reinterpret_cast<float*>(sw + sl.block + bl.qs), stream));
    kv_ptrs.resize(D.n_layers);
    for (int l = 0; l < D.n_layers; ++l) kv_ptrs[l] = sw + sl.kv + (size_t)l * sl.kv_layer;
    sio.ctx_kv = kv_ptrs.data();
  }

  // the model inputs of the first call from the initial state
  FlowArgs q = flow_args(fd);
  q.x = p->x; q.z_next = z; q.a_next = a;
  HIPCHECK(launch_flow_step(q, stream));
  // With caching the reuse decision lives in st on the device: a reused step's kernels
  // return at entry, the solver step applies vcur, and nothing waits for the host.
  if (caching || p->computed) HIPCHECK(launch_loop_init(st, stream));
  for (int i = 0; i < p->n_steps; ++i) {
    HIPCHECK(launch_fill(t_dev, io->B, p->t_sched[i], stream));
    {
      SkipScope scope(caching ? st : nullptr);
      TRY(step_run(*m, sio, w + lay.step, stream));
    }
    FlowArgs f = flow_args(fd);
    f.dt = p->t_sched[i + 1] - p->t_sched[i];
    f.x = p->x; f.z_next = z; f.a_next = a;
    f.v_video = io->v_video; f.v_action = io->v_action;
    if (caching) {
      f.v_in = vcur; f.v_out = vcur; f.skip = st;
    }
    if (unipc) {
      UnipcArgs u = uargs[i];
      u.f = f;
      HIPCHECK(launch_unipc_step(u, stream));
    } else {
      HIPCHECK(launch_flow_step(f, stream));
    }
    if (caching) HIPCHECK(launch_cosine(vcur, vprev, n, w + lay.cos, cs_dev, stream, st));
    if (caching || p->computed)
      HIPCHECK(launch_loop_decide(st, cs_dev, p->cache_tau, p->cache_window, p->computed, i, stream));
    if (caching) HIPCHECK(launch_copy_if(st + 2, vcur, vprev, n, stream));
  }
  return WAM_OK;
}

wam_status wam_chunk_positions(int32_t c, int32_t F, int32_t Hg, int32_t Wg, int32_t A, int32_t* pos) {
  CHECK(pos != nullptr, WAM_EINVAL, "pos is NULL");
  CHECK(c >= 0 && F >= 1 && Hg >= 1 && Wg >= 1 && A >= 0, WAM_EINVAL, "bad chunk geometry");
  int64_t i = 0;
  for (int f = 0; f < F; ++f)
    for (int r = 0; r < Hg; ++r)
      for (int s = 0; s < Wg; ++s, ++i) {
        pos[3 * i + 0] = F * c + f;
        pos[3 * i + 1] = r;
        pos[3 * i + 2] = s;
      }
  for (int j = 0; j < A; ++j, ++i) {
    pos[3 * i + 0] = F * c + F + j;
    pos[3 * i + 1] = 0;
    pos[3 * i + 2] = 0;
  }
  return WAM_OK;
}

wam_status wam_rope_tables(const int32_t* pos, int32_t L, int32_t Dh, double theta, float* cos_out,
                           float* sin_out) {
  CHECK(pos && cos_out && sin_out, WAM_EINVAL, "NULL pointer");
  CHECK(L >= 0 && Dh >= 6 && Dh % 2 == 0, WAM_EINVAL, "bad L=%d or Dh=%d", L, Dh);
  CHECK(theta > 0.0, WAM_EINVAL, "theta must be > 0");
  const int a = Dh / 6;
  const int seg[3] = {Dh - 4 * a, 2 * a, 2 * a};
  for (int64_t l = 0; l < L; ++l) {
    int p = 0;
    for (int ax = 0; ax < 3; ++ax)
      for (int i = 0; i < seg[ax] / 2; ++i, ++p) {
        const double ang = (double)pos[3 * l + ax] * std::pow(theta, -2.0 * i / seg[ax]);
        cos_out[l * (Dh / 2) + p] = (float)std::cos(ang);
        sin_out[l * (Dh / 2) + p] = (float)std::sin(ang);
      }
  }
  return WAM_OK;
}

}  // extern "C"
