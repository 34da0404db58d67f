// The denoising loop's own kernels for gfx950: the flow-matching solver steps (Euler and
// UniPC) with classifier-free guidance, the cosine similarity behind DiT caching, and the
// timestep fill.  All HBM-bound elementwise work over one chunk's latents and actions.
#include <mutex>

#include "common.h"
#include "kernels.h"

namespace wam {
namespace {

// Element k of the effective velocity of state sample j (k < n_video: the latent,
// else the action part).  With guidance (state sample 0 from step samples 0 = cond
// and 1 = uncond): v_u + s (v_c - v_u).
WAM_DEV float eff_velocity(const FlowArgs& a, bool reuse, int j, int64_t k) {
  if (reuse) return a.v_in[(int64_t)j * (a.n_video + a.n_action) + k];
  const bool vid = k < a.n_video;
  const float* base = vid ? a.v_video : a.v_action;
  const int64_t n = vid ? a.n_video : a.n_action;
  const int64_t kk = vid ? k : k - a.n_video;
  if (a.cfg) {
    const float vc = base[kk], vu = base[n + kk];
    return vu + a.cfg_scale * (vc - vu);
  }
  return base[(int64_t)j * n + kk];
}

// x <- x + dt v_eff (in place), v_eff optionally kept, and the bf16 model inputs of the
// next step rewritten from x for every step sample (both halves of a guidance pair).
__global__ __launch_bounds__(256) void flow_step_kernel(const FlowArgs a) {
  const int64_t n = a.n_video + a.n_action;
  const int nx = a.cfg ? 1 : a.B;
  const int64_t total = (int64_t)nx * n;
  // with the loop's flag, the velocity is reused while the flag is set
  const bool reuse = a.skip ? *a.skip > 0 : a.v_in != nullptr;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int j = (int)(e / n);
    const int64_t k = e - (int64_t)j * n;
    float x = a.x[e];
    if (a.v_video || a.v_action || a.v_in) {
      const float v = eff_velocity(a, reuse, j, k);
      if (a.v_out) a.v_out[e] = v;
      x = __builtin_fmaf(a.dt, v, x);
      a.x[e] = x;
    }
    const bf16 xb = (bf16)x;
    const int b0 = a.cfg ? 0 : j, b1 = a.cfg ? a.B : j + 1;
    for (int b = b0; b < b1; ++b) {
      if (k < a.n_video) static_cast<bf16*>(a.z_next)[(int64_t)b * a.n_video + k] = xb;
      else static_cast<bf16*>(a.a_next)[(int64_t)b * a.n_action + (k - a.n_video)] = xb;
    }
  }
}

// One UniPC step (corrector, then predictor) per element of the state; the weights are
// the host's, so the kernel is a fixed linear combination of at most five fp32 vectors.
// The history buffers are read before m_out is written, and m_out never aliases them.
__global__ __launch_bounds__(256) void unipc_step_kernel(const UnipcArgs a) {
  const FlowArgs& f = a.f;
  const int64_t n = f.n_video + f.n_action;
  const int nx = f.cfg ? 1 : f.B;
  const int64_t total = (int64_t)nx * n;
  const bool reuse = f.skip ? *f.skip > 0 : f.v_in != nullptr;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int j = (int)(e / n);
    const int64_t k = e - (int64_t)j * n;
    const float v = eff_velocity(f, reuse, j, k);
    if (f.v_out) f.v_out[e] = v;
    const float x = f.x[e];
    const float m = __builtin_fmaf(a.s_v, v, x);
    float h[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) h[q] = a.m_hist[q] ? a.m_hist[q][e] : 0.f;
    float xc = x;
    if (a.correct) {
      xc = __builtin_fmaf(a.c_x, a.x_last[e], a.c_new * m);
#pragma unroll
      for (int q = 0; q < 3; ++q) xc = __builtin_fmaf(a.c_m[q], h[q], xc);
    }
    float xn = __builtin_fmaf(a.p_x, xc, a.p_new * m);
#pragma unroll
    for (int q = 0; q < 2; ++q) xn = __builtin_fmaf(a.p_m[q], h[q], xn);
    a.x_last[e] = xc;
    a.m_out[e] = m;
    f.x[e] = xn;
    const bf16 xb = (bf16)xn;
    const int b0 = f.cfg ? 0 : j, b1 = f.cfg ? f.B : j + 1;
    for (int b = b0; b < b1; ++b) {
      if (k < f.n_video) static_cast<bf16*>(f.z_next)[(int64_t)b * f.n_video + k] = xb;
      else static_cast<bf16*>(f.a_next)[(int64_t)b * f.n_action + (k - f.n_video)] = xb;
    }
  }
}

// Deterministic cosine similarity: a fixed grid of COS_BLOCKS workgroups each writes its
// (a.b, a.a, b.b) partial sums in fp64, then one workgroup adds them in a fixed order.
constexpr int COS_BLOCKS = 512;

__global__ __launch_bounds__(256) void cos_partial_kernel(const float* __restrict__ x, const float* __restrict__ y,
                                                          int64_t n, double* __restrict__ part,
                                                          const int32_t* skip) {
  if (skip_step(skip)) return;
  double s[3] = {0.0, 0.0, 0.0};
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)COS_BLOCKS * 256) {
    const double u = x[i], v = y[i];
    s[0] += u * v;
    s[1] += u * u;
    s[2] += v * v;
  }
  __shared__ double red[3][256];
  for (int c = 0; c < 3; ++c) red[c][threadIdx.x] = s[c];
  __syncthreads();
  for (int o = 128; o >= 1; o >>= 1) {
    if ((int)threadIdx.x < o)
      for (int c = 0; c < 3; ++c) red[c][threadIdx.x] += red[c][threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x < 3) part[blockIdx.x * 3 + threadIdx.x] = red[threadIdx.x][0];
}

__global__ __launch_bounds__(256) void cos_final_kernel(const double* __restrict__ part, float* __restrict__ out,
                                                        const int32_t* skip) {
  if (skip_step(skip)) return;
  __shared__ double red[3][256];
  for (int c = 0; c < 3; ++c) {
    double v = 0.0;
    for (int i = threadIdx.x; i < COS_BLOCKS; i += 256) v += part[i * 3 + c];
    red[c][threadIdx.x] = v;
  }
  __syncthreads();
  for (int o = 128; o >= 1; o >>= 1) {
    if ((int)threadIdx.x < o)
      for (int c = 0; c < 3; ++c) red[c][threadIdx.x] += red[c][threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double den = sqrt(red[1][0]) * sqrt(red[2][0]);
    out[0] = den > 0.0 ? (float)(red[0][0] / den) : 0.f;
  }
}

__global__ void fill_kernel(float* p, int n, float v) {
  if ((int)threadIdx.x < n) p[threadIdx.x] = v;
}

// DiT caching decided on the device (state layout in kernels.h), so the loop needs no
// host round trip and can be captured in a graph.
__global__ void loop_init_kernel(int32_t* state) {
  if (threadIdx.x < 3) state[threadIdx.x] = 0;
}

__global__ void loop_decide_kernel(int32_t* state, const float* cs, float tau, int32_t window, int32_t* computed,
                                   int32_t i) {
  if (threadIdx.x != 0) return;
  const int32_t left = state[0], done = state[1];
  const int32_t c = left > 0 ? 0 : 1;
  if (left > 0) state[0] = left - 1;
  else if (window > 0 && done >= 1 && cs[0] > tau) state[0] = window;
  state[1] = done + c;
  state[2] = c;
  if (computed) computed[i] = c;
}

__global__ __launch_bounds__(256) void copy_if_kernel(const int32_t* flag, const float* __restrict__ src,
                                                      float* __restrict__ dst, int64_t n) {
  if (*flag == 0) return;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.x * 256) dst[e] = src[e];
}

}  // namespace

hipError_t launch_flow_step(const FlowArgs& a, hipStream_t s) {
  const int64_t total = (int64_t)(a.cfg ? 1 : a.B) * (a.n_video + a.n_action);
  if (total == 0) return hipSuccess;
  const int64_t want = (total + 255) / 256;
  const unsigned grid = (unsigned)(want < 4096 ? want : 4096);
  hipLaunchKernelGGL(flow_step_kernel, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_unipc_step(const UnipcArgs& a, hipStream_t s) {
  const int64_t total = (int64_t)(a.f.cfg ? 1 : a.f.B) * (a.f.n_video + a.f.n_action);
  if (total == 0) return hipSuccess;
  const int64_t want = (total + 255) / 256;
  const unsigned grid = (unsigned)(want < 4096 ? want : 4096);
  hipLaunchKernelGGL(unipc_step_kernel, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

size_t cosine_workspace_bytes() { return (size_t)COS_BLOCKS * 3 * sizeof(double); }

// The allocation-free cosine similarity keeps its partial sums in this file-scope device
// array: one copy per GPU, at its own address, held until the process ends.  Host code
// never passes the array's name to a kernel (on the host it is only a stand-in); it
// passes the device address hipGetSymbolAddress returns, looked up once per device.
static __device__ __align__(256) double scratch[COS_BLOCKS * 3];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];
}  // namespace

size_t cosine_static_scratch_bytes() { return sizeof(scratch); }

hipError_t cosine_static_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_cosine(const float* x, const float* y, int64_t n, void* ws, float* out, hipStream_t s,
                         const int32_t* skip) {
  double* part = static_cast<double*>(ws);
  hipLaunchKernelGGL(cos_partial_kernel, dim3(COS_BLOCKS), dim3(256), 0, s, x, y, n, part, skip);
  hipLaunchKernelGGL(cos_final_kernel, dim3(1), dim3(256), 0, s, part, out, skip);
  return hipGetLastError();
}

hipError_t launch_fill(float* p, int n, float v, hipStream_t s) {
  hipLaunchKernelGGL(fill_kernel, dim3(1), dim3(64), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t launch_loop_init(int32_t* state, hipStream_t s) {
  hipLaunchKernelGGL(loop_init_kernel, dim3(1), dim3(64), 0, s, state);
  return hipGetLastError();
}

hipError_t launch_loop_decide(int32_t* state, const float* cs, float tau, int32_t window, int32_t* computed,
                              int32_t i, hipStream_t s) {
  hipLaunchKernelGGL(loop_decide_kernel, dim3(1), dim3(64), 0, s, state, cs, tau, window, computed, i);
  return hipGetLastError();
}

hipError_t launch_copy_if(const int32_t* flag, const float* src, float* dst, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int64_t want = (n + 255) / 256;
  const unsigned grid = (unsigned)(want < 2048 ? want : 2048);
  hipLaunchKernelGGL(copy_if_kernel, dim3(grid), dim3(256), 0, s, flag, src, dst, n);
  return hipGetLastError();
}

}  // namespace wam
