// Constrained parameterization of the resonant modes (Sec. 3.1, last
// paragraph): unconstrained parameters are mapped into the valid ranges,
//   gamma = alpha_min + softplus(theta_gamma)     (damping above a floor)
//   omega = pi * sigmoid(theta_omega)             (frequency in (0, pi))
// with the chain rule for the backward, and an initialization whose mapped
// values have log-spaced half-lives ln 2 / gamma and periods 2 pi / omega.
// Elementwise over the [D][M] parameter bank; bound by launch latency.
#include "common.h"
#include "kernels.h"

namespace res {

// softplus(u) = max(u, 0) + log(1 + e^-|u|): no exponential overflows
__device__ __forceinline__ float softplus_f(float u) { return fmaxf(u, 0.f) + log1pf(expf(-fabsf(u))); }
// 1 / (1 + e^-u), as e^u / (1 + e^u) for u < 0
__device__ __forceinline__ float sigmoid_f(float u) {
  const float e = expf(-fabsf(u));
  return u >= 0.f ? 1.f / (1.f + e) : e / (1.f + e);
}

__global__ __launch_bounds__(256) void params_map_kernel(const float* __restrict__ tg, const float* __restrict__ tw,
                                                         int64_t n, float alpha_min, float* __restrict__ gamma,
                                                         float* __restrict__ omega) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    gamma[i] = alpha_min + softplus_f(tg[i]);
    omega[i] = (float)M_PI * sigmoid_f(tw[i]);
  }
}

__global__ __launch_bounds__(256) void params_map_bwd_kernel(const float* __restrict__ tg,
                                                             const float* __restrict__ tw,
                                                             const float* __restrict__ dg,
                                                             const float* __restrict__ dw, int64_t n,
                                                             float* __restrict__ dtg, float* __restrict__ dtw) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    // sigmoid (1 - sigmoid) = e^-|u| / (1 + e^-|u|)^2: no cancellation in 1 - sigmoid
    const float e = expf(-fabsf(tw[i])), q = 1.f + e;
    dtg[i] = dg[i] * sigmoid_f(tg[i]);
    dtw[i] = dw[i] * ((float)M_PI * (e / (q * q)));
  }
}

// theta for mode index k of n log-spaced timescales (float64, then rounded once):
// half-life hl_min (hl_max / hl_min)^(k / (n-1)), period per_max down to per_min
__global__ __launch_bounds__(256) void params_init_kernel(int D, int M, double hl_min, double hl_max,
                                                          double per_min, double per_max, double alpha_min,
                                                          float* __restrict__ tg, float* __restrict__ tw) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)D * M) return;
  const int n = M > 1 ? M : D;
  const int k = M > 1 ? (int)(i % M) : (int)(i / M);
  const double f = n > 1 ? (double)k / (double)(n - 1) : 0.5;
  const double hl = hl_min * pow(hl_max / hl_min, f);
  const double per = per_min * pow(per_max / per_min, 1.0 - f);
  const double g = log(2.0) / hl;
  double w = 2.0 * M_PI / per;
  if (w > M_PI * (1.0 - 1e-6)) w = M_PI * (1.0 - 1e-6);
  const double p = w / M_PI;
  tg[i] = (float)log(expm1(g - alpha_min));
  tw[i] = (float)log(p / (1.0 - p));
}

static unsigned elem_grid(int64_t n) {
  const int64_t g = (n + 255) / 256;
  return (unsigned)(g < 4096 ? (g > 0 ? g : 1) : 4096);
}

hipError_t launch_params_map(const float* tg, const float* tw, int64_t n, float alpha_min, float* gamma,
                             float* omega, hipStream_t st) {
  hipLaunchKernelGGL(params_map_kernel, dim3(elem_grid(n)), dim3(256), 0, st, tg, tw, n, alpha_min, gamma, omega);
  return hipGetLastError();
}

hipError_t launch_params_map_bwd(const float* tg, const float* tw, const float* dg, const float* dw, int64_t n,
                                 float* dtg, float* dtw, hipStream_t st) {
  hipLaunchKernelGGL(params_map_bwd_kernel, dim3(elem_grid(n)), dim3(256), 0, st, tg, tw, dg, dw, n, dtg, dtw);
  return hipGetLastError();
}

hipError_t launch_params_init(int64_t D, int64_t M, double hl_min, double hl_max, double per_min, double per_max,
                              double alpha_min, float* tg, float* tw, hipStream_t st) {
  const int64_t n = D * M;
  hipLaunchKernelGGL(params_init_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, (int)D, (int)M,
                     hl_min, hl_max, per_min, per_max, alpha_min, tg, tw);
  return hipGetLastError();
}

}  // namespace res
