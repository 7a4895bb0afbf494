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

// ---------------------------------------------------------------------------
// Diagnostics of a mode bank (Sec. 3.5): half-lives ln 2 / gamma [D][M], state
// energy decay exp(-2 gamma t) [D][M][T], and the magnitude spectrum of the
// length-T impulse response K[tau] = Re sum_m c_m lambda_m^tau (Sec. 3.1 kernel),
//   S[k][d] = |sum_{tau < T} K[tau] e^{-2 pi i k tau / T}|,  k = 0 .. T/2,
// in closed form: with w = e^{-2 pi i k / T} (so w^T = 1) each mode's geometric
// sum is (1 - lambda^T) / (1 - lambda w), and K is half the sum of c lambda^tau
// and its conjugate, so
//   S = |(1/2) sum_m [c (1 - lambda^T) / (1 - lambda w) + conj(c) (1 - conj(lambda)^T) / (1 - conj(lambda) w)]|,
// O(M) per bin in float64 instead of an impulse response and an FFT.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void diag_decay_kernel(const float* __restrict__ gamma, int64_t DM, int64_t T,
                                                         float* __restrict__ hl, float* __restrict__ en) {
  const int64_t n = en ? DM * T : DM;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t dm = en ? e / T : e;
    const double g = (double)gamma[dm];
    if (en) en[e] = (float)exp(-2.0 * g * (double)(e % T));
    if (hl && (!en || e % T == 0)) hl[dm] = (float)(0.69314718055994530942 / g);
  }
}

__global__ __launch_bounds__(256) void diag_spectrum_kernel(const float* __restrict__ gamma,
                                                            const float* __restrict__ omega,
                                                            const float* __restrict__ amp,
                                                            const float* __restrict__ phase, int64_t D, int64_t M,
                                                            int64_t T, float* __restrict__ spec) {
  const int64_t nk = T / 2 + 1;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < nk * D; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = e / D, d = e % D;
    double ws, wc;
    sincos(-2.0 * 3.14159265358979323846 * (double)k / (double)T, &ws, &wc);
    double sr = 0.0, si = 0.0;
    for (int64_t m = 0; m < M; ++m) {
      const int64_t i = d * M + m;
      const double g = (double)gamma[i], om = (double)omega[i];
      double ls, lc, ts, tc, ps, pc;
      sincos(om, &ls, &lc);
      sincos(om * (double)T, &ts, &tc);
      sincos((double)phase[i], &ps, &pc);
      const double r1 = exp(-g), rT = exp(-g * (double)T), a = (double)amp[i];
      const double cr = a * pc, ci = a * ps;
      const double lr = r1 * lc, li = r1 * ls, Tr = rT * tc, Ti = rT * ts;
      // mode term c (1 - lambda^T) / (1 - lambda w), then the conjugate pole and weight
#pragma unroll
      for (int cj = 0; cj < 2; ++cj) {
        const double sgn = cj ? -1.0 : 1.0;
        const double nr = cr * (1.0 - Tr) - (sgn * ci) * (-sgn * Ti);
        const double ni = cr * (-sgn * Ti) + (sgn * ci) * (1.0 - Tr);
        const double dr = 1.0 - (lr * wc - (sgn * li) * ws), di = -(lr * ws + (sgn * li) * wc);
        const double q = dr * dr + di * di;
        sr += 0.5 * (nr * dr + ni * di) / q;
        si += 0.5 * (ni * dr - nr * di) / q;
      }
    }
    spec[k * D + d] = (float)sqrt(sr * sr + si * si);
  }
}

hipError_t launch_diagnostics(const float* gamma, const float* omega, const float* amp, const float* phase, int64_t D,
                              int64_t M, int64_t T, float* hl, float* en, float* spec, hipStream_t st) {
  if (hl || en) {
    const int64_t n = en ? D * M * T : D * M;
    hipLaunchKernelGGL(diag_decay_kernel, dim3(elem_grid(n)), dim3(256), 0, st, gamma, D * M, T, hl, en);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (spec) {
    const int64_t n = (T / 2 + 1) * D;
    hipLaunchKernelGGL(diag_spectrum_kernel, dim3(elem_grid(n)), dim3(256), 0, st, gamma, omega, amp, phase, D, M,
                       T, spec);
  }
  return hipGetLastError();
}

}  // namespace res
