// Quadratic causal reference mixer, the baseline of the kernel-tail benchmark
// (Sec. 5.3, Table 5): y[b,t,d] = sum_{s<=t} K_d[t-s] x[b,s,d], evaluated
// directly in O(L^2 D) multiply-adds, with the taps of the Sec. 3.1 kernel
//   K_d[tau] = sum_m a exp(-gamma tau) cos(omega tau + phi)
// tabulated once per call in float64 (rounded to float32) as [L][D].
//
// A block takes 64 output steps x 64 channels of one batch row; thread (g, c)
// owns channel c and the 16 steps 16 g .. 16 g + 15.  The input tiles up to the
// diagonal are visited in order: each stages 64 input rows and the 127 lags the
// tile pair needs in LDS, then every thread adds 64 x 16 products in float32.
// A comparison baseline, not part of the mixing path.
#include "common.h"
#include "kernels.h"

namespace res {

constexpr int QR_T = 64;  // output steps and input steps per tile
constexpr int QR_C = 64;  // channels per block

__global__ __launch_bounds__(256) void quad_taps_kernel(const float* __restrict__ gamma,
                                                        const float* __restrict__ omega,
                                                        const float* __restrict__ amp,
                                                        const float* __restrict__ phase, int64_t L, int D, int M,
                                                        float* __restrict__ K) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < L * D; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t tau = i / D;
    const int d = (int)(i % D);
    double k = 0.0;
    for (int m = 0; m < M; ++m) {
      const double g = gamma[d * M + m], w = omega[d * M + m], a = amp[d * M + m], p = phase[d * M + m];
      k += a * exp(-g * (double)tau) * cos(w * (double)tau + p);
    }
    K[i] = (float)k;
  }
}

__global__ __launch_bounds__(256) void quad_mix_kernel(const float* __restrict__ x, const float* __restrict__ K,
                                                       float* __restrict__ y, int64_t L, int D) {
  __shared__ float xs[QR_T][QR_C];
  __shared__ float ks[2 * QR_T][QR_C];  // lags lag0 .. lag0 + 127
  const int c = threadIdx.x % QR_C, g = threadIdx.x / QR_C;
  const int64_t T0 = (int64_t)blockIdx.x * QR_T;
  const int d0 = blockIdx.y * QR_C;
  const int64_t b = blockIdx.z;
  const int d = d0 + c;
  float acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  for (int64_t s0 = 0; s0 <= T0; s0 += QR_T) {
    const int64_t lag0 = T0 - s0 - QR_T;  // ks[j] = K[lag0 + j]
    __syncthreads();                      // the previous tile's reads are done
    for (int r = g; r < QR_T; r += 4) {
      const int64_t s = s0 + r;
      xs[r][c] = (s < L && d < D) ? x[(b * L + s) * D + d] : 0.f;
    }
    for (int r = g; r < 2 * QR_T; r += 4) {
      const int64_t lag = lag0 + r;
      ks[r][c] = (lag >= 0 && lag < L && d < D) ? K[lag * D + d] : 0.f;
    }
    __syncthreads();
    for (int s = 0; s < QR_T; ++s) {
      const float xv = xs[s][c];
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[i] = fmaf(ks[16 * g + i - s + QR_T][c], xv, acc[i]);
    }
  }
  if (d >= D) return;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int64_t t = T0 + 16 * g + i;
    if (t < L) y[(b * L + t) * D + d] = acc[i];
  }
}

size_t quad_workspace_bytes(int64_t L, int64_t D) { return (size_t)(L * D) * sizeof(float); }

hipError_t launch_quad_reference(const float* x, float* y, int64_t B, int64_t L, int64_t D, int64_t M,
                                 const float* gamma, const float* omega, const float* amp, const float* phase,
                                 float* K, hipStream_t st) {
  const int64_t n = L * D;
  const unsigned tg = (unsigned)((n + 255) / 256 < 8192 ? (n + 255) / 256 : 8192);
  hipLaunchKernelGGL(quad_taps_kernel, dim3(tg), dim3(256), 0, st, gamma, omega, amp, phase, L, (int)D, (int)M, K);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 grid((unsigned)((L + QR_T - 1) / QR_T), (unsigned)((D + QR_C - 1) / QR_C), (unsigned)B);
  hipLaunchKernelGGL(quad_mix_kernel, grid, dim3(256), 0, st, x, K, y, L, (int)D);
  return hipGetLastError();
}

}  // namespace res
