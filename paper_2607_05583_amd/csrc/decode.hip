// Batched recurrent decode step (Sec. 3.3): state <- lambda state + x_t,
// y_t = Re sum_m c state, for every (b, d) at once.
//
// A block covers 4 consecutive channels x 64 batch rows.  The block's 4*M
// (channel, mode) constants are computed once in float64 and split into a
// float32 pair lambda = hi + lo, so that a long run of steps does not drift by
// the rounding of a single float32 pole.  Each thread owns one (b, d): its M
// complex modes (M*8 bytes, contiguous) stay in registers for the update.
#include "common.h"
#include "kernels.h"

namespace res {

constexpr int DEC_CH = 4;
constexpr int DEC_ROWS = 64;

template <typename TX, typename TY>
__global__ __launch_bounds__(DEC_CH* DEC_ROWS) void decode_kernel(
    const TX* __restrict__ x, TY* __restrict__ y, int B, int D, int M,
    const float* __restrict__ gamma, const float* __restrict__ omega,
    const float* __restrict__ amp, const float* __restrict__ phase, float* __restrict__ state) {
  __shared__ float2 lhi[DEC_CH][RES_M_MAX_DEV], llo[DEC_CH][RES_M_MAX_DEV], cs[DEC_CH][RES_M_MAX_DEV];
  const int tid = threadIdx.x;
  const int d0 = blockIdx.x * DEC_CH;
  const int b0 = blockIdx.y * DEC_ROWS;
  for (int t = tid; t < DEC_CH * M; t += blockDim.x) {
    const int dl = t / M, m = t % M, d = d0 + dl;
    float2 hi = make_float2(0.f, 0.f), lo = hi, c = hi;
    if (d < D) {
      const double g = gamma[d * M + m], w = omega[d * M + m];
      const double a = amp[d * M + m], ph = phase[d * M + m];
      double s, co;
      sincos(w, &s, &co);
      const double e = exp(-g);
      const double lr = e * co, lim = e * s;
      hi = make_float2((float)lr, (float)lim);
      lo = make_float2((float)(lr - (double)hi.x), (float)(lim - (double)hi.y));
      sincos(ph, &s, &co);
      c = make_float2((float)(a * co), (float)(a * s));
    }
    lhi[dl][m] = hi;
    llo[dl][m] = lo;
    cs[dl][m] = c;
  }
  __syncthreads();
  const int dl = tid % DEC_CH;
  const int b = b0 + tid / DEC_CH;
  const int d = d0 + dl;
  if (b >= B || d >= D) return;
  const size_t row = (size_t)b * D + d;
  const float xv = to_f32(x[row]);
  float2* st = reinterpret_cast<float2*>(state) + row * M;
  float yv = 0.f;
  for (int m = 0; m < M; ++m) {
    const float2 h = st[m];
    const float2 hi = lhi[dl][m], lo = llo[dl][m], c = cs[dl][m];
    const float2 t = cmul(lo, h);
    float2 hn;
    hn.x = fmaf(hi.x, h.x, fmaf(-hi.y, h.y, t.x + xv));
    hn.y = fmaf(hi.x, h.y, fmaf(hi.y, h.x, t.y));
    st[m] = hn;
    yv = fmaf(c.x, hn.x, fmaf(-c.y, hn.y, yv));
  }
  y[row] = from_f32<TY>(yv);
}

template <typename TX, typename TY>
hipError_t launch_decode(int64_t B, int64_t D, int64_t M, const void* x, void* y,
                         const float* gamma, const float* omega, const float* amp,
                         const float* phase, float* state, hipStream_t st) {
  const dim3 grid((unsigned)((D + DEC_CH - 1) / DEC_CH), (unsigned)((B + DEC_ROWS - 1) / DEC_ROWS));
  hipLaunchKernelGGL((decode_kernel<TX, TY>), grid, dim3(DEC_CH * DEC_ROWS), 0, st,
                     reinterpret_cast<const TX*>(x), reinterpret_cast<TY*>(y), (int)B, (int)D,
                     (int)M, gamma, omega, amp, phase, state);
  return hipGetLastError();
}

template hipError_t launch_decode<float, float>(int64_t, int64_t, int64_t, const void*, void*,
                                                const float*, const float*, const float*,
                                                const float*, float*, hipStream_t);
template hipError_t launch_decode<bf16_t, bf16_t>(int64_t, int64_t, int64_t, const void*, void*,
                                                  const float*, const float*, const float*,
                                                  const float*, float*, hipStream_t);
template hipError_t launch_decode<bf16_t, float>(int64_t, int64_t, int64_t, const void*, void*,
                                                 const float*, const float*, const float*,
                                                 const float*, float*, hipStream_t);

}  // namespace res
