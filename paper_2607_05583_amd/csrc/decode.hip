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

// One mode's update h <- (hi + lo) h + x and its readout term, with explicit
// fused multiply-adds so that every decode kernel rounds alike.
__device__ __forceinline__ float2 mode_step(float2 h, float2 hi, float2 lo, float xv) {
  const float tx = fmaf(lo.x, h.x, -(lo.y * h.y));
  const float ty = fmaf(lo.x, h.y, lo.y * h.x);
  return make_float2(fmaf(hi.x, h.x, fmaf(-hi.y, h.y, tx + xv)), fmaf(hi.x, h.y, fmaf(hi.y, h.x, ty)));
}
__device__ __forceinline__ float mode_readout(float2 c, float2 hn, float yv) {
  return fmaf(c.x, hn.x, fmaf(-c.y, hn.y, yv));
}

// The decode constants of one (channel, mode): lambda = exp(-gamma) e^{i omega}
// in float64, split into float32 hi + lo, and c = a e^{i phi}.  Every decode
// kernel and the constants table take them from here, so they agree bitwise.
__device__ __forceinline__ void decode_consts(float g32, float w32, float a32, float p32, float2& hi, float2& lo,
                                              float2& c) {
  const double g = g32, w = w32, a = a32, ph = p32;
  double s, co;
  sincos(w, &s, &co);
  const double e = exp(-g);
  const double lr = e * co, lim = e * s;
  hi = make_float2((float)lr, (float)lim);
  lo = make_float2((float)(lr - (double)hi.x), (float)(lim - (double)hi.y));
  sincos(ph, &s, &co);
  c = make_float2((float)(a * co), (float)(a * s));
}

template <typename TX, typename TY, int MF>
__global__ __launch_bounds__(DEC_CH* DEC_ROWS) void decode_kernel(
    const TX* __restrict__ x, TY* __restrict__ y, int B, int D, int M,
    const float* __restrict__ gamma, const float* __restrict__ omega,
    const float* __restrict__ amp, const float* __restrict__ phase, float* __restrict__ state) {
  __shared__ float2 lhi[DEC_CH][RES_M_MAX_DEV], llo[DEC_CH][RES_M_MAX_DEV], cs[DEC_CH][RES_M_MAX_DEV];
  const int tid = threadIdx.x;
  const int d0 = blockIdx.x * DEC_CH;
  const int b0 = blockIdx.y * DEC_ROWS;
  // MF > 0: M == MF is known, and the thread's state (MF complex modes) and
  // drive are loaded before the constants are computed, so their latency
  // overlaps that work
  float4 hv[MF > 0 ? MF / 2 : 1];
  float xf = 0.f;
  if (MF > 0) {
    const int dlf = tid % DEC_CH, bf = b0 + tid / DEC_CH, df = d0 + dlf;
    if (bf < B && df < D) {
      const size_t rowf = (size_t)bf * D + df;
      xf = to_f32(x[rowf]);
      const float4* sv = reinterpret_cast<const float4*>(state) + rowf * (MF / 2);
#pragma unroll
      for (int i = 0; i < MF / 2; ++i) hv[i] = sv[i];
    }
  }
  for (int t = tid; t < DEC_CH * M; t += blockDim.x) {
    const int dl = t / M, m = t % M, d = d0 + dl;
    float2 hi = make_float2(0.f, 0.f), lo = hi, c = hi;
    if (d < D) decode_consts(gamma[d * M + m], omega[d * M + m], amp[d * M + m], phase[d * M + m], hi, lo, c);
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
  float yv = 0.f;
  if (MF > 0) {
    float4* sv = reinterpret_cast<float4*>(state) + row * (MF / 2);
#pragma unroll
    for (int i = 0; i < MF / 2; ++i) {
      float h[4] = {hv[i].x, hv[i].y, hv[i].z, hv[i].w};
      float hn[4];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int m = 2 * i + j;
        const float2 r = mode_step(make_float2(h[2 * j], h[2 * j + 1]), lhi[dl][m], llo[dl][m], xf);
        hn[2 * j] = r.x;
        hn[2 * j + 1] = r.y;
        yv = mode_readout(cs[dl][m], r, yv);
      }
      sv[i] = make_float4(hn[0], hn[1], hn[2], hn[3]);
    }
    y[row] = from_f32<TY>(yv);
    return;
  }
  const float xv = to_f32(x[row]);
  float2* st = reinterpret_cast<float2*>(state) + row * M;
  for (int m = 0; m < M; ++m) {
    const float2 hn = mode_step(st[m], lhi[dl][m], llo[dl][m], xv);
    st[m] = hn;
    yv = mode_readout(cs[dl][m], hn, yv);
  }
  y[row] = from_f32<TY>(yv);
}

template <typename TX, typename TY>
hipError_t launch_decode(int64_t B, int64_t D, int64_t M, const void* x, void* y,
                         const float* gamma, const float* omega, const float* amp,
                         const float* phase, float* state, hipStream_t st) {
  const dim3 grid((unsigned)((D + DEC_CH - 1) / DEC_CH), (unsigned)((B + DEC_ROWS - 1) / DEC_ROWS));
  if (M == 8 && ((uintptr_t)state & 15) == 0)  // 16-byte state loads
    hipLaunchKernelGGL((decode_kernel<TX, TY, 8>), grid, dim3(DEC_CH * DEC_ROWS), 0, st,
                       reinterpret_cast<const TX*>(x), reinterpret_cast<TY*>(y), (int)B, (int)D,
                       (int)M, gamma, omega, amp, phase, state);
  else
    hipLaunchKernelGGL((decode_kernel<TX, TY, 0>), grid, dim3(DEC_CH * DEC_ROWS), 0, st,
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

// ---------------------------------------------------------------------------
// Decode from a constants table.  resonator_decode_constants evaluates the
// constants of every (channel, mode) once (decode_consts) into
// tab[d][m] = (hi.re, hi.im, lo.re, lo.im, c.re, c.im); the step kernel then
// reads them instead of evaluating float64 exp and sincos per call.  A work-group
// is one wave: 64 consecutive channels of one batch row (each thread one (b, d),
// its modes in registers), so the wave's state (4 KB at M = 8), constants and
// drive and output rows are contiguous; a step over B x D needs B D / 64
// work-groups (256 at B64 D256).  The arithmetic and its order are
// decode_kernel's, so a step from the table gives the bits of
// resonator_decode_step.
// ---------------------------------------------------------------------------
constexpr int DTB_CH = 64;
constexpr int DTB_ROWS = 1;

__global__ void decode_consts_kernel(int D, int M, const float* __restrict__ gamma, const float* __restrict__ omega,
                                     const float* __restrict__ amp, const float* __restrict__ phase,
                                     float* __restrict__ tab) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= D * M) return;
  float2 hi, lo, c;
  decode_consts(gamma[i], omega[i], amp[i], phase[i], hi, lo, c);
  float2* t = reinterpret_cast<float2*>(tab) + (size_t)i * 3;
  t[0] = hi;
  t[1] = lo;
  t[2] = c;
}

hipError_t launch_decode_consts(int64_t D, int64_t M, const float* gamma, const float* omega, const float* amp,
                                const float* phase, float* tab, hipStream_t st) {
  const int n = (int)(D * M);
  hipLaunchKernelGGL(decode_consts_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, (int)D, (int)M,
                     gamma, omega, amp, phase, tab);
  return hipGetLastError();
}

template <typename TX, typename TY, int MF>
__global__ __launch_bounds__(DTB_CH* DTB_ROWS) void decode_tab_kernel(const TX* __restrict__ x,
                                                                     TY* __restrict__ y, int B, int D, int M,
                                                                     const float* __restrict__ tab,
                                                                     float* __restrict__ state) {
  const int tid = threadIdx.x;
  const int dl = tid % DTB_CH;
  const int b = blockIdx.y * DTB_ROWS + tid / DTB_CH;
  const int d = blockIdx.x * DTB_CH + dl;
  if (b >= B || d >= D) return;
  const size_t row = (size_t)b * D + d;
  const float2* t = reinterpret_cast<const float2*>(tab) + (size_t)d * M * 3;
  float yv = 0.f;
  if (MF > 0) {
    // all loads first: drive, state (16-byte pieces), constants
    const float xv = to_f32(x[row]);
    float4* sv = reinterpret_cast<float4*>(state) + row * (MF / 2);
    const float4* tv = reinterpret_cast<const float4*>(t);
    float4 hv[MF > 0 ? MF / 2 : 1], cv[MF > 0 ? MF * 3 / 2 : 1];
#pragma unroll
    for (int i = 0; i < MF / 2; ++i) hv[i] = sv[i];
#pragma unroll
    for (int i = 0; i < MF * 3 / 2; ++i) cv[i] = tv[i];
    const float* cf = reinterpret_cast<const float*>(cv);
#pragma unroll
    for (int i = 0; i < MF / 2; ++i) {
      float h[4] = {hv[i].x, hv[i].y, hv[i].z, hv[i].w};
      float hn[4];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int m = 2 * i + j;
        const float* k = cf + 6 * m;
        const float2 r = mode_step(make_float2(h[2 * j], h[2 * j + 1]), make_float2(k[0], k[1]),
                                   make_float2(k[2], k[3]), xv);
        hn[2 * j] = r.x;
        hn[2 * j + 1] = r.y;
        yv = mode_readout(make_float2(k[4], k[5]), r, yv);
      }
      sv[i] = make_float4(hn[0], hn[1], hn[2], hn[3]);
    }
    y[row] = from_f32<TY>(yv);
    return;
  }
  const float xv = to_f32(x[row]);
  float2* st = reinterpret_cast<float2*>(state) + row * M;
  for (int m = 0; m < M; ++m) {
    const float2 hn = mode_step(st[m], t[3 * m], t[3 * m + 1], xv);
    st[m] = hn;
    yv = mode_readout(t[3 * m + 2], hn, yv);
  }
  y[row] = from_f32<TY>(yv);
}

template <typename TX, typename TY>
hipError_t launch_decode_tab(int64_t B, int64_t D, int64_t M, const void* x, void* y, const float* tab,
                             float* state, hipStream_t st) {
  const dim3 grid((unsigned)((D + DTB_CH - 1) / DTB_CH), (unsigned)((B + DTB_ROWS - 1) / DTB_ROWS));
  if (M == 8 && ((uintptr_t)state & 15) == 0 && ((uintptr_t)tab & 15) == 0)  // 16-byte loads
    hipLaunchKernelGGL((decode_tab_kernel<TX, TY, 8>), grid, dim3(DTB_CH * DTB_ROWS), 0, st,
                       reinterpret_cast<const TX*>(x), reinterpret_cast<TY*>(y), (int)B, (int)D, (int)M, tab,
                       state);
  else
    hipLaunchKernelGGL((decode_tab_kernel<TX, TY, 0>), grid, dim3(DTB_CH * DTB_ROWS), 0, st,
                       reinterpret_cast<const TX*>(x), reinterpret_cast<TY*>(y), (int)B, (int)D, (int)M, tab,
                       state);
  return hipGetLastError();
}
#define RES_DECODE_TAB_INST(TX, TY)                                                                      \
  template hipError_t launch_decode_tab<TX, TY>(int64_t, int64_t, int64_t, const void*, void*, const float*, \
                                                float*, hipStream_t);
RES_DECODE_TAB_INST(float, float)
RES_DECODE_TAB_INST(bf16_t, bf16_t)
RES_DECODE_TAB_INST(bf16_t, float)
#undef RES_DECODE_TAB_INST

// ---------------------------------------------------------------------------
// Several decode steps in one launch, for drives known in advance (a prompt
// chunk, drafted tokens to verify).  Step n applies the update and readout of
// decode_kernel with the same constants and in the same order, so N steps here
// give the same bits as N single steps.  A thread owns one (b, d) and keeps its
// M modes in registers for all N steps; a wave covers 64 consecutive channels
// of one batch row, so every step's drive and output rows are coalesced, and
// the next step's drive is loaded before the current step is computed.
// ---------------------------------------------------------------------------
constexpr int DMS_CH = 64;
constexpr int DMS_ROWS = 4;

template <typename TX, typename TY, int MM>
__global__ __launch_bounds__(DMS_CH* DMS_ROWS) void decode_steps_kernel(
    const TX* __restrict__ x, TY* __restrict__ y, int B, int64_t N, int D, int M,
    const float* __restrict__ gamma, const float* __restrict__ omega, const float* __restrict__ amp,
    const float* __restrict__ phase, float* __restrict__ state) {
  __shared__ float2 lhi[DMS_CH][MM], llo[DMS_CH][MM], cs[DMS_CH][MM];
  const int tid = threadIdx.x;
  const int d0 = blockIdx.x * DMS_CH;
  const int b0 = blockIdx.y * DMS_ROWS;
  for (int t = tid; t < DMS_CH * M; t += blockDim.x) {
    const int dl = t / M, m = t % M, d = d0 + dl;
    float2 hi = make_float2(0.f, 0.f), lo = hi, c = hi;
    if (d < D) decode_consts(gamma[d * M + m], omega[d * M + m], amp[d * M + m], phase[d * M + m], hi, lo, c);
    lhi[dl][m] = hi;
    llo[dl][m] = lo;
    cs[dl][m] = c;
  }
  __syncthreads();
  const int dl = tid % DMS_CH;
  const int b = b0 + tid / DMS_CH;
  const int d = d0 + dl;
  if (b >= B || d >= D) return;  // no barrier follows
  float2 h[MM], hi[MM], lo[MM], c[MM];
  float2* st = reinterpret_cast<float2*>(state) + ((size_t)b * D + d) * M;
#pragma unroll
  for (int m = 0; m < MM; ++m) {
    if (m < M) {
      h[m] = st[m];
      hi[m] = lhi[dl][m];
      lo[m] = llo[dl][m];
      c[m] = cs[dl][m];
    }
  }
  const TX* xr = x + (size_t)b * N * D + d;
  TY* yr = y + (size_t)b * N * D + d;
  // Drives of the next DPF steps are loaded while the current DPF are computed.
  // Past the last step the index is clamped to it (the value is not used), so
  // the loads are unconditional and none waits behind a branch.
  constexpr int DPF = 8;
  TX xb[DPF];
#pragma unroll
  for (int j = 0; j < DPF; ++j) xb[j] = xr[(j < N ? (int64_t)j : N - 1) * D];
  for (int64_t n0 = 0; n0 < N; n0 += DPF) {
    TX xn[DPF];
#pragma unroll
    for (int j = 0; j < DPF; ++j) {
      const int64_t nn = n0 + DPF + j;
      xn[j] = xr[(nn < N ? nn : N - 1) * D];
    }
#pragma unroll
    for (int j = 0; j < DPF; ++j) {
      if (n0 + j < N) {
        float yv = 0.f;
#pragma unroll
        for (int m = 0; m < MM; ++m) {
          if (m < M) {
            h[m] = mode_step(h[m], hi[m], lo[m], to_f32(xb[j]));
            yv = mode_readout(c[m], h[m], yv);
          }
        }
        yr[(n0 + j) * D] = from_f32<TY>(yv);
      }
    }
#pragma unroll
    for (int j = 0; j < DPF; ++j) xb[j] = xn[j];
  }
#pragma unroll
  for (int m = 0; m < MM; ++m)
    if (m < M) st[m] = h[m];
}

template <typename TX, typename TY>
hipError_t launch_decode_steps(int64_t B, int64_t N, int64_t D, int64_t M, const void* x, void* y,
                               const float* gamma, const float* omega, const float* amp,
                               const float* phase, float* state, hipStream_t st) {
  const dim3 grid((unsigned)((D + DMS_CH - 1) / DMS_CH), (unsigned)((B + DMS_ROWS - 1) / DMS_ROWS));
  if (M <= 8)
    hipLaunchKernelGGL((decode_steps_kernel<TX, TY, 8>), grid, dim3(DMS_CH * DMS_ROWS), 0, st,
                       reinterpret_cast<const TX*>(x), reinterpret_cast<TY*>(y), (int)B, N, (int)D,
                       (int)M, gamma, omega, amp, phase, state);
  else
    hipLaunchKernelGGL((decode_steps_kernel<TX, TY, RES_M_MAX_DEV>), grid, dim3(DMS_CH * DMS_ROWS), 0, st,
                       reinterpret_cast<const TX*>(x), reinterpret_cast<TY*>(y), (int)B, N, (int)D,
                       (int)M, gamma, omega, amp, phase, state);
  return hipGetLastError();
}

#define RES_DECODE_STEPS_INST(TX, TY)                                                                   \
  template hipError_t launch_decode_steps<TX, TY>(int64_t, int64_t, int64_t, int64_t, const void*, void*, \
                                                  const float*, const float*, const float*, const float*, \
                                                  float*, hipStream_t);
RES_DECODE_STEPS_INST(float, float)
RES_DECODE_STEPS_INST(bf16_t, bf16_t)
RES_DECODE_STEPS_INST(bf16_t, float)
#undef RES_DECODE_STEPS_INST

}  // namespace res
