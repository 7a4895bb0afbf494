// Mixer epilogue (Sec. 3.4): head coupling, sigmoid gate and causal depthwise
// local path around the resonant mixing output.
//
//   C = I + (lambda_c / sqrt(H)) tanh(Ct)                       coupling eq.
//   ybar[b,t,g dh + j] = sum_h C[g,h] y[b,t,h dh + j]           head mixing eq.
//   l[b,t,c] = sum_{k<K} w[c,k] v[b,t-k,c]   (zero before t = 0)  local path
//   z = sigmoid(gate) * ybar + s * l                            combine eq.
//
// Every kernel is bound by HBM traffic: the activations are read once from
// HBM; the H reads of a row for the head sum and the K reads for the local taps
// hit in L1/L2.  A thread owns VEC adjacent channels of one head (same j block
// in every head), so its loads are VEC-element vectors.
//
// Backward (loss sum(dz z)), with sg = sigmoid(gate), dyb = dz sg, dl = dz s:
//   dgate = dz ybar sg (1 - sg);  dy[h dh + j] = sum_g C[g,h] dyb[g dh + j];
//   dv[t] = sum_k w[k] dl[t+k];   and the parameter sums over (b, t)
//   dC[g,h] = sum dyb[g dh + j] y[h dh + j],  ds = sum dz l,  dw[k] = sum dl[t] v[t-k],
// reduced per block of rows (float32, fixed order), then over blocks (float64,
// fixed order), so they are bitwise reproducible.
#include "common.h"
#include "kernels.h"

namespace res {

template <typename T, int VEC> struct Vec;
template <> struct Vec<float, 1> {
  typedef float S;
  __device__ static void load(const float* p, float (&o)[1]) { o[0] = p[0]; }
  __device__ static void store(float* p, const float (&v)[1]) { p[0] = v[0]; }
};
template <> struct Vec<float, 2> {
  __device__ static void load(const float* p, float (&o)[2]) {
    const float2 u = *reinterpret_cast<const float2*>(p);
    o[0] = u.x, o[1] = u.y;
  }
  __device__ static void store(float* p, const float (&v)[2]) { *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]); }
};
template <> struct Vec<bf16_t, 1> {
  __device__ static void load(const bf16_t* p, float (&o)[1]) { o[0] = to_f32(p[0]); }
  __device__ static void store(bf16_t* p, const float (&v)[1]) { p[0] = from_f32<bf16_t>(v[0]); }
};
template <> struct Vec<bf16_t, 2> {
  __device__ static void load(const bf16_t* p, float (&o)[2]) {
    const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
    o[0] = __uint_as_float(u << 16), o[1] = __uint_as_float(u & 0xFFFF0000u);
  }
  __device__ static void store(bf16_t* p, const float (&v)[2]) {
    const uint32_t u = (uint32_t)from_f32<bf16_t>(v[0]) | ((uint32_t)from_f32<bf16_t>(v[1]) << 16);
    *reinterpret_cast<uint32_t*>(p) = u;
  }
};

__device__ __forceinline__ float sigmoidf_(float u) { return 1.f / (1.f + __expf(-u)); }

// C = I + (lambda_c / sqrt(H)) tanh(Ct) into LDS (all threads; the caller syncs)
__device__ __forceinline__ void coupling_to_lds(float* sC, const float* Ct, float lambda_c, int H) {
  const float scale = lambda_c / sqrtf((float)H);
  for (int i = threadIdx.x; i < H * H; i += blockDim.x)
    sC[i] = (i / H == i % H ? 1.f : 0.f) + scale * tanhf(Ct[i]);
}

// One work item = (row r = b L + t, channels c .. c+VEC-1 of head g).
template <typename T, int VEC>
__global__ __launch_bounds__(256) void epi_fwd_kernel(const T* __restrict__ y, const T* __restrict__ gate,
                                                      const T* __restrict__ v, T* __restrict__ z, int64_t rows,
                                                      int64_t L, int H, int dh, int K, const float* __restrict__ Ct,
                                                      float lambda_c, const float* __restrict__ w,
                                                      const float* __restrict__ s) {
  __shared__ float sC[EPI_H_MAX * EPI_H_MAX];
  coupling_to_lds(sC, Ct, lambda_c, H);
  __syncthreads();
  typedef Vec<T, VEC> V;
  const int D = H * dh, gpr = D / VEC;  // channel groups per row
  for (int64_t it = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; it < rows * gpr;
       it += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = it / gpr;
    const int c = (int)(it % gpr) * VEC, g = c / dh, j = c % dh;
    const T* yr = y + r * D;
    float acc[VEC], u[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
    for (int h = 0; h < H; ++h) {
      V::load(yr + h * dh + j, u);
      const float ch = sC[g * H + h];
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] = fmaf(ch, u[e], acc[e]);
    }
    float gt[VEC], out[VEC];
    V::load(gate + r * D + c, gt);
#pragma unroll
    for (int e = 0; e < VEC; ++e) out[e] = sigmoidf_(gt[e]) * acc[e];
    if (K > 0) {
      const int64_t t = r % L;
      float l[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) l[e] = 0.f;
      for (int k = 0; k < K && k <= t; ++k) {
        V::load(v + (r - k) * D + c, u);
#pragma unroll
        for (int e = 0; e < VEC; ++e) l[e] = fmaf(w[(c + e) * K + k], u[e], l[e]);
      }
#pragma unroll
      for (int e = 0; e < VEC; ++e) out[e] = fmaf(s[c + e], l[e], out[e]);
    }
    V::store(z + r * D + c, out);
  }
}

// dy, dgate, dv (elementwise over the same work items)
template <typename T, int VEC>
__global__ __launch_bounds__(256) void epi_bwd_act_kernel(const T* __restrict__ y, const T* __restrict__ gate,
                                                          const T* __restrict__ dz, T* __restrict__ dy,
                                                          T* __restrict__ dgate, T* __restrict__ dv, int64_t rows,
                                                          int64_t L, int H, int dh, int K,
                                                          const float* __restrict__ Ct, float lambda_c,
                                                          const float* __restrict__ w,
                                                          const float* __restrict__ s) {
  __shared__ float sC[EPI_H_MAX * EPI_H_MAX];
  coupling_to_lds(sC, Ct, lambda_c, H);
  __syncthreads();
  typedef Vec<T, VEC> V;
  const int D = H * dh, gpr = D / VEC;
  for (int64_t it = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; it < rows * gpr;
       it += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = it / gpr;
    const int c = (int)(it % gpr) * VEC, g = c / dh, j = c % dh;
    const int64_t o = r * D;
    float ybar[VEC], dyh[VEC], u[VEC], gt[VEC], dzz[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) ybar[e] = dyh[e] = 0.f;
    // ybar of this head, and dy of this head (head index g plays h in dy)
    for (int q = 0; q < H; ++q) {
      V::load(y + o + q * dh + j, u);
      const float cgq = sC[g * H + q];
#pragma unroll
      for (int e = 0; e < VEC; ++e) ybar[e] = fmaf(cgq, u[e], ybar[e]);
      V::load(gate + o + q * dh + j, gt);
      V::load(dz + o + q * dh + j, dzz);
      const float cqg = sC[q * H + g];
#pragma unroll
      for (int e = 0; e < VEC; ++e) dyh[e] = fmaf(cqg, dzz[e] * sigmoidf_(gt[e]), dyh[e]);
    }
    V::load(gate + o + c, gt);
    V::load(dz + o + c, dzz);
    float dg[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const float sg = sigmoidf_(gt[e]);
      dg[e] = dzz[e] * ybar[e] * sg * (1.f - sg);
    }
    V::store(dy + o + c, dyh);
    V::store(dgate + o + c, dg);
    if (K > 0) {
      const int64_t t = r % L;
      float dvv[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) dvv[e] = 0.f;
      for (int k = 0; k < K && t + k < L; ++k) {
        V::load(dz + o + (int64_t)k * D + c, u);
#pragma unroll
        for (int e = 0; e < VEC; ++e) dvv[e] = fmaf(w[(c + e) * K + k] * s[c + e], u[e], dvv[e]);
      }
      V::store(dv + o + c, dvv);
    }
  }
}

// Parameter sums over a block of EPI_ROWS rows of one batch row: one thread per
// channel (looping over channel blocks of blockDim.x), rows in order; the head
// sums dC[g, h] over j then go through LDS in a fixed order.  Partial layout per
// block: [H*H dC | D ds | D*K dw] float32.
template <typename T>
__global__ __launch_bounds__(256) void epi_bwd_param_kernel(const T* __restrict__ y, const T* __restrict__ gate,
                                                            const T* __restrict__ v, const T* __restrict__ dz,
                                                            int64_t L, int H, int dh, int K,
                                                            const float* __restrict__ w,
                                                            const float* __restrict__ s,
                                                            float* __restrict__ part) {
  __shared__ float sdc[256 * EPI_H_MAX];  // per thread: its row of dC contributions
  const int D = H * dh;
  const int64_t nblk_t = (L + EPI_ROWS - 1) / EPI_ROWS;
  const int64_t b = blockIdx.x / nblk_t, t0 = (blockIdx.x % nblk_t) * EPI_ROWS;
  const int nr = (int)(L - t0 < EPI_ROWS ? L - t0 : EPI_ROWS);
  const int P = H * H + D + D * K;
  float* out = part + (size_t)blockIdx.x * P;
  for (int cb = 0; cb < D; cb += blockDim.x) {
    const int c = cb + threadIdx.x;
    const bool live = c < D;
    const int j = live ? c % dh : 0;
    // accumulators in registers: loops fully unrolled to the maxima, guarded by H, K
    float dc[EPI_H_MAX], dw[EPI_K_MAX], ds = 0.f;
#pragma unroll
    for (int h = 0; h < EPI_H_MAX; ++h) dc[h] = 0.f;
#pragma unroll
    for (int k = 0; k < EPI_K_MAX; ++k) dw[k] = 0.f;
    if (live) {
      const float sc = K > 0 ? s[c] : 0.f;
      for (int i = 0; i < nr; ++i) {
        const int64_t t = t0 + i, o = (b * L + t) * D;
        const float dzz = to_f32(dz[o + c]);
        const float dyb = dzz * sigmoidf_(to_f32(gate[o + c]));
#pragma unroll
        for (int h = 0; h < EPI_H_MAX; ++h)
          if (h < H) dc[h] = fmaf(dyb, to_f32(y[o + h * dh + j]), dc[h]);
        if (K > 0) {
          const float dl = dzz * sc;
          float l = 0.f;
#pragma unroll
          for (int k = 0; k < EPI_K_MAX; ++k) {
            if (k < K && k <= t) {
              const float vv = to_f32(v[o - (int64_t)k * D + c]);
              l = fmaf(w[c * K + k], vv, l);
              dw[k] = fmaf(dl, vv, dw[k]);
            }
          }
          ds = fmaf(dzz, l, ds);
        }
      }
      if (K > 0) {
        out[H * H + c] = ds;
#pragma unroll
        for (int k = 0; k < EPI_K_MAX; ++k)
          if (k < K) out[H * H + D + c * K + k] = dw[k];
      }
    }
    // dC[g, h] += sum over this channel block's channels of head g, in order
#pragma unroll
    for (int h = 0; h < EPI_H_MAX; ++h)
      if (h < H) sdc[threadIdx.x * EPI_H_MAX + h] = live ? dc[h] : 0.f;
    __syncthreads();
    for (int e = threadIdx.x; e < H * H; e += blockDim.x) {
      const int gg = e / H, h = e % H;
      float acc = cb == 0 ? 0.f : out[e];
      for (int q = 0; q < (int)blockDim.x; ++q) {
        const int cc = cb + q;
        if (cc < D && cc / dh == gg) acc += sdc[q * EPI_H_MAX + h];
      }
      out[e] = acc;
    }
    __syncthreads();
  }
}

// Sum of the block partials in float64, in a fixed order, then the chain rule of
// the coupling map.  A block takes 16 partial columns; its 16 row groups each sum
// every 16th block partial (two interleaved accumulators), and the row groups
// are added in order.
__global__ __launch_bounds__(256) void epi_bwd_reduce_kernel(const float* __restrict__ part, int64_t nblk, int H,
                                                             int D, int K, const float* __restrict__ Ct,
                                                             float lambda_c, float* __restrict__ dCt,
                                                             float* __restrict__ dw, float* __restrict__ ds,
                                                             double* __restrict__ lam_terms) {
  const int P = H * H + D + D * K;
  const int cl = threadIdx.x % 16, rg = threadIdx.x / 16;
  const int col = blockIdx.x * 16 + cl;
  __shared__ double s_acc[256];
  double a0 = 0.0, a1 = 0.0;
  if (col < P) {
    int64_t k = rg;
    for (; k + 16 < nblk; k += 32) {
      a0 += part[(size_t)k * P + col];
      a1 += part[(size_t)(k + 16) * P + col];
    }
    if (k < nblk) a0 += part[(size_t)k * P + col];
  }
  s_acc[threadIdx.x] = a0 + a1;
  __syncthreads();
  if (rg != 0 || col >= P) return;
  double acc = 0.0;
  for (int r = 0; r < 16; ++r) acc += s_acc[r * 16 + cl];
  if (col < H * H) {
    const double th = tanh((double)Ct[col]);
    dCt[col] = (float)(acc * (double)lambda_c / sqrt((double)H) * (1.0 - th * th));
    lam_terms[col] = acc * th;
  } else if (col < H * H + D) {
    if (K > 0) ds[col - H * H] = (float)acc;
  } else {
    dw[col - H * H - D] = (float)acc;
  }
}

// dlambda_c = sum_{g,h} dC[g,h] tanh(Ct[g,h]) / sqrt(H), summed in order (one thread)
__global__ void epi_bwd_lambda_kernel(const double* __restrict__ lam_terms, int H, float* __restrict__ dlambda_c) {
  double u = 0.0;
  for (int i = 0; i < H * H; ++i) u += lam_terms[i];
  *dlambda_c = (float)(u / sqrt((double)H));
}

// ---------------------------------------------------------------------------
static unsigned epi_grid(int64_t items) {
  const int64_t g = (items + 255) / 256;
  return (unsigned)(g < 8192 ? (g > 0 ? g : 1) : 8192);
}

template <typename T>
hipError_t launch_epi_fwd(const void* y, const void* gate, const void* v, void* z, int64_t B, int64_t L, int H,
                          int dh, int K, const float* Ct, float lambda_c, const float* w, const float* s, int vec,
                          hipStream_t st) {
  const int64_t rows = B * L;
  const int64_t items = rows * (int64_t)(H * dh / vec);
  if (vec == 2)
    hipLaunchKernelGGL((epi_fwd_kernel<T, 2>), dim3(epi_grid(items)), dim3(256), 0, st, (const T*)y,
                       (const T*)gate, (const T*)v, (T*)z, rows, L, H, dh, K, Ct, lambda_c, w, s);
  else
    hipLaunchKernelGGL((epi_fwd_kernel<T, 1>), dim3(epi_grid(items)), dim3(256), 0, st, (const T*)y,
                       (const T*)gate, (const T*)v, (T*)z, rows, L, H, dh, K, Ct, lambda_c, w, s);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_epi_bwd(const void* y, const void* gate, const void* v, const void* dz, void* dy, void* dgate,
                          void* dv, int64_t B, int64_t L, int H, int dh, int K, const float* Ct, float lambda_c,
                          const float* w, const float* s, float* dCt, float* dlambda_c, float* dw, float* ds,
                          float* part, int vec, hipStream_t st) {
  const int64_t rows = B * L;
  const int64_t items = rows * (int64_t)(H * dh / vec);
  if (vec == 2)
    hipLaunchKernelGGL((epi_bwd_act_kernel<T, 2>), dim3(epi_grid(items)), dim3(256), 0, st, (const T*)y,
                       (const T*)gate, (const T*)dz, (T*)dy, (T*)dgate, (T*)dv, rows, L, H, dh, K, Ct, lambda_c, w,
                       s);
  else
    hipLaunchKernelGGL((epi_bwd_act_kernel<T, 1>), dim3(epi_grid(items)), dim3(256), 0, st, (const T*)y,
                       (const T*)gate, (const T*)dz, (T*)dy, (T*)dgate, (T*)dv, rows, L, H, dh, K, Ct, lambda_c, w,
                       s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t nblk = B * ((L + EPI_ROWS - 1) / EPI_ROWS);
  hipLaunchKernelGGL((epi_bwd_param_kernel<T>), dim3((unsigned)nblk), dim3(256), 0, st, (const T*)y, (const T*)gate, (const T*)v, (const T*)dz, L, H, dh, K, w, s, part);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int P = H * H + H * dh + H * dh * K;
  double* lam_terms = reinterpret_cast<double*>(part + epi_part_floats(B, L, H, dh, K));
  hipLaunchKernelGGL(epi_bwd_reduce_kernel, dim3((unsigned)((P + 15) / 16)), dim3(256), 0, st, part, nblk, H,
                     H * dh, K, Ct, lambda_c, dCt, dw, ds, lam_terms);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(epi_bwd_lambda_kernel, dim3(1), dim3(1), 0, st, lam_terms, H, dlambda_c);
  return hipGetLastError();
}

template hipError_t launch_epi_fwd<float>(const void*, const void*, const void*, void*, int64_t, int64_t, int, int,
                                          int, const float*, float, const float*, const float*, int, hipStream_t);
template hipError_t launch_epi_fwd<bf16_t>(const void*, const void*, const void*, void*, int64_t, int64_t, int, int,
                                           int, const float*, float, const float*, const float*, int, hipStream_t);
template hipError_t launch_epi_bwd<float>(const void*, const void*, const void*, const void*, void*, void*, void*,
                                          int64_t, int64_t, int, int, int, const float*, float, const float*,
                                          const float*, float*, float*, float*, float*, float*, int, hipStream_t);
template hipError_t launch_epi_bwd<bf16_t>(const void*, const void*, const void*, const void*, void*, void*, void*,
                                           int64_t, int64_t, int, int, int, const float*, float, const float*,
                                           const float*, float*, float*, float*, float*, float*, int, hipStream_t);

}  // namespace res
