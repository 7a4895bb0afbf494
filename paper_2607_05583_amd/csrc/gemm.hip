// Grouped linear projection (Sec. 3.1 drive/gate projection, Sec. 3.4 output
// projection): y[:, g-th output slice] = x[:, g-th input slice] W[g], for G
// groups of a block-diagonal weight.  A plain GEMM, so it goes to rocBLAS as one
// strided-batched GEMM over the groups (float32 accumulation).
//
// Row-major x [N, d_in] is, column-major, x^T [d_in, N] with leading dimension
// d_in, and group g's slice starts d_in / G elements further; row-major W[g]
// [d_in/G, d_out/G] is, column-major, W[g]^T; so y^T_g = W[g]^T x^T_g with
// m = d_out/G, n = N, k = d_in/G, and y^T_g starts d_out / G further.
#include <mutex>

#include <rocblas/rocblas.h>

#include "common.h"
#include "kernels.h"

namespace res {

namespace {
constexpr int MAX_DEVICES = 64;
rocblas_handle g_handle[MAX_DEVICES] = {};
std::mutex g_handle_mu;

rocblas_handle handle_for(int dev) {
  std::lock_guard<std::mutex> lk(g_handle_mu);
  if (!g_handle[dev] && rocblas_create_handle(&g_handle[dev]) != rocblas_status_success) g_handle[dev] = nullptr;
  return g_handle[dev];
}
}  // namespace

// 0 on success; otherwise a message for the caller's error report
const char* launch_grouped_linear(const void* x, const void* W, void* y, int64_t N, int64_t d_in, int64_t d_out,
                                  int64_t G, bool bf16, hipStream_t st) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return "no current HIP device";
  rocblas_handle h = handle_for(dev);
  if (!h) return "rocblas_create_handle failed";
  if (rocblas_set_stream(h, st) != rocblas_status_success) return "rocblas_set_stream failed";
  const rocblas_datatype t = bf16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
  const int64_t di = d_in / G, dq = d_out / G;
  const float alpha = 1.f, beta = 0.f;
  const rocblas_status s = rocblas_gemm_strided_batched_ex(
      h, rocblas_operation_none, rocblas_operation_none, (rocblas_int)dq, (rocblas_int)N, (rocblas_int)di, &alpha,
      W, t, (rocblas_int)dq, (rocblas_stride)(di * dq), x, t, (rocblas_int)d_in, (rocblas_stride)di, &beta, y, t,
      (rocblas_int)d_out, (rocblas_stride)dq, y, t, (rocblas_int)d_out, (rocblas_stride)dq, (rocblas_int)G,
      rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
  return s == rocblas_status_success ? nullptr : rocblas_status_to_string(s);
}

// Backward of the grouped projection, in the same column-major view:
//   data:   dx^T_g [di x N] = W[g] [di x dq] dy^T_g [dq x N]    (A = W^T stored, transposed)
//   weight: dW[g]^T [dq x di] = dy^T_g [dq x N] x_g [N x di]      (B = x^T stored, transposed)
// accumulate adds into the output (beta = 1) instead of overwriting it.
const char* launch_grouped_linear_bwd_data(const void* dy, const void* W, void* dx, int64_t N, int64_t d_in,
                                           int64_t d_out, int64_t G, bool bf16, bool accumulate, hipStream_t st) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return "no current HIP device";
  rocblas_handle h = handle_for(dev);
  if (!h) return "rocblas_create_handle failed";
  if (rocblas_set_stream(h, st) != rocblas_status_success) return "rocblas_set_stream failed";
  const rocblas_datatype t = bf16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
  const int64_t di = d_in / G, dq = d_out / G;
  const float alpha = 1.f, beta = accumulate ? 1.f : 0.f;
  const rocblas_status s = rocblas_gemm_strided_batched_ex(
      h, rocblas_operation_transpose, rocblas_operation_none, (rocblas_int)di, (rocblas_int)N, (rocblas_int)dq,
      &alpha, W, t, (rocblas_int)dq, (rocblas_stride)(di * dq), dy, t, (rocblas_int)d_out, (rocblas_stride)dq, &beta,
      dx, t, (rocblas_int)d_in, (rocblas_stride)di, dx, t, (rocblas_int)d_in, (rocblas_stride)di, (rocblas_int)G,
      rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
  return s == rocblas_status_success ? nullptr : rocblas_status_to_string(s);
}

const char* launch_grouped_linear_bwd_weight(const void* x, const void* dy, float* dW, int64_t N, int64_t d_in,
                                             int64_t d_out, int64_t G, bool bf16, bool accumulate, hipStream_t st) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return "no current HIP device";
  rocblas_handle h = handle_for(dev);
  if (!h) return "rocblas_create_handle failed";
  if (rocblas_set_stream(h, st) != rocblas_status_success) return "rocblas_set_stream failed";
  const rocblas_datatype t = bf16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
  const int64_t di = d_in / G, dq = d_out / G;
  const float alpha = 1.f, beta = accumulate ? 1.f : 0.f;
  const rocblas_status s = rocblas_gemm_strided_batched_ex(
      h, rocblas_operation_none, rocblas_operation_transpose, (rocblas_int)dq, (rocblas_int)di, (rocblas_int)N,
      &alpha, dy, t, (rocblas_int)d_out, (rocblas_stride)dq, x, t, (rocblas_int)d_in, (rocblas_stride)di, &beta, dW,
      rocblas_datatype_f32_r, (rocblas_int)dq, (rocblas_stride)(di * dq), dW, rocblas_datatype_f32_r,
      (rocblas_int)dq, (rocblas_stride)(di * dq), (rocblas_int)G, rocblas_datatype_f32_r, rocblas_gemm_algo_standard,
      0, 0);
  return s == rocblas_status_success ? nullptr : rocblas_status_to_string(s);
}

// Dense [d_in][d_out] copy of a block-diagonal weight W [G][d_in/G][d_out/G]
// (zeros off the diagonal blocks): one dense GEMM then gives exactly the grouped
// product (the zero blocks add exact zeros to float32 sums) with the library's
// efficient tile shapes, where G small GEMMs of d/G columns would not.
template <typename T>
__global__ __launch_bounds__(256) void block_diag_kernel(const T* __restrict__ W, T* __restrict__ Wd,
                                                         int64_t d_in, int64_t d_out, int64_t G) {
  const int64_t di = d_in / G, dq = d_out / G;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < d_in * d_out;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e / d_out, j = e % d_out, gi = i / di, gj = j / dq;
    Wd[e] = gi == gj ? W[(gi * di + i % di) * dq + j % dq] : T(0);
  }
}

hipError_t launch_block_diag(const void* W, void* Wd, int64_t d_in, int64_t d_out, int64_t G, bool bf16,
                             hipStream_t st) {
  const int64_t n = d_in * d_out;
  const unsigned grid = (unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  if (bf16)
    hipLaunchKernelGGL(block_diag_kernel<bf16_t>, dim3(grid), dim3(256), 0, st, (const bf16_t*)W, (bf16_t*)Wd, d_in,
                       d_out, G);
  else
    hipLaunchKernelGGL(block_diag_kernel<float>, dim3(grid), dim3(256), 0, st, (const float*)W, (float*)Wd, d_in,
                       d_out, G);
  return hipGetLastError();
}

// The inverse for float32 gradients: the G diagonal blocks of a dense
// [d_in][d_out] product into W [G][d_in/G][d_out/G] (added when accumulate).
// With the dense weight gradient x^T dy as one GEMM of d_in x d_out, this gives
// the grouped weight gradients from the library's efficient tile shapes, where G
// batched GEMMs of d/G x d/G over a long contraction would not.
__global__ __launch_bounds__(256) void block_extract_kernel(const float* __restrict__ Wd, float* __restrict__ W,
                                                            int64_t d_in, int64_t d_out, int64_t G, int accumulate) {
  const int64_t di = d_in / G, dq = d_out / G;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < d_in * dq;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = e / dq, j = e % dq, g = r / di;  // W[g][r % di][j], row r of the dense product
    const float v = Wd[r * d_out + g * dq + j];
    W[e] = accumulate ? W[e] + v : v;
  }
}

hipError_t launch_block_extract(const float* Wd, float* W, int64_t d_in, int64_t d_out, int64_t G, bool accumulate,
                                hipStream_t st) {
  const int64_t n = d_in * (d_out / G);
  const unsigned grid = (unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  hipLaunchKernelGGL(block_extract_kernel, dim3(grid), dim3(256), 0, st, Wd, W, d_in, d_out, G, (int)accumulate);
  return hipGetLastError();
}

// Split-K grouped weight gradient.  The contraction over N rows (tokens) is cut
// into S chunks of Nc rows; one strided-batched GEMM gives the S dense partial
// products P[s] = x_s^T dy_s [d_in][d_out] (float32) with S x (d_in/64) x
// (d_out/64) output tiles in flight, where one long GEMM has only the last two
// factors; a second kernel sums the partials of the diagonal blocks in a fixed
// order (deterministic) into W [G][d_in/G][d_out/G].
int64_t splitk_rows(int64_t N) {
  const int64_t nc = (N + SPLITK_TARGET - 1) / SPLITK_TARGET;
  return nc < SPLITK_MIN_ROWS ? SPLITK_MIN_ROWS : nc;
}
int64_t splitk_parts(int64_t N) {
  const int64_t nc = splitk_rows(N);
  return (N + nc - 1) / nc;
}

__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ P, float* __restrict__ W,
                                                            int64_t d_in, int64_t d_out, int64_t G, int64_t S,
                                                            int accumulate) {
  const int64_t di = d_in / G, dq = d_out / G, slab = d_in * d_out;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < d_in * dq;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = e / dq, j = e % dq, g = r / di;
    const float* src = P + r * d_out + g * dq + j;
    float v = 0.f;
#pragma unroll 8
    for (int64_t q = 0; q < S; ++q) v += src[q * slab];  // loads issued ahead, sums in order
    W[e] = accumulate ? W[e] + v : v;
  }
}

const char* launch_grouped_linear_bwd_weight_splitk(const void* x, const void* dy, float* dW, int64_t N,
                                                    int64_t d_in, int64_t d_out, int64_t G, bool bf16,
                                                    bool accumulate, float* P, hipStream_t st) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return "no current HIP device";
  rocblas_handle h = handle_for(dev);
  if (!h) return "rocblas_create_handle failed";
  if (rocblas_set_stream(h, st) != rocblas_status_success) return "rocblas_set_stream failed";
  const rocblas_datatype t = bf16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
  const size_t es = bf16 ? 2 : 4;
  const int64_t nc = splitk_rows(N), full = N / nc, rem = N - full * nc, S = full + (rem > 0 ? 1 : 0);
  const float alpha = 1.f, beta = 0.f;
  // column-major: P[s]^T [d_out x d_in] = dy_s^T [d_out x nc] (x_s^T)^T, as the unsplit weight gradient with G = 1
  if (full > 0) {
    const rocblas_status s = rocblas_gemm_strided_batched_ex(
        h, rocblas_operation_none, rocblas_operation_transpose, (rocblas_int)d_out, (rocblas_int)d_in,
        (rocblas_int)nc, &alpha, dy, t, (rocblas_int)d_out, (rocblas_stride)(nc * d_out), x, t, (rocblas_int)d_in,
        (rocblas_stride)(nc * d_in), &beta, P, rocblas_datatype_f32_r, (rocblas_int)d_out,
        (rocblas_stride)(d_in * d_out), P, rocblas_datatype_f32_r, (rocblas_int)d_out, (rocblas_stride)(d_in * d_out),
        (rocblas_int)full, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
    if (s != rocblas_status_success) return rocblas_status_to_string(s);
  }
  if (rem > 0) {
    const char* dyr = static_cast<const char*>(dy) + (size_t)(full * nc * d_out) * es;
    const char* xr = static_cast<const char*>(x) + (size_t)(full * nc * d_in) * es;
    float* Pr = P + (size_t)(full * d_in * d_out);
    const rocblas_status s = rocblas_gemm_ex(
        h, rocblas_operation_none, rocblas_operation_transpose, (rocblas_int)d_out, (rocblas_int)d_in,
        (rocblas_int)rem, &alpha, dyr, t, (rocblas_int)d_out, xr, t, (rocblas_int)d_in, &beta, Pr,
        rocblas_datatype_f32_r, (rocblas_int)d_out, Pr, rocblas_datatype_f32_r, (rocblas_int)d_out,
        rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
    if (s != rocblas_status_success) return rocblas_status_to_string(s);
  }
  const int64_t n = d_in * (d_out / G);
  const unsigned grid = (unsigned)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3(grid), dim3(256), 0, st, P, dW, d_in, d_out, G, S, (int)accumulate);
  return hipGetLastError() == hipSuccess ? nullptr : "split-K reduce launch";
}

}  // namespace res
