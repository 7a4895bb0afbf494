// The paper's own prefill path as a comparison variant (Sec. 3.2): per channel,
// the causal convolution y = K * x evaluated with zero-padded FFTs,
//   y = IFFT( FFT(x padded to n) . FFT(K padded to n) )[0 : L],  n = next power of two >= 2L
// (n >= 2L - 1, so the circular product has no wrap-around), in float32, with
// rocFFT.  Not part of the mixing path: a baseline for the chunked scan.
//
// Steps: the taps K_d[tau], tau < L, in float64 (rounded to float32) into a
// padded [D][n+2] buffer;
// x [B][L][D] transposed into a padded time-major [B*D][n+2] buffer (LDS tiles);
// batched in-place real FFTs of both; the spectra multiplied (with the 1/n of
// the inverse); the inverse real FFT; the first L steps transposed back.
// rocFFT plans are made once per (n, batch) and device and kept.
#include <map>
#include <mutex>
#include <tuple>

#include <rocfft/rocfft.h>

#include "common.h"
#include "kernels.h"

namespace res {

namespace {
std::mutex g_fft_mu;
bool g_fft_ready = false;
struct FftPlans {
  rocfft_plan fwd = nullptr, inv = nullptr;
  size_t work = 0;
};
std::map<std::tuple<int, size_t, size_t>, FftPlans> g_plans;  // (device, n, batch)

const char* make_plan(rocfft_plan* p, bool forward, size_t n, size_t batch, size_t* work) {
  rocfft_plan_description d = nullptr;
  if (rocfft_plan_description_create(&d) != rocfft_status_success) return "rocfft description";
  const size_t one = 1, rdist = n + 2, cdist = n / 2 + 1;
  rocfft_status s;
  if (forward)
    s = rocfft_plan_description_set_data_layout(d, rocfft_array_type_real, rocfft_array_type_hermitian_interleaved,
                                                nullptr, nullptr, 1, &one, rdist, 1, &one, cdist);
  else
    s = rocfft_plan_description_set_data_layout(d, rocfft_array_type_hermitian_interleaved, rocfft_array_type_real,
                                                nullptr, nullptr, 1, &one, cdist, 1, &one, rdist);
  if (s == rocfft_status_success)
    s = rocfft_plan_create(p, rocfft_placement_inplace,
                           forward ? rocfft_transform_type_real_forward : rocfft_transform_type_real_inverse,
                           rocfft_precision_single, 1, &n, batch, d);
  rocfft_plan_description_destroy(d);
  if (s != rocfft_status_success) return "rocfft_plan_create";
  size_t w = 0;
  if (rocfft_plan_get_work_buffer_size(*p, &w) != rocfft_status_success) return "rocfft work size";
  *work = w;
  return nullptr;
}

// plans for `batch` transforms of length n on the current device
const char* plans_for(size_t n, size_t batch, FftPlans** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return "no current HIP device";
  std::lock_guard<std::mutex> lk(g_fft_mu);
  if (!g_fft_ready) {
    if (rocfft_setup() != rocfft_status_success) return "rocfft_setup";
    g_fft_ready = true;
  }
  auto key = std::make_tuple(dev, n, batch);
  auto it = g_plans.find(key);
  if (it == g_plans.end()) {
    FftPlans pl;
    size_t w1 = 0, w2 = 0;
    if (const char* e = make_plan(&pl.fwd, true, n, batch, &w1)) return e;
    if (const char* e = make_plan(&pl.inv, false, n, batch, &w2)) return e;
    pl.work = w1 > w2 ? w1 : w2;
    it = g_plans.emplace(key, pl).first;
  }
  *out = &it->second;
  return nullptr;
}

const char* run_plan(rocfft_plan p, void* buf, void* work, size_t work_bytes, hipStream_t st) {
  rocfft_execution_info info = nullptr;
  if (rocfft_execution_info_create(&info) != rocfft_status_success) return "rocfft execution info";
  rocfft_status s = rocfft_execution_info_set_stream(info, st);
  if (s == rocfft_status_success && work_bytes > 0) s = rocfft_execution_info_set_work_buffer(info, work, work_bytes);
  void* bufs[1] = {buf};
  if (s == rocfft_status_success) s = rocfft_execute(p, bufs, nullptr, info);
  rocfft_execution_info_destroy(info);
  return s == rocfft_status_success ? nullptr : "rocfft_execute";
}
}  // namespace

size_t fft_next_pow2(int64_t L) {
  size_t n = 1;
  while (n < (size_t)(2 * L)) n <<= 1;
  return n;
}

// Taps K_d[tau] = Re sum_m c_m lambda_m^tau into [D][rows] (zero for tau >= L).
// A wave covers 64 FT_KS consecutive taps of one channel; lane l holds taps
// tau0 + l + 64 k, k < FT_KS (coalesced stores).  Per mode it evaluates
// c lambda^tau0 directly in float64 and steps by lambda^64 (at most FT_KS
// products, so about FT_KS 2^-53 relative error before the float32 rounding).
constexpr int FT_KS = 32;
constexpr int FT_SPAN = 4 * 64 * FT_KS;  // taps per 256-thread block

__global__ __launch_bounds__(256) void fft_taps_kernel(const float* __restrict__ gamma, const float* __restrict__ omega,
                                                       const float* __restrict__ amp, const float* __restrict__ phase,
                                                       int64_t L, int M, int64_t rows, int64_t nb,
                                                       float* __restrict__ Kp) {
  const int64_t d = blockIdx.x / nb, j = blockIdx.x % nb;
  const int lane = threadIdx.x % 64;
  const int64_t wave0 = j * FT_SPAN + (int64_t)(threadIdx.x / 64) * (64 * FT_KS);
  const int64_t t0 = wave0 + lane;
  double acc[FT_KS];
#pragma unroll
  for (int k = 0; k < FT_KS; ++k) acc[k] = 0.0;
  if (wave0 < L)
    for (int m = 0; m < M; ++m) {
      const double g = gamma[d * M + m], w = omega[d * M + m], a = amp[d * M + m], p = phase[d * M + m];
      double sn, cs, s1, c1;
      sincos(w * (double)t0 + p, &sn, &cs);
      const double e = a * exp(-g * (double)t0);
      double zr = e * cs, zi = e * sn;
      sincos(w * 64.0, &s1, &c1);
      const double e1 = exp(-g * 64.0), sr = e1 * c1, si = e1 * s1;
#pragma unroll
      for (int k = 0; k < FT_KS; ++k) {
        acc[k] += zr;
        const double nr = zr * sr - zi * si;
        zi = zr * si + zi * sr;
        zr = nr;
      }
    }
  float* out = Kp + d * rows;
#pragma unroll
  for (int k = 0; k < FT_KS; ++k) {
    const int64_t t = t0 + 64 * k;
    if (t < rows) out[t] = t < L ? (float)acc[k] : 0.f;
  }
}

// [B][L][D] -> [B][D][rows] (zero for t >= L), 32 x 32 tiles through LDS
__global__ __launch_bounds__(256) void fft_pack_kernel(const float* __restrict__ x, float* __restrict__ Xp, int64_t L,
                                                       int D, int64_t rows) {
  __shared__ float tile[32][33];
  const int64_t t0 = (int64_t)blockIdx.x * 32;
  const int d0 = blockIdx.y * 32;
  const int64_t b = blockIdx.z;
  const int tx = threadIdx.x % 32, ty = threadIdx.x / 32;  // 32 x 8
  for (int r = ty; r < 32; r += 8) {
    const int64_t t = t0 + r;
    const int d = d0 + tx;
    tile[r][tx] = (t < L && d < D) ? x[(b * L + t) * D + d] : 0.f;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int d = d0 + r;
    const int64_t t = t0 + tx;
    if (d < D && t < rows) Xp[(b * D + d) * rows + t] = tile[tx][r];
  }
}

// [B][D][rows] -> [B][L][D], the first L steps
__global__ __launch_bounds__(256) void fft_unpack_kernel(const float* __restrict__ Yp, float* __restrict__ y, int64_t L,
                                                         int D, int64_t rows) {
  __shared__ float tile[32][33];
  const int64_t t0 = (int64_t)blockIdx.x * 32;
  const int d0 = blockIdx.y * 32;
  const int64_t b = blockIdx.z;
  const int tx = threadIdx.x % 32, ty = threadIdx.x / 32;
  for (int r = ty; r < 32; r += 8) {
    const int d = d0 + r;
    const int64_t t = t0 + tx;
    tile[r][tx] = (d < D && t < L) ? Yp[(b * D + d) * rows + t] : 0.f;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int64_t t = t0 + r;
    const int d = d0 + tx;
    if (t < L && d < D) y[(b * L + t) * D + d] = tile[tx][r];
  }
}

// X[b d][k] *= K[d][k] / n  (interleaved complex, n/2 + 1 bins per row)
__global__ __launch_bounds__(256) void fft_mul_kernel(float2* __restrict__ X, const float2* __restrict__ K, int64_t BD,
                                                      int D, int64_t bins, float inv_n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < BD * bins; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t bd = i / bins, k = i % bins;
    const int d = (int)(bd % D);
    const float2 a = X[i], c = K[(int64_t)d * bins + k];
    X[i] = make_float2((a.x * c.x - a.y * c.y) * inv_n, (a.x * c.y + a.y * c.x) * inv_n);
  }
}

// workspace: Xp [B*D][n+2] | Kp [D][n+2] | rocFFT work (both plan sets)
const char* fft_workspace_bytes(int64_t B, int64_t L, int64_t D, size_t* bytes) {
  const size_t n = fft_next_pow2(L), rows = n + 2;
  FftPlans *px = nullptr, *pk = nullptr;
  if (const char* e = plans_for(n, (size_t)(B * D), &px)) return e;
  if (const char* e = plans_for(n, (size_t)D, &pk)) return e;
  const size_t w = px->work > pk->work ? px->work : pk->work;
  *bytes = ((size_t)(B * D) * rows + (size_t)D * rows) * sizeof(float) + ((w + 255) & ~(size_t)255) + 256;
  return nullptr;
}

const char* launch_fft_reference(const float* x, float* y, int64_t B, int64_t L, int64_t D, int64_t M,
                                 const float* gamma, const float* omega, const float* amp, const float* phase,
                                 void* ws, hipStream_t st) {
  const size_t n = fft_next_pow2(L);
  const int64_t rows = (int64_t)n + 2, bins = (int64_t)n / 2 + 1;
  FftPlans *px = nullptr, *pk = nullptr;
  if (const char* e = plans_for(n, (size_t)(B * D), &px)) return e;
  if (const char* e = plans_for(n, (size_t)D, &pk)) return e;
  float* Xp = reinterpret_cast<float*>(ws);
  float* Kp = Xp + (size_t)(B * D) * rows;
  char* work = reinterpret_cast<char*>(Kp + (size_t)D * rows);
  work = reinterpret_cast<char*>(((uintptr_t)work + 255) & ~(uintptr_t)255);
  const size_t wb = px->work > pk->work ? px->work : pk->work;
  {
    const int64_t nb = (rows + FT_SPAN - 1) / FT_SPAN;
    hipLaunchKernelGGL(fft_taps_kernel, dim3((unsigned)(D * nb)), dim3(256), 0, st, gamma, omega, amp, phase, L,
                       (int)M, rows, nb, Kp);
    if (hipGetLastError() != hipSuccess) return "taps launch";
  }
  hipLaunchKernelGGL(fft_pack_kernel, dim3((unsigned)((rows + 31) / 32), (unsigned)((D + 31) / 32), (unsigned)B),
                     dim3(256), 0, st, x, Xp, L, (int)D, rows);
  if (hipGetLastError() != hipSuccess) return "pack launch";
  if (const char* e = run_plan(pk->fwd, Kp, work, wb, st)) return e;
  if (const char* e = run_plan(px->fwd, Xp, work, wb, st)) return e;
  {
    const int64_t nm = B * D * bins;
    const unsigned g = (unsigned)((nm + 255) / 256 < 8192 ? (nm + 255) / 256 : 8192);
    hipLaunchKernelGGL(fft_mul_kernel, dim3(g), dim3(256), 0, st, reinterpret_cast<float2*>(Xp),
                       reinterpret_cast<const float2*>(Kp), B * D, (int)D, bins, 1.f / (float)n);
  }
  if (hipGetLastError() != hipSuccess) return "spectrum product launch";
  if (const char* e = run_plan(px->inv, Xp, work, wb, st)) return e;
  hipLaunchKernelGGL(fft_unpack_kernel, dim3((unsigned)((L + 31) / 32), (unsigned)((D + 31) / 32), (unsigned)B),
                     dim3(256), 0, st, Xp, y, L, (int)D, rows);
  if (hipGetLastError() != hipSuccess) return "unpack launch";
  return nullptr;
}

}  // namespace res
